"""Replays a plan's action list on integer "states" (test helper).

Each buffer holds the index t of the state x_t it contains. The replay
checks what makes a plan correct, independently of how it was built:
  * a forward step t reads a buffer holding x_{t-1} and writes a buffer
    other than the caller's x0 and its own source;
  * the seed comes exactly once, after x_T was written, before any adjoint;
  * adjoint steps run T, T-1, ..., 1, each reading a buffer that holds
    x_{t-1} at that moment when the step's adjoint needs state;
  * the x_T buffer is not read again after the seed (it may alias g_T);
  * checkpoint slots used stay within the allowed count;
  * a fused forward run (FWD2, steps t-n+1..t, n >= 2) reads x_{t-n} and
    leaves x_{t-n+1}..x_{t-1} nowhere, so any later use of them fails the
    checks above; a fused adjoint run (ADJ2, steps t..t-n+1) only appears
    for state-free adjoints;
  * a pipelined forward run (FWDW, steps t-n+1..t) reads x_{t-n} and leaves
    only x_t behind; a pipelined reverse run (ADJW, steps t..t-n+1) is
    state-free;
  * every action's step count n matches its op.
Returns the forward-step count and the set of slots touched.
"""
X0, W0, W1, XT, SLOT0 = 0, 1, 2, 3, 4
FWD, SEED, ADJ, FWD2, ADJ2, FWDW, ADJW = 0, 1, 2, 3, 4, 5, 6
NONE = -1


def replay(actions, T, needs_state, max_slots):
    holds = {X0: 0}
    seeded = False
    next_adj = T
    nfwd = 0
    slots = set()
    for k, (op, t, src, dst, n) in enumerate(actions):
        if op in (FWD, FWD2, FWDW):
            if op == FWD:
                assert n == 1, f"action {k}: step count {n}"
            elif op == FWD2:
                assert n >= 2, f"action {k}: step count {n}"
            assert n >= 1
            assert not (seeded and src == XT), f"action {k}: reads x_T buffer after the seed"
            assert holds.get(src) == t - n, f"action {k}: FWD {t} reads buffer {src} holding {holds.get(src)}"
            assert dst not in (X0, src, NONE), f"action {k}: bad destination {dst}"
            assert 1 <= t <= T
            if dst == XT:
                assert t == T, f"action {k}: only x_T goes to the x_T buffer"
            if dst >= SLOT0:
                slots.add(dst)
            holds[dst] = t
            nfwd += n
        elif op == SEED:
            assert n == 0
            assert not seeded, "seeded twice"
            assert holds.get(src) == T, f"seed reads buffer {src} holding {holds.get(src)}"
            seeded = True
            if T > 0:
                assert src == XT
                holds[XT] = None  # now holds g_T
        elif op == ADJ:
            assert n == 1
            assert seeded, "adjoint before seed"
            assert t == next_adj, f"adjoint {t} out of order (expected {next_adj})"
            if needs_state:
                assert holds.get(src) == t - 1, f"ADJ {t} reads buffer {src} holding {holds.get(src)}"
            else:
                assert src == NONE
            next_adj -= 1
        elif op == ADJ2:
            assert n >= 2
            assert seeded and not needs_state and src == NONE
            assert t == next_adj and t >= n, f"fused adjoint {t} out of order"
            next_adj -= n
        elif op == ADJW:
            assert seeded and not needs_state and src == NONE
            assert t == next_adj and 1 <= n <= t, f"pipelined adjoint {t}/{n} out of order"
            next_adj -= n
        else:
            raise AssertionError(f"unknown op {op}")
    assert seeded
    assert next_adj == 0, f"adjoints missing below {next_adj + 1}"
    assert len(slots) <= max_slots, f"{len(slots)} slots used, {max_slots} allowed"
    assert all(SLOT0 <= s < SLOT0 + max(max_slots, 0) for s in slots)
    return nfwd, slots
