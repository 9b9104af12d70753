"""Checkpoint planner of the product library, through the C-ABI (CPU only).

adst_plan / adst_plan_actions never touch the GPU. Every action list is
replayed by tests/plan_checker.py, and its forward-step count is compared
with the oracle's schedule definitions (oracle/checkpoint.py).
"""
import pytest

import paper_2509_02197_amd as adst
from oracle import checkpoint as cp
from tests.plan_checker import replay

AC = adst.ADST_ALLENCAHN3D7
F64 = adst.ADST_F64


def prob(kind=AC, dims=(4, 3, 2), dtype=F64, flags=0):
    return adst.make_problem(kind, dtype, dims, flags=flags)


def budget_for(slots, p=None):
    p = p or prob()
    S = p.n[0] * p.n[1] * p.n[2] * (8 if p.dtype == F64 else 4)
    return slots * S


@pytest.mark.parametrize("sched", [adst.ADST_SCHED_BINOMIAL, adst.ADST_SCHED_UNIFORM])
def test_schedules_replay_and_match_definitions(sched):
    p = prob()
    for T in range(0, 41):
        for slots in list(range(0, 9)) + [T, T + 5]:
            acts = adst.adst_plan_actions(p, T, budget_for(slots), sched)
            info = adst.adst_plan(p, T, budget_for(slots), sched)
            c = min(slots, cp.store_all_slots(T)) + 1
            nfwd, used = replay(acts, T, True, min(slots, cp.store_all_slots(T)))
            if sched == adst.ADST_SCHED_BINOMIAL:
                expect = cp.forward_steps_binomial(T, c)
            else:
                expect = cp.forward_steps_uniform(T, c)
            assert nfwd == expect, (T, slots, nfwd, expect)
            assert info.fwd_steps_total == nfwd
            assert info.recompute_steps == nfwd - T
            assert info.slots == len(used)
            assert info.n_actions == len(acts)


@pytest.mark.parametrize("T,slots", [(100, 10), (50, 8), (200, 16), (200, 7), (300, 3), (500, 40)])
def test_binomial_large(T, slots):
    p = prob()
    acts = adst.adst_plan_actions(p, T, budget_for(slots), adst.ADST_SCHED_BINOMIAL)
    nfwd, used = replay(acts, T, True, slots)
    assert nfwd == cp.forward_steps_binomial(T, slots + 1)
    assert len(used) <= slots


def test_binomial_counts_of_the_named_workloads():
    """Forward-step totals at the budgets of the four large workloads."""
    W = adst.workloads.WORKLOADS
    cases = {
        "allencahn3d7_f64_512cube_T50": 90,
        "vardiff2d9_f32_8192x8192_T200": 411,
        "allencahn3d7_f64_1024cube_T200": 581,
    }
    for name, fwd in cases.items():
        w = W[name]
        p = adst.make_problem(w.kind, w.dtype, adst.workloads.dims_of(w.shape))
        info = adst.adst_plan(p, w.steps, w.budget_bytes, adst.ADST_SCHED_BINOMIAL, w.want_dK)
        assert info.fwd_steps_total == fwd, name
    # Jacobi at the 10-snapshot budget with the tape forced: c = 11
    w = W["jacobi2d5_f64_4096x4096_T100"]
    p = adst.make_problem(w.kind, w.dtype, adst.workloads.dims_of(w.shape),
                          flags=adst.ADST_FORCE_TAPE)
    info = adst.adst_plan(p, w.steps, w.budget_bytes, adst.ADST_SCHED_BINOMIAL)
    assert info.slots <= 10 and info.fwd_steps_total == 210
    info = adst.adst_plan(p, w.steps, w.budget_bytes, adst.ADST_SCHED_UNIFORM)
    assert info.fwd_steps_total == 541
    # 64 GB (decimal) over 8 GiB states leaves 7 slots
    w = W["allencahn3d7_f64_1024cube_T200"]
    p = adst.make_problem(w.kind, w.dtype, adst.workloads.dims_of(w.shape))
    info = adst.adst_plan(p, w.steps, w.budget_bytes, adst.ADST_SCHED_BINOMIAL)
    assert info.slots == 7 and info.slot_bytes_peak <= w.budget_bytes


def test_store_all():
    p = prob()
    for T in range(0, 30):
        acts = adst.adst_plan_actions(p, T, budget_for(T), adst.ADST_SCHED_STORE_ALL)
        nfwd, used = replay(acts, T, True, cp.store_all_slots(T))
        assert nfwd == T and len(used) == cp.store_all_slots(T)


def test_linear_kind_elides_the_tape():
    """A step whose adjoint reads no state needs nothing stored at any budget."""
    p = prob(adst.ADST_JACOBI2D5, (6, 5, 1))
    for sched in range(4):
        for slots in (0, 3, 100):
            acts = adst.adst_plan_actions(p, 37, budget_for(slots, p), sched)
            nfwd, used = replay(acts, 37, False, 0)
            assert nfwd == 37 and not used
    # the coefficient field's gradient makes the variable-coefficient kind read state
    p = prob(adst.ADST_VARDIFF2D9, (6, 5, 1))
    assert adst.adst_plan(p, 10, 0, 0, grads=0).needs_state == 0
    assert adst.adst_plan(p, 10, 0, 0, grads=adst.ADST_GRAD_COEFF).needs_state == 1
    # forcing the tape makes a linear kind use the schedule
    p = prob(adst.ADST_JACOBI2D5, (6, 5, 1), flags=adst.ADST_FORCE_TAPE)
    acts = adst.adst_plan_actions(p, 37, budget_for(3, p), adst.ADST_SCHED_BINOMIAL)
    nfwd, _ = replay(acts, 37, True, 3)
    assert nfwd == cp.forward_steps_binomial(37, 4)


GS = adst.ADST_GAUSSSEIDEL2D5


def gs_levels(nx, ny, itemsize, phases):
    """Wavefront launches of one pipelined run: tiles of 64 lanes x 16 bytes
    by 32 rows, levels tau = I + 3 J + 3 s."""
    V = 16 // itemsize
    nb = -(-nx // V)
    nti, ntj = -(-(ny + 63) // 32), -(-nb // 64)
    return (nti - 1) + 3 * (ntj - 1) + 3 * (phases - 1) + 1


@pytest.mark.parametrize("dims,dtype", [((6, 5, 1), F64), ((400, 400, 1), F64),
                                        ((4096, 4096, 1), F64), ((301, 70, 1), adst.ADST_F32)])
def test_in_place_kind_plans_one_pipelined_run_each_way(dims, dtype):
    """The Gauss-Seidel kind is linear: at every budget and schedule the plan
    is one pipelined forward run to x_T, the seed and one pipelined reverse
    run, with nothing stored and no work states."""
    p = prob(GS, dims, dtype)
    isz = 8 if dtype == F64 else 4
    n = dims[0] * dims[1]
    for T in (1, 2, 7, 100):
        for sched in range(4):
            for slots in (0, 5):
                acts = adst.adst_plan_actions(p, T, budget_for(slots, p), sched)
                assert acts == [(adst.ADST_OP_FWDW, T, adst.ADST_BUF_X0, adst.ADST_BUF_XT, T),
                                (adst.ADST_OP_SEED, T, adst.ADST_BUF_XT, adst.ADST_BUF_NONE, 0),
                                (adst.ADST_OP_ADJW, T, adst.ADST_BUF_NONE, adst.ADST_BUF_NONE, T)]
                nfwd, used = replay(acts, T, False, 0)
                assert nfwd == T and not used
        info = adst.adst_plan(p, T, 0, adst.ADST_SCHED_AUTO)
        assert info.workspace_bytes == 16384 and info.fwd_workspace_bytes == 0
        assert info.fwd_launches == info.adj_launches == 1
        assert info.fwd_kernels == gs_levels(dims[0], dims[1], isz, T)
        assert info.adj_kernels == gs_levels(dims[0], dims[1], isz, T + 1)
        # read and write every point once per step each way, plus the seed
        assert info.alg_bytes == n * isz * (2 * T + 2 * T + 2)


def test_in_place_kind_with_forced_tape_uses_the_schedule():
    p = prob(GS, (9, 7, 1), flags=adst.ADST_FORCE_TAPE)
    S = 9 * 7 * 8
    stride = -(-S // 4096) * 4096
    for sched, slots in ((adst.ADST_SCHED_BINOMIAL, 3), (adst.ADST_SCHED_UNIFORM, 3),
                         (adst.ADST_SCHED_STORE_ALL, 35)):
        acts = adst.adst_plan_actions(p, 37, budget_for(slots, p), sched)
        nfwd, used = replay(acts, 37, True, slots)
        info = adst.adst_plan(p, 37, budget_for(slots, p), sched)
        assert info.fwd_steps_total == nfwd and info.adj_kernels == 37 * gs_levels(9, 7, 8, 2)
        assert info.fwd_kernels == nfwd * gs_levels(9, 7, 8, 1)
        # work states and slots, but no second gradient buffer
        assert info.workspace_bytes == 16384 + (2 + info.slots) * stride
    assert nfwd == 37


def test_auto_picks_store_all_when_it_fits():
    p = prob()
    info = adst.adst_plan(p, 20, budget_for(18), adst.ADST_SCHED_AUTO)
    assert info.sched == adst.ADST_SCHED_STORE_ALL and info.recompute_steps == 0
    info = adst.adst_plan(p, 20, budget_for(17), adst.ADST_SCHED_AUTO)
    assert info.sched == adst.ADST_SCHED_BINOMIAL and info.recompute_steps > 0
    info = adst.adst_plan(p, 20, 0, adst.ADST_SCHED_AUTO)  # never fails on budget
    assert info.slots == 0 and info.fwd_steps_total == cp.forward_steps_binomial(20, 1)


def test_store_all_over_budget_is_an_error():
    p = prob()
    with pytest.raises(adst.AdstError) as e:
        adst.adst_plan(p, 20, budget_for(17), adst.ADST_SCHED_STORE_ALL)
    assert e.value.status == adst.ADST_ERR_BUDGET
    assert "store-all" in adst.adst_last_error()


def test_budget_counts_whole_slots_only():
    p = prob()
    S = budget_for(1)
    assert adst.adst_plan(p, 50, 3 * S - 1, adst.ADST_SCHED_BINOMIAL).slots <= 2
    assert adst.adst_plan(p, 50, 3 * S, adst.ADST_SCHED_BINOMIAL).slots == 3


def fused_forward_adjoint_pairs(acts, indices=False):
    """Forward actions the library runs inside the next adjoint launch: a
    single step or a fused run of up to three whose output is the next
    adjoint step's x_{t-1} and that no later action reads before it is
    written again (their count, or their indices)."""
    FWD, ADJ, SEED = adst.ADST_OP_FWD, adst.ADST_OP_ADJ, adst.ADST_OP_SEED
    reads_ops = (FWD, adst.ADST_OP_FWD2, adst.ADST_OP_FWDW, ADJ, SEED)
    writes_ops = (FWD, adst.ADST_OP_FWD2, adst.ADST_OP_FWDW)
    found = []
    for i in range(len(acts) - 1):
        f, g = acts[i], acts[i + 1]
        fwd = (f[0] == FWD and f[4] == 1) or (f[0] == adst.ADST_OP_FWD2 and 2 <= f[4] <= 3)
        if not (fwd and g[0] == ADJ and g[2] == f[3] and g[1] == f[1] + 1 and f[3] != f[2]):
            continue
        ok = True
        for a in acts[i + 2:]:
            if a[0] in reads_ops and a[2] == f[3]:
                ok = False
                break
            if a[0] in writes_ops and a[3] == f[3]:
                break
        if ok:
            found.append(i)
    return found if indices else len(found)


def test_workspace_and_bytes():
    p = prob(dims=(100, 30, 7))
    S = 100 * 30 * 7 * 8
    stride = -(-S // 4096) * 4096
    info = adst.adst_plan(p, 12, 4 * S, adst.ADST_SCHED_BINOMIAL)
    assert info.state_bytes == S
    assert info.workspace_bytes == 16384 + (3 + info.slots) * stride
    assert info.fwd_workspace_bytes == S
    # Allen-Cahn: 8 B per point per forward launch read and 8 per state it
    # writes (a fused run writes one, a store-through run each of its
    # states), 24 per adjoint, 16 for the seed; a recomputed step whose
    # state only the next adjoint step reads runs inside that adjoint launch
    # and moves nothing of its own
    n = 100 * 30 * 7
    acts = adst.adst_plan_actions(p, 12, 4 * S, adst.ADST_SCHED_BINOMIAL)
    fused = fused_forward_adjoint_pairs(acts)
    assert fused > 0
    assert info.fwd_kernels < info.fwd_launches - fused
    assert info.fwd_alg_bytes == n * (8 * info.fwd_kernels + 8 * (info.fwd_launches - fused))
    assert info.alg_bytes == info.fwd_alg_bytes + n * (24 * 12 + 16)
    # without fusion every forward action moves its own bytes
    pn = prob(dims=(100, 30, 7), flags=adst.ADST_NO_FUSE)
    info = adst.adst_plan(pn, 12, 4 * S, adst.ADST_SCHED_BINOMIAL)
    assert info.fwd_kernels == info.fwd_launches == info.fwd_steps_total
    assert info.fwd_alg_bytes == n * 16 * info.fwd_steps_total
    assert adst.adst_plan(p, 0, 0, 0).workspace_bytes == 16384


@pytest.mark.parametrize("kind,dtype,dims,grads,depth,bytes_in", [
    (adst.ADST_ALLENCAHN3D7, adst.ADST_F64, (10, 9, 8), 0, 3, 8),
    (adst.ADST_VARDIFF2D9, adst.ADST_F32, (10, 9, 1), adst.ADST_GRAD_COEFF, 2, 8),
])
def test_store_through_runs(kind, dtype, dims, grads, depth, bytes_in):
    # store-all: one chain x0 -> slot -> ... -> work -> x_T through all T
    # single steps, taken up to `depth` steps per launch
    isz = 8 if dtype == adst.ADST_F64 else 4
    n = dims[0] * dims[1] * dims[2]
    T = 8
    p = adst.make_problem(kind, dtype, dims)
    info = adst.adst_plan(p, T, 20 * n * isz, adst.ADST_SCHED_STORE_ALL, grads)
    assert info.fwd_launches == T and info.fwd_kernels == -(-T // depth)
    assert info.fwd_alg_bytes == n * (bytes_in * info.fwd_kernels + isz * T)
    # one launch per step without fusion or with the limiter
    for q in (adst.make_problem(kind, dtype, dims, flags=adst.ADST_NO_FUSE),
              adst.make_problem(kind, dtype, dims, lim=(0.0, 1.0))):
        i = adst.adst_plan(q, T, 20 * n * isz, adst.ADST_SCHED_STORE_ALL, grads)
        assert i.fwd_kernels == T and i.fwd_alg_bytes == n * (bytes_in + isz) * T


def test_store_through_runs_counted_like_the_executor():
    # binomial plans: the launches fwd_kernels counts are the runs of chained
    # single steps (up to three, into buffers other than the run's input)
    # and the fused actions
    p = adst.make_problem(adst.ADST_ALLENCAHN3D7, adst.ADST_F64, (10, 9, 8))
    S = 10 * 9 * 8 * 8
    for T, slots in ((8, 3), (13, 4), (23, 5), (40, 6)):
        acts = adst.adst_plan_actions(p, T, slots * S, adst.ADST_SCHED_BINOMIAL)
        info = adst.adst_plan(p, T, slots * S, adst.ADST_SCHED_BINOMIAL)
        fused = set(fused_forward_adjoint_pairs(acts, indices=True))
        kernels, i = 0, 0
        while i < len(acts):
            a = acts[i]
            if i in fused:  # runs inside the next adjoint launch
                i += 1
                continue
            if a[0] in (adst.ADST_OP_FWD, adst.ADST_OP_FWD2):
                kernels += 1
            r = 1
            if a[0] == adst.ADST_OP_FWD:
                while r < 3 and i + r < len(acts):
                    b, prev = acts[i + r], acts[i + r - 1]
                    if b[0] != adst.ADST_OP_FWD or b[2] != prev[3] or b[1] != prev[1] + 1:
                        break
                    if i + r in fused:
                        break
                    if b[3] == a[2] or any(acts[i + k][3] == b[3] for k in range(r)):
                        break
                    r += 1
            i += r
        assert info.fwd_kernels == kernels


def test_zero_steps_plan():
    acts = adst.adst_plan_actions(prob(), 0, 0, adst.ADST_SCHED_AUTO)
    assert acts == [(adst.ADST_OP_SEED, 0, adst.ADST_BUF_X0, adst.ADST_BUF_NONE, 0)]


@pytest.mark.parametrize("kind,flags,sched,slots", [
    (adst.ADST_JACOBI2D5, 0, adst.ADST_SCHED_AUTO, 0),
    (adst.ADST_JACOBI2D5, adst.ADST_FORCE_TAPE, adst.ADST_SCHED_BINOMIAL, 3),
    (adst.ADST_JACOBI2D5, adst.ADST_FORCE_TAPE, adst.ADST_SCHED_UNIFORM, 3),
    (adst.ADST_JACOBI2D5, adst.ADST_FORCE_TAPE, adst.ADST_SCHED_STORE_ALL, 100),
    (adst.ADST_VARDIFF2D9, 0, adst.ADST_SCHED_BINOMIAL, 2),
    (adst.ADST_ALLENCAHN3D7, 0, adst.ADST_SCHED_BINOMIAL, 3),
    (adst.ADST_ALLENCAHN3D7, 0, adst.ADST_SCHED_UNIFORM, 2),
])
def test_fused_plans_replay_with_the_same_step_counts(kind, flags, sched, slots):
    """Temporal blocking changes launches, never which states are computed:
    fused plans replay, take the same forward steps, and fewer launches."""
    for T in list(range(0, 23)) + [64, 100]:
        dims = (6, 5, 4) if kind == AC else (6, 5, 1)
        p = prob(kind, dims, flags=flags)
        pn = prob(kind, dims, flags=flags | adst.ADST_NO_FUSE)
        want_dK = kind == adst.ADST_VARDIFF2D9
        b = budget_for(slots, p)
        fused = adst.adst_plan_actions(p, T, b, sched, want_dK)
        plain = adst.adst_plan_actions(pn, T, b, sched, want_dK)
        ns = bool(flags & adst.ADST_FORCE_TAPE) or want_dK or kind == AC
        nf, _ = replay(fused, T, ns, slots)
        np_, _ = replay(plain, T, ns, slots)
        assert nf == np_
        assert not any(op in (adst.ADST_OP_FWD2, adst.ADST_OP_ADJ2) for op, *_ in plain)
        info, infon = adst.adst_plan(p, T, b, sched, want_dK), adst.adst_plan(pn, T, b, sched, want_dK)
        assert info.fwd_steps_total == infon.fwd_steps_total == nf
        assert info.fwd_launches <= infon.fwd_launches == infon.fwd_steps_total
        assert info.adj_launches <= infon.adj_launches == T
        depth = {adst.ADST_JACOBI2D5: 6, AC: 3, adst.ADST_VARDIFF2D9: 2}[kind]
        assert all(a[4] <= depth for a in fused if a[0] == adst.ADST_OP_FWD2)
        assert all(a[4] <= depth for a in fused if a[0] == adst.ADST_OP_ADJ2)


def _runs_into_slots(acts):
    """(steps per launch of each run whose last launch writes a slot)."""
    FWD, FWD2, SLOT0 = adst.ADST_OP_FWD, adst.ADST_OP_FWD2, adst.ADST_BUF_SLOT0
    runs, cur = [], []
    for i, a in enumerate(acts):
        if a[0] not in (FWD, FWD2):
            cur = []
            continue
        prev = acts[i - 1] if i else None
        chained = (cur and prev[0] in (FWD, FWD2) and prev[3] == a[2]
                   and prev[1] == a[1] - a[4] and prev[3] < SLOT0)
        cur = cur + [a[4]] if chained else [a[4]]
        if a[3] >= SLOT0:
            runs.append(cur)
            cur = []
    return runs


@pytest.mark.parametrize("T,slots", [(40, 6), (64, 3), (100, 15), (200, 7), (200, 3)])
def test_allencahn_runs_into_slots_end_in_pairs(T, slots):
    """An Allen-Cahn run into a checkpoint slot that would end with a single
    step after a 3-step launch ends with two 2-step launches instead (two
    2-step launches cost less than a 3-step launch and a single step); which
    states are computed and kept, the step count and the launch count stay
    those of the plain split (the other kinds keep it)."""
    p = prob(dims=(6, 5, 4))
    b = budget_for(slots, p)
    acts = adst.adst_plan_actions(p, T, b, adst.ADST_SCHED_BINOMIAL)
    runs = _runs_into_slots(acts)
    assert runs and not any(len(r) >= 2 and r[-2:] == [3, 1] for r in runs)
    plain = [sum(r) for r in runs]
    assert all(r == [3] * ((n - 4) // 3) + [2, 2] for r, n in zip(runs, plain) if n % 3 == 1 and n > 3)
    assert all(r == [3] * (n // 3) + ([n % 3] if n % 3 else []) for r, n in zip(runs, plain)
               if n % 3 != 1 or n == 1)
    nf, _ = replay(acts, T, True, slots)
    pn = prob(dims=(6, 5, 4), flags=adst.ADST_NO_FUSE)
    plainacts = adst.adst_plan_actions(pn, T, b, adst.ADST_SCHED_BINOMIAL)
    kept = lambda L: [(a[1], a[3]) for a in L if a[0] in (adst.ADST_OP_FWD, adst.ADST_OP_FWD2)
                      and a[3] >= adst.ADST_BUF_SLOT0]
    assert kept(acts) == kept(plainacts)
    assert nf == cp.forward_steps_binomial(T, slots + 1)
    if (T, slots) == (200, 7):
        assert sum(1 for r in runs if r[-2:] == [2, 2]) == 14
    # Jacobi with a forced tape (six steps per launch) keeps the single step
    pj = prob(adst.ADST_JACOBI2D5, (6, 5, 1), flags=adst.ADST_FORCE_TAPE)
    runs = _runs_into_slots(adst.adst_plan_actions(pj, T, budget_for(slots, pj),
                                                   adst.ADST_SCHED_BINOMIAL))
    assert all(r == [6] * (sum(r) // 6) + ([sum(r) % 6] if sum(r) % 6 else []) for r in runs)


def test_elided_jacobi_fuses_everything():
    """Jacobi steps go up to six per launch, forward and adjoint; the
    remainder takes the last forward launch and the last adjoint launch."""
    p = prob(adst.ADST_JACOBI2D5, (6, 5, 1))
    info = adst.adst_plan(p, 100, 0, adst.ADST_SCHED_AUTO)
    assert info.fwd_launches == 17 and info.adj_launches == 17
    acts = adst.adst_plan_actions(p, 100, 0, adst.ADST_SCHED_AUTO)
    assert [a[4] for a in acts if a[0] == adst.ADST_OP_FWD2] == [6] * 16 + [4]
    assert [a[4] for a in acts if a[0] == adst.ADST_OP_ADJ2] == [6] * 16 + [4]
    info = adst.adst_plan(p, 7, 0, adst.ADST_SCHED_AUTO)
    assert info.fwd_launches == 2 and info.adj_launches == 2
    acts = adst.adst_plan_actions(p, 7, 0, adst.ADST_SCHED_AUTO)
    assert [a[0] for a in acts] == [adst.ADST_OP_FWD2, adst.ADST_OP_FWD, adst.ADST_OP_SEED,
                                    adst.ADST_OP_ADJ2, adst.ADST_OP_ADJ]
    # Allen-Cahn fuses forward chains; its adjoint reads state, so it does not
    info = adst.adst_plan(prob(), 30, budget_for(4), adst.ADST_SCHED_BINOMIAL)
    assert info.fwd_launches < info.fwd_steps_total and info.adj_launches == 30
    pn = prob(flags=adst.ADST_NO_FUSE)
    info = adst.adst_plan(pn, 30, budget_for(4), adst.ADST_SCHED_BINOMIAL)
    assert info.fwd_launches == info.fwd_steps_total
