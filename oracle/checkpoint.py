"""Checkpoint-schedule cost definitions (TEST INFRASTRUCTURE ONLY).

These are the plain definitions the planner's forward-step counts are checked
against. The store/recompute trade-off is the paper's Sec. IV; for a single
time loop with uniform step cost and a known step count the optimal schedule
is the binomial one of Revolve (cited in the paper's related work,
"Prior Research on AD Checkpointing").

Conventions: ``c`` is the number of checkpoints *including* the one holding
x0 (x0 is the caller's array and costs no slot); a step's adjoint needs only
its input state x_{t-1}; the state x_{T-1} is still in hand after the forward
sweep, so the first adjoint step needs no restore.
"""
from functools import lru_cache
from math import comb


@lru_cache(maxsize=None)
def _cost_table(L: int, C: int):
    """Bottom-up table of the dynamic programme in ``binomial_cost``:
    tab[c][l] for 1 <= l <= L, 1 <= c <= C."""
    tab = [[0] * (L + 1) for _ in range(C + 1)]
    for l in range(1, L + 1):
        tab[1][l] = l * (l - 1) // 2
    for c in range(2, C + 1):
        for l in range(2, L + 1):
            tab[c][l] = min(m + tab[c - 1][l - m] + tab[c][m] for m in range(1, l))
    return tab


def binomial_cost(l: int, c: int) -> int:
    """G(l, c): fewest forward steps that make every input state
    x_{i}, ..., x_{i+l-1} of l consecutive steps available, in reverse order,
    starting from a checkpoint at x_i with c checkpoints in total.

    Dynamic programme over the first split m (place a new checkpoint at
    x_{i+m}, reverse the right part with one checkpoint fewer, then the left
    part with all of them):
        G(1, c) = 0
        G(l, 1) = l (l - 1) / 2            (recompute every state from x_i)
        G(l, c) = min_{1 <= m < l} m + G(l - m, c - 1) + G(m, c)
    """
    if l < 1 or c < 1:
        raise ValueError("binomial_cost needs l >= 1 and c >= 1")
    c = min(c, l)  # more checkpoints than steps cannot help
    # round the table size up so that many queries share one table
    L = -(-l // 128) * 128
    C = -(-c // 8) * 8
    return _cost_table(L, C)[c][l]


def binomial_closed_form(l: int, c: int) -> int:
    """Griewank's closed form for the same quantity (Revolve):
    with beta(s, r) = C(s + r, s) and r the integer with
    beta(c, r - 1) < l <= beta(c, r),  G(l, c) = r l - beta(c + 1, r - 1)."""
    if l < 1 or c < 1:
        raise ValueError("needs l >= 1 and c >= 1")
    r = 0
    while comb(c + r, c) < l:
        r += 1
    return r * l - comb(c + 1 + r - 1, c + 1)


def forward_steps_binomial(T: int, c: int) -> int:
    """Forward steps of one forward+VJP call under the binomial schedule:
    G(T, c) to make every x_{t-1} available plus the one step to x_T."""
    return 0 if T == 0 else binomial_cost(T, c) + 1


def forward_steps_store_all(T: int) -> int:
    """Every state is computed once."""
    return T


def store_all_slots(T: int) -> int:
    """Slots store-all needs: x_1..x_{T-2}; x_0 is the caller's, x_{T-1}
    stays in hand after the sweep."""
    return max(T - 2, 0)


def uniform_checkpoints(T: int, c: int):
    """Uniform schedule: interval k = ceil(T / c), checkpoints at the
    multiples of k below T - 1 (x_{T-1} is in hand, x_0 is free)."""
    if T <= 1:
        return 1, []
    k = -(-T // c)
    return k, [s for s in range(k, T - 1, k)]


def forward_steps_uniform(T: int, c: int) -> int:
    """Forward steps of the uniform schedule: the sweep, then for every
    adjoint step t < T a one-level recompute of x_{t-1} from the nearest
    checkpoint at or below it."""
    if T == 0:
        return 0
    k, cps = uniform_checkpoints(T, c)
    base = set([0] + cps)
    total = T
    for t in range(T - 1, 0, -1):
        s = t - 1
        b = max(q for q in base if q <= s)
        total += s - b
    return total
