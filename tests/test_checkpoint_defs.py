"""Pins of the checkpoint-cost definitions used to check the planner (CPU).

The dynamic programme for the binomial schedule is pinned to Griewank's
closed form (Revolve, cited in the paper's related work) and to small cases
worked out by hand; the uniform count is pinned by hand.
"""
import pytest

from oracle import checkpoint as cp


def test_binomial_dp_equals_closed_form():
    for c in range(1, 21):
        for l in range(1, 301):
            assert cp.binomial_cost(l, c) == cp.binomial_closed_form(l, c), (l, c)


@pytest.mark.parametrize("T,c,recompute", [
    # T=3, c=1: sweep x0->x3 (x2 in hand), then x1 recomputed from x0: 1
    (3, 1, 1),
    # T=3, c=2: keep x1, x2 in hand: nothing recomputed
    (3, 2, 0),
    # T=4, c=2: one checkpoint besides x0; one state must be recomputed
    (4, 2, 1),
    # T=10, c=3 (binomial r=2 regime: 10 <= C(5,3)): G = 2*10 - C(5,4) = 15
    (10, 3, 6),
    (7, 7, 0), (7, 20, 0), (1, 1, 0), (2, 1, 0),
])
def test_binomial_hand_cases(T, c, recompute):
    assert cp.forward_steps_binomial(T, c) - T == recompute


def test_single_checkpoint_recomputes_triangle():
    # c = 1: every x_{t-1}, t < T, is recomputed from x0: sum_{s<T-1} s
    for T in range(1, 40):
        assert cp.forward_steps_binomial(T, 1) == T + (T - 1) * (T - 2) // 2


def test_uniform_hand_case():
    # T=10, c=3: k=4, checkpoints {0,4,8}; recompute of x_s is s mod 4 for
    # s = 0..8 (x9 in hand): 0+1+2+3+0+1+2+3+0 = 12
    assert cp.uniform_checkpoints(10, 3) == (4, [4, 8])
    assert cp.forward_steps_uniform(10, 3) == 22


def test_store_all_slots():
    assert [cp.store_all_slots(T) for T in range(5)] == [0, 0, 0, 1, 2]
    assert cp.forward_steps_binomial(50, cp.store_all_slots(50) + 1) == 50
