"""Store/recompute selection for general programs (the paper's Sec. IV),
through the C-ABI (CPU only).

The oracle (oracle/ilp.py) enumerates all assignments; it is pinned by the
paper's own worked example (Listing 1: the solver stores A1 and A2 and
recomputes A0, Sec. IV-A and V-D) and by a case worked by hand. The product
solver (branch and bound) must return the same choice on random programs
with several control-flow paths.
"""
import os

import numpy as np
import pytest

import paper_2509_02197_amd as adst
from oracle import checkpoint as cp
from oracle import ilp as oilp
from tests.ilp_util import read_ilp_case

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def product_solve(arrays, events, limit):
    A = [(a["size"], a["overhead"], a["cost"]) for a in arrays]
    return adst.adst_ilp_solve(A, events, limit)


def test_listing1_oracle_matches_the_paper():
    arrays, events, limit, (store, cost) = read_ilp_case(os.path.join(GOLDEN, "ilp_listing1.txt"))
    v, c, pk = oilp.solve(arrays, events, limit)
    assert v == store and c == cost
    # storing everything breaks the limit, so exactly one array is recomputed
    assert oilp.peak(arrays, events, [1, 1, 1]) > limit


def test_listing1_product_matches_the_paper():
    arrays, events, limit, (store, cost) = read_ilp_case(os.path.join(GOLDEN, "ilp_listing1.txt"))
    v, info = product_solve(arrays, events, limit)
    assert v == store
    assert info.objective == cost and info.peak <= limit and info.paths == 1
    # at a generous limit nothing is recomputed; below every choice it fails
    v, info = product_solve(arrays, events, 1000)
    assert v == [1, 1, 1] and info.objective == 0
    with pytest.raises(adst.AdstError) as e:
        product_solve(arrays, events, 300)
    assert e.value.status == adst.ADST_ERR_BUDGET


def test_hand_case():
    """Worked by hand. Base 10; A0 (size 30, cost 5) is produced and dropped
    before A1 (size 20, cost 1) is produced; the backward pass rebuilds A1,
    releases it, then rebuilds A0. Measurements:
        10, 40, 40-30(1-v0), +20, -20(1-v1), +20(1-v1), +0, -20, +30(1-v0), +0, -30
    Peaks: store both 60; recompute A1 only 60 (A0 is held when A1 is
    produced); recompute A0 only 40; both 40. At limit 55 the cheaper A1 does
    not help: the optimum recomputes A0 (cost 5, peak 40)."""
    arrays = [{"size": 30, "overhead": 0, "cost": 5}, {"size": 20, "overhead": 0, "cost": 1}]
    events = [("alloc", 10), ("produce", 0), ("drop", 0), ("produce", 1), ("drop", 1),
              ("recompute", 1), ("recompute_done", 1), ("release", 1),
              ("recompute", 0), ("recompute_done", 0), ("release", 0)]
    assert [oilp.peak(arrays, events, v) for v in ([1, 1], [1, 0], [0, 1], [0, 0])] == \
        [60, 60, 40, 40]
    assert oilp.solve(arrays, events, 55) == ([0, 1], 5, 40)
    assert oilp.solve(arrays, events, 60) == ([1, 1], 0, 60)
    pv, info = product_solve(arrays, events, 55)
    assert pv == [0, 1] and info.objective == 5 and info.peak == 40


def random_program(rng, n, npaths):
    arrays = [{"size": int(rng.integers(5, 60)), "overhead": int(rng.integers(0, 60)),
               "cost": int(rng.integers(1, 40))} for _ in range(n)]
    events = []
    for p in range(npaths):
        if p:
            events.append(("path",))
        used = sorted(rng.choice(n, size=int(rng.integers(1, n + 1)), replace=False).tolist())
        events.append(("alloc", int(rng.integers(0, 50))))
        live = []
        for i in used:
            events.append(("produce", i))
            if rng.random() < 0.5:
                events.append(("alloc", int(rng.integers(0, 40))))
            live.append(i)
            if rng.random() < 0.7:
                events.append(("drop", live.pop(0)))
        for i in live:
            events.append(("drop", i))
        if rng.random() < 0.5:
            events.append(("free", int(rng.integers(0, 30))))
        for i in reversed(used):
            events.append(("recompute", i))
            events.append(("recompute_done", i))
            if rng.random() < 0.5:
                events.append(("alloc", 7))
                events.append(("free", 7))
            events.append(("release", i))
    return arrays, events


@pytest.mark.parametrize("seed", range(40))
def test_branch_and_bound_equals_enumeration(seed):
    rng = np.random.Generator(np.random.PCG64(1000 + seed))
    n = int(rng.integers(1, 10))
    arrays, events = random_program(rng, n, int(rng.integers(1, 4)))
    # recomputing can raise the peak (its overhead), so bracket the limits by
    # the peaks of a few assignments
    peaks = [oilp.peak(arrays, events, v) for v in ([0] * n, [1] * n)]
    peaks += [oilp.peak(arrays, events, rng.integers(0, 2, n).tolist()) for _ in range(4)]
    lo, hi = int(min(peaks)), int(max(peaks))
    for limit in sorted({lo - 1, lo, (lo + hi) // 2, hi - 1, hi, int(rng.integers(lo, hi + 1))}):
        ref = oilp.solve(arrays, events, limit)
        if ref is None:
            with pytest.raises(adst.AdstError) as e:
                product_solve(arrays, events, limit)
            assert e.value.status == adst.ADST_ERR_BUDGET
            continue
        v, info = product_solve(arrays, events, limit)
        assert v == ref[0], (limit, v, ref)
        assert info.objective == ref[1] and info.peak == ref[2]


def test_control_flow_paths_all_constrain():
    """Two branches forward different arrays (the paper's Sec. IV-B): the
    choice must satisfy the limit on both paths."""
    arrays = [{"size": 50, "overhead": 0, "cost": 10},   # C on the first path
              {"size": 50, "overhead": 50, "cost": 30},  # D on the second path
              {"size": 50, "overhead": 0, "cost": 20}]   # E, on both
    events = [("alloc", 100), ("produce", 0), ("produce", 2), ("drop", 0), ("drop", 2),
              ("alloc", 50), ("recompute", 2), ("recompute_done", 2), ("release", 2),
              ("recompute", 0), ("recompute_done", 0), ("release", 0),
              ("path",),
              ("alloc", 100), ("produce", 1), ("produce", 2), ("drop", 1), ("drop", 2),
              ("alloc", 50), ("recompute", 2), ("recompute_done", 2), ("release", 2),
              ("recompute", 1), ("recompute_done", 1), ("release", 1)]
    for limit in (200, 250, 300, 350):
        ref = oilp.solve(arrays, events, limit)
        if ref is None:
            with pytest.raises(adst.AdstError):
                product_solve(arrays, events, limit)
            continue
        v, info = product_solve(arrays, events, limit)
        assert v == ref[0] and info.paths == 2
        for path in oilp.measurements(arrays, events, v):
            assert max(path) <= limit


def test_argument_errors():
    arrays = [(10, 0, 1)]
    with pytest.raises(adst.AdstError) as e:
        adst.adst_ilp_solve(arrays, [("produce", 3)], 100)
    assert e.value.status == adst.ADST_ERR_ARG
    with pytest.raises(adst.AdstError) as e:
        adst.adst_ilp_solve(arrays, [("alloc", -5)], 100)
    assert e.value.status == adst.ADST_ERR_ARG
    with pytest.raises(adst.AdstError) as e:
        adst.adst_ilp_solve([(10, -1, 1)], [], 100)
    assert e.value.status == adst.ADST_ERR_ARG
    with pytest.raises(adst.AdstError) as e:
        adst.adst_ilp_solve([(1, 0, 1)] * 49, [], 100)
    assert e.value.status == adst.ADST_ERR_ARG
    v, info = adst.adst_ilp_solve([], [("alloc", 5)], 10)
    assert v == [] and info.peak == 5


def chain_program(T):
    """The time loop under the per-array cost model: x_t (t = 1..T-1) is a
    forwarded state; recomputing it reruns t steps from the program input
    x_0 with one intermediate state alive. Sizes in states, costs in steps."""
    arrays = [{"size": 1, "overhead": 1 if t >= 2 else 0, "cost": t} for t in range(1, T)]
    events = []
    for t in range(1, T):
        events.append(("produce", t - 1))
        if t >= 2:
            events.append(("drop", t - 2))
    events.append(("drop", T - 2))
    for t in range(T - 1, 0, -1):
        events += [("recompute", t - 1), ("recompute_done", t - 1), ("release", t - 1)]
    return arrays, events


@pytest.mark.parametrize("T,slots", [(12, 3), (16, 5), (20, 6)])
def test_uniform_chain_binomial_beats_per_array_choice(T, slots):
    """On one loop of identical steps the per-array program recomputes each
    dropped state from x_0, while the binomial schedule (Revolve, cited in
    the related work) restarts from the nearest checkpoint: the binomial
    forward-step count is never higher. Memory counted in states, with two
    states of working space beside the checkpoints."""
    arrays, events = chain_program(T)
    v, info = product_solve(arrays, events, slots + 2)
    ilp_steps = T + info.objective
    assert info.peak <= slots + 2
    assert cp.forward_steps_binomial(T, slots + 1) <= ilp_steps
