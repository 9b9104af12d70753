"""Gradients of the scalar step constants on the GPU vs the CPU oracle,
through the C-ABI (needs an MI355X).

Bars: dL/dp within relative 1e-12 (fp64) / 1e-5 (fp32) of the oracle's
store-all sum (both sum g_t[c] * dF_c/dp in double; only the order of the
sum and, in fp32, the adjoint's rounding differ); bit-identical across
budgets and schedules; asking for them changes no other output's bits.
"""
import numpy as np
import pytest

import oracle
import paper_2509_02197_amd as adst
from tests.gpu_util import NP_DTYPE, TOL, gpu_vjp, rel, say

pytestmark = pytest.mark.gpu

J, AC, VD = adst.ADST_JACOBI2D5, adst.ADST_ALLENCAHN3D7, adst.ADST_VARDIFF2D9
F64, F32 = adst.ADST_F64, adst.ADST_F32
HALF_SQ, DOT_W, DIFF, SEED = (adst.ADST_LOSS_HALF_SQ, adst.ADST_LOSS_DOT_W,
                              adst.ADST_LOSS_HALF_SQ_DIFF, adst.ADST_LOSS_SEED)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    adst.lib()


def inputs(kind, dtype, shape, seed):
    r = np.random.Generator(np.random.PCG64(seed))
    lo = -1.0 if kind == AC else 0.0
    dt = NP_DTYPE[dtype]
    return {"x0": r.uniform(lo, 1, shape).astype(dt),
            "K": r.uniform(0.5, 1.5, shape).astype(dt) if kind == VD else None,
            "aux": r.standard_normal(shape).astype(dt)}


def check(kind, dtype, inp, T, loss, dK, g):
    dx0, dk, xT, L, dp = oracle.vjp(kind, inp["x0"], K=inp["K"], steps=T, loss=loss,
                                    aux=inp["aux"], want_dK=dK, want_dp=True)
    tol = TOL[dtype]
    assert np.array_equal(g["xT"], xT)
    assert rel(g["dx0"], dx0) <= tol
    if dK:
        assert rel(g["dK"], dk) <= tol
    for k in range(2):
        e = abs(g["dparams"][k] - dp[k]) / max(abs(dp[k]), 1e-300)
        say(f"  dparams[{k}] gpu {g['dparams'][k]:.17g} oracle {dp[k]:.17g} rel {e:.2e}")
        if dp[k] == 0.0:
            assert g["dparams"][k] == 0.0
        else:
            assert e <= tol, (k, g["dparams"][k], dp[k])


CASES = [
    (J, F64, (64, 64), 10, HALF_SQ, False, None),
    (J, F64, (333, 517), 7, DIFF, False, 2),
    (J, F32, (130, 70), 5, SEED, False, None),
    (J, F64, (1, 1), 3, HALF_SQ, False, None),
    (J, F64, (2, 9), 4, DOT_W, False, 1),
    (AC, F64, (39, 45, 67), 6, DOT_W, False, 2),
    (AC, F32, (17, 33, 65), 4, DIFF, False, None),
    (AC, F64, (1, 1, 1), 5, SEED, False, 0),
    (AC, F64, (3, 1, 200), 5, HALF_SQ, False, 1),
    (VD, F32, (257, 300), 9, DIFF, True, 2),
    (VD, F64, (70, 129), 6, DOT_W, False, None),
    (VD, F64, (1, 7), 3, DIFF, True, 0),
]


@pytest.mark.parametrize("kind,dtype,shape,T,loss,dK,slots", CASES)
def test_dparams_match_oracle(kind, dtype, shape, T, loss, dK, slots):
    say(f"dparams kind={kind} dtype={dtype} shape={shape} T={T} loss={loss} slots={slots}")
    inp = inputs(kind, dtype, shape, 1)
    budget = None if slots is None else slots * inp["x0"].nbytes
    g = gpu_vjp(kind, inp, T, loss, budget, adst.ADST_SCHED_AUTO, dK, want_dparams=True)
    assert g["info"]["needs_state"] == 1
    check(kind, dtype, inp, T, loss, dK, g)


@pytest.mark.parametrize("kind,dtype,shape,T,loss,dK", [
    (J, F64, (90, 130), 15, HALF_SQ, False), (AC, F64, (20, 30, 70), 13, DOT_W, False),
    (AC, F32, (70, 20, 30), 7, HALF_SQ, False), (VD, F32, (100, 130), 17, DIFF, True),
    (VD, F64, (70, 600), 9, DOT_W, False)])
def test_dparams_bitwise_across_schedules(kind, dtype, shape, T, loss, dK):
    say(f"dparams schedules kind={kind} shape={shape} T={T}")
    inp = inputs(kind, dtype, shape, 2)
    S = inp["x0"].nbytes
    ref = gpu_vjp(kind, inp, T, loss, None, adst.ADST_SCHED_STORE_ALL, dK, want_dparams=True)
    check(kind, dtype, inp, T, loss, dK, ref)
    for budget, sched in ((0, adst.ADST_SCHED_BINOMIAL), (2 * S, adst.ADST_SCHED_BINOMIAL),
                          (3 * S, adst.ADST_SCHED_UNIFORM)):
        g = gpu_vjp(kind, inp, T, loss, budget, sched, dK, want_dparams=True)
        assert g["info"]["recompute_steps"] > 0
        assert np.array_equal(g["dparams"], ref["dparams"]), (budget, sched)
        assert np.array_equal(g["dx0"], ref["dx0"])
    # asking for the constants' gradients leaves the other outputs' bits alone
    plain = gpu_vjp(kind, inp, T, loss, None, adst.ADST_SCHED_AUTO, dK)
    assert np.array_equal(plain["dx0"], ref["dx0"]) and plain["loss"] == ref["loss"]
    if dK:
        assert np.array_equal(plain["dK"], ref["dK"])


def test_dparams_zero_steps_and_trace():
    inp = inputs(AC, F64, (6, 7, 8), 3)
    g = gpu_vjp(AC, inp, 0, DOT_W, want_dparams=True)
    assert np.array_equal(g["dparams"], np.zeros(2))
    g = gpu_vjp(AC, inp, 6, DOT_W, 2 * inp["x0"].nbytes, adst.ADST_SCHED_BINOMIAL,
                flags=adst.ADST_TRACE, want_dparams=True)
    assert g["info"]["ms_dparams"] > 0 and g["info"]["ms_adj"] > 0
    check(AC, F64, inp, 6, DOT_W, False, g)
