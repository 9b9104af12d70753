"""The per-step limiter (a data-dependent branch at every point) on the GPU
vs the CPU oracle, through the C-ABI (needs an MI355X).

Bars as for the unlimited steps: forward states bit-identical (the branch
is decided on identical bits), gradients within 1e-12 (fp64) / 1e-5 (fp32),
every schedule bit-identical; infinite bounds reproduce the unlimited bits.
"""
import numpy as np
import pytest

import oracle
import paper_2509_02197_amd as adst
from tests.gpu_util import NP_DTYPE, TOL, dev, gpu_vjp, rel, say

pytestmark = pytest.mark.gpu

J, AC, VD = adst.ADST_JACOBI2D5, adst.ADST_ALLENCAHN3D7, adst.ADST_VARDIFF2D9
F64, F32 = adst.ADST_F64, adst.ADST_F32
HALF_SQ, DOT_W, DIFF, SEED = (adst.ADST_LOSS_HALF_SQ, adst.ADST_LOSS_DOT_W,
                              adst.ADST_LOSS_HALF_SQ_DIFF, adst.ADST_LOSS_SEED)
LIM = {J: (0.35, 0.65), AC: (-0.45, 0.5), VD: (0.3, 0.7)}


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


FORWARD_CASES = [(J, F64, (64, 64), 10), (J, F32, (130, 70), 5), (J, F64, (333, 517), 7),
                 (AC, F64, (39, 45, 67), 6), (AC, F32, (17, 33, 65), 4), (VD, F32, (257, 300), 9),
                 (VD, F64, (70, 129), 6), (J, F64, (2, 9), 4)]


@pytest.mark.parametrize("kind,dtype,shape,T", FORWARD_CASES)
def test_limited_forward_bitwise(kind, dtype, shape, T):
    say(f"limited forward kind={kind} dtype={dtype} shape={shape} T={T}")
    inp = inputs(kind, dtype, shape, 1)
    g = adst.forward(kind, dev(inp["x0"]), dev(inp["K"]), T, lim=LIM[kind]).cpu().numpy()
    ref = oracle.forward(kind, inp["x0"], K=inp["K"], steps=T, lim=LIM[kind])
    assert np.array_equal(g, ref)
    if min(shape) > 2:  # the limiter changed the trajectory
        assert not np.array_equal(ref, oracle.forward(kind, inp["x0"], K=inp["K"], steps=T))


VJP_CASES = [
    (J, F64, (64, 64), 10, HALF_SQ, False, False),
    (J, F64, (333, 517), 7, DIFF, False, True),
    (J, F32, (130, 70), 5, SEED, False, False),
    (AC, F64, (39, 45, 67), 6, DOT_W, False, True),
    (AC, F32, (17, 33, 65), 4, DIFF, False, False),
    (VD, F32, (257, 300), 9, DIFF, True, True),
    (VD, F64, (70, 129), 6, DOT_W, True, False),
    (J, F64, (2, 9), 4, DOT_W, False, False),
]


@pytest.mark.parametrize("kind,dtype,shape,T,loss,dK,dp", VJP_CASES)
def test_limited_vjp_matches_oracle(kind, dtype, shape, T, loss, dK, dp):
    say(f"limited vjp kind={kind} dtype={dtype} shape={shape} T={T} loss={loss} dK={dK} dp={dp}")
    inp = inputs(kind, dtype, shape, 2)
    g = gpu_vjp(kind, inp, T, loss, 2 * inp["x0"].nbytes, adst.ADST_SCHED_AUTO, dK,
                want_dparams=dp, lim=LIM[kind])
    assert g["info"]["needs_state"] == 1
    ref = oracle.vjp(kind, inp["x0"], K=inp["K"], steps=T, loss=loss, aux=inp["aux"],
                     want_dK=dK, want_dp=True, lim=LIM[kind])
    tol = TOL[dtype]
    assert np.array_equal(g["xT"], ref[2])
    e = rel(g["dx0"], ref[0])
    say(f"  dx0 rel {e:.2e}")
    assert e <= tol
    if dK:
        assert rel(g["dK"], ref[1]) <= tol
    assert abs(g["loss"] - ref[3]) <= tol * max(abs(ref[3]), 1e-300)
    if dp:
        for k in range(2):
            if ref[4][k] == 0.0:
                assert g["dparams"][k] == 0.0
            else:
                assert abs(g["dparams"][k] - ref[4][k]) <= tol * abs(ref[4][k])


@pytest.mark.parametrize("kind,dtype,shape,T,loss", [(J, F64, (90, 130), 15, HALF_SQ),
                                                     (AC, F64, (20, 30, 70), 13, DOT_W),
                                                     (VD, F32, (100, 130), 11, DIFF)])
def test_limited_schedules_bitwise(kind, dtype, shape, T, loss):
    inp = inputs(kind, dtype, shape, 3)
    S = inp["x0"].nbytes
    ref = gpu_vjp(kind, inp, T, loss, None, adst.ADST_SCHED_STORE_ALL, lim=LIM[kind])
    for budget, sched in ((0, adst.ADST_SCHED_BINOMIAL), (2 * S, adst.ADST_SCHED_BINOMIAL),
                          (3 * S, adst.ADST_SCHED_UNIFORM)):
        g = gpu_vjp(kind, inp, T, loss, budget, sched, lim=LIM[kind])
        assert g["info"]["recompute_steps"] > 0
        assert np.array_equal(g["dx0"], ref["dx0"]) and g["loss"] == ref["loss"]


@pytest.mark.parametrize("kind,dtype,shape,T,loss", [(J, F64, (64, 70), 9, HALF_SQ),
                                                     (AC, F64, (9, 10, 11), 5, DOT_W)])
def test_infinite_bounds_give_the_unlimited_bits(kind, dtype, shape, T, loss):
    inp = inputs(kind, dtype, shape, 4)
    a = gpu_vjp(kind, inp, T, loss)
    b = gpu_vjp(kind, inp, T, loss, lim=(-np.inf, np.inf))
    assert np.array_equal(a["xT"], b["xT"]) and np.array_equal(a["dx0"], b["dx0"])


# The Jacobi adjoint under the limiter alone masks and transposes in one
# register-marching pass; asking for the constants' gradients as well takes
# the separate mask pass and the tiled adjoint. Both must give the same
# dx0 bits. Shapes put the column strips (124 output columns in fp64, 248
# in fp32), the row chunks (6 rows at each end of a strip, 12 between them
# in the first and last strip and 128 in the others: heights 140/141 and
# 268/269 over three or more strips) and the element path (odd widths)
# against the ring, plus grids narrower than a strip and a few rows tall.
FUSED_LIM_SHAPES = [
    (F64, (50, 124)), (F64, (49, 125)), (F64, (97, 248)), (F64, (3, 300)), (F64, (300, 3)),
    (F64, (5, 4)), (F64, (61, 351)), (F32, (50, 248)), (F32, (13, 249)), (F32, (100, 497)),
    (F32, (7, 5)), (F64, (204, 380)), (F64, (205, 373)), (F64, (410, 130)), (F32, (211, 750)),
    (F64, (140, 380)), (F64, (141, 373)), (F64, (268, 130)), (F32, (269, 750)),
]


@pytest.mark.parametrize("dtype,shape", FUSED_LIM_SHAPES)
def test_fused_limiter_adjoint_matches_two_pass(dtype, shape):
    say(f"fused limiter adjoint dtype={dtype} shape={shape}")
    inp = inputs(J, dtype, shape, 5)
    T, loss = 6, DOT_W
    a = gpu_vjp(J, inp, T, loss, 2 * inp["x0"].nbytes, adst.ADST_SCHED_BINOMIAL, lim=LIM[J])
    b = gpu_vjp(J, inp, T, loss, 2 * inp["x0"].nbytes, adst.ADST_SCHED_BINOMIAL, lim=LIM[J],
                want_dparams=True)
    assert np.array_equal(a["dx0"], b["dx0"]) and a["loss"] == b["loss"]
    ref = oracle.vjp(J, inp["x0"], steps=T, loss=loss, aux=inp["aux"], lim=LIM[J])
    assert rel(a["dx0"], ref[0]) <= TOL[dtype]


def test_fused_limiter_adjoint_full_grid():
    """4096^2 f64, the benchmark's limiter leg: the one-pass masked adjoint
    and the two-pass one give the same bits."""
    say("fused limiter adjoint 4096x4096 T=8")
    inp = inputs(J, F64, (4096, 4096), 6)
    S = inp["x0"].nbytes
    a = gpu_vjp(J, inp, 8, HALF_SQ, 2 * S, adst.ADST_SCHED_BINOMIAL, lim=(0.3, 0.7),
                want_xT=False)
    b = gpu_vjp(J, inp, 8, HALF_SQ, 2 * S, adst.ADST_SCHED_BINOMIAL, lim=(0.3, 0.7),
                want_xT=False, want_dparams=True)
    assert np.array_equal(a["dx0"], b["dx0"]) and a["loss"] == b["loss"]


# The Allen-Cahn adjoint applies the branch mask as it reads g (the step's
# value re-evaluated at every cell it reads: its own, the six neighbours'
# and the LDS ring's); with the constants' gradients it keeps the separate
# mask pass. Shapes put the edges of its 64 x 16 x 256 tiles (64 x 8 x 32
# for the constants' variant), ragged tails in every axis and one-plane and
# one-row grids against the ring.
FUSED_LIM_AC_SHAPES = [
    (F64, (39, 45, 67)), (F64, (33, 9, 65)), (F64, (1, 20, 70)), (F64, (40, 1, 3)),
    (F64, (3, 4, 5)), (F32, (17, 33, 65)), (F32, (64, 16, 128)),
    (F64, (64, 28, 112)), (F64, (65, 29, 113)), (F64, (130, 15, 57)), (F32, (129, 14, 56)),
    (F64, (33, 17, 64)), (F64, (31, 32, 65)),
    (F64, (256, 6, 64)), (F64, (258, 9, 40)), (F32, (513, 5, 33)),
]


@pytest.mark.parametrize("dtype,shape", FUSED_LIM_AC_SHAPES)
def test_fused_limiter_allencahn_matches_two_pass(dtype, shape):
    say(f"fused limiter allen-cahn dtype={dtype} shape={shape}")
    inp = inputs(AC, dtype, shape, 7)
    T, loss = 7, DOT_W
    a = gpu_vjp(AC, inp, T, loss, 2 * inp["x0"].nbytes, adst.ADST_SCHED_BINOMIAL, lim=LIM[AC])
    b = gpu_vjp(AC, inp, T, loss, 2 * inp["x0"].nbytes, adst.ADST_SCHED_BINOMIAL, lim=LIM[AC],
                want_dparams=True)
    assert np.array_equal(a["dx0"], b["dx0"]) and a["loss"] == b["loss"]
    ref = oracle.vjp(AC, inp["x0"], steps=T, loss=loss, aux=inp["aux"], lim=LIM[AC])
    assert rel(a["dx0"], ref[0]) <= TOL[dtype]


def test_fused_limiter_allencahn_full_grid():
    """512^3 f64, the benchmark's Allen-Cahn limiter leg: the masked adjoint
    (streaming stores at this size) and the two-pass one give the same bits."""
    say("fused limiter allen-cahn 512^3 T=4")
    inp = inputs(AC, F64, (512, 512, 512), 8)
    S = inp["x0"].nbytes
    a = gpu_vjp(AC, inp, 4, DOT_W, 2 * S, adst.ADST_SCHED_BINOMIAL, lim=(-0.9, 0.9),
                want_xT=False)
    b = gpu_vjp(AC, inp, 4, DOT_W, 2 * S, adst.ADST_SCHED_BINOMIAL, lim=(-0.9, 0.9),
                want_xT=False, want_dparams=True)
    assert np.array_equal(a["dx0"], b["dx0"]) and a["loss"] == b["loss"]
