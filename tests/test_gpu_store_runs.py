"""Store-through forward launches (needs an MI355X): a run of chained single
forward steps whose every state is kept (the store-all runs of the binomial
schedule, and the whole store-all schedule) is taken by one launch that
writes each state of the run, up to three steps (Allen-Cahn) or two
(variable coefficients) per launch.

The shapes put grids narrower than one tile, exact tiles, tiles plus one and
ragged tails against the fused kernels' output tiles (Allen-Cahn 56 x 14 over
32 planes and 60 x 28 over 64 planes; variable coefficients 252 x 8), and
one-plane and one-row grids. Plans: store-all (one chain through every
step) and binomial plans whose budgets leave store-all runs of several
lengths.

Bars: dx0, dK, x_T and the loss bit-identical to one launch per step
(ADST_NO_FUSE) and to every other schedule; within relative L2 1e-12 (fp64)
/ 1e-5 (fp32) of the oracle; the plan's forward launch count below the
unfused one.
"""
import numpy as np
import pytest

import oracle
import paper_2509_02197_amd as adst
from tests.gpu_util import NP_DTYPE, TOL, gpu_vjp, rel, say

pytestmark = pytest.mark.gpu

AC, VD = adst.ADST_ALLENCAHN3D7, adst.ADST_VARDIFF2D9
F64, F32 = adst.ADST_F64, adst.ADST_F32

CASES = [
    (AC, F64, (1, 1, 1)), (AC, F64, (3, 15, 63)), (AC, F64, (33, 14, 62)),
    (AC, F64, (65, 13, 61)), (AC, F64, (40, 29, 125)), (AC, F32, (17, 33, 130)),
    (AC, F64, (64, 28, 60)), (AC, F64, (66, 57, 113)),
    (VD, F32, (1, 7)), (VD, F32, (9, 253)), (VD, F32, (17, 504)), (VD, F32, (33, 1000)),
    (VD, F64, (25, 505)), (VD, F64, (12, 3)),
]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    adst.lib()


def _inputs(kind, dtype, shape, seed):
    r = np.random.Generator(np.random.PCG64(seed))
    t = NP_DTYPE[dtype]
    if kind == AC:
        return {"x0": r.uniform(-1.0, 1.0, shape).astype(t),
                "aux": r.standard_normal(shape).astype(t)}
    return {"x0": r.uniform(0.0, 1.0, shape).astype(t),
            "K": r.uniform(0.5, 1.5, shape).astype(t),
            "aux": r.uniform(0.0, 1.0, shape).astype(t)}


@pytest.mark.parametrize("kind,dtype,shape", CASES)
def test_store_runs_bitwise_and_oracle(kind, dtype, shape):
    inp = _inputs(kind, dtype, shape, 61)
    loss = adst.ADST_LOSS_DOT_W if kind == AC else adst.ADST_LOSS_HALF_SQ_DIFF
    want_dK = kind == VD
    T = 13
    S = inp["x0"].nbytes
    dx0, dK, xT, L = oracle.vjp(kind, inp["x0"], K=inp.get("K"), steps=T, loss=loss,
                                aux=inp["aux"], want_dK=want_dK)
    ref = None
    for sched, slots in ((adst.ADST_SCHED_STORE_ALL, T), (adst.ADST_SCHED_BINOMIAL, 5),
                         (adst.ADST_SCHED_BINOMIAL, 3)):
        say(f"store runs kind={kind} dtype={dtype} shape={shape} sched={sched} slots={slots}")
        a = gpu_vjp(kind, inp, T, loss, slots * S, sched, want_dK=want_dK)
        b = gpu_vjp(kind, inp, T, loss, slots * S, sched, want_dK=want_dK,
                    flags=adst.ADST_NO_FUSE)
        assert a["info"]["fwd_kernels"] < b["info"]["fwd_kernels"], sched
        assert a["info"]["fwd_alg_bytes"] < b["info"]["fwd_alg_bytes"], sched
        for k in ("dx0", "xT") + (("dK",) if want_dK else ()):
            assert np.array_equal(a[k], b[k]), (sched, k)
        assert a["loss"] == b["loss"]
        if ref is None:
            ref = a
            assert np.array_equal(a["xT"], xT)
            assert rel(a["dx0"], dx0) <= TOL[dtype]
            if want_dK:
                assert rel(a["dK"], dK) <= TOL[dtype]
            assert abs(a["loss"] - L) <= TOL[dtype] * max(abs(L), 1.0)
        else:
            for k in ("dx0", "xT") + (("dK",) if want_dK else ()):
                assert np.array_equal(a[k], ref[k]), (sched, k)


@pytest.mark.parametrize("kind,dtype,shape,T,flags,dparams", [
    (AC, F64, (5, 15, 63), 1, 0, False), (AC, F64, (5, 15, 63), 2, 0, False),
    (AC, F64, (5, 15, 63), 3, 0, False), (AC, F64, (5, 15, 63), 4, 0, False),
    (AC, F64, (33, 14, 62), 7, 0, True),
    (VD, F32, (9, 253), 3, 0, False), (VD, F32, (9, 253), 6, 0, True),
    (VD, F32, (17, 504), 5, adst.ADST_FORCE_TAPE, False),
])
def test_store_runs_short_forced_and_dparams(kind, dtype, shape, T, flags, dparams):
    # runs of every length up to the depth, the constants' gradients (whose
    # adjoint reads the stored states) and a forced tape for the linear
    # variable-coefficient step without dK: all bit-identical to one launch
    # per step
    inp = _inputs(kind, dtype, shape, 62)
    loss = adst.ADST_LOSS_DOT_W if kind == AC else adst.ADST_LOSS_HALF_SQ_DIFF
    want_dK = kind == VD and not flags
    S = inp["x0"].nbytes
    say(f"store runs short kind={kind} dtype={dtype} shape={shape} T={T} flags={flags} dp={dparams}")
    kw = dict(want_dK=want_dK, want_dparams=dparams)
    a = gpu_vjp(kind, inp, T, loss, T * S, adst.ADST_SCHED_STORE_ALL, flags=flags, **kw)
    b = gpu_vjp(kind, inp, T, loss, T * S, adst.ADST_SCHED_STORE_ALL,
                flags=flags | adst.ADST_NO_FUSE, **kw)
    if T >= 2:
        assert a["info"]["fwd_kernels"] < b["info"]["fwd_kernels"]
    keys = ("dx0", "xT") + (("dK",) if want_dK else ()) + (("dparams",) if dparams else ())
    for k in keys:
        assert np.array_equal(a[k], b[k]), k
    assert a["loss"] == b["loss"]
    dx0, _, xT, _ = oracle.vjp(kind, inp["x0"], K=inp.get("K"), steps=T, loss=loss,
                               aux=inp["aux"], want_dK=want_dK)
    assert np.array_equal(a["xT"], xT)
    assert rel(a["dx0"], dx0) <= TOL[dtype]
