"""Temporal blocking of the variable-coefficient kind, two forward steps per
launch, against one launch per step and against the oracle (needs an
MI355X).

A fused launch has each 256-thread workgroup own 252 output columns and 8
rows: the first step runs on the tile plus a one-cell ring, the second on
the tile. The shapes put grids narrower and shorter than a tile, exact
tiles, tiles plus one and ragged tails against 252 columns and 8 rows, rows
whose length is not a multiple of the 16-byte vector (element loads) and
one-row and one-column grids. Step counts cover one fused launch, a fused
launch after a single step, and longer runs.

Bars: forward states bit-identical to the single steps and to the oracle;
the gradients (dx0 and dK) of a binomial plan, whose recomputation runs take
fused launches, bit-identical to the single steps and within relative L2
1e-12 (fp64) / 1e-5 (fp32) of the oracle.
"""
import numpy as np
import pytest

import oracle
import paper_2509_02197_amd as adst
from tests.gpu_util import NP_DTYPE, TOL, dev, gpu_vjp, rel, say

pytestmark = pytest.mark.gpu

VD = adst.ADST_VARDIFF2D9
F64, F32 = adst.ADST_F64, adst.ADST_F32
STEPS = (2, 3, 4, 7, 10)

# (dtype, numpy shape (ny, nx))
SHAPES = [
    (F32, (1, 1)), (F32, (1, 7)), (F32, (7, 1)), (F32, (3, 3)), (F32, (8, 252)),
    (F32, (9, 253)), (F32, (17, 504)), (F32, (16, 505)), (F32, (40, 256)), (F32, (33, 1000)),
    (F32, (5, 250)), (F32, (70, 129)),
    (F64, (8, 252)), (F64, (9, 254)), (F64, (25, 505)), (F64, (12, 3)),
]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    adst.lib()


def _inputs(dtype, shape, seed):
    r = np.random.Generator(np.random.PCG64(seed))
    t = NP_DTYPE[dtype]
    return {"x0": r.uniform(0.0, 1.0, shape).astype(t),
            "K": r.uniform(0.5, 1.5, shape).astype(t),
            "aux": r.uniform(0.0, 1.0, shape).astype(t)}


@pytest.mark.parametrize("dtype,shape", SHAPES)
def test_fused_forward_bitwise(dtype, shape):
    inp = _inputs(dtype, shape, 51)
    xd, kd = dev(inp["x0"]), dev(inp["K"])
    for T in STEPS:
        say(f"vardiff fused forward dtype={dtype} shape={shape} T={T}")
        a = adst.forward(VD, xd, kd, T).cpu().numpy()
        b = adst.forward(VD, xd, kd, T, flags=adst.ADST_NO_FUSE).cpu().numpy()
        assert np.array_equal(a, b), T
        assert np.array_equal(a, oracle.forward(VD, inp["x0"], K=inp["K"], steps=T)), T


@pytest.mark.parametrize("dtype,shape", [(F32, (33, 505)), (F64, (25, 300)), (F32, (9, 7))])
def test_fused_recomputation_gradient(dtype, shape):
    inp = _inputs(dtype, shape, 52)
    T = 21
    budget = 3 * inp["x0"].nbytes
    say(f"vardiff fused recompute dtype={dtype} shape={shape} T={T}")
    kw = dict(budget=budget, sched=adst.ADST_SCHED_BINOMIAL, want_dK=True)
    a = gpu_vjp(VD, inp, T, adst.ADST_LOSS_HALF_SQ_DIFF, **kw)
    b = gpu_vjp(VD, inp, T, adst.ADST_LOSS_HALF_SQ_DIFF, flags=adst.ADST_NO_FUSE, **kw)
    assert a["info"]["fwd_launches"] < b["info"]["fwd_launches"] == b["info"]["fwd_steps_total"]
    for key in ("dx0", "dK", "xT"):
        assert np.array_equal(a[key], b[key]), key
    assert a["loss"] == b["loss"]
    dx0, dK, xT, _ = oracle.vjp(VD, inp["x0"], K=inp["K"], steps=T,
                                loss=adst.ADST_LOSS_HALF_SQ_DIFF, aux=inp["aux"], want_dK=True)
    assert np.array_equal(a["xT"], xT)
    assert rel(a["dx0"], dx0) <= TOL[dtype]
    assert rel(a["dK"], dK) <= TOL[dtype]
