"""Temporal blocking of the Allen-Cahn kind, up to three forward steps per
launch, against one launch per step and against the oracle (needs an MI355X).

A launch of n steps has each workgroup evaluate the n steps on a region of
each plane while marching in z: two steps on 64 x 16 regions (four waves of
four rows) over 32-plane chunks with 56 x 14 output tiles, three steps on
64 x 32 regions (sixteen waves of two rows) over 64-plane chunks with
60 x 28 output tiles. The shapes put grids narrower than one tile,
exact tiles, tiles plus one and ragged tails against these sizes in every
axis, and runs of 1 to 3 planes. Step counts cover one launch of each depth
and runs that split into full launches and a shorter remainder.

Bars: forward states bit-identical to the single steps and to the oracle;
the gradient of a binomial plan (whose recomputation runs take fused
launches) bit-identical to the single steps and within relative L2 1e-12
(fp64) / 1e-5 (fp32) of the oracle.
"""
import numpy as np
import pytest

import oracle
import paper_2509_02197_amd as adst
from tests.gpu_util import NP_DTYPE, TOL, dev, gpu_vjp, rel, say

pytestmark = pytest.mark.gpu

AC = adst.ADST_ALLENCAHN3D7
F64, F32 = adst.ADST_F64, adst.ADST_F32
STEPS = (2, 3, 4, 5, 6, 7, 8, 11)

# (dtype, numpy shape (nz, ny, nx))
SHAPES = [
    (F64, (1, 1, 1)), (F64, (3, 4, 5)), (F64, (2, 30, 70)), (F64, (33, 12, 60)),
    (F64, (32, 18, 58)), (F64, (33, 19, 59)), (F64, (65, 14, 62)), (F64, (40, 37, 130)),
    (F64, (70, 15, 63)), (F64, (5, 40, 200)), (F64, (64, 13, 61)),
    (F32, (17, 33, 130)), (F32, (33, 19, 117)), (F32, (4, 4, 4)),
    (F64, (65, 28, 60)), (F64, (64, 29, 121)), (F64, (9, 57, 120)), (F32, (66, 56, 61)),
]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    adst.lib()


def _x0(dtype, shape, seed):
    r = np.random.Generator(np.random.PCG64(seed))
    return r.uniform(-1.0, 1.0, shape).astype(NP_DTYPE[dtype])


@pytest.mark.parametrize("dtype,shape", SHAPES)
def test_fused_forward_bitwise(dtype, shape):
    x0 = _x0(dtype, shape, 41)
    xd = dev(x0)
    for T in STEPS:
        say(f"allen-cahn fused forward dtype={dtype} shape={shape} T={T}")
        a = adst.forward(AC, xd, None, T).cpu().numpy()
        b = adst.forward(AC, xd, None, T, flags=adst.ADST_NO_FUSE).cpu().numpy()
        assert np.array_equal(a, b), T
        assert np.array_equal(a, oracle.forward(AC, x0, steps=T)), T


@pytest.mark.parametrize("dtype,shape", [(F64, (33, 19, 59)), (F64, (40, 37, 130)),
                                         (F32, (33, 19, 117))])
def test_fused_recomputation_gradient(dtype, shape):
    r = np.random.Generator(np.random.PCG64(42))
    inp = {"x0": _x0(dtype, shape, 43),
           "aux": r.standard_normal(shape).astype(NP_DTYPE[dtype])}
    T = 23
    budget = 3 * inp["x0"].nbytes
    say(f"allen-cahn fused recompute dtype={dtype} shape={shape} T={T}")
    a = gpu_vjp(AC, inp, T, adst.ADST_LOSS_DOT_W, budget, adst.ADST_SCHED_BINOMIAL)
    b = gpu_vjp(AC, inp, T, adst.ADST_LOSS_DOT_W, budget, adst.ADST_SCHED_BINOMIAL,
                flags=adst.ADST_NO_FUSE)
    assert a["info"]["fwd_launches"] < b["info"]["fwd_launches"] == b["info"]["fwd_steps_total"]
    assert np.array_equal(a["dx0"], b["dx0"]) and np.array_equal(a["xT"], b["xT"])
    assert a["loss"] == b["loss"]
    dx0, _, xT, _ = oracle.vjp(AC, inp["x0"], steps=T, loss=adst.ADST_LOSS_DOT_W, aux=inp["aux"])
    assert np.array_equal(a["xT"], xT)
    e = rel(a["dx0"], dx0)
    assert e <= TOL[dtype], e
