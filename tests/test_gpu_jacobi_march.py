"""Temporal blocking of the Jacobi kind, up to six steps per launch, against
one launch per step and against the oracle (needs an MI355X).

A launch of n >= 3 steps marches one wave down a strip of columns with the n
time levels in registers; strips overlap by whole 16-byte vectors of halo
and each chunk of rows recomputes n rows above and below itself. The shapes
put strip edges, chunk edges and the vector width against the grid's fixed
ring: widths around one strip (120 or 116 output columns in fp64, 248 or 240
in fp32, for 3-4 and 5-6 steps), heights around the row chunks (6 rows at
each end of a strip; between them 12-row chunks in the first and last strip
and 48-row chunks in the others, so heights 60/61 over three or more strips
put a chunk edge on the last rows, and 54/55 one 12-row edge-strip chunk
boundary), widths that are not a multiple of the vector (element loads and
stores) and grids narrower than the halo.
Step counts cover one launch of each depth and runs that split into several
launches with a shorter remainder.

Bars: forward states bit-identical to the single steps and to the oracle;
gradients bit-identical to the single steps and within relative L2 1e-12
(fp64) / 1e-5 (fp32) of the oracle.
"""
import numpy as np
import pytest

import oracle
import paper_2509_02197_amd as adst
from tests.gpu_util import NP_DTYPE, TOL, dev, gpu_vjp, rel, say

pytestmark = pytest.mark.gpu

J = adst.ADST_JACOBI2D5
F64, F32 = adst.ADST_F64, adst.ADST_F32
STEPS = (3, 4, 5, 6, 7, 8, 11, 13)

# (dtype, numpy shape (ny, nx))
SHAPES = [
    (F64, (1, 1)), (F64, (2, 2)), (F64, (3, 3)), (F64, (4, 5)), (F64, (13, 7)),
    (F64, (50, 120)), (F64, (49, 121)), (F64, (12, 116)), (F64, (13, 117)),
    (F64, (48, 128)), (F64, (60, 236)), (F64, (97, 240)), (F64, (25, 241)),
    (F64, (3, 1000)), (F64, (1000, 3)), (F64, (130, 4)), (F64, (61, 350)),
    (F64, (54, 370)), (F64, (55, 361)), (F64, (60, 370)), (F64, (61, 365)),
    (F32, (50, 248)), (F32, (11, 249)), (F32, (49, 240)), (F32, (24, 496)),
    (F32, (4, 4)), (F32, (7, 5)), (F32, (37, 1021)), (F32, (100, 250)),
]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    adst.lib()


def _x0(dtype, shape, seed):
    r = np.random.Generator(np.random.PCG64(seed))
    return r.uniform(0.0, 1.0, shape).astype(NP_DTYPE[dtype])


@pytest.mark.parametrize("dtype,shape", SHAPES)
def test_fused_forward_bitwise(dtype, shape):
    x0 = _x0(dtype, shape, 31)
    xd = dev(x0)
    for T in STEPS:
        say(f"march forward dtype={dtype} shape={shape} T={T}")
        a = adst.forward(J, xd, None, T).cpu().numpy()
        b = adst.forward(J, xd, None, T, flags=adst.ADST_NO_FUSE).cpu().numpy()
        assert np.array_equal(a, b), T
        assert np.array_equal(a, oracle.forward(J, x0, steps=T)), T


@pytest.mark.parametrize("dtype,shape", SHAPES)
def test_fused_adjoint_bitwise(dtype, shape):
    r = np.random.Generator(np.random.PCG64(32))
    inp = {"x0": _x0(dtype, shape, 33),
           "aux": r.standard_normal(shape).astype(NP_DTYPE[dtype])}
    for T in STEPS:
        say(f"march adjoint dtype={dtype} shape={shape} T={T}")
        a = gpu_vjp(J, inp, T, adst.ADST_LOSS_DOT_W)
        b = gpu_vjp(J, inp, T, adst.ADST_LOSS_DOT_W, flags=adst.ADST_NO_FUSE)
        depth = 6 if shape[1] > 4 else 2  # the marching adjoint needs nx > 16 bytes
        assert a["info"]["adj_launches"] == -(-T // depth)
        assert np.array_equal(a["dx0"], b["dx0"]), T
        assert np.array_equal(a["xT"], b["xT"]), T
        dx0, _, xT, _ = oracle.vjp(J, inp["x0"], steps=T, loss=adst.ADST_LOSS_DOT_W,
                                   aux=inp["aux"])
        assert np.array_equal(a["xT"], xT)
        e = rel(a["dx0"], dx0)
        assert e <= TOL[dtype], (T, e)


def test_headline_grid_fused_equals_single_steps():
    """The 4096^2 grid in the launch configuration the benchmark times: 100
    steps as sixteen 6-step launches and one 4-step launch each way, the
    same bits as 100 single-step launches."""
    import torch
    say("march 4096x4096 T=100 fused vs single")
    x0 = _x0(F64, (4096, 4096), 34)
    inp = {"x0": x0}
    a = gpu_vjp(J, inp, 100, adst.ADST_LOSS_HALF_SQ)
    assert a["info"]["fwd_launches"] == 17 and a["info"]["adj_launches"] == 17
    b = gpu_vjp(J, inp, 100, adst.ADST_LOSS_HALF_SQ, flags=adst.ADST_NO_FUSE)
    assert np.array_equal(a["xT"], b["xT"]) and np.array_equal(a["dx0"], b["dx0"])
    assert a["loss"] == b["loss"]
    # forward alone, from adst_forward's launch sequence (remainder first)
    xT = adst.forward(J, dev(x0), None, 100)
    torch.cuda.synchronize()
    assert np.array_equal(xT.cpu().numpy(), a["xT"])
