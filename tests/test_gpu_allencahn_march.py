"""The Allen-Cahn z-march kernels: recomputed forward steps (one, or a
fused run of two or three) run inside the adjoint launch that reads their
result (x_{t-1} formed on chip, never stored), against one launch per step
and against the oracle (needs an MI355X).

The plain adjoint launch owns a 64 x 16 region of every plane (64 lanes by
four waves of four rows; 64 x 32, eight waves of four rows, where a plane
holds 4 MiB or more); the fused
forward-adjoint launches own a 64 x 16 region (one or two levels) or a
64 x 32 region of eight waves (three levels), and their output tile is the
region less n-1 cells per side for n forward levels (56 columns wide for
two); all march over 64-plane chunks, and the forward steps' neighbours come
from a one-cell ring read with the region. The shapes put grids narrower
than one tile, exact tiles, tiles plus one and ragged tails against these
sizes in every axis, with one to three planes, grids with planes of over
4 MiB (one of a single plane), and planes of exactly 4 MiB and one row less,
either side of the rule that picks the region.

Bars: gradients of binomial plans (whose adjoint steps read states a
single recomputed step produced) bit-identical to one launch per step and
within relative L2 1e-12 (fp64) / 1e-5 (fp32) of the oracle; x_T bit for
bit.
"""
import numpy as np
import pytest

import oracle
import paper_2509_02197_amd as adst
from tests.gpu_util import NP_DTYPE, TOL, gpu_vjp, rel, say

pytestmark = pytest.mark.gpu

AC = adst.ADST_ALLENCAHN3D7
F64, F32 = adst.ADST_F64, adst.ADST_F32

SHAPES = [
    (F64, (1, 1, 1)), (F64, (2, 3, 70)), (F64, (3, 16, 64)), (F64, (65, 17, 65)),
    (F64, (64, 16, 128)), (F64, (9, 33, 129)), (F64, (20, 15, 63)), (F64, (5, 1, 200)),
    (F64, (7, 50, 1)), (F32, (17, 31, 97)), (F32, (66, 16, 64)),
    (F64, (4, 32, 64)), (F64, (70, 65, 66)), (F32, (3, 96, 130)),
    (F64, (3, 515, 1030)), (F32, (2, 1057, 1100)), (F64, (5, 28, 60)), (F64, (66, 29, 61)),
    # one plane of over 4 MiB; planes of exactly 4 MiB (the taller region) and
    # one row less (the 64 x 16 region)
    (F64, (1, 515, 1030)), (F64, (2, 512, 1024)), (F64, (2, 511, 1024)),
]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    adst.lib()


@pytest.mark.parametrize("dtype,shape", SHAPES)
@pytest.mark.parametrize("T,slots", [(9, 2), (23, 3), (30, 2)])
def test_forward_adjoint_launch(dtype, shape, T, slots):
    r = np.random.Generator(np.random.PCG64(44))
    inp = {"x0": r.uniform(-1.0, 1.0, shape).astype(NP_DTYPE[dtype]),
           "aux": r.standard_normal(shape).astype(NP_DTYPE[dtype])}
    budget = slots * inp["x0"].nbytes
    say(f"allen-cahn forward+adjoint dtype={dtype} shape={shape} T={T} slots={slots}")
    a = gpu_vjp(AC, inp, T, adst.ADST_LOSS_DOT_W, budget, adst.ADST_SCHED_BINOMIAL,
                flags=adst.ADST_TRACE)
    names = {k["name"]: k["launches"] for k in adst.adst_trace_kernels()}
    fused = {n: names.get(f"ac_march<fwd{n}+adj>", 0) for n in (1, 2, 3)}
    assert fused[1] > 0, names
    if T >= 23:
        assert fused[2] > 0, names  # fused runs of two steps before an adjoint step
    if T >= 30:
        assert fused[3] > 0, names
    assert a["info"]["adj_kernels"] == T
    b = gpu_vjp(AC, inp, T, adst.ADST_LOSS_DOT_W, budget, adst.ADST_SCHED_BINOMIAL,
                flags=adst.ADST_NO_FUSE)
    assert np.array_equal(a["dx0"], b["dx0"]) and np.array_equal(a["xT"], b["xT"])
    assert a["loss"] == b["loss"]
    dx0, _, xT, L = oracle.vjp(AC, inp["x0"], steps=T, loss=adst.ADST_LOSS_DOT_W,
                               aux=inp["aux"])
    assert np.array_equal(a["xT"], xT)
    e = rel(a["dx0"], dx0)
    say(f"  dx0 rel L2 {e:.3e}; fused launches {fused}")
    assert e <= TOL[dtype]
