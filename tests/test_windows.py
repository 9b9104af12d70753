"""The windowed oracle reproduces the full-grid oracle exactly (CPU)."""
import numpy as np
import pytest

import oracle
from oracle import ALLENCAHN3D7, DOT_W, HALF_SQ, HALF_SQ_DIFF, JACOBI2D5, VARDIFF2D9
from tests.windows import sample_points, window_forward, window_vjp


def _inputs(shape, kind, seed, dtype):
    r = np.random.Generator(np.random.PCG64(seed))
    lo = -1.0 if kind == ALLENCAHN3D7 else 0.0
    return {"x0": r.uniform(lo, 1, shape).astype(dtype),
            "K": r.uniform(0.5, 1.5, shape).astype(dtype) if kind == VARDIFF2D9 else None,
            "aux": r.standard_normal(shape).astype(dtype)}


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
@pytest.mark.parametrize("kind,shape,T,loss,dK", [
    (JACOBI2D5, (61, 70), 5, HALF_SQ, False),
    (ALLENCAHN3D7, (23, 21, 25), 3, DOT_W, False),
    (VARDIFF2D9, (50, 47), 6, HALF_SQ_DIFF, True),
])
def test_window_equals_full_oracle(kind, shape, T, loss, dK, dtype):
    # exact in either precision: the window holds the same operations in the
    # same order for the sampled point (the full-size fp32 workload relies on
    # it as the fp64 ones do)
    inp = _inputs(shape, kind, 3, dtype)
    full_dx0, full_dK, full_xT, _ = oracle.vjp(kind, inp["x0"], K=inp["K"], steps=T, loss=loss,
                                              aux=inp["aux"], want_dK=dK)
    for p in sample_points(shape, 16, 4):
        d, k = window_vjp(kind, inp, T, p, loss, dK)
        assert d == full_dx0[p], p
        if dK:
            assert k == full_dK[p], p
        assert window_forward(kind, inp, T, p) == full_xT[p], p
