"""The caller's inputs are read-only (x0, K, loss_aux): after adst_vjp they
hold the bits they held before, whatever the loss, schedule, limiter or
gradient set. For the dot-product and explicit-seed losses the first adjoint
step reads g_T from loss_aux itself, so those two losses must give the same
bits as each other, and the same gradient as the oracle (needs an MI355X)."""
import numpy as np
import pytest

import oracle
import paper_2509_02197_amd as adst
from tests.gpu_util import NP_DTYPE, TOL, rel, say

pytestmark = pytest.mark.gpu

J, AC, VD, GS = (adst.ADST_JACOBI2D5, adst.ADST_ALLENCAHN3D7, adst.ADST_VARDIFF2D9,
                 adst.ADST_GAUSSSEIDEL2D5)
F64, F32 = adst.ADST_F64, adst.ADST_F32
HALF_SQ, DOT_W, DIFF, SEED = (adst.ADST_LOSS_HALF_SQ, adst.ADST_LOSS_DOT_W,
                              adst.ADST_LOSS_HALF_SQ_DIFF, adst.ADST_LOSS_SEED)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    adst.lib()


def _inputs(kind, dtype, shape, seed):
    r = np.random.Generator(np.random.PCG64(seed))
    dt = NP_DTYPE[dtype]
    lo = -1.0 if kind == AC else 0.0
    return {"x0": r.uniform(lo, 1, shape).astype(dt),
            "K": r.uniform(0.5, 1.5, shape).astype(dt) if kind == VD else None,
            "aux": r.standard_normal(shape).astype(dt)}


# kind, dtype, shape, T, slots (None: store-all), sched, want_dK, flags, limiter, dparams
CASES = [
    (AC, F64, (9, 20, 70), 11, 3, adst.ADST_SCHED_BINOMIAL, False, 0, None, False),
    (AC, F32, (5, 17, 64), 7, 2, adst.ADST_SCHED_UNIFORM, False, 0, None, False),
    (AC, F64, (6, 19, 66), 9, 2, adst.ADST_SCHED_BINOMIAL, False, 0, (-0.45, 0.5), False),
    (AC, F64, (6, 19, 66), 9, 2, adst.ADST_SCHED_BINOMIAL, False, 0, None, True),
    (J, F64, (70, 130), 13, None, adst.ADST_SCHED_AUTO, False, 0, None, False),
    (J, F64, (70, 130), 13, 3, adst.ADST_SCHED_BINOMIAL, False, adst.ADST_FORCE_TAPE, None, False),
    (J, F64, (70, 130), 8, 3, adst.ADST_SCHED_BINOMIAL, False, 0, (0.35, 0.65), False),
    (VD, F32, (65, 260), 9, 3, adst.ADST_SCHED_BINOMIAL, True, 0, None, False),
    (VD, F64, (33, 70), 6, 2, adst.ADST_SCHED_BINOMIAL, True, 0, (0.3, 0.7), True),
    (GS, F64, (40, 50), 5, None, adst.ADST_SCHED_AUTO, False, 0, None, False),
]


def _run(case, loss, inp):
    import torch
    kind, dtype, shape, T, slots, sched, want_dK, flags, lim, dp = case
    x0 = torch.from_numpy(inp["x0"]).cuda()
    K = None if inp["K"] is None else torch.from_numpy(inp["K"]).cuda()
    aux = torch.from_numpy(inp["aux"]).cuda()
    before = [t.clone() for t in (x0, K, aux) if t is not None]
    budget = None if slots is None else slots * inp["x0"].nbytes
    out = adst.vjp(kind, x0, K, T, loss, aux, budget, sched, want_dK, flags=flags, lim=lim,
                   want_dparams=dp)
    torch.cuda.synchronize()
    after = [t for t in (x0, K, aux) if t is not None]
    for b, a in zip(before, after):
        assert torch.equal(b, a), "an input changed"
    return {k: (v.detach().cpu().numpy() if torch.is_tensor(v) else v)
            for k, v in out.items() if k in ("dx0", "dK", "xT", "loss", "dparams")}


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"k{c[0]}-{c[2]}-T{c[3]}-l{c[8]}-dp{c[9]}")
def test_inputs_stay_untouched(case):
    kind, dtype, shape, T = case[:4]
    say(f"inputs kind={kind} shape={shape} T={T} case={case[4:]}")
    inp = _inputs(kind, dtype, shape, 77)
    res = {loss: _run(case, loss, inp) for loss in (HALF_SQ, DOT_W, DIFF, SEED)}
    # g_T = loss_aux and L = sum aux * x_T for both: the same bits
    for k in ("dx0", "dK", "xT", "loss", "dparams"):
        a, b = res[DOT_W][k], res[SEED][k]
        assert (a is None and b is None) or np.array_equal(a, b), k
    # the dot-product loss against the oracle
    want_dK = case[6]
    ref = oracle.vjp(kind, inp["x0"], inp["K"], steps=T, loss=DOT_W, aux=inp["aux"],
                     want_dK=want_dK, lim=case[8])
    assert rel(res[DOT_W]["dx0"], ref[0]) <= TOL[dtype]
