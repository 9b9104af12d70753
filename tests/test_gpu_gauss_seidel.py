"""The in-place Gauss-Seidel kind on the GPU vs the CPU oracle, through the
C-ABI (needs an MI355X).

Bars as for the other kinds: forward states bit-identical to the oracle
(any order that updates a point after its W and S neighbours and before its
E and N neighbours gives the same bits, so the wavefront evaluation must
reproduce the row-major sweep exactly); gradients and loss within relative
L2 1e-12 (fp64) / 1e-5 (fp32); the pipelined plan and every forced-tape
schedule bit-identical to each other.

Full size (4096^2, 100 sweeps): the forward state against the oracle's whole
sweep, and the gradient through the adjoint identity <dx0, v> = <g, J v>,
J v being the (bit-pinned) forward map of v: the map x0 -> x_T is linear.
At the paper's case-study size (400^2, 100 sweeps) the oracle's whole
gradient is compared.
"""
import numpy as np
import pytest

import oracle
import paper_2509_02197_amd as adst
from paper_2509_02197_amd.workloads import WORKLOADS, make_inputs
from tests.gpu_util import NP_DTYPE, TOL, dev, gpu_vjp, rel, say

pytestmark = pytest.mark.gpu

GS = adst.ADST_GAUSSSEIDEL2D5
F64, F32 = adst.ADST_F64, adst.ADST_F32
HALF_SQ, DOT_W, DIFF, SEED = (adst.ADST_LOSS_HALF_SQ, adst.ADST_LOSS_DOT_W,
                              adst.ADST_LOSS_HALF_SQ_DIFF, adst.ADST_LOSS_SEED)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    adst.lib()


def inputs(dtype, shape, seed):
    r = np.random.Generator(np.random.PCG64(seed))
    dt = NP_DTYPE[dtype]
    return {"x0": r.uniform(0, 1, shape).astype(dt), "K": None,
            "aux": r.standard_normal(shape).astype(dt)}


def check(dtype, inp, T, loss, g):
    dx0, _, xT, L = oracle.vjp(GS, inp["x0"], steps=T, loss=loss, aux=inp["aux"])
    tol = TOL[dtype]
    if g["xT"] is not None:
        assert np.array_equal(g["xT"], xT), "forward state differs from the oracle"
    e = rel(g["dx0"], dx0)
    say(f"  dx0 rel L2 {e:.3e}")
    assert e <= tol, f"dx0 rel L2 {e:.3e}"
    assert abs(g["loss"] - L) <= tol * max(abs(L), 1e-300), (g["loss"], L)


# shapes as (ny, nx): several tiles in both directions, ragged edges (nx not
# a multiple of the 16-byte block), thin grids, grids without interior points
FORWARD_CASES = [
    (F64, (64, 64), 10), (F64, (333, 517), 7), (F32, (130, 70), 5), (F64, (1, 1), 3),
    (F64, (2, 9), 4), (F64, (9, 2), 4), (F64, (3, 3), 2), (F64, (5, 1001), 6),
    (F64, (1001, 5), 6), (F32, (257, 301), 9), (F64, (400, 400), 100), (F32, (64, 8), 40),
    (F64, (129, 130), 31),
]


@pytest.mark.parametrize("dtype,shape,T", FORWARD_CASES)
def test_forward_bitwise(dtype, shape, T):
    say(f"gs forward dtype={dtype} shape={shape} T={T}")
    inp = inputs(dtype, shape, 1)
    g = adst.forward(GS, dev(inp["x0"]), None, T).cpu().numpy()
    ref = oracle.forward(GS, inp["x0"], steps=T)
    assert np.array_equal(g, ref)


VJP_CASES = [
    (F64, (64, 64), 10, HALF_SQ), (F64, (333, 517), 7, DIFF), (F32, (130, 70), 5, DIFF),
    (F64, (1, 1), 3, HALF_SQ), (F64, (2, 9), 4, DOT_W), (F64, (9, 2), 4, SEED),
    (F64, (3, 3), 1, HALF_SQ), (F64, (4, 4), 2, SEED), (F64, (5, 1001), 6, DOT_W),
    (F64, (1001, 5), 6, HALF_SQ), (F32, (257, 301), 9, HALF_SQ), (F64, (129, 130), 31, SEED),
    (F64, (70, 66), 1, DIFF),
]


@pytest.mark.parametrize("dtype,shape,T,loss", VJP_CASES)
def test_vjp_matches_oracle(dtype, shape, T, loss):
    say(f"gs vjp dtype={dtype} shape={shape} T={T} loss={loss}")
    inp = inputs(dtype, shape, 2)
    g = gpu_vjp(GS, inp, T, loss)
    assert g["info"]["fwd_launches"] == 1 and g["info"]["adj_launches"] == 1
    check(dtype, inp, T, loss, g)


@pytest.mark.parametrize("dtype,shape,T,loss", [(F64, (90, 130), 7, DIFF), (F32, (77, 300), 5,
                                                                             HALF_SQ)])
def test_without_xT_output_runs_in_dx0(dtype, shape, T, loss):
    """With no xT buffer the forward sweeps land in dx0 and the seed and the
    reverse sweeps run there in place: same bits."""
    inp = inputs(dtype, shape, 3)
    a = gpu_vjp(GS, inp, T, loss)
    b = gpu_vjp(GS, inp, T, loss, want_xT=False)
    assert b["xT"] is None
    assert np.array_equal(a["dx0"], b["dx0"]) and a["loss"] == b["loss"]


@pytest.mark.parametrize("dtype,shape,T,loss", [(F64, (90, 130), 13, HALF_SQ),
                                                (F32, (66, 257), 9, DIFF),
                                                (F64, (7, 5), 6, DOT_W)])
def test_forced_tape_schedules_give_the_pipelined_bits(dtype, shape, T, loss):
    """Forcing a tape runs one sweep (forward) or one reverse sweep per
    action, with recomputation from checkpoints; the per-point arithmetic is
    the same as in the pipelined runs, so every schedule gives the same bits."""
    say(f"gs schedules dtype={dtype} shape={shape} T={T}")
    inp = inputs(dtype, shape, 4)
    S = inp["x0"].nbytes
    ref = gpu_vjp(GS, inp, T, loss)
    check(dtype, inp, T, loss, ref)
    runs = [("store-all", None, adst.ADST_SCHED_STORE_ALL), ("binomial0", 0, adst.ADST_SCHED_BINOMIAL),
            ("binomial2", 2 * S, adst.ADST_SCHED_BINOMIAL), ("uniform3", 3 * S, adst.ADST_SCHED_UNIFORM)]
    for name, budget, sched in runs:
        g = gpu_vjp(GS, inp, T, loss, budget, sched, flags=adst.ADST_FORCE_TAPE)
        assert g["info"]["adj_launches"] == T
        if name != "store-all" and T > 2:
            assert g["info"]["recompute_steps"] > 0
        for key in ("dx0", "xT"):
            assert np.array_equal(g[key], ref[key]), (name, key)
        assert g["loss"] == ref["loss"], name


def test_zero_steps():
    inp = inputs(F64, (20, 30), 5)
    g = gpu_vjp(GS, inp, 0, DIFF)
    assert np.array_equal(g["dx0"], inp["x0"] - inp["aux"])
    assert np.array_equal(g["xT"], inp["x0"])


def test_trace_and_kernel_counts():
    inp = inputs(F64, (200, 300), 6)
    g = gpu_vjp(GS, inp, 9, HALF_SQ, flags=adst.ADST_TRACE)
    info = g["info"]
    assert info["ms_fwd_sweep"] > 0 and info["ms_adj"] > 0 and info["ms_seed"] > 0
    assert info["fwd_kernels"] > 9 and info["adj_kernels"] > info["fwd_kernels"]
    check(F64, inp, 9, HALF_SQ, g)


def test_repeat_calls_same_bits():
    inp = inputs(F64, (150, 170), 7)
    a = gpu_vjp(GS, inp, 11, SEED)
    b = gpu_vjp(GS, inp, 11, SEED)
    assert np.array_equal(a["dx0"], b["dx0"]) and np.array_equal(a["xT"], b["xT"])


def test_paper_case_study_size_whole_gradient():
    """The Seidel2d case study's size (N = 400, 100 time steps): the oracle's
    whole store-all gradient."""
    w = WORKLOADS["gaussseidel2d5_f64_400x400_T100"]
    say(f"fullsize {w.name}")
    inp = make_inputs(w)
    g = gpu_vjp(w.kind, inp, w.steps, w.loss, w.budget_bytes, w.sched)
    assert g["info"]["slots"] == 0 and g["info"]["recompute_steps"] == 0
    check(w.dtype, inp, w.steps, w.loss, g)


def test_4096_T100_forward_and_adjoint_identity():
    w = WORKLOADS["gaussseidel2d5_f64_4096x4096_T100"]
    say(f"fullsize {w.name}")
    inp = make_inputs(w)
    g = gpu_vjp(w.kind, inp, w.steps, w.loss, w.budget_bytes, w.sched)
    assert g["info"]["workspace_bytes"] == 16384
    say("  oracle forward over the whole grid")
    xT = oracle.forward(w.kind, inp["x0"], steps=w.steps)
    assert np.array_equal(g["xT"], xT)
    L = 0.5 * np.sum(xT * xT)
    assert abs(g["loss"] - L) <= 1e-12 * L
    # <dx0, v> = <x_T, J v> for the loss 0.5 |x_T|^2, J v the forward map of v
    r = np.random.Generator(np.random.PCG64(11))
    for k in range(2):
        v = r.standard_normal(w.shape)
        Jv = adst.forward(w.kind, dev(v), None, w.steps).cpu().numpy()
        lhs, rhs = float(np.sum(g["dx0"] * v)), float(np.sum(xT * Jv))
        say(f"  direction {k}: <dx0, v> = {lhs:.15e}, <x_T, J v> = {rhs:.15e}")
        assert abs(lhs - rhs) <= 1e-12 * max(abs(rhs), 1e-300)
