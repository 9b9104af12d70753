"""GPU path vs the CPU oracle, through the C-ABI (needs an MI355X).

Bars: forward states bit-identical to the oracle (same evaluation order, no
contraction on either side); gradients and loss within relative L2 1e-12 in
fp64 and 1e-5 in fp32 (the adjoint sums in gather order, the oracle in
scatter order); every budget and schedule bit-identical to every other.
"""
import numpy as np
import pytest

import oracle
import paper_2509_02197_amd as adst
from paper_2509_02197_amd.workloads import WORKLOADS, make_inputs
from tests.gpu_util import NP_DTYPE, TOL, dev, gpu_vjp, rel, say

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


def inputs(kind, dtype, shape, seed=0):
    r = np.random.Generator(np.random.PCG64(seed))
    lo = -1.0 if kind == AC else 0.0
    dt = NP_DTYPE[dtype]
    return {"x0": r.uniform(lo, 1, shape).astype(dt),
            "K": r.uniform(0.5, 1.5, shape).astype(dt) if kind == VD else None,
            "aux": r.standard_normal(shape).astype(dt)}


def oracle_vjp(kind, inp, T, loss, dK):
    return oracle.vjp(kind, inp["x0"], K=inp["K"], steps=T, loss=loss, aux=inp["aux"],
                      want_dK=dK)


def check_against_oracle(kind, dtype, inp, T, loss, dK, g):
    dx0, dk, xT, L = oracle_vjp(kind, inp, T, loss, dK)
    tol = TOL[dtype]
    assert np.array_equal(g["xT"], xT), "forward state differs from the oracle"
    e = rel(g["dx0"], dx0)
    assert e <= tol, f"dx0 rel L2 {e:.3e}"
    if dK:
        e = rel(g["dK"], dk)
        assert e <= tol, f"dK rel L2 {e:.3e}"
    assert abs(g["loss"] - L) <= tol * max(abs(L), 1e-300), (g["loss"], L)


FORWARD_CASES = [
    (J, F64, (64, 64), 10), (J, F64, (333, 517), 7), (J, F32, (130, 70), 5), (J, F64, (1, 1), 3),
    (J, F64, (2, 9), 4), (AC, F64, (39, 45, 67), 6), (AC, F32, (17, 33, 65), 4),
    (AC, F64, (1, 1, 1), 5), (AC, F64, (3, 1, 200), 3), (VD, F32, (257, 300), 9),
    (VD, F64, (70, 129), 6), (VD, F32, (1, 7), 3), (VD, F64, (2, 2), 2),
]


@pytest.mark.parametrize("kind,dtype,shape,T", FORWARD_CASES)
def test_forward_bitwise(kind, dtype, shape, T):
    say(f"forward kind={kind} dtype={dtype} shape={shape} T={T}")
    inp = inputs(kind, dtype, shape, 1)
    g = adst.forward(kind, dev(inp["x0"]), dev(inp["K"]), T).cpu().numpy()
    ref = oracle.forward(kind, inp["x0"], K=inp["K"], steps=T)
    assert np.array_equal(g, ref)


VJP_CASES = [
    (J, F64, (64, 64), 10, HALF_SQ, False),
    (J, F64, (333, 517), 7, HALF_SQ, False),
    (J, F32, (130, 70), 5, DIFF, False),
    (J, F64, (1, 1), 3, HALF_SQ, False),
    (J, F64, (2, 9), 4, DOT_W, False),
    (J, F64, (3, 3), 1, HALF_SQ, False),
    (AC, F64, (39, 45, 67), 6, DOT_W, False),
    (AC, F64, (1, 1, 1), 4, SEED, False),
    (AC, F64, (3, 1, 200), 5, HALF_SQ, False),
    (AC, F32, (17, 33, 65), 4, DIFF, False),
    (VD, F32, (257, 300), 9, DIFF, True),
    (VD, F64, (70, 129), 6, DOT_W, True),
    (VD, F32, (64, 65), 5, HALF_SQ, False),
    (VD, F64, (1, 7), 3, DIFF, True),
    (VD, F64, (2, 2), 2, SEED, True),
]


@pytest.mark.parametrize("kind,dtype,shape,T,loss,dK", VJP_CASES)
def test_vjp_matches_oracle(kind, dtype, shape, T, loss, dK):
    say(f"vjp kind={kind} dtype={dtype} shape={shape} T={T} loss={loss} dK={dK}")
    inp = inputs(kind, dtype, shape, 2)
    g = gpu_vjp(kind, inp, T, loss, want_dK=dK)
    check_against_oracle(kind, dtype, inp, T, loss, dK, g)


SCHEDULE_CASES = [
    (AC, F64, (20, 30, 70), 13, DOT_W, False, 0),
    (AC, F32, (9, 16, 130), 11, HALF_SQ, False, 0),
    (VD, F32, (100, 130), 17, DIFF, True, 0),
    (VD, F64, (33, 70), 9, DOT_W, True, 0),
    (J, F64, (90, 130), 15, HALF_SQ, False, adst.ADST_FORCE_TAPE),
]


@pytest.mark.parametrize("kind,dtype,shape,T,loss,dK,flags", SCHEDULE_CASES)
def test_bitwise_identical_across_budgets_and_schedules(kind, dtype, shape, T, loss, dK, flags):
    say(f"schedules kind={kind} dtype={dtype} shape={shape} T={T}")
    inp = inputs(kind, dtype, shape, 3)
    S = inp["x0"].nbytes
    runs = [("store-all", None, adst.ADST_SCHED_STORE_ALL)]
    for slots in (0, 1, 2, 3, 5):
        runs.append((f"binomial{slots}", slots * S, adst.ADST_SCHED_BINOMIAL))
    for slots in (1, 3):
        runs.append((f"uniform{slots}", slots * S, adst.ADST_SCHED_UNIFORM))
    runs.append(("auto-small", 2 * S, adst.ADST_SCHED_AUTO))
    ref = None
    for name, budget, sched in runs:
        g = gpu_vjp(kind, inp, T, loss, budget, sched, dK, flags)
        if ref is None:
            ref = g
            check_against_oracle(kind, dtype, inp, T, loss, dK, g)
            continue
        assert g["info"]["recompute_steps"] > 0 or name.startswith("binomial5") or T <= 2
        for key in ("dx0", "dK", "xT"):
            if ref[key] is not None:
                assert np.array_equal(g[key], ref[key]), (name, key)
        assert g["loss"] == ref["loss"], name
    # the same call again gives the same bits
    g = gpu_vjp(kind, inp, T, loss, 0, adst.ADST_SCHED_BINOMIAL, dK, flags)
    assert np.array_equal(g["dx0"], ref["dx0"])


def test_force_tape_gives_same_bits_as_elided():
    inp = inputs(J, F64, (70, 90), 4)
    a = gpu_vjp(J, inp, 12, HALF_SQ, 0, adst.ADST_SCHED_AUTO)
    b = gpu_vjp(J, inp, 12, HALF_SQ, 3 * inp["x0"].nbytes, adst.ADST_SCHED_BINOMIAL,
                flags=adst.ADST_FORCE_TAPE)
    assert a["info"]["recompute_steps"] == 0 and b["info"]["recompute_steps"] > 0
    assert np.array_equal(a["dx0"], b["dx0"]) and a["loss"] == b["loss"]


@pytest.mark.parametrize("kind,dtype,shape,dK", [
    (J, F64, (20, 30), False), (AC, F64, (5, 6, 7), False), (VD, F32, (40, 33), True)])
def test_zero_steps(kind, dtype, shape, dK):
    inp = inputs(kind, dtype, shape, 5)
    g = gpu_vjp(kind, inp, 0, DIFF, want_dK=dK)
    assert np.array_equal(g["dx0"], inp["x0"] - inp["aux"])
    assert np.array_equal(g["xT"], inp["x0"])
    if dK:
        assert np.array_equal(g["dK"], np.zeros_like(inp["x0"]))
    check_against_oracle(kind, dtype, inp, 0, DIFF, dK, g)


def test_trace_fills_phase_times():
    # 23 steps in two slots: recomputation runs of their own remain beside
    # the steps that run inside adjoint launches
    inp = inputs(AC, F64, (16, 32, 64), 6)
    g = gpu_vjp(AC, inp, 23, DOT_W, 2 * inp["x0"].nbytes, adst.ADST_SCHED_BINOMIAL,
                flags=adst.ADST_TRACE)
    info = g["info"]
    assert info["ms_fwd_sweep"] > 0 and info["ms_adj"] > 0 and info["ms_seed"] > 0
    assert info["ms_fwd_recompute"] > 0
    assert info["ms_total"] >= info["ms_adj"]
    check_against_oracle(AC, F64, inp, 23, DOT_W, False, g)


def test_workspace_reuse_between_calls():
    """A workspace is clobbered, never read before written: a dirty one from
    another call gives the same bits as a fresh one."""
    inp = inputs(VD, F32, (120, 77), 7)
    a = gpu_vjp(VD, inp, 8, DIFF, 2 * inp["x0"].nbytes, adst.ADST_SCHED_BINOMIAL, True,
                keep_ws=True)
    ws = a["ws"]
    ws.fill_(0xA5)
    b = gpu_vjp(VD, inp, 8, DIFF, 2 * inp["x0"].nbytes, adst.ADST_SCHED_BINOMIAL, True, ws=ws)
    assert np.array_equal(a["dx0"], b["dx0"]) and np.array_equal(a["dK"], b["dK"])


FUSION_CASES = [
    # kind, dtype, shape, T, loss, dK, flags, sched, slots (None = unlimited)
    (J, F64, (64, 64), 10, HALF_SQ, False, 0, adst.ADST_SCHED_AUTO, None),
    (J, F64, (333, 517), 7, HALF_SQ, False, 0, adst.ADST_SCHED_AUTO, None),
    (J, F32, (130, 70), 9, DIFF, False, 0, adst.ADST_SCHED_AUTO, None),
    (J, F64, (1, 1), 5, HALF_SQ, False, 0, adst.ADST_SCHED_AUTO, None),
    (J, F64, (2, 9), 4, DOT_W, False, 0, adst.ADST_SCHED_AUTO, None),
    (J, F64, (3, 3), 3, HALF_SQ, False, 0, adst.ADST_SCHED_AUTO, None),
    (J, F64, (5, 260), 6, HALF_SQ, False, 0, adst.ADST_SCHED_AUTO, None),
    (J, F64, (517, 253), 11, SEED, False, 0, adst.ADST_SCHED_AUTO, None),
    (J, F64, (90, 130), 15, HALF_SQ, False, adst.ADST_FORCE_TAPE, adst.ADST_SCHED_BINOMIAL, 2),
    (J, F32, (77, 300), 13, DIFF, False, adst.ADST_FORCE_TAPE, adst.ADST_SCHED_UNIFORM, 3),
    (VD, F32, (257, 300), 9, DIFF, True, 0, adst.ADST_SCHED_BINOMIAL, 2),
    (VD, F64, (70, 129), 6, DOT_W, False, 0, adst.ADST_SCHED_AUTO, None),
    (VD, F32, (1, 7), 3, DIFF, True, 0, adst.ADST_SCHED_BINOMIAL, 1),
    (VD, F64, (3, 300), 5, HALF_SQ, False, 0, adst.ADST_SCHED_AUTO, None),
    (VD, F32, (66, 517), 12, DIFF, True, 0, adst.ADST_SCHED_UNIFORM, 2),
    (AC, F64, (39, 45, 67), 9, DOT_W, False, 0, adst.ADST_SCHED_BINOMIAL, 2),
    (AC, F32, (17, 33, 130), 11, DIFF, False, 0, adst.ADST_SCHED_UNIFORM, 2),
    (AC, F64, (70, 15, 63), 8, HALF_SQ, False, 0, adst.ADST_SCHED_BINOMIAL, 1),
    (AC, F64, (1, 1, 1), 6, SEED, False, 0, adst.ADST_SCHED_BINOMIAL, 0),
    (AC, F64, (3, 1, 200), 7, HALF_SQ, False, 0, adst.ADST_SCHED_BINOMIAL, 1),
    (AC, F64, (33, 14, 62), 5, DOT_W, False, 0, adst.ADST_SCHED_BINOMIAL, 0),
    (AC, F64, (33, 17, 129), 6, DOT_W, False, 0, adst.ADST_SCHED_BINOMIAL, 2),
    (AC, F64, (20, 32, 256), 5, HALF_SQ, False, 0, adst.ADST_SCHED_UNIFORM, 2),
    (AC, F32, (9, 16, 128), 4, DIFF, False, 0, adst.ADST_SCHED_BINOMIAL, 1),
]


@pytest.mark.parametrize("kind,dtype,shape,T,loss,dK,flags,sched,slots", FUSION_CASES)
def test_fused_launches_match_single_steps_bitwise(kind, dtype, shape, T, loss, dK, flags, sched,
                                                   slots):
    """Temporal blocking (several steps per launch) gives the bits of one launch
    per step, and both match the oracle."""
    say(f"fusion kind={kind} dtype={dtype} shape={shape} T={T} flags={flags} sched={sched}")
    inp = inputs(kind, dtype, shape, 8)
    budget = None if slots is None else slots * inp["x0"].nbytes
    a = gpu_vjp(kind, inp, T, loss, budget, sched, dK, flags)
    b = gpu_vjp(kind, inp, T, loss, budget, sched, dK, flags | adst.ADST_NO_FUSE)
    assert b["info"]["fwd_launches"] == b["info"]["fwd_steps_total"]
    assert a["info"]["fwd_launches"] <= b["info"]["fwd_launches"]
    if kind == J and T >= 2 and not flags:
        assert a["info"]["fwd_launches"] < b["info"]["fwd_launches"]
        assert a["info"]["adj_launches"] < b["info"]["adj_launches"]
    for key in ("dx0", "dK", "xT"):
        if a[key] is not None:
            assert np.array_equal(a[key], b[key]), key
    assert a["loss"] == b["loss"]
    check_against_oracle(kind, dtype, inp, T, loss, dK, a)


@pytest.mark.parametrize("kind,dtype,shape,T", [
    (J, F64, (130, 257), 9), (J, F32, (64, 64), 1), (AC, F64, (20, 17, 33), 5),
    (VD, F32, (70, 129), 4), (J, F64, (7, 9), 0),
])
def test_half_square_without_xT_output(kind, dtype, shape, T):
    """Without an x_T output, x_T is written straight into g_T's buffer and
    the half-square seed only reduces the loss there: the same bits as with
    the output."""
    say(f"half-square seed without xT kind={kind} dtype={dtype} shape={shape} T={T}")
    inp = inputs(kind, dtype, shape, 12)
    a = gpu_vjp(kind, inp, T, HALF_SQ, want_xT=True)
    b = gpu_vjp(kind, inp, T, HALF_SQ, want_xT=False)
    assert np.array_equal(a["dx0"], b["dx0"]) and a["loss"] == b["loss"]
    check_against_oracle(kind, dtype, inp, T, HALF_SQ, False, a)
