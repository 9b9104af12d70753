"""Observability and memory safety of adst_vjp on the GPU: the per-launch
trace statistics agree with the plan, ADST_LOG prints the plan, and no
launch writes outside the buffers it was given (guard bands around the
workspace and every caller array keep their fill pattern; inputs keep
their bits)."""
import os
import subprocess
import sys

import numpy as np
import pytest

import paper_2509_02197_amd as adst
from tests.gpu_util import say

pytestmark = pytest.mark.gpu
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

F64, F32 = adst.ADST_F64, adst.ADST_F32
CASES = [
    # kind, dtype, shape, T, loss, budget in states, sched, dK, flags, lim, dparams
    (adst.ADST_ALLENCAHN3D7, F64, (21, 35, 70), 30, adst.ADST_LOSS_DOT_W, 4,
     adst.ADST_SCHED_BINOMIAL, False, 0, None, False),
    (adst.ADST_JACOBI2D5, F64, (133, 301), 23, adst.ADST_LOSS_HALF_SQ, 3, adst.ADST_SCHED_AUTO,
     False, 0, None, False),
    (adst.ADST_JACOBI2D5, F64, (133, 301), 23, adst.ADST_LOSS_HALF_SQ, 3,
     adst.ADST_SCHED_UNIFORM, False, adst.ADST_FORCE_TAPE, None, False),
    (adst.ADST_VARDIFF2D9, F32, (130, 270), 17, adst.ADST_LOSS_HALF_SQ_DIFF, 3,
     adst.ADST_SCHED_BINOMIAL, True, 0, None, False),
    (adst.ADST_VARDIFF2D9, F32, (130, 270), 9, adst.ADST_LOSS_HALF_SQ_DIFF, 2,
     adst.ADST_SCHED_BINOMIAL, True, 0, (0.2, 0.8), True),
    (adst.ADST_JACOBI2D5, F64, (70, 129), 11, adst.ADST_LOSS_HALF_SQ, 2,
     adst.ADST_SCHED_BINOMIAL, False, 0, (0.3, 0.7), False),
    (adst.ADST_GAUSSSEIDEL2D5, F64, (90, 150), 7, adst.ADST_LOSS_HALF_SQ, 0,
     adst.ADST_SCHED_AUTO, False, 0, None, False),
]


def _inputs(kind, dtype, shape, seed=3):
    r = np.random.Generator(np.random.PCG64(seed))
    dt = np.float64 if dtype == F64 else np.float32
    lo = -1.0 if kind == adst.ADST_ALLENCAHN3D7 else 0.0
    return (r.uniform(lo, 1, shape).astype(dt),
            r.uniform(0.5, 1.5, shape).astype(dt) if kind == adst.ADST_VARDIFF2D9 else None,
            r.standard_normal(shape).astype(dt))


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    adst.lib()


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"k{c[0]}-{c[1]}-{c[2]}-s{c[6]}-f{c[8]}")
def test_trace_statistics_match_the_plan(case):
    import torch
    kind, dtype, shape, T, loss, nst, sched, want_dK, flags, lim, dp = case
    say(f"trace kind={kind} shape={shape} T={T} sched={sched} flags={flags} lim={lim}")
    x0, K, aux = (None if a is None else torch.from_numpy(a).cuda()
                  for a in _inputs(kind, dtype, shape))
    S = x0.numel() * x0.element_size()
    out = adst.vjp(kind, x0, K, T, loss, aux, nst * S, sched, want_dK,
                   flags=flags | adst.ADST_TRACE, lim=lim, want_dparams=dp)
    info = out["info"]
    ks = adst.adst_trace_kernels()
    fwd = sum(k["launches"] for k in ks if k["phase"] in ("forward sweep", "recomputation"))
    adj = sum(k["launches"] for k in ks if k["phase"] == "adjoint" and k["name"] != "limit_mask")
    assert fwd == info.fwd_kernels and adj == info.adj_kernels
    small = sum(k["alg_bytes_sum"] for k in ks if k["name"] in ("finalize_loss", "dparam_finalize"))
    total = sum(k["alg_bytes_sum"] for k in ks)
    assert total - small == info.alg_bytes
    phases = {k: sum(q["ms_sum"] for q in ks if q["phase"] == p) for k, p in
              (("ms_adj", "adjoint"), ("ms_seed", "loss and seed"))}
    assert abs(phases["ms_adj"] - info.ms_adj) <= 1e-3 * max(info.ms_adj, 1)
    for k in ks:
        assert k["launches"] >= 1 and k["ms_sum"] > 0 and k["ms_min"] <= k["ms_max"]
    # an untraced call leaves the statistics of the last traced one alone
    adst.vjp(kind, x0, K, T, loss, aux, nst * S, sched, want_dK, flags=flags, lim=lim,
             want_dparams=dp)
    torch.cuda.synchronize()
    assert adst.adst_trace_kernels() == ks


def test_adst_log_prints_the_plan():
    code = (
        "import torch, paper_2509_02197_amd as a\n"
        "x = torch.rand(5, 9, 70, dtype=torch.float64, device='cuda')\n"
        "w = torch.randn(5, 9, 70, dtype=torch.float64, device='cuda')\n"
        "a.vjp(a.ADST_ALLENCAHN3D7, x, None, 6, a.ADST_LOSS_DOT_W, w, 2 * x.numel() * 8,"
        " a.ADST_SCHED_BINOMIAL)\n"
        "torch.cuda.synchronize()\n")
    env = dict(os.environ, ADST_LOG="2", PYTHONPATH=ROOT)
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True,
                       timeout=120, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [ln for ln in r.stderr.splitlines() if ln.startswith("adst plan:")]
    assert len(lines) == 1
    assert "allencahn3d7 f64 70x9x5 T=6" in lines[0] and "sched=binomial slots=2 (c=3)" in lines[0]
    acts = [ln for ln in r.stderr.splitlines() if ln.strip().split(" ")[-1].startswith("n=")]
    assert any(" SEED " in a for a in acts) and sum(" ADJ " in a for a in acts) == 6


GUARD = 1 << 16  # bytes of guard band on each side


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"k{c[0]}-{c[1]}-{c[2]}-s{c[6]}-f{c[8]}")
def test_no_write_outside_the_given_buffers(case):
    import torch
    kind, dtype, shape, T, loss, nst, sched, want_dK, flags, lim, dp = case
    say(f"guard kind={kind} shape={shape} T={T} sched={sched} flags={flags}")
    x0h, Kh, auxh = _inputs(kind, dtype, shape)
    S = x0h.nbytes
    prob = adst.make_problem(kind, dtype, adst._dims(shape), None, flags, lim)
    grads = (adst.ADST_GRAD_COEFF if want_dK else 0) | (adst.ADST_GRAD_PARAMS if dp else 0)
    info = adst.adst_plan(prob, T, nst * S, sched, grads)
    sizes = {"x0": S, "K": S, "aux": S, "dx0": S, "dK": S, "xT": S, "L": 8, "dp": 16,
             "ws": info.workspace_bytes}
    # one arena: [guard][buf][guard][buf]...[guard], each buffer 256-byte aligned
    offs, pos = {}, GUARD
    for k, n in sizes.items():
        offs[k] = pos
        pos += (n + 255) // 256 * 256 + GUARD
    pattern = np.frombuffer(np.array([0x7ff4dead5a5a5a5a], dtype=np.uint64).tobytes() * (pos // 8),
                            dtype=np.uint8)
    arena = torch.from_numpy(pattern.copy()).cuda()
    base = arena.data_ptr()

    def put(name, a):
        if a is not None:
            arena[offs[name]:offs[name] + a.nbytes].copy_(torch.from_numpy(a.view(np.uint8).reshape(-1)))
    put("x0", x0h)
    put("K", Kh)
    put("aux", auxh)
    before = arena.cpu().numpy().copy()
    p = lambda k: base + offs[k]  # noqa: E731
    adst.adst_vjp(prob, p("x0"), p("K") if Kh is not None else None, T, loss, p("aux"), nst * S,
                  sched, p("dx0"), p("dK") if want_dK else None, p("xT"), p("L"),
                  p("dp") if dp else None, p("ws"), info.workspace_bytes)
    torch.cuda.synchronize()
    after = arena.cpu().numpy()
    written = {"dx0", "xT", "L", "ws"} | ({"dK"} if want_dK else set()) | ({"dp"} if dp else set())
    keep = np.ones(pos, dtype=bool)
    for k in written:
        keep[offs[k]:offs[k] + sizes[k]] = False
    bad = np.nonzero((after != before) & keep)[0]
    assert bad.size == 0, f"bytes changed outside the outputs, first at arena offset {bad[0]}"
    # the outputs were written (no NaN pattern left in dx0)
    dx0 = after[offs["dx0"]:offs["dx0"] + S].view(x0h.dtype)
    assert np.all(np.isfinite(dx0))
