"""Parity at the full sizes of the five workloads, in the launch
configuration the benchmark times (needs an MI355X and a few minutes).

Where the oracle can afford it, it computes sampled outputs one by one on
windows (tests/windows.py; exact for the sampled points). Where it cannot
(1024^3 for 200 steps), properties that hold at any size are checked:
bit-identity across budgets, a central finite difference of the loss along
a random direction, and sampled forward states.
"""
import numpy as np
import pytest

import oracle
import paper_2509_02197_amd as adst
from paper_2509_02197_amd.workloads import WORKLOADS, make_inputs
from tests.gpu_util import TOL, dev, gpu_vjp, rel, say
from tests.windows import sample_points, window_forward, window_vjp

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    adst.lib()


def _sampled_parity(w, inp, g, npts, seed):
    pts = sample_points(w.shape, npts, seed)
    got_d, ref_d, got_k, ref_k = [], [], [], []
    for p in pts:
        d, k = window_vjp(w.kind, inp, w.steps, p, w.loss, w.want_dK, params=w.params)
        got_d.append(g["dx0"][p])
        ref_d.append(d)
        if w.want_dK:
            got_k.append(g["dK"][p])
            ref_k.append(k)
        assert g["xT"][p] == window_forward(w.kind, inp, w.steps, p, params=w.params), p
    e = rel(got_d, ref_d)
    say(f"  {len(pts)} sampled points: dx0 rel L2 {e:.3e}")
    assert e <= TOL[w.dtype]
    if w.want_dK:
        e = rel(got_k, ref_k)
        say(f"  dK rel L2 {e:.3e}")
        assert e <= TOL[w.dtype]


def test_jacobi_4096_T100():
    w = WORKLOADS["jacobi2d5_f64_4096x4096_T100"]
    say(f"fullsize {w.name}")
    inp = make_inputs(w)
    g = gpu_vjp(w.kind, inp, w.steps, w.loss, w.budget_bytes, w.sched, w.want_dK)
    assert g["info"]["slots"] == 0 and g["info"]["recompute_steps"] == 0
    # whole forward state and loss against the oracle's forward sweep
    xT = oracle.forward(w.kind, inp["x0"], steps=w.steps)
    assert np.array_equal(g["xT"], xT)
    L = 0.5 * np.sum(xT * xT)
    assert abs(g["loss"] - L) <= 1e-12 * L
    _sampled_parity(w, inp, g, 12, 1)
    # the same gradient when the tape is forced through the 10-snapshot budget
    for sched in (adst.ADST_SCHED_BINOMIAL, adst.ADST_SCHED_UNIFORM):
        h = gpu_vjp(w.kind, inp, w.steps, w.loss, w.budget_bytes, sched, False,
                    adst.ADST_FORCE_TAPE)
        say(f"  forced tape sched={sched}: {h['info']['fwd_steps_total']} forward steps")
        assert h["info"]["slots"] <= 10 and h["info"]["recompute_steps"] > 0
        assert np.array_equal(h["dx0"], g["dx0"]) and h["loss"] == g["loss"]


def test_allencahn_512_T50():
    w = WORKLOADS["allencahn3d7_f64_512cube_T50"]
    say(f"fullsize {w.name}")
    inp = make_inputs(w)
    g = gpu_vjp(w.kind, inp, w.steps, w.loss, w.budget_bytes, w.sched, w.want_dK)
    assert g["info"]["slots"] == 8 and g["info"]["fwd_steps_total"] == 90
    _sampled_parity(w, inp, g, 9, 2)
    h = gpu_vjp(w.kind, inp, w.steps, w.loss, w.budget_bytes, adst.ADST_SCHED_UNIFORM)
    assert np.array_equal(h["dx0"], g["dx0"]) and h["loss"] == g["loss"]


def test_vardiff_8192_T200():
    w = WORKLOADS["vardiff2d9_f32_8192x8192_T200"]
    say(f"fullsize {w.name}")
    inp = make_inputs(w)
    g = gpu_vjp(w.kind, inp, w.steps, w.loss, w.budget_bytes, w.sched, w.want_dK)
    assert g["info"]["slots"] == 16 and g["info"]["fwd_steps_total"] == 411
    _sampled_parity(w, inp, g, 8, 3)
    h = gpu_vjp(w.kind, inp, w.steps, w.loss, 5 * w.state_bytes, adst.ADST_SCHED_BINOMIAL,
                w.want_dK)
    assert np.array_equal(h["dx0"], g["dx0"]) and np.array_equal(h["dK"], g["dK"])


def test_allencahn_1024_T200():
    import torch
    w = WORKLOADS["allencahn3d7_f64_1024cube_T200"]
    say(f"fullsize {w.name}")
    inp = make_inputs(w)
    x0, W = dev(inp["x0"]), dev(inp["aux"])
    del inp["aux"]
    a = adst.vjp(w.kind, x0, None, w.steps, w.loss, W, w.budget_bytes, w.sched)
    torch.cuda.synchronize()
    info = a["info"]
    say(f"  64 GB budget: {info.slots} slots, {info.fwd_steps_total} forward steps")
    assert info.slots == 7 and info.fwd_steps_total == 581
    dx0, L = a["dx0"], float(a["loss"])
    # sampled forward states near a corner
    p = (0, 0, 0)
    assert float(a["xT"][p]) == window_forward(w.kind, inp, w.steps, p, params=w.params)
    del a["xT"]
    # another budget gives the same bits
    b = adst.vjp(w.kind, x0, None, w.steps, w.loss, W, 32_000_000_000, w.sched, ws=a["ws"])
    torch.cuda.synchronize()
    say(f"  32 GB budget: {b['info'].slots} slots, {b['info'].fwd_steps_total} forward steps")
    assert b["info"].slots == 3
    assert torch.equal(b["dx0"], dx0) and float(b["loss"]) == L
    del b
    # central finite difference of L along a random direction
    gen = torch.Generator(device="cuda").manual_seed(9)
    v = torch.randn(x0.shape, dtype=torch.float64, device="cuda", generator=gen)
    h = 1e-4

    def loss_at(x):
        xT = adst.forward(w.kind, x, None, w.steps)
        return float(torch.dot(W.reshape(-1), xT.reshape(-1)))

    fd = (loss_at(x0 + h * v) - loss_at(x0 - h * v)) / (2 * h)
    ad = float(torch.dot(dx0.reshape(-1), v.reshape(-1)))
    say(f"  directional derivative: adjoint {ad:.12e} finite difference {fd:.12e}")
    assert abs(fd - ad) <= 1e-6 * abs(ad)
