"""The C-ABI library on a host without a GPU: it loads, exports every
function include/adst.h declares, and rejects every bad argument before
enqueueing anything (so these calls never reach the GPU; the pointers below
are never dereferenced).
"""
import ctypes
import os
import re

import pytest

import paper_2509_02197_amd as adst

def _gpu_visible():
    try:
        import torch
        return torch.cuda.device_count() > 0
    except Exception:
        return False


# The fake pointers below must never reach a kernel: run only where no GPU
# is visible, so that a validation gap can only ever fail on the host.
pytestmark = pytest.mark.skipif(_gpu_visible(), reason="host-only argument checks")

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "adst.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(adst_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    assert declared_functions() == sorted(adst.EXPORTED)


def test_library_exports_every_declared_function():
    lib = ctypes.CDLL(adst.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings():
    for s in range(6):
        assert adst.adst_status_str(s)
    assert adst.adst_status_str(99) == "unknown status"


def test_struct_layouts_match_header():
    # int32 x2, int64 x3, double x4, uint32 (+pad) = 72 bytes
    assert ctypes.sizeof(adst.adst_problem) == 72
    assert ctypes.sizeof(adst.adst_action) == 20
    # int32 x4, int64 x8, uint64 x6, float x6, uint64
    assert ctypes.sizeof(adst.adst_plan_info) == 4 * 4 + 8 * 8 + 6 * 8 + 6 * 4 + 8
    assert adst.adst_plan_info.fwd_alg_bytes.offset == 4 * 4 + 8 * 8 + 6 * 8 + 6 * 4


def _p(kind=adst.ADST_ALLENCAHN3D7, dims=(8, 8, 8), dtype=adst.ADST_F64, flags=0):
    return adst.make_problem(kind, dtype, dims, flags=flags)


def _status(fn, *a):
    try:
        fn(*a)
    except adst.AdstError as e:
        return e.status
    return adst.ADST_OK


@pytest.mark.parametrize("mutate,status", [
    (lambda p: setattr(p, "kind", 7), adst.ADST_ERR_ARG),
    (lambda p: setattr(p, "dtype", 3), adst.ADST_ERR_ARG),
    (lambda p: p.n.__setitem__(1, 0), adst.ADST_ERR_ARG),
    (lambda p: setattr(p, "flags", 0x80), adst.ADST_ERR_ARG),
    (lambda p: [p.n.__setitem__(i, 2000) for i in range(3)], adst.ADST_ERR_ARG),
])
def test_plan_rejects_bad_problems(mutate, status):
    p = _p()
    mutate(p)
    assert _status(adst.adst_plan, p, 10, 0, 0) == status
    assert adst.adst_last_error()


def test_plan_rejects_bad_scalars():
    assert _status(adst.adst_plan, _p(), -1, 0, 0) == adst.ADST_ERR_ARG
    assert _status(adst.adst_plan, _p(), 10, 0, 9) == adst.ADST_ERR_ARG
    info = adst.adst_plan_info()
    assert adst.lib().adst_plan(None, 3, 0, 0, 0, ctypes.byref(info)) == adst.ADST_ERR_ARG
    assert adst.lib().adst_plan(ctypes.byref(_p()), 3, 0, 0, 0, None) == adst.ADST_ERR_ARG


def test_plan_rejects_unsupported_combinations():
    # 2-D kinds with nz > 1
    assert _status(adst.adst_plan, _p(adst.ADST_JACOBI2D5, (8, 8, 2)), 5, 0, 0) == \
        adst.ADST_ERR_UNSUPPORTED
    assert _status(adst.adst_plan, _p(adst.ADST_VARDIFF2D9, (8, 8, 3)), 5, 0, 0) == \
        adst.ADST_ERR_UNSUPPORTED
    # a coefficient gradient for a kind without a coefficient field
    assert _status(adst.adst_plan, _p(), 5, 0, 0, True) == adst.ADST_ERR_UNSUPPORTED


# Fake, never-dereferenced device addresses: far apart unless a test wants overlap.
X0, K, AUX, DX0, DK, XT, LOSS, WS = (0x10000000 * (i + 1) for i in range(8))
BIG = 1 << 40


def _vjp(p, **kw):
    a = dict(x0=X0, coeff=None, steps=5, loss=adst.ADST_LOSS_HALF_SQ, loss_aux=None,
             budget=BIG, sched=0, dx0=DX0, dcoeff=None, xT=None, loss_dev=None, dparams=None,
             ws=WS, ws_bytes=BIG)
    a.update(kw)
    return _status(adst.adst_vjp, p, a["x0"], a["coeff"], a["steps"], a["loss"], a["loss_aux"],
                   a["budget"], a["sched"], a["dx0"], a["dcoeff"], a["xT"], a["loss_dev"],
                   a["dparams"], a["ws"], a["ws_bytes"], 0)


def test_vjp_argument_errors():
    p = _p()
    E = adst.ADST_ERR_ARG
    assert _vjp(p, dx0=None) == E
    assert _vjp(p, x0=None) == E
    assert _vjp(p, steps=-2) == E
    assert _vjp(p, loss=7) == E
    assert _vjp(p, loss=adst.ADST_LOSS_DOT_W) == E             # needs loss_aux
    assert _vjp(p, loss=adst.ADST_LOSS_HALF_SQ_DIFF) == E      # needs loss_aux
    assert _vjp(p, dx0=X0 + 8) == E                            # dx0 overlaps x0
    assert _vjp(p, xT=DX0 + 8) == E                            # xT overlaps dx0
    assert _vjp(p, loss_dev=WS + 64) == E                      # loss overlaps ws
    assert _vjp(p, loss=adst.ADST_LOSS_SEED, loss_aux=DX0) == E  # output overlaps input
    pv = _p(adst.ADST_VARDIFF2D9, (8, 8, 1))
    assert _vjp(pv) == E                                       # K missing
    assert _vjp(pv, coeff=K, dcoeff=K) == E                    # dK overlaps K
    assert _vjp(p, dparams=DX0 + 8) == E                       # dparams overlaps dx0
    assert _vjp(p, dparams=X0) == E                            # dparams overlaps x0
    # the constants' gradients are not built for the in-place kind
    assert _vjp(_p(adst.ADST_GAUSSSEIDEL2D5, (8, 8, 1)), dparams=LOSS) == \
        adst.ADST_ERR_UNSUPPORTED


def test_limiter_arguments():
    pj = _p(adst.ADST_JACOBI2D5, (8, 8, 1))
    assert adst.adst_plan(pj, 5, BIG, 0).needs_state == 0
    lim = adst.make_problem(adst.ADST_JACOBI2D5, adst.ADST_F64, (8, 8, 1), lim=(0.2, 0.8))
    info = adst.adst_plan(lim, 5, BIG, 0)
    assert info.needs_state == 1 and info.fwd_launches == info.fwd_steps_total  # no fused steps
    bad = adst.make_problem(adst.ADST_JACOBI2D5, adst.ADST_F64, (8, 8, 1), lim=(0.8, 0.2))
    assert _status(adst.adst_plan, bad, 5, 0, 0) == adst.ADST_ERR_ARG
    nan = adst.make_problem(adst.ADST_JACOBI2D5, adst.ADST_F64, (8, 8, 1), lim=(float("nan"), 1))
    assert _status(adst.adst_plan, nan, 5, 0, 0) == adst.ADST_ERR_ARG
    gs = adst.make_problem(adst.ADST_GAUSSSEIDEL2D5, adst.ADST_F64, (8, 8, 1), lim=(0, 1))
    assert _status(adst.adst_plan, gs, 5, 0, 0) == adst.ADST_ERR_UNSUPPORTED


def test_gradient_mask():
    pj = _p(adst.ADST_JACOBI2D5, (8, 8, 1))
    assert _status(adst.adst_plan, pj, 5, 0, 0, 4) == adst.ADST_ERR_ARG
    assert _status(adst.adst_plan, _p(adst.ADST_GAUSSSEIDEL2D5, (8, 8, 1)), 5, 0, 0,
                   adst.ADST_GRAD_PARAMS) == adst.ADST_ERR_UNSUPPORTED
    # the constants' partials read x_{t-1}: the linear kinds now keep a tape
    plain = adst.adst_plan(pj, 5, BIG, 0)
    withp = adst.adst_plan(pj, 5, BIG, 0, adst.ADST_GRAD_PARAMS)
    assert plain.needs_state == 0 and withp.needs_state == 1 and withp.slots == 3
    # their slots (one per adjoint workgroup and constant: an 8 x 8 grid is one
    # work item, so 2 doubles) sit after the checkpoint slots, 4 KiB aligned
    S = 8 * 8 * 8
    stride = -(-S // 4096) * 4096
    assert withp.workspace_bytes == 16384 + (3 + 3) * stride + 4096
    # bytes: every adjoint step also reads x_{t-1} for the partials
    assert withp.alg_bytes - (16 * 5 + 16 * 5 + 16) * 64 == 8 * 5 * 64
    # slot counts follow the adjoint's work items: Jacobi one per column strip
    # (124 columns in f64) and row chunk (12 rows in the two edge strips, 128
    # in the others, 6 at each end), Allen-Cahn 64 x 8 x 32 tiles, variable
    # coefficients 256 x 4 tiles (2 doubles per item, 4 KiB aligned)
    def march_items(nx, ny):
        ns = -(-nx // 124)
        chunks = lambda mid: 2 + -(-(ny - 12) // mid) if ny > 12 else 1
        nedge = 2 if ns >= 2 else 1
        return nedge * chunks(12) + (ns - nedge) * chunks(128)
    assert march_items(600, 100) == 2 * 10 + 3 * 3
    assert march_items(4096, 4096) == 2 * 343 + 32 * 34
    for kind, dims, tiles in [(adst.ADST_JACOBI2D5, (600, 100, 1), march_items(600, 100)),
                              (adst.ADST_JACOBI2D5, (4096, 4096, 1), march_items(4096, 4096)),
                              (adst.ADST_ALLENCAHN3D7, (65, 9, 33), 2 * 2 * 2),
                              (adst.ADST_VARDIFF2D9, (257, 9, 1), 2 * 3)]:
        dt = adst.ADST_F32 if kind == adst.ADST_VARDIFF2D9 else adst.ADST_F64
        pk = adst.make_problem(kind, dt, dims, flags=adst.ADST_FORCE_TAPE)
        a = adst.adst_plan(pk, 5, BIG, 0)
        b = adst.adst_plan(pk, 5, BIG, 0, adst.ADST_GRAD_PARAMS)
        assert a.slots == b.slots
        assert b.workspace_bytes - a.workspace_bytes == -(-16 * tiles // 4096) * 4096, kind


def test_vjp_budget_and_workspace_errors():
    p = _p()
    assert _vjp(p, budget=0, sched=adst.ADST_SCHED_STORE_ALL) == adst.ADST_ERR_BUDGET
    need = adst.adst_plan(p, 5, BIG, 0).workspace_bytes
    assert _vjp(p, ws_bytes=need - 1) == adst.ADST_ERR_WORKSPACE
    assert _vjp(p, ws=None) == adst.ADST_ERR_WORKSPACE
    assert _vjp(_p(adst.ADST_JACOBI2D5, (8, 8, 1)), dcoeff=DK) == adst.ADST_ERR_UNSUPPORTED


def test_forward_argument_errors():
    p = _p()

    def fwd(**kw):
        a = dict(x0=X0, coeff=None, steps=4, xT=XT, ws=WS, ws_bytes=BIG)
        a.update(kw)
        return _status(adst.adst_forward, p if "p" not in kw else kw["p"], a["x0"], a["coeff"],
                       a["steps"], a["xT"], a["ws"], a["ws_bytes"], 0)

    assert fwd(xT=None) == adst.ADST_ERR_ARG
    assert fwd(steps=-1) == adst.ADST_ERR_ARG
    assert fwd(xT=X0) == adst.ADST_ERR_ARG
    assert fwd(ws_bytes=10) == adst.ADST_ERR_WORKSPACE
    assert fwd(ws=XT + 16) == adst.ADST_ERR_ARG


# ---- the binding's tensor checks (before any plan or launch)
def _t(*shape, dtype=None):
    import torch
    return torch.zeros(*shape, dtype=dtype or torch.float64)


@pytest.mark.parametrize("make,msg", [
    (lambda: dict(x0=_t(8, 9).t()), "contiguous"),
    (lambda: dict(x0=_t(8, 9), coeff=_t(8, 9, dtype=__import__("torch").float32)), "dtype"),
    (lambda: dict(x0=_t(8, 9), coeff=_t(9, 8)), "shape"),
    (lambda: dict(x0=_t(8, 9), aux=_t(8, 18)[:, ::2]), "contiguous"),
    (lambda: dict(x0=_t(8, 9), aux=_t(1, 9).expand(8, 9)), "contiguous"),
    (lambda: dict(x0=_t(8, 9)), "GPU"),
    (lambda: dict(x0=_t(8, 9, dtype=__import__("torch").int32)), "dtype"),
])
def test_binding_rejects_bad_tensors(make, msg):
    kw = make()
    with pytest.raises((ValueError, TypeError), match=msg):
        adst.vjp(adst.ADST_VARDIFF2D9, kw.pop("x0"), kw.get("coeff"), 3,
                 adst.ADST_LOSS_HALF_SQ_DIFF, kw.get("aux"))
    if "aux" not in kw:
        kw2 = make()
        with pytest.raises((ValueError, TypeError), match=msg):
            adst.forward(adst.ADST_VARDIFF2D9, kw2.pop("x0"), kw2.get("coeff"), 3)
