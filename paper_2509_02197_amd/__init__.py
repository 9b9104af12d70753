"""adst: reverse-mode gradients of time-iterated stencils under a checkpoint
memory budget, on AMD MI355X (gfx950).

Thin ctypes binding of ``libadst.so`` (declared in ``include/adst.h``). The
functions keep the C names and only marshal arguments: tensors become device
pointers, the stream defaults to torch's current stream. Every step of the
path runs in the library's HIP kernels; there is no Python or CPU fallback,
and a missing library is an error.
"""
import ctypes
import os

from . import workloads  # noqa: F401  (seeded inputs; no method arithmetic)

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libadst.so")

# enums of adst.h
ADST_OK, ADST_ERR_ARG, ADST_ERR_BUDGET, ADST_ERR_WORKSPACE, ADST_ERR_UNSUPPORTED, ADST_ERR_HIP = range(6)
ADST_JACOBI2D5, ADST_ALLENCAHN3D7, ADST_VARDIFF2D9, ADST_GAUSSSEIDEL2D5 = 0, 1, 2, 3
ADST_F64, ADST_F32 = 0, 1
ADST_SCHED_AUTO, ADST_SCHED_STORE_ALL, ADST_SCHED_UNIFORM, ADST_SCHED_BINOMIAL = 0, 1, 2, 3
ADST_LOSS_HALF_SQ, ADST_LOSS_DOT_W, ADST_LOSS_HALF_SQ_DIFF, ADST_LOSS_SEED = 0, 1, 2, 3
ADST_FORCE_TAPE, ADST_TRACE, ADST_NO_FUSE, ADST_LIMIT = 0x1, 0x2, 0x4, 0x8
ADST_GRAD_COEFF, ADST_GRAD_PARAMS = 0x1, 0x2
ADST_OP_FWD, ADST_OP_SEED, ADST_OP_ADJ, ADST_OP_FWD2, ADST_OP_ADJ2, ADST_OP_FWDW, ADST_OP_ADJW = range(7)
ADST_BUF_NONE, ADST_BUF_X0, ADST_BUF_W0, ADST_BUF_W1, ADST_BUF_XT, ADST_BUF_SLOT0 = -1, 0, 1, 2, 3, 4

EXPORTED = ("adst_plan", "adst_plan_actions", "adst_forward", "adst_vjp", "adst_ilp_solve",
            "adst_trace_kernels", "adst_copy", "adst_vjp_static_ws", "adst_status_str",
            "adst_last_error")
ADST_STATIC_WS_BYTES = 64 << 20
PHASE_NAMES = ("forward sweep", "recomputation", "adjoint", "loss and seed", "constants")
ILP_EVENTS = {"alloc": 0, "free": 1, "produce": 2, "drop": 3, "recompute": 4,
              "recompute_done": 5, "release": 6, "path": 7}


class adst_problem(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("dtype", ctypes.c_int32), ("n", ctypes.c_int64 * 3),
                ("p", ctypes.c_double * 2), ("lim", ctypes.c_double * 2),
                ("flags", ctypes.c_uint32)]


class adst_action(ctypes.Structure):
    _fields_ = [("op", ctypes.c_int32), ("t", ctypes.c_int32), ("src", ctypes.c_int32),
                ("dst", ctypes.c_int32), ("n", ctypes.c_int32)]


class adst_plan_info(ctypes.Structure):
    _fields_ = [("steps", ctypes.c_int32), ("sched", ctypes.c_int32), ("slots", ctypes.c_int32),
                ("needs_state", ctypes.c_int32), ("fwd_steps_total", ctypes.c_int64),
                ("recompute_steps", ctypes.c_int64), ("adj_steps", ctypes.c_int64),
                ("n_actions", ctypes.c_int64), ("fwd_launches", ctypes.c_int64),
                ("adj_launches", ctypes.c_int64), ("fwd_kernels", ctypes.c_int64),
                ("adj_kernels", ctypes.c_int64), ("state_bytes", ctypes.c_uint64),
                ("budget_bytes", ctypes.c_uint64), ("slot_bytes_peak", ctypes.c_uint64),
                ("workspace_bytes", ctypes.c_uint64), ("fwd_workspace_bytes", ctypes.c_uint64),
                ("alg_bytes", ctypes.c_uint64), ("ms_fwd_sweep", ctypes.c_float),
                ("ms_fwd_recompute", ctypes.c_float), ("ms_adj", ctypes.c_float),
                ("ms_seed", ctypes.c_float), ("ms_total", ctypes.c_float),
                ("ms_dparams", ctypes.c_float), ("fwd_alg_bytes", ctypes.c_uint64)]

    def as_dict(self):
        return {f[0]: getattr(self, f[0]) for f in self._fields_}


class adst_ilp_array(ctypes.Structure):
    _fields_ = [("size", ctypes.c_double), ("overhead", ctypes.c_double),
                ("cost", ctypes.c_double)]


class adst_ilp_event(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("array", ctypes.c_int32), ("amount", ctypes.c_double)]


class adst_ilp_info(ctypes.Structure):
    _fields_ = [("objective", ctypes.c_double), ("peak", ctypes.c_double),
                ("measurements", ctypes.c_int64), ("nodes", ctypes.c_int64),
                ("paths", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class adst_kernel_stat(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 56), ("phase", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("launches", ctypes.c_int64),
                ("ms_sum", ctypes.c_double), ("ms_min", ctypes.c_double),
                ("ms_max", ctypes.c_double), ("alg_bytes_sum", ctypes.c_double)]


class AdstError(RuntimeError):
    def __init__(self, status, detail):
        self.status = status
        super().__init__(f"adst status {status}: {detail}")


_lib = None


def lib():
    """The loaded library. Built in-tree on first use if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        from . import build as _build
        _build.build()
    L = ctypes.CDLL(LIB_PATH)
    vp, u64, i32, i64 = ctypes.c_void_p, ctypes.c_uint64, ctypes.c_int32, ctypes.c_int64
    P = ctypes.POINTER
    L.adst_plan.argtypes = [P(adst_problem), i32, u64, i32, i32, P(adst_plan_info)]
    L.adst_plan_actions.argtypes = [P(adst_problem), i32, u64, i32, i32, P(adst_action), i64,
                                    P(i64)]
    L.adst_forward.argtypes = [P(adst_problem), vp, vp, i32, vp, vp, u64, vp]
    L.adst_vjp.argtypes = [P(adst_problem), vp, vp, i32, i32, vp, u64, i32, vp, vp, vp, vp, vp, vp,
                           u64, vp, P(adst_plan_info)]
    L.adst_ilp_solve.argtypes = [P(adst_ilp_array), i32, P(adst_ilp_event), i64, ctypes.c_double,
                                 P(i32), P(adst_ilp_info)]
    L.adst_vjp_static_ws.argtypes = [P(adst_problem), vp, vp, i32, i32, vp, u64, i32, vp, vp, vp,
                                     vp, vp, vp, P(adst_plan_info)]
    L.adst_trace_kernels.argtypes = [P(adst_kernel_stat), i32, P(i32)]
    L.adst_copy.argtypes = [vp, vp, u64, vp]
    for f in ("adst_plan", "adst_plan_actions", "adst_forward", "adst_vjp", "adst_ilp_solve",
              "adst_trace_kernels", "adst_copy", "adst_vjp_static_ws"):
        getattr(L, f).restype = ctypes.c_int
    L.adst_status_str.argtypes = [ctypes.c_int]
    L.adst_status_str.restype = ctypes.c_char_p
    L.adst_last_error.argtypes = []
    L.adst_last_error.restype = ctypes.c_char_p
    _lib = L
    return L


def adst_status_str(status):
    return lib().adst_status_str(status).decode()


def adst_last_error():
    return lib().adst_last_error().decode()


def _check(status):
    if status != ADST_OK:
        raise AdstError(status, f"{adst_status_str(status)}: {adst_last_error()}")


def make_problem(kind, dtype, dims, params=None, flags=0, lim=None):
    """dims = (nx, ny, nz) with nx fastest; lim = limiter bounds (lo, hi) or
    None (sets ADST_LIMIT)."""
    from .workloads import DEFAULT_PARAMS
    p = adst_problem()
    p.kind, p.dtype = kind, dtype
    for i in range(3):
        p.n[i] = int(dims[i])
    pp = params if params is not None else DEFAULT_PARAMS[kind]
    p.p[0], p.p[1] = float(pp[0]), float(pp[1])
    if lim is not None:
        p.lim[0], p.lim[1] = float(lim[0]), float(lim[1])
        flags |= ADST_LIMIT
    p.flags = flags
    return p


def _ptr(x):
    if x is None:
        return None
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    return int(x)


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if hasattr(stream, "cuda_stream"):
        return stream.cuda_stream
    return int(stream)


def adst_plan(prob, steps, mem_budget_bytes, sched, grads=0):
    info = adst_plan_info()
    _check(lib().adst_plan(ctypes.byref(prob), steps, mem_budget_bytes, sched, int(grads),
                           ctypes.byref(info)))
    return info


def adst_plan_actions(prob, steps, mem_budget_bytes, sched, grads=0):
    """The plan's action list as a list of (op, t, src, dst, n) tuples."""
    n = ctypes.c_int64(0)
    L = lib()
    _check(L.adst_plan_actions(ctypes.byref(prob), steps, mem_budget_bytes, sched,
                               int(grads), None, 0, ctypes.byref(n)))
    buf = (adst_action * max(n.value, 1))()
    _check(L.adst_plan_actions(ctypes.byref(prob), steps, mem_budget_bytes, sched,
                               int(grads), buf, n.value, ctypes.byref(n)))
    return [(a.op, a.t, a.src, a.dst, a.n) for a in buf[:n.value]]


def adst_forward(prob, x0, coeff, steps, xT, ws, ws_bytes, stream=None):
    _check(lib().adst_forward(ctypes.byref(prob), _ptr(x0), _ptr(coeff), steps, _ptr(xT),
                              _ptr(ws), ws_bytes, _stream(stream)))


def adst_vjp(prob, x0, coeff, steps, loss, loss_aux, mem_budget_bytes, sched, dx0, dcoeff, xT,
             loss_dev, dparams, ws, ws_bytes, stream=None, want_info=True):
    info = adst_plan_info() if want_info else None
    _check(lib().adst_vjp(ctypes.byref(prob), _ptr(x0), _ptr(coeff), steps, loss, _ptr(loss_aux),
                          mem_budget_bytes, sched, _ptr(dx0), _ptr(dcoeff), _ptr(xT),
                          _ptr(loss_dev), _ptr(dparams), _ptr(ws), ws_bytes, _stream(stream),
                          ctypes.byref(info) if info is not None else None))
    return info


def adst_vjp_static_ws(prob, x0, coeff, steps, loss, loss_aux, mem_budget_bytes, sched, dx0,
                       dcoeff, xT, loss_dev, dparams, stream=None, want_info=True):
    """adst_vjp with the library's static per-GPU workspace (no allocation;
    plans whose workspace exceeds ADST_STATIC_WS_BYTES are rejected)."""
    info = adst_plan_info() if want_info else None
    _check(lib().adst_vjp_static_ws(ctypes.byref(prob), _ptr(x0), _ptr(coeff), steps, loss,
                                    _ptr(loss_aux), mem_budget_bytes, sched, _ptr(dx0),
                                    _ptr(dcoeff), _ptr(xT), _ptr(loss_dev), _ptr(dparams),
                                    _stream(stream),
                                    ctypes.byref(info) if info is not None else None))
    return info


def adst_trace_kernels():
    """Per-kernel statistics of this thread's last adst_vjp call made with
    ADST_TRACE: a list of dicts (name, phase, launches, ms_sum, ms_min,
    ms_max, alg_bytes_sum)."""
    n = ctypes.c_int32(0)
    L = lib()
    _check(L.adst_trace_kernels(None, 0, ctypes.byref(n)))
    buf = (adst_kernel_stat * max(n.value, 1))()
    _check(L.adst_trace_kernels(buf, n.value, ctypes.byref(n)))
    return [{"name": s.name.decode(), "phase": PHASE_NAMES[s.phase], "launches": s.launches,
             "ms_sum": s.ms_sum, "ms_min": s.ms_min, "ms_max": s.ms_max,
             "alg_bytes_sum": s.alg_bytes_sum} for s in buf[:n.value]]


def adst_copy(dst, src, nbytes, stream=None):
    _check(lib().adst_copy(_ptr(dst), _ptr(src), int(nbytes), _stream(stream)))


def adst_ilp_solve(arrays, events, limit):
    """arrays: sequence of (size, overhead, cost); events: sequence of
    ("alloc"|"free", amount), (kind, array_index) or ("path",).
    Returns (store flags, adst_ilp_info)."""
    n = len(arrays)
    A = (adst_ilp_array * max(n, 1))()
    for k, (size, overhead, cost) in enumerate(arrays):
        A[k].size, A[k].overhead, A[k].cost = size, overhead, cost
    E = (adst_ilp_event * max(len(events), 1))()
    for k, ev in enumerate(events):
        E[k].kind = ILP_EVENTS[ev[0]]
        if ev[0] in ("alloc", "free"):
            E[k].amount = float(ev[1])
        elif ev[0] != "path":
            E[k].array = int(ev[1])
    store = (ctypes.c_int32 * max(n, 1))()
    info = adst_ilp_info()
    _check(lib().adst_ilp_solve(A, n, E, len(events), float(limit), store, ctypes.byref(info)))
    return [store[k] for k in range(n)], info


# ------------------------------------------------------------ conveniences
def _dtype_code(t):
    import torch
    if t.dtype == torch.float64:
        return ADST_F64
    if t.dtype == torch.float32:
        return ADST_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _dims(shape):
    if len(shape) == 2:
        return (shape[1], shape[0], 1)
    if len(shape) == 3:
        return (shape[2], shape[1], shape[0])
    raise ValueError(f"expected a 2-D or 3-D array, got {tuple(shape)}")


def _check_tensors(x0, **others):
    """The kernels read and write row-major, unpadded arrays of one dtype on
    one device: reject anything else before any plan or launch."""
    import torch
    if not torch.is_tensor(x0):
        raise ValueError("x0 must be a torch tensor")
    _dtype_code(x0)
    _dims(x0.shape)
    if not x0.is_contiguous():
        raise ValueError("x0 must be contiguous (row-major, unpadded)")
    for name, t in others.items():
        if t is None:
            continue
        if not torch.is_tensor(t):
            raise ValueError(f"{name} must be a torch tensor")
        if t.dtype != x0.dtype:
            raise ValueError(f"{name} has dtype {t.dtype}, x0 has {x0.dtype}")
        if tuple(t.shape) != tuple(x0.shape):
            raise ValueError(f"{name} has shape {tuple(t.shape)}, x0 has {tuple(x0.shape)}")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous (row-major, unpadded)")
        if t.device != x0.device:
            raise ValueError(f"{name} is on {t.device}, x0 on {x0.device}")
    if x0.device.type != "cuda":
        raise ValueError(f"x0 must be on a GPU, not {x0.device}")


def forward(kind, x0, coeff=None, steps=1, params=None, stream=None, lim=None, flags=0):
    """x_T on the device of x0 (torch tensors, row-major)."""
    import torch
    _check_tensors(x0, coeff=coeff)
    prob = make_problem(kind, _dtype_code(x0), _dims(x0.shape), params, flags, lim)
    xT = torch.empty_like(x0)
    info = adst_plan(prob, steps, 1 << 62, ADST_SCHED_STORE_ALL)
    ws = torch.empty(max(info.fwd_workspace_bytes, 1), dtype=torch.uint8, device=x0.device)
    adst_forward(prob, x0, coeff, steps, xT, ws, info.fwd_workspace_bytes, stream)
    return xT


def vjp(kind, x0, coeff=None, steps=1, loss=ADST_LOSS_HALF_SQ, aux=None, budget_bytes=None,
        sched=ADST_SCHED_AUTO, want_dcoeff=False, params=None, flags=0, stream=None, ws=None,
        want_xT=True, want_dparams=False, lim=None):
    """Allocate outputs and workspace with torch and run adst_vjp.

    budget_bytes=None means unlimited (store-all). Returns a dict with dx0,
    dK (or None), xT (None unless want_xT), loss (0-d device tensor),
    dparams (device double[2], or None unless want_dparams), info and the
    workspace."""
    import torch
    _check_tensors(x0, coeff=coeff, aux=aux)
    prob = make_problem(kind, _dtype_code(x0), _dims(x0.shape), params, flags, lim)
    if budget_bytes is None:
        budget_bytes = (1 << 63)
    grads = (ADST_GRAD_COEFF if want_dcoeff else 0) | (ADST_GRAD_PARAMS if want_dparams else 0)
    info = adst_plan(prob, steps, budget_bytes, sched, grads)
    if ws is None or ws.numel() < info.workspace_bytes:
        ws = torch.empty(info.workspace_bytes, dtype=torch.uint8, device=x0.device)
    dx0 = torch.empty_like(x0)
    dK = torch.empty_like(x0) if want_dcoeff else None
    xT = torch.empty_like(x0) if want_xT else None
    L = torch.empty((), dtype=torch.float64, device=x0.device)
    dp = torch.empty(2, dtype=torch.float64, device=x0.device) if want_dparams else None
    info = adst_vjp(prob, x0, coeff, steps, loss, aux, budget_bytes, sched, dx0, dK, xT, L, dp,
                    ws, ws.numel(), stream)
    return {"dx0": dx0, "dK": dK, "xT": xT, "loss": L, "dparams": dp, "info": info, "ws": ws}
