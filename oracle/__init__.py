"""Plain CPU oracle for the stencil VJP (TEST INFRASTRUCTURE ONLY).

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package. The product library never calls it.

``forward``, ``vjp`` and ``jvp`` wrap the store-all tape implementation in
``oracle.cpp`` (scatter-form reverse sweep; see that file's header for the
step definitions, the evaluation order and the loss conventions).
``checkpoint`` holds the checkpoint-count definitions used to check the
planner.
"""
import ctypes
import os

import numpy as np

JACOBI2D5, ALLENCAHN3D7, VARDIFF2D9, GAUSSSEIDEL2D5 = 0, 1, 2, 3
HALF_SQ, DOT_W, HALF_SQ_DIFF, SEED = 0, 1, 2, 3

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _build
        _build.build()
    lib = ctypes.CDLL(_LIB_PATH)
    vp, i64p, dp = ctypes.c_void_p, ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_double)
    ci = ctypes.c_int
    for suf in ("f64", "f32"):
        f = getattr(lib, "oracle_forward_" + suf)
        f.argtypes = [ci, i64p, dp, dp, vp, vp, ci, vp]
        f.restype = ci
        f = getattr(lib, "oracle_vjp_" + suf)
        f.argtypes = [ci, i64p, dp, dp, vp, vp, ci, ci, vp, vp, vp, vp, dp, dp]
        f.restype = ci
        f = getattr(lib, "oracle_jvp_" + suf)
        f.argtypes = [ci, i64p, dp, dp, vp, vp, vp, vp, dp, ci, vp, vp]
        f.restype = ci
    _lib = lib
    return lib


def default_params(kind):
    """The step constants of the kinds: Jacobi and Gauss-Seidel w = 0.2;
    Allen-Cahn diffusion 0.1 and cubic 0.1; variable-coefficient diffusion
    dt = 0.1."""
    return {JACOBI2D5: (0.2, 0.0), ALLENCAHN3D7: (0.1, 0.1), VARDIFF2D9: (0.1, 0.0),
            GAUSSSEIDEL2D5: (0.2, 0.0)}[kind]


def _suffix(dtype):
    dtype = np.dtype(dtype)
    if dtype == np.float64:
        return "f64"
    if dtype == np.float32:
        return "f32"
    raise TypeError(f"oracle supports float64/float32, not {dtype}")


def _dims(shape):
    """Row-major [nz][ny][nx] (or [ny][nx]) -> (nx, ny, nz)."""
    if len(shape) == 2:
        return (shape[1], shape[0], 1)
    if len(shape) == 3:
        return (shape[2], shape[1], shape[0])
    raise ValueError(f"expected a 2-D or 3-D array, got shape {shape}")


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _lim(lim):
    """Limiter bounds (lo, hi) as a C array, or None for no limiter."""
    return None if lim is None else (ctypes.c_double * 2)(float(lim[0]), float(lim[1]))


def _prep(x0, *others):
    x0 = np.ascontiguousarray(x0)
    out = [x0]
    for o in others:
        out.append(None if o is None else np.ascontiguousarray(o, dtype=x0.dtype))
    return out


def _args(kind, x0, params):
    n = (ctypes.c_int64 * 3)(*_dims(x0.shape))
    p = (ctypes.c_double * 2)(*(params if params is not None else default_params(kind)))
    return n, p


def forward(kind, x0, K=None, steps=1, params=None, lim=None):
    """x_T after ``steps`` forward steps (lim = limiter bounds (lo, hi))."""
    x0, K = _prep(x0, K)
    n, p = _args(kind, x0, params)
    xT = np.empty_like(x0)
    rc = getattr(_load(), "oracle_forward_" + _suffix(x0.dtype))(
        kind, n, p, _lim(lim), _ptr(x0), _ptr(K), steps, _ptr(xT))
    if rc:
        raise ValueError("oracle_forward rejected the problem")
    return xT


def vjp(kind, x0, K=None, steps=1, loss=HALF_SQ, aux=None, want_dK=False, params=None,
        want_dp=False, lim=None):
    """Store-all reverse-mode gradient. Returns (dx0, dK or None, x_T, L), and
    with want_dp also the gradients of the two step constants (dL/dp[0],
    dL/dp[1]) as a fifth element."""
    x0, K, aux = _prep(x0, K, aux)
    n, p = _args(kind, x0, params)
    dx0 = np.empty_like(x0)
    dK = np.empty_like(x0) if want_dK else None
    xT = np.empty_like(x0)
    L = ctypes.c_double(0.0)
    dpv = (ctypes.c_double * 2)(0.0, 0.0)
    rc = getattr(_load(), "oracle_vjp_" + _suffix(x0.dtype))(
        kind, n, p, _lim(lim), _ptr(x0), _ptr(K), steps, loss, _ptr(aux), _ptr(dx0), _ptr(dK),
        _ptr(xT), ctypes.byref(L), dpv if want_dp else None)
    if rc:
        raise ValueError("oracle_vjp rejected the problem")
    if want_dp:
        return dx0, dK, xT, L.value, (dpv[0], dpv[1])
    return dx0, dK, xT, L.value


def jvp(kind, x0, v, K=None, kappa=None, steps=1, params=None, pdot=None, lim=None):
    """Tangent-linear sweep. Returns (x_T, xdot_T) for direction (v, kappa,
    pdot), pdot the direction of the two step constants."""
    x0, v, K, kappa = _prep(x0, v, K, kappa)
    n, p = _args(kind, x0, params)
    xT = np.empty_like(x0)
    xdT = np.empty_like(x0)
    pd = None if pdot is None else (ctypes.c_double * 2)(*pdot)
    rc = getattr(_load(), "oracle_jvp_" + _suffix(x0.dtype))(
        kind, n, p, _lim(lim), _ptr(x0), _ptr(K), _ptr(v), _ptr(kappa), pd, steps, _ptr(xT),
        _ptr(xdT))
    if rc:
        raise ValueError("oracle_jvp rejected the problem")
    return xT, xdT
