"""Pins of the oracle's gradients of the scalar step constants (CPU only).

dL/dp accumulates, over every step t and point c, g_t[c] times the step's
partial dF_c/dp at x_{t-1} (a constant read by every update is a
multiply-read input, Sec. II). Pinned against:
  * closed forms from dense operators: x_T = M(p)^T x0, so
    dx_T/dp = sum_k M^(T-1-k) M'(p) M^k x0, with M and M' = dM/dp built
    from Kronecker path-graph adjacencies (and, for the in-place kind, the
    derivative of the matrix-splitting solve);
  * central finite differences of the loss in p (all kinds, nonlinear ones
    included);
  * the dot-product identity with the oracle's tangent sweep along p, itself
    checked against finite differences of the forward map.
"""
import numpy as np
import pytest

import oracle
from oracle import (ALLENCAHN3D7, DOT_W, GAUSSSEIDEL2D5, HALF_SQ, HALF_SQ_DIFF, JACOBI2D5, SEED,
                    VARDIFF2D9)
from tests import linalg_forms as lf


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def tangent_of_power(M, dM, x0, T):
    """d/dp (M^T x0) for M' = dM, by the recursion xd <- M xd + M' x."""
    x, xd = x0.copy(), np.zeros_like(x0)
    for _ in range(T):
        xd = M @ xd + dM @ x
        x = M @ x
    return x, xd


def interior_mask(ny, nx):
    yy, xx = np.divmod(np.arange(nx * ny), nx)
    return ((xx > 0) & (xx < nx - 1) & (yy > 0) & (yy < ny - 1)).astype(float)


@pytest.mark.parametrize("ny,nx,T", [(5, 6, 3), (9, 7, 8)])
def test_jacobi_dw_closed_form(ny, nx, T):
    w = 0.2
    x0 = rng(1).uniform(0, 1, (ny, nx)).reshape(-1)
    M = lf.jacobi_matrix(ny, nx, w)
    dM = interior_mask(ny, nx)[:, None] * (np.eye(nx * ny) + lf.grid2d_axis(ny, nx))
    xT, dxT = tangent_of_power(M, dM, x0, T)
    *_, dp = oracle.vjp(JACOBI2D5, x0.reshape(ny, nx), steps=T, loss=HALF_SQ, want_dp=True)
    ref = float(xT @ dxT)  # L = 0.5 |x_T|^2
    assert abs(dp[0] - ref) <= 1e-12 * abs(ref) and dp[1] == 0.0


@pytest.mark.parametrize("ny,nx,T", [(5, 6, 3), (8, 9, 6)])
def test_gauss_seidel_dw_closed_form(ny, nx, T):
    """M(w) = A(w)^-1 B(w) with A = I - wDL, B = wD(I+U) + (I-D):
    M' = A^-1 (B' - A' M) = A^-1 (D(I+U) + D L M)."""
    w = 0.2
    n = nx * ny
    x0 = rng(2).uniform(0, 1, (ny, nx)).reshape(-1)
    Y = rng(3).uniform(0, 1, n)
    D = np.diag(interior_mask(ny, nx))
    Adj = lf.grid2d_axis(ny, nx)
    L, U = np.tril(Adj, -1), np.triu(Adj, 1)
    M = lf.gauss_seidel_matrix(ny, nx, w)
    dM = np.linalg.solve(np.eye(n) - w * D @ L, D @ (np.eye(n) + U) + D @ L @ M)
    xT, dxT = tangent_of_power(M, dM, x0, T)
    *_, dp = oracle.vjp(GAUSSSEIDEL2D5, x0.reshape(ny, nx), steps=T, loss=HALF_SQ_DIFF,
                        aux=Y.reshape(ny, nx), want_dp=True)
    ref = float((xT - Y) @ dxT)
    assert abs(dp[0] - ref) <= 1e-12 * abs(ref) and dp[1] == 0.0


@pytest.mark.parametrize("shape,T", [((3, 4, 5), 4), ((2, 3, 6), 6)])
def test_allencahn_dD_and_dC_at_zero_cubic(shape, T):
    """With C = 0 the step is the heat operator M = I + D(A - 6I): dM/dD =
    A - 6I; and dL/dC = -sum_t <g_t, x_{t-1}^3>, g_t = (M^T)^(T-t) W."""
    nz, ny, nx = shape
    n = nx * ny * nz
    x0 = rng(4).uniform(-1, 1, n)
    W = rng(5).standard_normal(n)
    D = 0.1
    M = lf.heat3d_matrix(nz, ny, nx, D)
    dM = lf.grid3d_faces(nz, ny, nx) - 6.0 * np.eye(n)
    xT, dxT = tangent_of_power(M, dM, x0, T)
    states = [x0]
    for _ in range(T):
        states.append(M @ states[-1])
    dC = 0.0
    g = W.copy()
    for t in range(T, 0, -1):
        dC -= float(g @ states[t - 1] ** 3)
        g = M.T @ g
    *_, dp = oracle.vjp(ALLENCAHN3D7, x0.reshape(shape), steps=T, loss=DOT_W,
                        aux=W.reshape(shape), params=(D, 0.0), want_dp=True)
    assert abs(dp[0] - W @ dxT) <= 1e-12 * abs(W @ dxT)
    assert abs(dp[1] - dC) <= 1e-12 * abs(dC)


@pytest.mark.parametrize("ny,nx,T", [(5, 6, 4), (7, 9, 6)])
def test_vardiff_ddt_closed_form(ny, nx, T):
    """M(dt) = I + dt Lap(K): dM/ddt = Lap(K), the weighted graph Laplacian."""
    x0 = rng(6).uniform(0, 1, (ny, nx))
    K = rng(7).uniform(0.5, 1.5, (ny, nx))
    Y = rng(8).uniform(0, 1, (ny, nx)).reshape(-1)
    dt = 0.1
    M = lf.vardiff_matrix(K, dt)
    dM = (M - np.eye(nx * ny)) / dt
    xT, dxT = tangent_of_power(M, dM, x0.reshape(-1), T)
    *_, dp = oracle.vjp(VARDIFF2D9, x0, K=K, steps=T, loss=HALF_SQ_DIFF, aux=Y.reshape(ny, nx),
                        want_dp=True)
    ref = float((xT - Y) @ dxT)
    assert abs(dp[0] - ref) <= 1e-12 * abs(ref) and dp[1] == 0.0


def _loss(kind, x0, K, T, loss, aux, params):
    xT = oracle.forward(kind, x0, K=K, steps=T, params=params)
    if loss == HALF_SQ:
        return 0.5 * np.sum(xT * xT)
    if loss == HALF_SQ_DIFF:
        return 0.5 * np.sum((xT - aux) ** 2)
    return np.sum(aux * xT)


FD_CASES = [
    (JACOBI2D5, (6, 7), 5, HALF_SQ, (0.2, 0.0), (0,)),
    (GAUSSSEIDEL2D5, (6, 7), 5, HALF_SQ, (0.2, 0.0), (0,)),
    (ALLENCAHN3D7, (3, 4, 5), 4, DOT_W, (0.1, 0.1), (0, 1)),
    (ALLENCAHN3D7, (2, 3, 4), 5, HALF_SQ, (0.05, 0.6), (0, 1)),  # strong cubic
    (VARDIFF2D9, (6, 5), 4, HALF_SQ_DIFF, (0.1, 0.0), (0,)),
]


@pytest.mark.parametrize("kind,shape,T,loss,params,which", FD_CASES)
def test_fd_in_each_constant(kind, shape, T, loss, params, which):
    r = rng(10)
    lo = -1.0 if kind == ALLENCAHN3D7 else 0.0
    x0 = r.uniform(lo, 1, shape)
    K = r.uniform(0.5, 1.5, shape) if kind == VARDIFF2D9 else None
    aux = r.standard_normal(shape)
    *_, dp = oracle.vjp(kind, x0, K=K, steps=T, loss=loss, aux=aux, params=params, want_dp=True)
    for k in which:
        h = 1e-6 * max(abs(params[k]), 1.0)
        pp, pm = list(params), list(params)
        pp[k] += h
        pm[k] -= h
        fd = (_loss(kind, x0, K, T, loss, aux, pp) - _loss(kind, x0, K, T, loss, aux, pm)) / (2 * h)
        assert abs(fd - dp[k]) <= 1e-7 * max(abs(fd), 1e-12), (k, fd, dp[k])


DOT_CASES = [
    (JACOBI2D5, (13, 17), 6), (GAUSSSEIDEL2D5, (13, 17), 6), (ALLENCAHN3D7, (5, 6, 7), 5),
    (VARDIFF2D9, (11, 15), 5),
]


@pytest.mark.parametrize("kind,shape,T", DOT_CASES)
def test_dot_product_identity_along_the_constants(kind, shape, T):
    """<xdot_T, w> with xdot the tangent along (v = 0, pdot) equals
    pdot . dL/dp for the cotangent w (loss SEED)."""
    r = rng(11)
    lo = -1.0 if kind == ALLENCAHN3D7 else 0.0
    x0 = r.uniform(lo, 1, shape)
    K = r.uniform(0.5, 1.5, shape) if kind == VARDIFF2D9 else None
    w = r.standard_normal(shape)
    pdot = (0.7, -1.3) if kind == ALLENCAHN3D7 else (0.7, 0.0)
    _, xd = oracle.jvp(kind, x0, np.zeros(shape), K=K, kappa=None if K is None else np.zeros(shape),
                       steps=T, pdot=pdot)
    *_, dp = oracle.vjp(kind, x0, K=K, steps=T, loss=SEED, aux=w, want_dp=True)
    lhs = float(np.sum(xd * w))
    rhs = pdot[0] * dp[0] + pdot[1] * dp[1]
    assert abs(lhs - rhs) <= 1e-12 * max(abs(lhs), 1e-30)


@pytest.mark.parametrize("kind,shape,T", DOT_CASES)
def test_tangent_along_the_constants_matches_fd(kind, shape, T):
    r = rng(12)
    lo = -1.0 if kind == ALLENCAHN3D7 else 0.0
    x0 = r.uniform(lo, 1, shape)
    K = r.uniform(0.5, 1.5, shape) if kind == VARDIFF2D9 else None
    base = oracle.default_params(kind)
    pdot = (0.7, -1.3) if kind == ALLENCAHN3D7 else (0.7, 0.0)
    _, xd = oracle.jvp(kind, x0, np.zeros(shape), K=K, kappa=None if K is None else np.zeros(shape),
                       steps=T, pdot=pdot)
    h = 1e-7
    pp = (base[0] + h * pdot[0], base[1] + h * pdot[1])
    pm = (base[0] - h * pdot[0], base[1] - h * pdot[1])
    fd = (oracle.forward(kind, x0, K=K, steps=T, params=pp) -
          oracle.forward(kind, x0, K=K, steps=T, params=pm)) / (2 * h)
    assert np.linalg.norm(xd - fd) <= 1e-6 * np.linalg.norm(fd)


def test_zero_steps_and_f32():
    x0 = rng(13).uniform(0, 1, (7, 9))
    *_, dp = oracle.vjp(JACOBI2D5, x0, steps=0, loss=HALF_SQ, want_dp=True)
    assert dp == (0.0, 0.0)
    *_, d64 = oracle.vjp(VARDIFF2D9, x0, K=np.ones_like(x0) + x0, steps=8, loss=HALF_SQ,
                         want_dp=True)
    *_, d32 = oracle.vjp(VARDIFF2D9, x0.astype(np.float32), K=(np.ones_like(x0) + x0).astype(np.float32),
                         steps=8, loss=HALF_SQ, want_dp=True)
    assert abs(d32[0] - d64[0]) <= 1e-4 * abs(d64[0])
