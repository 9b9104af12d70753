"""Pins of the oracle's limiter (a data-dependent branch in every step)
(CPU only).

Each step's new value y becomes lo if y < lo, hi if y > hi, and is kept
otherwise; its derivative is that of the branch taken (1 where kept, 0
where clamped), which the reverse sweep recovers by re-evaluating y from
x_{t-1}. Pinned against:
  * an independent dense formulation of the linear kinds: x_t =
    clip(M x_{t-1}, lo, hi) with numpy, masks m_t = (lo <= M x_{t-1} <= hi),
    dx0 = (diag(m_1) M)^T ... (diag(m_T) M)^T g (checked to stay clear of the
    bounds so the two formulations take the same branches);
  * central finite differences away from the kinks, nonlinear kind included;
  * the dot-product identity with the tangent sweep through the branches;
  * invariants: infinite bounds change nothing (bit for bit); bounds the
    values never leave change nothing; a collapsed interval [c, c] clamps
    everything, so nothing flows back.
"""
import numpy as np
import pytest

import oracle
from oracle import (ALLENCAHN3D7, DOT_W, GAUSSSEIDEL2D5, HALF_SQ, HALF_SQ_DIFF, JACOBI2D5, SEED,
                    VARDIFF2D9)
from tests import linalg_forms as lf


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def dense_limited(M, x0, T, lo, hi, g_of_xT):
    """x_T and dx0 of the limited linear map, with the smallest distance of
    any pre-limiter value to a bound."""
    xs, masks, margin = [x0], [], np.inf
    for _ in range(T):
        y = M @ xs[-1]
        masks.append(((y >= lo) & (y <= hi)).astype(float))
        # values exactly on a bound (a value clamped earlier and carried by an
        # identity row) are exact in both formulations; the rest must be clear
        dist = np.minimum(np.abs(y - lo), np.abs(y - hi))
        if np.any(dist > 0):
            margin = min(margin, np.min(dist[dist > 0]))
        xs.append(np.clip(y, lo, hi))
    g = g_of_xT(xs[-1])
    for t in range(T, 0, -1):
        g = M.T @ (masks[t - 1] * g)
    active = sum(float(np.sum(1 - m)) for m in masks)
    return xs[-1], g, margin, active


@pytest.mark.parametrize("ny,nx,T,lim", [(6, 7, 5, (0.35, 0.65)), (9, 11, 8, (0.3, 0.7))])
def test_jacobi_limited_dense_form(ny, nx, T, lim):
    x0 = rng(1).uniform(0, 1, (ny, nx))
    M = lf.jacobi_matrix(ny, nx)
    xT, dx0, margin, active = dense_limited(M, x0.reshape(-1), T, *lim, lambda x: x)
    assert margin > 1e-9 and active > 0  # the branch matters and both sides take the same one
    d, _, x, _ = oracle.vjp(JACOBI2D5, x0, steps=T, loss=HALF_SQ, lim=lim)
    assert np.max(np.abs(x.reshape(-1) - xT)) < 1e-14
    assert np.linalg.norm(d.reshape(-1) - dx0) <= 1e-13 * np.linalg.norm(dx0)


@pytest.mark.parametrize("ny,nx,T,lim", [(7, 6, 6, (0.3, 0.7))])
def test_vardiff_limited_dense_form(ny, nx, T, lim):
    x0 = rng(2).uniform(0, 1, (ny, nx))
    K = rng(3).uniform(0.5, 1.5, (ny, nx))
    Y = rng(4).uniform(0, 1, (ny, nx)).reshape(-1)
    M = lf.vardiff_matrix(K)
    xT, dx0, margin, active = dense_limited(M, x0.reshape(-1), T, *lim, lambda x: x - Y)
    assert margin > 1e-9 and active > 0
    d, _, x, _ = oracle.vjp(VARDIFF2D9, x0, K=K, steps=T, loss=HALF_SQ_DIFF,
                            aux=Y.reshape(ny, nx), lim=lim)
    assert np.max(np.abs(x.reshape(-1) - xT)) < 1e-14
    assert np.linalg.norm(d.reshape(-1) - dx0) <= 1e-13 * np.linalg.norm(dx0)


def test_allencahn_linear_part_limited_dense_form():
    shape = (3, 4, 5)
    x0 = rng(5).uniform(-1, 1, shape)
    W = rng(6).standard_normal(shape).reshape(-1)
    M = lf.heat3d_matrix(*shape, D=0.1)
    lim = (-0.25, 0.3)
    xT, dx0, margin, active = dense_limited(M, x0.reshape(-1), 4, *lim, lambda x: W)
    assert margin > 1e-9 and active > 0
    d, _, x, _ = oracle.vjp(ALLENCAHN3D7, x0, steps=4, loss=DOT_W, aux=W.reshape(shape),
                            params=(0.1, 0.0), lim=lim)
    assert np.max(np.abs(x.reshape(-1) - xT)) < 1e-14
    assert np.linalg.norm(d.reshape(-1) - dx0) <= 1e-13 * np.linalg.norm(dx0)


def _loss(kind, x0, K, T, loss, aux, lim):
    xT = oracle.forward(kind, x0, K=K, steps=T, lim=lim)
    if loss == HALF_SQ:
        return 0.5 * np.sum(xT * xT)
    return np.sum(aux * xT)


@pytest.mark.parametrize("kind,shape,lim,loss", [
    (JACOBI2D5, (6, 5), (0.3, 0.7), HALF_SQ),
    (ALLENCAHN3D7, (3, 4, 5), (-0.5, 0.55), DOT_W),
    (VARDIFF2D9, (6, 5), (0.25, 0.75), DOT_W),
])
def test_fd_away_from_the_kinks(kind, shape, lim, loss):
    r = rng(7)
    lo = -1.0 if kind == ALLENCAHN3D7 else 0.0
    x0 = r.uniform(lo, 1, shape)
    K = r.uniform(0.5, 1.5, shape) if kind == VARDIFF2D9 else None
    aux = r.standard_normal(shape)
    T = 4
    # every pre-limiter value along the trajectory stays clear of the bounds
    x = x0.copy()
    clamped = 0
    for _ in range(T):
        y = oracle.forward(kind, x, K=K, steps=1)
        dist = np.minimum(np.abs(y - lim[0]), np.abs(y - lim[1]))
        assert np.min(dist[dist > 0]) > 1e-5  # exact hits: clamped values carried over
        clamped += int(np.sum((y < lim[0]) | (y > lim[1])))
        x = oracle.forward(kind, x, K=K, steps=1, lim=lim)
    assert clamped > 0
    dx0, *_ = oracle.vjp(kind, x0, K=K, steps=T, loss=loss, aux=aux, lim=lim)
    h = 1e-7
    fd = np.zeros_like(x0)
    for idx in np.ndindex(*shape):
        xp, xm = x0.copy(), x0.copy()
        xp[idx] += h
        xm[idx] -= h
        fd[idx] = (_loss(kind, xp, K, T, loss, aux, lim) - _loss(kind, xm, K, T, loss, aux, lim)) / (2 * h)
    assert np.max(np.abs(fd - dx0)) <= 1e-6 * max(np.max(np.abs(fd)), 1e-30)


@pytest.mark.parametrize("kind,shape,lim", [
    (JACOBI2D5, (13, 17), (0.4, 0.6)), (ALLENCAHN3D7, (5, 6, 7), (-0.3, 0.35)),
    (VARDIFF2D9, (11, 15), (0.3, 0.7))])
def test_dot_product_identity_through_the_branches(kind, shape, lim):
    r = rng(8)
    lo = -1.0 if kind == ALLENCAHN3D7 else 0.0
    x0 = r.uniform(lo, 1, shape)
    K = r.uniform(0.5, 1.5, shape) if kind == VARDIFF2D9 else None
    v, w = r.standard_normal(shape), r.standard_normal(shape)
    kap = np.zeros(shape) if K is not None else None
    _, xd = oracle.jvp(kind, x0, v, K=K, kappa=kap, steps=6, lim=lim)
    dx0, *_ = oracle.vjp(kind, x0, K=K, steps=6, loss=SEED, aux=w, lim=lim)
    lhs, rhs = float(np.sum(xd * w)), float(np.sum(v * dx0))
    assert abs(lhs - rhs) <= 1e-12 * max(abs(lhs), 1e-30)


def test_invariants():
    x0 = rng(9).uniform(0, 1, (20, 23))
    K = rng(10).uniform(0.5, 1.5, (20, 23))
    for kind, kk in ((JACOBI2D5, None), (VARDIFF2D9, K)):
        a = oracle.vjp(kind, x0, K=kk, steps=9, loss=HALF_SQ)
        b = oracle.vjp(kind, x0, K=kk, steps=9, loss=HALF_SQ, lim=(-np.inf, np.inf))
        c = oracle.vjp(kind, x0, K=kk, steps=9, loss=HALF_SQ, lim=(0.0, 1.0))  # never left
        for u, v in ((a, b), (a, c)):
            assert np.array_equal(u[0], v[0]) and np.array_equal(u[2], v[2])
    # a collapsed interval clamps every value: x_T is constant, no gradient flows
    dx0, _, xT, _ = oracle.vjp(JACOBI2D5, x0, steps=3, loss=HALF_SQ, lim=(0.5, 0.5))
    assert np.all(xT == 0.5) and np.all(dx0 == 0.0)
    # the in-place kind has no limiter
    with pytest.raises(ValueError):
        oracle.forward(GAUSSSEIDEL2D5, x0, steps=1, lim=(0.0, 1.0))
