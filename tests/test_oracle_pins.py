"""Pins of the CPU oracle against facts fixed by mathematics (CPU only).

The paper prints no stencil gradient, so each part of the oracle is pinned
to something other than itself:
  * closed forms of the linear steps (dense operators built from Kronecker
    products, numpy matrix powers): x_T = M^T x0 and dx0 = (M^T)^T g_T;
  * the textbook 9-point Laplacian for K = 1;
  * central finite differences of the forward map (oracle.forward only);
  * the adjoint dot-product identity <J v, w> = <v, J^T w> with the oracle's
    own tangent-linear sweep, itself checked against finite differences;
  * invariants (fixed points, conservation, zero stays zero, symmetric
    operators) and hand-derived cases.
"""
import os

import numpy as np
import pytest

import oracle
from oracle import (ALLENCAHN3D7, DOT_W, GAUSSSEIDEL2D5, HALF_SQ, HALF_SQ_DIFF, JACOBI2D5, SEED,
                    VARDIFF2D9)
from tests import linalg_forms as lf

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    nb = np.linalg.norm(b)
    return np.linalg.norm(a - b) / (nb if nb > 0 else 1.0)


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


# ---------------------------------------------------------------- closed forms
@pytest.mark.parametrize("ny,nx,T", [(3, 3, 1), (9, 11, 7), (16, 16, 10)])
def test_jacobi_closed_form(ny, nx, T):
    x0 = rng(1).uniform(0, 1, (ny, nx))
    M = lf.jacobi_matrix(ny, nx)
    MT = np.linalg.matrix_power(M, T)
    xT_ref = (MT @ x0.reshape(-1)).reshape(ny, nx)
    dx0_ref = (MT.T @ xT_ref.reshape(-1)).reshape(ny, nx)  # HALF_SQ: g_T = x_T
    dx0, _, xT, L = oracle.vjp(JACOBI2D5, x0, steps=T, loss=HALF_SQ)
    assert rel(xT, xT_ref) < 1e-13
    assert rel(dx0, dx0_ref) < 1e-13
    assert abs(L - 0.5 * np.sum(xT_ref ** 2)) <= 1e-13 * abs(L)


@pytest.mark.parametrize("ny,nx,T", [(3, 3, 1), (4, 4, 1), (9, 11, 7), (16, 13, 10), (2, 7, 3)])
def test_gauss_seidel_closed_form(ny, nx, T):
    """x_T = M^T x0 and dx0 = (M^T)^T (x_T - Y) with M the matrix-splitting
    form of one in-place sweep (a triangular solve, not a loop over points)."""
    x0 = rng(8).uniform(0, 1, (ny, nx))
    Y = rng(9).uniform(0, 1, (ny, nx))
    M = lf.gauss_seidel_matrix(ny, nx)
    MT = np.linalg.matrix_power(M, T)
    xT_ref = MT @ x0.reshape(-1)
    dx0_ref = MT.T @ (xT_ref - Y.reshape(-1))
    dx0, _, xT, _ = oracle.vjp(GAUSSSEIDEL2D5, x0, steps=T, loss=HALF_SQ_DIFF, aux=Y)
    assert rel(xT.reshape(-1), xT_ref) < 1e-13
    assert rel(dx0.reshape(-1), dx0_ref) < 1e-13
    # the in-place sweep is not the Jacobi step
    if ny >= 4 and nx >= 4:
        J = np.linalg.matrix_power(lf.jacobi_matrix(ny, nx), T)
        assert rel(J @ x0.reshape(-1), xT_ref) > 1e-3


def test_gauss_seidel_converges_to_harmonic():
    """With w = 1/5 the fixed point satisfies 4 x[c] = sum of the four
    neighbours: many sweeps reach the discrete harmonic function with the
    ring as Dirichlet data (Gauss-Seidel converges for this system)."""
    x0 = rng(41).uniform(0, 1, (9, 12))
    ref = lf.laplace_dirichlet_solution(x0)
    xT = oracle.forward(GAUSSSEIDEL2D5, x0, steps=1500)
    assert np.max(np.abs(xT - ref)) < 1e-12


@pytest.mark.parametrize("shape,T", [((3, 4, 5), 4), ((6, 5, 7), 6), ((1, 1, 1), 3)])
def test_allencahn_linear_part_closed_form(shape, T):
    """With the cubic coefficient set to 0 the step is the 3-D heat step
    with zero ghost values: a Kronecker-sum operator."""
    nz, ny, nx = shape
    x0 = rng(2).uniform(-1, 1, shape)
    W = rng(3).standard_normal(shape)
    M = lf.heat3d_matrix(nz, ny, nx, D=0.1)
    MT = np.linalg.matrix_power(M, T)
    xT_ref = MT @ x0.reshape(-1)
    dx0_ref = MT.T @ W.reshape(-1)  # DOT_W: g_T = W
    dx0, _, xT, L = oracle.vjp(ALLENCAHN3D7, x0, steps=T, loss=DOT_W, aux=W, params=(0.1, 0.0))
    assert rel(xT.reshape(-1), xT_ref) < 1e-13
    assert rel(dx0.reshape(-1), dx0_ref) < 1e-13
    assert abs(L - W.reshape(-1) @ xT_ref) <= 1e-12 * max(1.0, abs(L))


@pytest.mark.parametrize("ny,nx,T", [(5, 6, 4), (12, 9, 8)])
def test_vardiff_closed_form_variable_K(ny, nx, T):
    """The step is linear in x for fixed K: x_T = M(K)^T x0."""
    x0 = rng(4).uniform(0, 1, (ny, nx))
    K = rng(5).uniform(0.5, 1.5, (ny, nx))
    Y = rng(6).uniform(0, 1, (ny, nx))
    M = lf.vardiff_matrix(K, dt=0.1)
    MT = np.linalg.matrix_power(M, T)
    xT_ref = MT @ x0.reshape(-1)
    dx0_ref = MT.T @ (xT_ref - Y.reshape(-1))  # HALF_SQ_DIFF: g_T = x_T - Y
    dx0, _, xT, _ = oracle.vjp(VARDIFF2D9, x0, K=K, steps=T, loss=HALF_SQ_DIFF, aux=Y)
    assert rel(xT.reshape(-1), xT_ref) < 1e-13
    assert rel(dx0.reshape(-1), dx0_ref) < 1e-13


def test_vardiff_K1_is_textbook_nine_point():
    """With K = 1 the conservative edge form is the isotropic 9-point
    Laplacian (4*axis + diagonal - 20*centre)/6 on interior points."""
    x = rng(7).uniform(0, 1, (10, 13))
    K = np.ones_like(x)
    dt = 0.1
    x1 = oracle.forward(VARDIFF2D9, x, K=K, steps=1, params=(dt, 0.0))
    ref = x[1:-1, 1:-1] + dt * lf.nine_point_laplacian_interior(x)
    assert np.max(np.abs(x1[1:-1, 1:-1] - ref)) < 1e-15


# ------------------------------------------------------- finite differences
def _loss_value(loss, xT, aux):
    if loss == HALF_SQ:
        return 0.5 * np.sum(xT * xT)
    if loss == HALF_SQ_DIFF:
        d = xT - aux
        return 0.5 * np.sum(d * d)
    return np.sum(aux * xT)


def _fd_check(kind, x0, K, T, loss, aux, want_dK, params=None, h=1e-5, tol=1e-7):
    dx0, dK, _, _ = oracle.vjp(kind, x0, K=K, steps=T, loss=loss, aux=aux, want_dK=want_dK,
                               params=params)

    def f(x, k):
        return _loss_value(loss, oracle.forward(kind, x, K=k, steps=T, params=params), aux)

    fd = np.zeros_like(x0)
    for idx in np.ndindex(*x0.shape):
        xp, xm = x0.copy(), x0.copy()
        xp[idx] += h
        xm[idx] -= h
        fd[idx] = (f(xp, K) - f(xm, K)) / (2 * h)
    scale = max(np.max(np.abs(fd)), 1e-30)
    assert np.max(np.abs(fd - dx0)) <= tol * scale, np.max(np.abs(fd - dx0)) / scale
    if want_dK:
        fdk = np.zeros_like(K)
        for idx in np.ndindex(*K.shape):
            kp, km = K.copy(), K.copy()
            kp[idx] += h
            km[idx] -= h
            fdk[idx] = (f(x0, kp) - f(x0, km)) / (2 * h)
        scale = max(np.max(np.abs(fdk)), 1e-30)
        assert np.max(np.abs(fdk - dK)) <= tol * scale, np.max(np.abs(fdk - dK)) / scale


def test_fd_jacobi():
    _fd_check(JACOBI2D5, rng(10).uniform(0, 1, (6, 5)), None, 4, HALF_SQ, None, False)


@pytest.mark.parametrize("loss", [HALF_SQ, HALF_SQ_DIFF])
def test_fd_gauss_seidel(loss):
    aux = rng(19).uniform(0, 1, (5, 7))
    _fd_check(GAUSSSEIDEL2D5, rng(18).uniform(0, 1, (5, 7)), None, 5, loss, aux, False)


@pytest.mark.parametrize("loss", [DOT_W, HALF_SQ, HALF_SQ_DIFF])
def test_fd_allencahn(loss):
    x0 = rng(11).uniform(-1, 1, (3, 4, 5))
    aux = rng(12).standard_normal((3, 4, 5))
    _fd_check(ALLENCAHN3D7, x0, None, 3, loss, aux, False)


def test_fd_allencahn_strong_cubic():
    """A larger cubic coefficient makes the nonlinear adjoint dominate."""
    x0 = rng(13).uniform(-1, 1, (2, 3, 4))
    aux = rng(14).standard_normal((2, 3, 4))
    _fd_check(ALLENCAHN3D7, x0, None, 4, DOT_W, aux, False, params=(0.05, 0.6))


@pytest.mark.parametrize("loss", [HALF_SQ_DIFF, DOT_W])
def test_fd_vardiff_dx0_and_dK(loss):
    x0 = rng(15).uniform(0, 1, (6, 5))
    K = rng(16).uniform(0.5, 1.5, (6, 5))
    aux = rng(17).uniform(0, 1, (6, 5))
    _fd_check(VARDIFF2D9, x0, K, 4, loss, aux, True)


# ------------------------------------------------ tangent and dot product
@pytest.mark.parametrize("kind,shape,T,withK", [
    (JACOBI2D5, (13, 17), 6, False),
    (GAUSSSEIDEL2D5, (13, 17), 6, False),
    (ALLENCAHN3D7, (5, 6, 7), 5, False),
    (VARDIFF2D9, (11, 15), 5, True),
])
def test_jvp_matches_fd(kind, shape, T, withK):
    r = rng(20)
    lo = -1.0 if kind == ALLENCAHN3D7 else 0.0
    x0 = r.uniform(lo, 1, shape)
    K = r.uniform(0.5, 1.5, shape) if withK else None
    v = r.standard_normal(shape)
    kap = r.standard_normal(shape) if withK else None
    _, xd = oracle.jvp(kind, x0, v, K=K, kappa=kap, steps=T)
    h = 1e-6
    Kp = K + h * kap if withK else None
    Km = K - h * kap if withK else None
    fd = (oracle.forward(kind, x0 + h * v, K=Kp, steps=T) -
          oracle.forward(kind, x0 - h * v, K=Km, steps=T)) / (2 * h)
    assert rel(xd, fd) < 1e-7


@pytest.mark.parametrize("kind,shape,T,withK", [
    (JACOBI2D5, (13, 17), 6, False),
    (JACOBI2D5, (40, 33), 20, False),
    (GAUSSSEIDEL2D5, (13, 17), 6, False),
    (GAUSSSEIDEL2D5, (40, 33), 20, False),
    (ALLENCAHN3D7, (5, 6, 7), 5, False),
    (ALLENCAHN3D7, (9, 8, 10), 12, False),
    (VARDIFF2D9, (11, 15), 5, True),
    (VARDIFF2D9, (30, 41), 16, True),
])
def test_dot_product_identity(kind, shape, T, withK):
    """<J (v, kappa), w> = <v, dx0> + <kappa, dK> with (dx0, dK) the VJP of
    the cotangent w (loss SEED)."""
    r = rng(21)
    lo = -1.0 if kind == ALLENCAHN3D7 else 0.0
    x0 = r.uniform(lo, 1, shape)
    K = r.uniform(0.5, 1.5, shape) if withK else None
    v = r.standard_normal(shape)
    kap = r.standard_normal(shape) if withK else None
    w = r.standard_normal(shape)
    _, xd = oracle.jvp(kind, x0, v, K=K, kappa=kap, steps=T)
    dx0, dK, _, _ = oracle.vjp(kind, x0, K=K, steps=T, loss=SEED, aux=w, want_dK=withK)
    lhs = np.sum(xd * w)
    rhs = np.sum(v * dx0) + (np.sum(kap * dK) if withK else 0.0)
    assert abs(lhs - rhs) <= 1e-12 * max(abs(lhs), 1e-30)


# ---------------------------------------------------------------- invariants
@pytest.mark.parametrize("kind", [JACOBI2D5, GAUSSSEIDEL2D5])
def test_ones_fixed_point(kind):
    """0.2 rounds so that 5 * 0.2 == 1 exactly: constants stay put."""
    x = np.ones((20, 30))
    assert np.array_equal(oracle.forward(kind, x, steps=25), x)


def test_vardiff_constant_fixed_point_and_conservation():
    K = rng(30).uniform(0.5, 1.5, (25, 19))
    c = np.full((25, 19), 0.375)
    assert np.array_equal(oracle.forward(VARDIFF2D9, c, K=K, steps=13), c)
    x0 = rng(31).uniform(0, 1, (25, 19))
    xT = oracle.forward(VARDIFF2D9, x0, K=K, steps=40)
    assert abs(xT.sum() - x0.sum()) <= 1e-12 * x0.sum()
    # the maximum principle of a non-negative-coefficient scheme
    assert xT.max() <= x0.max() and xT.min() >= x0.min()


def test_vardiff_unit_seed_gives_unit_dx0_and_zero_dK():
    """The adjoint of a conservative scheme maps constants to themselves and
    a constant cotangent sees no flux, so dK vanishes."""
    x0 = rng(32).uniform(0, 1, (12, 14))
    K = rng(33).uniform(0.5, 1.5, (12, 14))
    one = np.ones_like(x0)
    dx0, dK, _, _ = oracle.vjp(VARDIFF2D9, x0, K=K, steps=9, loss=SEED, aux=one, want_dK=True)
    assert np.max(np.abs(dx0 - 1.0)) < 1e-14
    assert np.max(np.abs(dK)) < 1e-14


def test_allencahn_zero_stays_zero():
    z = np.zeros((4, 5, 6))
    assert np.array_equal(oracle.forward(ALLENCAHN3D7, z, steps=7), z)


@pytest.mark.parametrize("kind,shape,params,withK", [
    (ALLENCAHN3D7, (4, 5, 6), (0.1, 0.0), False),
    (VARDIFF2D9, (9, 7), (0.1, 0.0), True),
])
def test_linear_part_symmetric(kind, shape, params, withK):
    """<M u, v> = <u, M v>: the Dirichlet-ghost 7-point and the no-flux
    edge-form 9-point operators are symmetric."""
    r = rng(34)
    K = r.uniform(0.5, 1.5, shape) if withK else None
    u, v = r.standard_normal(shape), r.standard_normal(shape)
    Mu = oracle.forward(kind, u, K=K, steps=1, params=params)
    Mv = oracle.forward(kind, v, K=K, steps=1, params=params)
    assert abs(np.sum(Mu * v) - np.sum(u * Mv)) < 1e-13 * np.sum(np.abs(Mu * v))


@pytest.mark.parametrize("kind,shape,withK", [
    (JACOBI2D5, (5, 7), False), (ALLENCAHN3D7, (2, 3, 4), False), (VARDIFF2D9, (6, 5), True),
    (GAUSSSEIDEL2D5, (4, 6), False)])
def test_zero_steps_returns_seed(kind, shape, withK):
    r = rng(35)
    x0 = r.uniform(0, 1, shape)
    K = r.uniform(0.5, 1.5, shape) if withK else None
    Y = r.uniform(0, 1, shape)
    dx0, dK, xT, L = oracle.vjp(kind, x0, K=K, steps=0, loss=HALF_SQ_DIFF, aux=Y, want_dK=withK)
    assert np.array_equal(dx0, x0 - Y)
    assert np.array_equal(xT, x0)
    if withK:
        assert np.array_equal(dK, np.zeros_like(x0))


# ---------------------------------------------------------------- hand cases
def _read_golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                rows.append([float(v) for v in line.split()])
    return np.array(rows)


def test_jacobi_3x3_hand_case():
    """3x3 grid, one step, L = 0.5 sum x_1^2: only the centre is interior,
    so g0[centre] = 0.2 x1[centre], g0[edge] = x1[edge] + 0.2 x1[centre],
    g0[corner] = x1[corner]; worked out by hand in the golden file."""
    x0 = np.arange(1.0, 10.0).reshape(3, 3)
    expect = _read_golden("jacobi_3x3_T1.txt")
    dx0, _, xT, L = oracle.vjp(JACOBI2D5, x0, steps=1, loss=HALF_SQ)
    assert np.array_equal(xT, expect[0:3])
    assert np.array_equal(dx0, expect[3:6])
    assert L == 142.5


def test_gauss_seidel_4x4_hand_case():
    """4x4 grid, one sweep, w = 1/4 so every value is a dyadic rational and
    exact in binary. Interior points in row-major order (y, x):
      (1,1): C 0, E 0, N 0, S 2, W 5                  -> 7/4
      (1,2): C 0, E 6, N 0, S 3, W x'(1,1) = 7/4      -> 43/16
      (2,1): C 0, E 0, N 10, S x'(1,1) = 7/4, W 7     -> 75/16
      (2,2): C 0, E 8, N 11, S x'(1,2), W x'(2,1)     -> 211/32
    For the gradient of x'(2,2) (loss SEED, cotangent e_(2,2)): x0(2,2)
    enters through C (1/4), through E of (2,1) and through N of (1,2)
    (1/4 * 1/4 each), so dx0(2,2) = 3/8; the ring point (3,2) only through
    N of (2,2): 1/4. x0(1,1), x0(0,1) and x0(1,0) reach x'(2,2) only through
    x'(1,1) (as its C, S and W), then along (1,2) -> (2,2) or (2,1) -> (2,2):
    2 * (1/4)^3 each; the corner x0(0,0) is read by nothing: 0."""
    x0 = np.array([[1, 2, 3, 4], [5, 0, 0, 6], [7, 0, 0, 8], [9, 10, 11, 12]], dtype=float)
    x1 = oracle.forward(GAUSSSEIDEL2D5, x0, steps=1, params=(0.25, 0.0))
    expect = x0.copy()
    expect[1, 1], expect[1, 2], expect[2, 1], expect[2, 2] = 7 / 4, 43 / 16, 75 / 16, 211 / 32
    assert np.array_equal(x1, expect)
    e = np.zeros_like(x0)
    e[2, 2] = 1.0
    dx0, _, _, _ = oracle.vjp(GAUSSSEIDEL2D5, x0, steps=1, loss=SEED, aux=e, params=(0.25, 0.0))
    assert dx0[2, 2] == 3 / 8 and dx0[3, 2] == 1 / 4
    assert dx0[1, 1] == dx0[0, 1] == dx0[1, 0] == 2 / 64
    assert dx0[0, 0] == 0.0


def test_allencahn_single_point_is_scalar_map():
    """On a 1x1x1 grid every neighbour is a zero ghost value and the step is
    the scalar map x' = (1-6D) x - C x^3 with derivative (1-6D) - 3 C x^2;
    the VJP is the product of the derivatives along the trajectory."""
    D, C = 0.1, 0.1
    x = 0.7
    xs = [x]
    for _ in range(5):
        x = (1 - 6 * D) * x - C * x ** 3
        xs.append(x)
    grad = 1.0
    for xt in reversed(xs[:-1]):
        grad *= (1 - 6 * D) - 3 * C * xt ** 2
    dx0, _, xT, _ = oracle.vjp(ALLENCAHN3D7, np.full((1, 1, 1), 0.7), steps=5, loss=SEED,
                               aux=np.ones((1, 1, 1)))
    assert abs(xT[0, 0, 0] - xs[-1]) < 1e-15
    assert abs(dx0[0, 0, 0] - grad) < 1e-15


# ------------------------------------------------------------- precisions
@pytest.mark.parametrize("kind,shape,T,withK", [
    (JACOBI2D5, (33, 47), 12, False),
    (GAUSSSEIDEL2D5, (33, 47), 12, False),
    (ALLENCAHN3D7, (9, 10, 11), 8, False),
    (VARDIFF2D9, (37, 29), 20, True),
])
def test_f32_tracks_f64(kind, shape, T, withK):
    """The single-precision instantiation computes the same quantities."""
    r = rng(40)
    lo = -1.0 if kind == ALLENCAHN3D7 else 0.0
    x0 = r.uniform(lo, 1, shape).astype(np.float32)
    K = r.uniform(0.5, 1.5, shape).astype(np.float32) if withK else None
    Y = r.uniform(0, 1, shape).astype(np.float32)
    d32, k32, x32, L32 = oracle.vjp(kind, x0, K=K, steps=T, loss=HALF_SQ_DIFF, aux=Y,
                                    want_dK=withK)
    d64, k64, x64, L64 = oracle.vjp(kind, x0.astype(np.float64),
                                    K=None if K is None else K.astype(np.float64), steps=T,
                                    loss=HALF_SQ_DIFF, aux=Y.astype(np.float64), want_dK=withK)
    assert d32.dtype == np.float32
    assert rel(x32, x64) < 1e-6
    assert rel(d32, d64) < 1e-5
    assert abs(L32 - L64) <= 1e-5 * abs(L64)
    if withK:
        assert rel(k32, k64) < 1e-4
