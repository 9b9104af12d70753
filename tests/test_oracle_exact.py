"""Exact rational pins of the oracle (CPU only).

Each stencil program is evaluated here in exact rational arithmetic (Python
`fractions.Fraction`) on grids of two to four points per side, for at most
three steps, from dyadic inputs. Its derivatives come from forward-mode dual
numbers over the rationals: every input direction (each point of x0, each
point of K, the two step constants) is carried through the steps at once as
a tangent vector, and the gradient of the loss is the tangent's inner
product with dL/dx_T. That route shares nothing with the oracle's
store-all reverse sweep in scatter form (Sec. II, Sec. III-C): a transposed
neighbour, a dropped term, a wrong sign or a missing clear in the reverse
sweep shows up as a mismatch.

The step definitions are the stencil programs themselves (the unmodified
programs whose gradient is taken, Sec. I): Jacobi x'[c] = w(x[c]+W+E+S+N) on
interior points with the ring held; Allen-Cahn x' = (x + D lap x) - C x^3
with zero ghosts; variable-coefficient diffusion x' = x + dt sum_n
c_n (K[c]+K[n]) (x[n]-x[c]) (c_n = 1/3 on axis and 1/12 on diagonal edges,
the float64 values of those fractions, taken here as exact rationals, since
the program rounds them once); the in-place Gauss-Seidel sweep in row-major
order; the optional limiter clamping every new value to [lo, hi].

Where every value the program forms is a dyadic rational with few bits
(constants 1/4, 1/8, 1/16, inputs k/8), float64 holds them all exactly and
the oracle must return the exact result bit for bit. Otherwise each result
must lie within a few units in the last place of the largest entry of the
exact one (the programs are a handful of additions and products deep).
"""
from fractions import Fraction as Fr

import numpy as np
import pytest

import oracle

EPS = 2.0 ** -52


class Dual:
    """A rational value with a tangent vector (one entry per direction)."""
    __slots__ = ("v", "d")

    def __init__(self, v, d):
        self.v = v
        self.d = d

    @staticmethod
    def const(v, n):
        return Dual(Fr(v), [Fr(0)] * n)

    def __add__(self, o):
        return Dual(self.v + o.v, [a + b for a, b in zip(self.d, o.d)])

    def __sub__(self, o):
        return Dual(self.v - o.v, [a - b for a, b in zip(self.d, o.d)])

    def __mul__(self, o):
        return Dual(self.v * o.v, [self.v * b + o.v * a for a, b in zip(self.d, o.d)])


def clamp(y, lim, n):
    """The limiter: its derivative is that of the branch taken."""
    if lim is None:
        return y
    lo, hi = Fr(lim[0]), Fr(lim[1])
    if y.v < lo:
        return Dual.const(lo, n)
    if y.v > hi:
        return Dual.const(hi, n)
    return y


def exact_run(kind, x0, K, steps, params, lim):
    """x_T as Duals, tangents along (x0 points, K points, p0, p1)."""
    shape = x0.shape
    npts = x0.size
    nd = npts * (2 if K is not None else 1) + 2
    flat = x0.reshape(-1)
    x = []
    for i in range(npts):
        d = [Fr(0)] * nd
        d[i] = Fr(1)
        x.append(Dual(Fr(float(flat[i])), d))
    Kd = None
    if K is not None:
        Kd = []
        for i, v in enumerate(K.reshape(-1)):
            d = [Fr(0)] * nd
            d[npts + i] = Fr(1)
            Kd.append(Dual(Fr(float(v)), d))
    p = []
    for j in range(2):
        d = [Fr(0)] * nd
        d[nd - 2 + j] = Fr(1)
        p.append(Dual(Fr(float(params[j])), d))
    zero = Dual.const(0, nd)

    if len(shape) == 2:
        ny, nx = shape
        nz = 1
    else:
        nz, ny, nx = shape

    def at(k, j, i):
        return (k * ny + j) * nx + i

    def inside(k, j, i):
        return 0 <= k < nz and 0 <= j < ny and 0 <= i < nx

    def ring(j, i):
        return j == 0 or i == 0 or j == ny - 1 or i == nx - 1

    for _ in range(steps):
        if kind == oracle.GAUSSSEIDEL2D5:
            for j in range(1, ny - 1):
                for i in range(1, nx - 1):
                    s = x[at(0, j, i)] + x[at(0, j, i + 1)] + x[at(0, j + 1, i)] + \
                        x[at(0, j - 1, i)] + x[at(0, j, i - 1)]
                    x[at(0, j, i)] = p[0] * s
            continue
        new = []
        for k in range(nz):
            for j in range(ny):
                for i in range(nx):
                    c = x[at(k, j, i)]
                    if kind == oracle.JACOBI2D5:
                        if ring(j, i):
                            y = c
                        else:
                            y = p[0] * (c + x[at(0, j, i - 1)] + x[at(0, j, i + 1)] +
                                        x[at(0, j - 1, i)] + x[at(0, j + 1, i)])
                    elif kind == oracle.ALLENCAHN3D7:
                        lap = zero
                        for dk, dj, di in ((0, 0, -1), (0, 0, 1), (0, -1, 0), (0, 1, 0),
                                           (-1, 0, 0), (1, 0, 0)):
                            if inside(k + dk, j + dj, i + di):
                                lap = lap + x[at(k + dk, j + dj, i + di)]
                        lap = lap - Dual.const(6, nd) * c
                        y = (c + p[0] * lap) - p[1] * c * c * c
                    else:  # VARDIFF2D9
                        acc = zero
                        for dj in (-1, 0, 1):
                            for di in (-1, 0, 1):
                                if (dj or di) and inside(0, j + dj, i + di):
                                    cn = Fr(1.0 / 3.0) if dj == 0 or di == 0 else Fr(1.0 / 12.0)
                                    n = at(0, j + dj, i + di)
                                    acc = acc + Dual.const(cn, nd) * (Kd[at(0, j, i)] + Kd[n]) * \
                                        (x[n] - c)
                        y = c + p[0] * acc
                    new.append(clamp(y, lim, nd))
        x = new
    return x, npts, nd


def exact_vjp(kind, x0, K, steps, loss, aux, params, lim=None):
    """(dx0, dK or None, x_T, L, (dL/dp0, dL/dp1)) as exact rationals."""
    xT, npts, nd = exact_run(kind, x0, K, steps, params, lim)
    a = None if aux is None else [Fr(float(v)) for v in aux.reshape(-1)]
    L = Fr(0)
    grad = [Fr(0)] * nd
    for c in range(npts):
        v = xT[c].v
        if loss == oracle.HALF_SQ:
            L += v * v / 2
            seed = v
        elif loss == oracle.HALF_SQ_DIFF:
            d = v - a[c]
            L += d * d / 2
            seed = d
        else:  # DOT_W
            L += a[c] * v
            seed = a[c]
        if seed:
            for q in range(nd):
                if xT[c].d[q]:
                    grad[q] += seed * xT[c].d[q]
    dx0 = grad[:npts]
    dK = grad[npts:2 * npts] if K is not None else None
    return dx0, dK, [x.v for x in xT], L, (grad[nd - 2], grad[nd - 1])


def dyadic(rng, shape, lo=-8, hi=8, den=8):
    return rng.integers(lo, hi + 1, size=shape).astype(np.float64) / den


def check(got, exact, exact_bits, name, ulps=32):
    got = np.asarray(got, dtype=np.float64).reshape(-1)
    ref = np.array([float(v) for v in exact])  # correctly rounded
    if exact_bits:
        assert np.array_equal(got, ref), f"{name}: not the exact result"
    else:
        scale = max(float(max(abs(v) for v in exact)), 1e-300)
        err = float(np.max(np.abs(got - ref)))
        assert err <= ulps * EPS * scale, f"{name}: off by {err / (EPS * scale):.1f} ulp of max"


def compare(kind, shape, steps, loss, params, exact_bits, seed, lim=None, with_K=False,
            ulps=32):
    rng = np.random.default_rng(seed)
    x0 = dyadic(rng, shape)
    K = dyadic(rng, shape, 4, 12) if with_K else None   # K in [1/2, 3/2]
    aux = dyadic(rng, shape) if loss != oracle.HALF_SQ else None
    dx0, dK, xT, L, dp = oracle.vjp(kind, x0, K=K, steps=steps, loss=loss, aux=aux,
                                    want_dK=with_K, params=params, want_dp=True, lim=lim)
    e_dx0, e_dK, e_xT, e_L, e_dp = exact_vjp(kind, x0, K, steps, loss, aux, params, lim)
    tag = f"kind {kind} {shape} T={steps} loss {loss}"
    check(xT, e_xT, exact_bits, tag + " x_T", ulps)
    check(dx0, e_dx0, exact_bits, tag + " dx0", ulps)
    if with_K:
        check(dK, e_dK, exact_bits, tag + " dK", ulps)
    check([L], [e_L], exact_bits, tag + " L", ulps)
    # the constants' gradient exists per constant the step reads
    nparam = 2 if kind == oracle.ALLENCAHN3D7 else 1
    for j in range(nparam):
        check([dp[j]], [e_dp[j]], exact_bits, tag + f" dL/dp{j}", ulps)


LOSSES = (oracle.HALF_SQ, oracle.DOT_W, oracle.HALF_SQ_DIFF)


@pytest.mark.parametrize("shape", [(2, 2), (3, 3), (3, 4), (4, 4)])
@pytest.mark.parametrize("steps", [1, 2, 3])
@pytest.mark.parametrize("loss", LOSSES)
def test_jacobi_dyadic_exact(shape, steps, loss):
    compare(oracle.JACOBI2D5, shape, steps, loss, (0.25, 0.0), True, 11 + steps)


@pytest.mark.parametrize("shape", [(3, 3), (4, 4), (4, 3)])
@pytest.mark.parametrize("steps", [1, 2, 3])
def test_gauss_seidel_dyadic_exact(shape, steps):
    compare(oracle.GAUSSSEIDEL2D5, shape, steps, oracle.HALF_SQ, (0.25, 0.0), True, 21 + steps)


@pytest.mark.parametrize("shape", [(2, 2, 2), (3, 3, 3), (2, 3, 4)])
@pytest.mark.parametrize("loss", LOSSES)
def test_allencahn_dyadic_exact_one_step(shape, loss):
    # one step forms x^3 C with 13-bit values: every value exact in float64
    compare(oracle.ALLENCAHN3D7, shape, 1, loss, (0.125, 0.0625), True, 31)


@pytest.mark.parametrize("shape", [(2, 2, 2), (3, 3, 3), (4, 4, 4)])
@pytest.mark.parametrize("steps", [2, 3])
def test_allencahn_dyadic_rounded(shape, steps):
    compare(oracle.ALLENCAHN3D7, shape, steps, oracle.DOT_W, (0.125, 0.0625), False, 41)


@pytest.mark.parametrize("shape", [(2, 2), (3, 3), (4, 4)])
@pytest.mark.parametrize("steps", [1, 2, 3])
@pytest.mark.parametrize("loss", [oracle.HALF_SQ, oracle.HALF_SQ_DIFF])
def test_vardiff_rounded_weights(shape, steps, loss):
    # the 1/3 and 1/12 edge weights are not dyadic: rounding enters
    compare(oracle.VARDIFF2D9, shape, steps, loss, (0.125, 0.0), False, 51, with_K=True)


@pytest.mark.parametrize("kind,shape", [(oracle.JACOBI2D5, (4, 4)),
                                        (oracle.GAUSSSEIDEL2D5, (4, 4)),
                                        (oracle.ALLENCAHN3D7, (3, 3, 3))])
@pytest.mark.parametrize("steps", [1, 3])
def test_default_constants(kind, shape, steps):
    # w = 0.2, D = C = 0.1 are not dyadic: the oracle rounds, the rationals do not
    compare(kind, shape, steps, oracle.HALF_SQ, oracle.default_params(kind), False, 61)


@pytest.mark.parametrize("steps", [1, 2, 3])
def test_jacobi_limiter_dyadic_exact(steps):
    # bounds the dyadic values cross: some points clamp, some keep their branch
    compare(oracle.JACOBI2D5, (4, 4), steps, oracle.HALF_SQ, (0.25, 0.0), True, 71,
            lim=(-0.25, 0.375))


def test_dual_numbers_pin_themselves():
    # the tangent of a product and a clamp, by hand: d(x*x*x)/dx = 3x^2
    x = Dual(Fr(3, 8), [Fr(1)])
    y = x * x * x
    assert y.v == Fr(27, 512) and y.d == [Fr(27, 64)]
    assert clamp(y, (0.0, 0.03125), 1).d == [Fr(0)]
