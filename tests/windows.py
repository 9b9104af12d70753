"""Sampled gradients at full size, computed by the oracle on small windows.

Every step reads only neighbours at L-infinity distance 1, so dx0[p] and
dK[p] depend only on inputs within distance 2T of p (T forward steps reach
x_T, then T adjoint steps bring the cotangent back). Cutting the grid to the
window of radius 2T+1 around p changes values only near the window's
artificial edges, which cannot reach p in 2T steps, and the oracle performs
the same operations in the same order for every point near p. So the
windowed result equals the full-grid oracle at p exactly, while costing a
window instead of the whole grid.
"""
import numpy as np

import oracle


def window_slices(shape, point, radius):
    return tuple(slice(max(0, p - radius), min(n, p + radius + 1)) for p, n in zip(point, shape))


def window_vjp(kind, inputs, steps, point, loss, want_dK, params=None):
    """(dx0[point], dK[point] or None) for the full problem, by the oracle."""
    x0 = inputs["x0"]
    sl = window_slices(x0.shape, point, 2 * steps + 1)
    local = tuple(p - s.start for p, s in zip(point, sl))

    def sub(a):
        return None if a is None else np.ascontiguousarray(a[sl])

    dx0, dK, _, _ = oracle.vjp(kind, sub(x0), K=sub(inputs.get("K")), steps=steps, loss=loss,
                               aux=sub(inputs.get("aux")), want_dK=want_dK, params=params)
    return dx0[local], (dK[local] if want_dK else None)


def window_forward(kind, inputs, steps, point, params=None):
    """x_T[point] by the oracle on the window of radius T+1."""
    x0 = inputs["x0"]
    sl = window_slices(x0.shape, point, steps + 1)
    local = tuple(p - s.start for p, s in zip(point, sl))
    K = inputs.get("K")
    xT = oracle.forward(kind, np.ascontiguousarray(x0[sl]),
                        K=None if K is None else np.ascontiguousarray(K[sl]), steps=steps,
                        params=params)
    return xT[local]


def sample_points(shape, count, seed):
    """Corners, edge midpoints and random interior points of a grid."""
    pts = set()
    for corner in np.ndindex(*(2,) * len(shape)):
        pts.add(tuple(0 if c == 0 else n - 1 for c, n in zip(corner, shape)))
    pts.add(tuple(n // 2 for n in shape))
    pts.add(tuple(0 if i == 0 else n // 3 for i, n in enumerate(shape)))
    rng = np.random.Generator(np.random.PCG64(seed))
    while len(pts) < count:
        pts.add(tuple(int(rng.integers(0, n)) for n in shape))
    return sorted(pts)
