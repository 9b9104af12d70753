"""Dense matrix forms of the linear stencil steps, built from graph algebra.

These are test fixtures, independent of the oracle's loops: each operator is
assembled from Kronecker products of 1-D path-graph adjacencies (the textbook
construction of grid Laplacians), so a wrong neighbour, sign or boundary rule
in the oracle shows up as a mismatch. Index order is row-major, x fastest.
"""
import numpy as np


def path_adjacency(n):
    """Adjacency of the path graph on n vertices."""
    a = np.zeros((n, n))
    i = np.arange(n - 1)
    a[i, i + 1] = 1.0
    a[i + 1, i] = 1.0
    return a


def grid2d_axis(ny, nx):
    """Axis-neighbour adjacency of an ny-by-nx grid."""
    return np.kron(np.eye(ny), path_adjacency(nx)) + np.kron(path_adjacency(ny), np.eye(nx))


def grid2d_diag(ny, nx):
    """Diagonal-neighbour adjacency of an ny-by-nx grid."""
    return np.kron(path_adjacency(ny), path_adjacency(nx))


def grid3d_faces(nz, ny, nx):
    """Face-neighbour adjacency of an nz-by-ny-by-nx grid."""
    iz, iy, ix = np.eye(nz), np.eye(ny), np.eye(nx)
    return (np.kron(np.kron(iz, iy), path_adjacency(nx)) +
            np.kron(np.kron(iz, path_adjacency(ny)), ix) +
            np.kron(np.kron(path_adjacency(nz), iy), ix))


def jacobi_matrix(ny, nx, w=0.2):
    """One Jacobi step: rows of interior points average the point and its four
    neighbours with weight w; rows of the outer ring are identity."""
    n = nx * ny
    yy, xx = np.divmod(np.arange(n), nx)
    interior = ((xx > 0) & (xx < nx - 1) & (yy > 0) & (yy < ny - 1)).astype(float)
    avg = w * (np.eye(n) + grid2d_axis(ny, nx))
    return interior[:, None] * avg + np.diag(1.0 - interior)


def gauss_seidel_matrix(ny, nx, w=0.2):
    """One in-place Gauss-Seidel sweep in row-major order as the textbook
    matrix splitting. Split the axis adjacency A = L + U into its strictly
    lower part L (the W and S neighbours, which precede a point in row-major
    order and so already hold new values) and strictly upper part U (E and
    N, still old). With D the interior indicator, one sweep solves
        (I - w D L) x' = (w D (I + U) + (I - D)) x,
    a unit lower-triangular system (ring rows are identity rows)."""
    n = nx * ny
    yy, xx = np.divmod(np.arange(n), nx)
    interior = ((xx > 0) & (xx < nx - 1) & (yy > 0) & (yy < ny - 1)).astype(float)
    A = grid2d_axis(ny, nx)
    L = np.tril(A, -1)
    U = np.triu(A, 1)
    D = np.diag(interior)
    lhs = np.eye(n) - w * D @ L
    rhs = w * D @ (np.eye(n) + U) + (np.eye(n) - D)
    return np.linalg.solve(lhs, rhs)


def laplace_dirichlet_solution(ring):
    """Discrete harmonic function of the 5-point Laplacian with the ring of
    `ring` as Dirichlet data (interior values of `ring` ignored): solves
    4 u[c] - sum of the 4 neighbours = 0 on interior points."""
    ny, nx = ring.shape
    n = nx * ny
    yy, xx = np.divmod(np.arange(n), nx)
    interior = (xx > 0) & (xx < nx - 1) & (yy > 0) & (yy < ny - 1)
    lap = 4.0 * np.eye(n) - grid2d_axis(ny, nx)
    M = np.where(interior[:, None], lap, np.eye(n))
    b = np.where(interior, 0.0, ring.reshape(-1))
    return np.linalg.solve(M, b).reshape(ny, nx)


def heat3d_matrix(nz, ny, nx, D=0.1):
    """The linear part of the Allen-Cahn step, I + D * (A - 6 I), with
    out-of-grid neighbours reading zero (Dirichlet ghost values)."""
    n = nx * ny * nz
    return np.eye(n) + D * (grid3d_faces(nz, ny, nx) - 6.0 * np.eye(n))


def vardiff_matrix(K2d, dt=0.1):
    """The variable-coefficient step I + dt * L(K), L the weighted graph
    Laplacian of the 8-neighbour grid with edge weight c*(K_m + K_n),
    c = 1/3 on axis edges and 1/12 on diagonal edges (no-flux boundary:
    only in-grid edges exist)."""
    ny, nx = K2d.shape
    k = K2d.reshape(-1)
    ksum = k[:, None] + k[None, :]
    wts = (1.0 / 3.0) * grid2d_axis(ny, nx) * ksum + (1.0 / 12.0) * grid2d_diag(ny, nx) * ksum
    lap = wts - np.diag(wts.sum(axis=1))
    return np.eye(nx * ny) + dt * lap


def nine_point_laplacian_interior(x):
    """Textbook isotropic 9-point Laplacian (4*axis + diagonal - 20*centre)/6
    on interior points of a 2-D array (unit spacing)."""
    c = x[1:-1, 1:-1]
    axis = x[1:-1, :-2] + x[1:-1, 2:] + x[:-2, 1:-1] + x[2:, 1:-1]
    diag = x[:-2, :-2] + x[:-2, 2:] + x[2:, :-2] + x[2:, 2:]
    return (4.0 * axis + diag - 20.0 * c) / 6.0
