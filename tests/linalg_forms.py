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
