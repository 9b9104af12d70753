"""Seeded synthetic workloads: shapes, step counts, budgets and input arrays.

This module holds none of the method's arithmetic. It only names the
workloads and draws their inputs, so that the GPU path, the CPU oracle and
the benchmark all see the same arrays.

Random numbers: numpy's PCG64 bit generator seeded per array; uniform and
normal draws are taken in float64 and rounded to float32 for float32 arrays.
Arrays are row-major [nz][ny][nx] ([ny][nx] for 2-D kinds).
"""
from dataclasses import dataclass, field
from typing import Dict, Optional, Tuple

import numpy as np

JACOBI2D5, ALLENCAHN3D7, VARDIFF2D9, GAUSSSEIDEL2D5 = 0, 1, 2, 3
F64, F32 = 0, 1
HALF_SQ, DOT_W, HALF_SQ_DIFF, SEED = 0, 1, 2, 3
SCHED_AUTO, SCHED_STORE_ALL, SCHED_UNIFORM, SCHED_BINOMIAL = 0, 1, 2, 3

KIND_NAMES = {JACOBI2D5: "jacobi2d5", ALLENCAHN3D7: "allencahn3d7", VARDIFF2D9: "vardiff2d9",
              GAUSSSEIDEL2D5: "gaussseidel2d5"}
DEFAULT_PARAMS = {JACOBI2D5: (0.2, 0.0), ALLENCAHN3D7: (0.1, 0.1), VARDIFF2D9: (0.1, 0.0),
                  GAUSSSEIDEL2D5: (0.2, 0.0)}


@dataclass(frozen=True)
class Dist:
    """One input array: distribution and seed."""
    kind: str  # "uniform" or "normal"
    seed: int
    lo: float = 0.0
    hi: float = 1.0


@dataclass(frozen=True)
class Workload:
    name: str
    kind: int
    dtype: int
    shape: Tuple[int, ...]   # row-major
    steps: int
    loss: int
    budget_bytes: int        # checkpoint-slot bytes
    sched: int
    want_dK: bool
    x0: Dist
    K: Optional[Dist] = None
    aux: Optional[Dist] = None
    params: Tuple[float, float] = (0.0, 0.0)
    notes: str = ""

    @property
    def npoints(self) -> int:
        return int(np.prod(self.shape))

    @property
    def itemsize(self) -> int:
        return 8 if self.dtype == F64 else 4

    @property
    def state_bytes(self) -> int:
        return self.npoints * self.itemsize

    def with_(self, **kw) -> "Workload":
        d = dict(self.__dict__)
        d.update(kw)
        return Workload(**d)


GiB = 1 << 30

WORKLOADS: Dict[str, Workload] = {
    # 2-D 5-point Jacobi, fp64, 64x64, 10 steps, store-all.
    "jacobi2d5_f64_64x64_T10": Workload(
        "jacobi2d5_f64_64x64_T10", JACOBI2D5, F64, (64, 64), 10, HALF_SQ,
        budget_bytes=9 * 64 * 64 * 8, sched=SCHED_STORE_ALL, want_dK=False,
        x0=Dist("uniform", 0), params=DEFAULT_PARAMS[JACOBI2D5]),
    # Same stencil at 4096x4096, 100 steps; budget of 10 snapshots (1.34 GB).
    "jacobi2d5_f64_4096x4096_T100": Workload(
        "jacobi2d5_f64_4096x4096_T100", JACOBI2D5, F64, (4096, 4096), 100, HALF_SQ,
        budget_bytes=10 * 4096 * 4096 * 8, sched=SCHED_AUTO, want_dK=False,
        x0=Dist("uniform", 1), params=DEFAULT_PARAMS[JACOBI2D5]),
    # 3-D 7-point Allen-Cahn, fp64, 512^3, 50 steps; 8 snapshots (8.6 GB).
    "allencahn3d7_f64_512cube_T50": Workload(
        "allencahn3d7_f64_512cube_T50", ALLENCAHN3D7, F64, (512, 512, 512), 50, DOT_W,
        budget_bytes=8 * GiB, sched=SCHED_AUTO, want_dK=False,
        x0=Dist("uniform", 2, -1.0, 1.0), aux=Dist("normal", 3),
        params=DEFAULT_PARAMS[ALLENCAHN3D7]),
    # 2-D 9-point variable-coefficient diffusion, fp32, 8192^2, 200 steps,
    # gradients for x0 and K; 16 snapshots (4.29 GB).
    "vardiff2d9_f32_8192x8192_T200": Workload(
        "vardiff2d9_f32_8192x8192_T200", VARDIFF2D9, F32, (8192, 8192), 200, HALF_SQ_DIFF,
        budget_bytes=16 * 8192 * 8192 * 4, sched=SCHED_AUTO, want_dK=True,
        x0=Dist("uniform", 4), K=Dist("uniform", 5, 0.5, 1.5), aux=Dist("uniform", 6),
        params=DEFAULT_PARAMS[VARDIFF2D9]),
    # 3-D Allen-Cahn at 1024^3 (8.6 GB per state), 200 steps, 64 GB budget
    # (7 snapshots), binomial schedule.
    "allencahn3d7_f64_1024cube_T200": Workload(
        "allencahn3d7_f64_1024cube_T200", ALLENCAHN3D7, F64, (1024, 1024, 1024), 200, DOT_W,
        budget_bytes=64_000_000_000, sched=SCHED_BINOMIAL, want_dK=False,
        x0=Dist("uniform", 7, -1.0, 1.0), aux=Dist("normal", 8),
        params=DEFAULT_PARAMS[ALLENCAHN3D7]),
    # In-place 5-point Gauss-Seidel, fp64, at the size of the paper's Seidel2d
    # case study (N = 400, 100 time steps, Sec. V-B). Linear: nothing is
    # stored at any budget.
    "gaussseidel2d5_f64_400x400_T100": Workload(
        "gaussseidel2d5_f64_400x400_T100", GAUSSSEIDEL2D5, F64, (400, 400), 100, HALF_SQ,
        budget_bytes=0, sched=SCHED_AUTO, want_dK=False,
        x0=Dist("uniform", 9), params=DEFAULT_PARAMS[GAUSSSEIDEL2D5]),
    # The same sweep on a grid that fills the GPU (128 MiB per state).
    "gaussseidel2d5_f64_4096x4096_T100": Workload(
        "gaussseidel2d5_f64_4096x4096_T100", GAUSSSEIDEL2D5, F64, (4096, 4096), 100, HALF_SQ,
        budget_bytes=0, sched=SCHED_AUTO, want_dK=False,
        x0=Dist("uniform", 10), params=DEFAULT_PARAMS[GAUSSSEIDEL2D5]),
}

# The workload the headline metric is quoted on: the largest that fits one
# GPU, and the one whose budget binds (store-all would need 1.7 TB).
HEADLINE = "allencahn3d7_f64_1024cube_T200"


def draw(d: Dist, shape, dtype: int) -> np.ndarray:
    """Draw one array: float64 draws from PCG64(seed), rounded for float32."""
    rng = np.random.Generator(np.random.PCG64(d.seed))
    if d.kind == "uniform":
        a = rng.uniform(d.lo, d.hi, size=shape)
    elif d.kind == "normal":
        a = rng.standard_normal(size=shape)
    else:
        raise ValueError(d.kind)
    return np.ascontiguousarray(a.astype(np.float64 if dtype == F64 else np.float32))


def make_inputs(w: Workload, shape=None) -> Dict[str, Optional[np.ndarray]]:
    """x0, K (or None) and the loss's aux array (or None) for workload w,
    optionally at another shape (same distributions and seeds)."""
    shape = tuple(shape) if shape is not None else w.shape
    return {
        "x0": draw(w.x0, shape, w.dtype),
        "K": draw(w.K, shape, w.dtype) if w.K is not None else None,
        "aux": draw(w.aux, shape, w.dtype) if w.aux is not None else None,
    }


def dims_of(shape) -> Tuple[int, int, int]:
    """Row-major shape -> (nx, ny, nz)."""
    if len(shape) == 2:
        return (shape[1], shape[0], 1)
    return (shape[2], shape[1], shape[0])
