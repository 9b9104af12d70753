// gfx950 kernels of the stencil VJP: forward steps, adjoint steps in gather
// (transposed-stencil) form, loss/seed with a wave64 reduction, and small
// utilities. Built with -ffp-contract=off: every expression rounds in the
// order written, so a forward step is bit-identical wherever it runs (sweep
// or recomputation) and matches the documented evaluation order.
//
// Every kernel is bandwidth-bound (well under 1 flop per byte in fp64), so
// the design goal is coalesced 64-wide rows and few re-reads; there is no
// dense contraction and no matrix-core use.
//
// Adjoints are written in gather form: each output point g_{t-1}[m] collects
// sum_c J_t[c][m] g_t[c] from the points c whose stencil reads m (the reversed
// map of the paper's Sec. III-C has the same range as the forward map; where
// that reversed map scatters into input gradients with accumulation, the
// gather form gives one writer per point, needs no atomics, and is
// deterministic).

#include <hip/hip_runtime.h>

#include "adst.h"
#include "kernels.h"

namespace adst {
namespace {

constexpr int kBX = 64;  // one wavefront along x
constexpr int kBY = 4;   // four wavefronts per block
constexpr int kThreads = kBX * kBY;

struct Tile2 {
  int i, j;
};

__device__ inline Tile2 tile2(int tiles_x) {
  const int b = blockIdx.x;
  return {(b % tiles_x) * kBX + (int)threadIdx.x, (b / tiles_x) * kBY + (int)threadIdx.y};
}

struct Tile3 {
  int i, j, k;
};

__device__ inline Tile3 tile3(int tiles_x, int tiles_y) {
  int b = blockIdx.x;
  const int bx = b % tiles_x;
  b /= tiles_x;
  const int by = b % tiles_y;
  const int bz = b / tiles_y;
  return {bx * kBX + (int)threadIdx.x, by * kBY + (int)threadIdx.y, bz};
}

// ------------------------------------------------------------- Jacobi 2-D
// Forward: interior x'[c] = w*((((x[c]+x[W])+x[E])+x[S])+x[N]); ring copied.
template <class R>
__global__ __launch_bounds__(kThreads) void fwd_jacobi2d5(const R* __restrict__ x,
                                                          R* __restrict__ y, int nx, int ny,
                                                          int tiles_x, R w) {
  const Tile2 t = tile2(tiles_x);
  if (t.i >= nx || t.j >= ny) return;
  const int c = t.j * nx + t.i;
  if (t.i > 0 && t.i < nx - 1 && t.j > 0 && t.j < ny - 1) {
    R s = x[c];
    s += x[c - 1];
    s += x[c + 1];
    s += x[c - nx];
    s += x[c + nx];
    y[c] = w * s;
  } else {
    y[c] = x[c];
  }
}

// Adjoint (gather): with gi(q) = g[q] on interior q and 0 elsewhere,
//   interior m: g'[m] = w * (g[m] + sum_{q in nbr(m)} gi(q))
//   ring m:     g'[m] = g[m] + w * sum_{q in nbr(m)} gi(q)
// Points two or more cells from the edge see only interior neighbours.
template <class R>
__global__ __launch_bounds__(kThreads) void adj_jacobi2d5(const R* __restrict__ g,
                                                          R* __restrict__ gp, int nx, int ny,
                                                          int tiles_x, R w) {
  const Tile2 t = tile2(tiles_x);
  if (t.i >= nx || t.j >= ny) return;
  const int i = t.i, j = t.j;
  const int c = j * nx + i;
  if (i >= 2 && i <= nx - 3 && j >= 2 && j <= ny - 3) {
    R s = g[c];
    s += g[c - 1];
    s += g[c + 1];
    s += g[c - nx];
    s += g[c + nx];
    gp[c] = w * s;
    return;
  }
  auto gi = [&](int a, int b) -> R {
    return (a > 0 && a < nx - 1 && b > 0 && b < ny - 1) ? g[b * nx + a] : R(0);
  };
  R s = gi(i - 1, j);
  s += gi(i + 1, j);
  s += gi(i, j - 1);
  s += gi(i, j + 1);
  const bool interior = i > 0 && i < nx - 1 && j > 0 && j < ny - 1;
  gp[c] = interior ? w * (g[c] + s) : g[c] + w * s;
}

// ------------------------------------------------------- Allen-Cahn 3-D
// Forward, zero ghost values:
//   lap = (((((x[-x]+x[+x])+x[-y])+x[+y])+x[-z])+x[+z]) - 6*a
//   x'  = (a + D*lap) - C*((a*a)*a)
template <class R>
__global__ __launch_bounds__(kThreads) void fwd_allencahn3d7(const R* __restrict__ x,
                                                             R* __restrict__ y, int nx, int ny,
                                                             int nz, int tiles_x, int tiles_y,
                                                             R D, R C) {
  const Tile3 t = tile3(tiles_x, tiles_y);
  if (t.i >= nx || t.j >= ny) return;
  const int plane = nx * ny;
  const int c = t.k * plane + t.j * nx + t.i;
  const R a = x[c];
  const R xm = t.i > 0 ? x[c - 1] : R(0);
  const R xp = t.i < nx - 1 ? x[c + 1] : R(0);
  const R ym = t.j > 0 ? x[c - nx] : R(0);
  const R yp = t.j < ny - 1 ? x[c + nx] : R(0);
  const R zm = t.k > 0 ? x[c - plane] : R(0);
  const R zp = t.k < nz - 1 ? x[c + plane] : R(0);
  R lap = xm + xp;
  lap += ym;
  lap += yp;
  lap += zm;
  lap += zp;
  lap = lap - R(6) * a;
  y[c] = (a + D * lap) - C * ((a * a) * a);
}

// Adjoint: dx'[m]/dx[m] = (1 - 6D) - 3C x[m]^2 (the nonlinear term's adjoint,
// fused), dx'[c]/dx[m] = D for each in-grid face neighbour c of m. The
// Laplacian with zero ghosts is symmetric, so the gather reads g at m's own
// neighbours:  g'[m] = (k0 - k1*x[m]^2) * g[m] + D * sum_nbr g.
template <class R>
__global__ __launch_bounds__(kThreads) void adj_allencahn3d7(const R* __restrict__ x,
                                                             const R* __restrict__ g,
                                                             R* __restrict__ gp, int nx, int ny,
                                                             int nz, int tiles_x, int tiles_y,
                                                             R D, R k0, R k1) {
  const Tile3 t = tile3(tiles_x, tiles_y);
  if (t.i >= nx || t.j >= ny) return;
  const int plane = nx * ny;
  const int c = t.k * plane + t.j * nx + t.i;
  const R gm = t.i > 0 ? g[c - 1] : R(0);
  const R gpx = t.i < nx - 1 ? g[c + 1] : R(0);
  const R gym = t.j > 0 ? g[c - nx] : R(0);
  const R gyp = t.j < ny - 1 ? g[c + nx] : R(0);
  const R gzm = t.k > 0 ? g[c - plane] : R(0);
  const R gzp = t.k < nz - 1 ? g[c + plane] : R(0);
  R s = gm + gpx;
  s += gym;
  s += gyp;
  s += gzm;
  s += gzp;
  const R a = x[c];
  gp[c] = (k0 - k1 * (a * a)) * g[c] + D * s;
}

// ------------------------------------------ variable-coefficient diffusion 2-D
// Neighbour order (-1,0),(+1,0),(0,-1),(0,+1),(-1,-1),(+1,-1),(-1,+1),(+1,+1);
// the first four carry weight ca (1/3), the last four cd (1/12).
__constant__ int kNbrDx[8] = {-1, 1, 0, 0, -1, 1, -1, 1};
__constant__ int kNbrDy[8] = {0, 0, -1, 1, -1, -1, 1, 1};

// Forward: acc = sum over in-grid n of (c_n*(K[c]+K[n]))*(x[n]-x[c]),
// x' = x[c] + dt*acc.
template <class R>
__global__ __launch_bounds__(kThreads) void fwd_vardiff2d9(const R* __restrict__ x,
                                                           const R* __restrict__ K,
                                                           R* __restrict__ y, int nx, int ny,
                                                           int tiles_x, R dt, R ca, R cd) {
  const Tile2 t = tile2(tiles_x);
  if (t.i >= nx || t.j >= ny) return;
  const int i = t.i, j = t.j;
  const int c = j * nx + i;
  const R xc = x[c], Kc = K[c];
  R acc = R(0);
  if (i > 0 && i < nx - 1 && j > 0 && j < ny - 1) {
#pragma unroll
    for (int n = 0; n < 8; ++n) {
      const int m = c + kNbrDy[n] * nx + kNbrDx[n];
      const R cn = n < 4 ? ca : cd;
      acc += (cn * (Kc + K[m])) * (x[m] - xc);
    }
  } else {
#pragma unroll
    for (int n = 0; n < 8; ++n) {
      const int a = i + kNbrDx[n], b = j + kNbrDy[n];
      if (a < 0 || a >= nx || b < 0 || b >= ny) continue;
      const int m = b * nx + a;
      const R cn = n < 4 ? ca : cd;
      acc += (cn * (Kc + K[m])) * (x[m] - xc);
    }
  }
  y[c] = xc + dt * acc;
}

// Adjoint (the operator is symmetric in x):
//   g'[m] = g[m] + dt * sum_n (c_n*(K[m]+K[n]))*(g[n]-g[m])
//   dK[m] += dt * sum_n (c_n*(x[n]-x[m]))*(g[m]-g[n])      (x = x_{t-1})
// the second line being the coefficient-field gradient of step t, fused.
template <class R, bool WANT_DK>
__global__ __launch_bounds__(kThreads) void adj_vardiff2d9(const R* __restrict__ x,
                                                           const R* __restrict__ K,
                                                           const R* __restrict__ g,
                                                           R* __restrict__ gp, R* __restrict__ dK,
                                                           int dk_first, int nx, int ny,
                                                           int tiles_x, R dt, R ca, R cd) {
  const Tile2 t = tile2(tiles_x);
  if (t.i >= nx || t.j >= ny) return;
  const int i = t.i, j = t.j;
  const int c = j * nx + i;
  const R gc = g[c], Kc = K[c];
  const R xc = WANT_DK ? x[c] : R(0);
  R ag = R(0), ak = R(0);
  const bool interior = i > 0 && i < nx - 1 && j > 0 && j < ny - 1;
#pragma unroll
  for (int n = 0; n < 8; ++n) {
    const int a = i + kNbrDx[n], b = j + kNbrDy[n];
    if (!interior && (a < 0 || a >= nx || b < 0 || b >= ny)) continue;
    const int m = b * nx + a;
    const R cn = n < 4 ? ca : cd;
    const R gn = g[m];
    ag += (cn * (Kc + K[m])) * (gn - gc);
    if (WANT_DK) ak += (cn * (x[m] - xc)) * (gc - gn);
  }
  gp[c] = gc + dt * ag;
  if (WANT_DK) dK[c] = (dk_first ? R(0) : dK[c]) + dt * ak;
}

// --------------------------------------------------------------- loss, seed
// Sum over the 256 threads of a block: a wave64 butterfly, then the four
// wave sums in a fixed order. Valid in thread 0.
__device__ inline double block_sum(double v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  __shared__ double wave_sum[kThreads / 64];
  const int tid = threadIdx.y * kBX + threadIdx.x;
  if ((tid & 63) == 0) wave_sum[tid >> 6] = v;
  __syncthreads();
  return ((wave_sum[0] + wave_sum[1]) + wave_sum[2]) + wave_sum[3];
}

template <class R, int LOSS>
__global__ __launch_bounds__(kThreads) void seed_loss(const R* x, const R* __restrict__ aux, R* g,
                                                      R* __restrict__ xcopy, int64_t n,
                                                      double* __restrict__ partials) {
  const int tid = threadIdx.y * kBX + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  double acc = 0.0;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + tid; i < n; i += stride) {
    const R xv = x[i];
    R gv;
    double term;
    if (LOSS == ADST_LOSS_HALF_SQ) {
      gv = xv;
      term = 0.5 * ((double)xv * (double)xv);
    } else if (LOSS == ADST_LOSS_HALF_SQ_DIFF) {
      const R d = xv - aux[i];
      gv = d;
      term = 0.5 * ((double)d * (double)d);
    } else {  // DOT_W, SEED
      const R a = aux[i];
      gv = a;
      term = (double)a * (double)xv;
    }
    if (xcopy) xcopy[i] = xv;
    g[i] = gv;
    acc += term;
  }
  const double s = block_sum(acc);
  if (tid == 0) partials[blockIdx.x] = s;
}

__global__ __launch_bounds__(kThreads) void finalize_loss(const double* __restrict__ partials,
                                                          int nparts, double* __restrict__ out) {
  const int tid = threadIdx.y * kBX + threadIdx.x;
  double acc = 0.0;
  for (int i = tid; i < nparts; i += kThreads) acc += partials[i];
  const double s = block_sum(acc);
  if (tid == 0) *out = s;
}

// --------------------------------------------------------------- utilities
__global__ __launch_bounds__(kThreads) void fill_zero_u32(uint32_t* __restrict__ p, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.y * kBX + threadIdx.x; i < n;
       i += stride)
    p[i] = 0u;
}

__global__ __launch_bounds__(kThreads) void copy_u32(uint32_t* __restrict__ d,
                                                     const uint32_t* __restrict__ s, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.y * kBX + threadIdx.x; i < n;
       i += stride)
    d[i] = s[i];
}

int grid_for(int64_t n, int64_t per_block, int64_t cap) {
  int64_t b = (n + per_block - 1) / per_block;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return (int)b;
}

template <class R>
hipError_t forward_t(const StepShape& s, const void* xv, const void* Kv, void* yv,
                     hipStream_t st) {
  const R* x = static_cast<const R*>(xv);
  R* y = static_cast<R*>(yv);
  const dim3 block(kBX, kBY);
  const int tx = (s.nx + kBX - 1) / kBX, ty = (s.ny + kBY - 1) / kBY;
  const dim3 grid((unsigned)((int64_t)tx * ty * s.nz));
  switch (s.kind) {
    case ADST_JACOBI2D5:
      fwd_jacobi2d5<R><<<grid, block, 0, st>>>(x, y, s.nx, s.ny, tx, R(s.p0));
      break;
    case ADST_ALLENCAHN3D7:
      fwd_allencahn3d7<R><<<grid, block, 0, st>>>(x, y, s.nx, s.ny, s.nz, tx, ty, R(s.p0),
                                                  R(s.p1));
      break;
    case ADST_VARDIFF2D9:
      fwd_vardiff2d9<R><<<grid, block, 0, st>>>(x, static_cast<const R*>(Kv), y, s.nx, s.ny, tx,
                                                R(s.p0), R(1) / R(3), R(1) / R(12));
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <class R>
hipError_t adjoint_t(const StepShape& s, const void* xv, const void* Kv, const void* gv,
                     void* gpv, void* dKv, bool dk_first, hipStream_t st) {
  const R* x = static_cast<const R*>(xv);
  const R* K = static_cast<const R*>(Kv);
  const R* g = static_cast<const R*>(gv);
  R* gp = static_cast<R*>(gpv);
  R* dK = static_cast<R*>(dKv);
  const dim3 block(kBX, kBY);
  const int tx = (s.nx + kBX - 1) / kBX, ty = (s.ny + kBY - 1) / kBY;
  const dim3 grid((unsigned)((int64_t)tx * ty * s.nz));
  switch (s.kind) {
    case ADST_JACOBI2D5:
      adj_jacobi2d5<R><<<grid, block, 0, st>>>(g, gp, s.nx, s.ny, tx, R(s.p0));
      break;
    case ADST_ALLENCAHN3D7: {
      const R D = R(s.p0), C = R(s.p1);
      const R k0 = R(1) + D * R(-6), k1 = R(3) * C;
      adj_allencahn3d7<R><<<grid, block, 0, st>>>(x, g, gp, s.nx, s.ny, s.nz, tx, ty, D, k0, k1);
      break;
    }
    case ADST_VARDIFF2D9:
      if (dK)
        adj_vardiff2d9<R, true><<<grid, block, 0, st>>>(x, K, g, gp, dK, dk_first ? 1 : 0, s.nx,
                                                        s.ny, tx, R(s.p0), R(1) / R(3),
                                                        R(1) / R(12));
      else
        adj_vardiff2d9<R, false><<<grid, block, 0, st>>>(x, K, g, gp, nullptr, 0, s.nx, s.ny, tx,
                                                         R(s.p0), R(1) / R(3), R(1) / R(12));
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <class R>
hipError_t seed_t(int32_t loss, int64_t n, const void* xv, const void* auxv, void* gv,
                  void* xcopyv, double* partials, hipStream_t st) {
  const R* x = static_cast<const R*>(xv);
  const R* aux = static_cast<const R*>(auxv);
  R* g = static_cast<R*>(gv);
  R* xcopy = static_cast<R*>(xcopyv);
  const dim3 block(kBX, kBY);
  const dim3 grid(seed_partials(n));
  switch (loss) {
    case ADST_LOSS_HALF_SQ:
      seed_loss<R, ADST_LOSS_HALF_SQ><<<grid, block, 0, st>>>(x, aux, g, xcopy, n, partials);
      break;
    case ADST_LOSS_HALF_SQ_DIFF:
      seed_loss<R, ADST_LOSS_HALF_SQ_DIFF><<<grid, block, 0, st>>>(x, aux, g, xcopy, n, partials);
      break;
    case ADST_LOSS_DOT_W:
    case ADST_LOSS_SEED:
      seed_loss<R, ADST_LOSS_DOT_W><<<grid, block, 0, st>>>(x, aux, g, xcopy, n, partials);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_forward(const StepShape& s, const void* x, const void* K, void* y,
                          hipStream_t stream) {
  return s.dtype == ADST_F64 ? forward_t<double>(s, x, K, y, stream)
                             : forward_t<float>(s, x, K, y, stream);
}

hipError_t launch_adjoint(const StepShape& s, const void* x, const void* K, const void* g_next,
                          void* g_prev, void* dK, bool dk_first, hipStream_t stream) {
  return s.dtype == ADST_F64
             ? adjoint_t<double>(s, x, K, g_next, g_prev, dK, dk_first, stream)
             : adjoint_t<float>(s, x, K, g_next, g_prev, dK, dk_first, stream);
}

int32_t seed_partials(int64_t n) { return grid_for(n, 8 * kThreads, kMaxSeedPartials); }

hipError_t launch_seed(int32_t dtype, int32_t loss, int64_t n, const void* x, const void* aux,
                       void* g, void* xcopy, double* partials, hipStream_t stream) {
  return dtype == ADST_F64 ? seed_t<double>(loss, n, x, aux, g, xcopy, partials, stream)
                           : seed_t<float>(loss, n, x, aux, g, xcopy, partials, stream);
}

hipError_t launch_finalize(const double* partials, int32_t nparts, double* loss,
                           hipStream_t stream) {
  finalize_loss<<<dim3(1), dim3(kBX, kBY), 0, stream>>>(partials, nparts, loss);
  return hipGetLastError();
}

hipError_t launch_fill_zero(void* p, int64_t bytes, hipStream_t stream) {
  const int64_t n = bytes / 4;
  if (n == 0) return hipSuccess;
  fill_zero_u32<<<dim3(grid_for(n, kThreads * 4, 65536)), dim3(kBX, kBY), 0, stream>>>(
      static_cast<uint32_t*>(p), n);
  return hipGetLastError();
}

hipError_t launch_copy(void* dst, const void* src, int64_t bytes, hipStream_t stream) {
  const int64_t n = bytes / 4;
  if (n == 0) return hipSuccess;
  copy_u32<<<dim3(grid_for(n, kThreads * 4, 65536)), dim3(kBX, kBY), 0, stream>>>(
      static_cast<uint32_t*>(dst), static_cast<const uint32_t*>(src), n);
  return hipGetLastError();
}

}  // namespace adst
