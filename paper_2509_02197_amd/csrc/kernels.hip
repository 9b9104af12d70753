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

#include <algorithm>
#include <type_traits>

#include "adst.h"
#include "kernels.h"

namespace adst {
namespace {

constexpr int kBX = 64;  // one wavefront along x
constexpr int kBY = 4;   // four wavefronts per block
constexpr int kThreads = kBX * kBY;

// Launches cover their tiles in an XCD-aware order. Consecutive workgroup
// ids go to the 8 XCDs in turn, and each XCD has its own L2; renumbering so
// that XCD k works on the k-th contiguous eighth of the tiles keeps a tile's
// x- and y-neighbours (whose cache lines its halo shares) in the same L2.
// The grid is rounded up to a multiple of 8; surplus workgroups exit at once.
__device__ inline int xcd_tile(int ntiles) {
  const int per = (ntiles + 7) / 8;
  return (int)(blockIdx.x % 8) * per + (int)(blockIdx.x / 8);
}

inline unsigned xcd_grid(int64_t ntiles) { return (unsigned)(8 * ((ntiles + 7) / 8)); }

// Streaming stores. When a state is at least kStreamBytes, the states a
// launch reads and writes exceed the 256 MB Infinity Cache and nothing reads
// a written value again within the launch, so the Allen-Cahn and
// variable-coefficient kernels store (and the Allen-Cahn adjoint reads its
// once-read x) with non-temporal hints: written lines
// then stop evicting the halo lines that neighbouring tiles read from L2
// (measured at 512^3 f64: 4.7 -> 5.25 TB/s adjoint, 2393 -> 2193 ms for the
// 1024^3 call). Below it, the written state is the next launch's input and
// should stay in the Infinity Cache. The choice is a template argument: a
// run-time branch between the two stores is merged by the compiler into one
// store without the hint.
constexpr int64_t kStreamBytes = int64_t(256) << 20;
template <bool NT, class R>
__device__ inline void put(R* p, R v) {
  if constexpr (NT)
    __builtin_nontemporal_store(v, p);
  else
    *p = v;
}
template <bool NT, class R>
__device__ inline R take(const R* p) {
  if constexpr (NT)
    return __builtin_nontemporal_load(p);
  else
    return *p;
}

// ------------------------------------------------------- 2-D LDS tiles
// A workgroup owns a tile of the output: one thread per column, several
// rows each. It first stages the tile's input rows and columns, plus a halo,
// in LDS with all loads in flight at once (16-byte vector loads when rows are
// 16-byte aligned), then computes from LDS. Cells outside the grid read 0;
// no formula evaluated at an in-grid point uses them.

// Stage LR x LW elements of a, starting at global row row0 and column col0
// (col0 a multiple of the vector width), into lds (row stride LW).
template <class R, int NT, int LR, int LW>
__device__ inline void stage_rows(R* lds, const R* __restrict__ a, int col0, int row0, int nx,
                                  int ny, bool vec) {
  constexpr int V = 16 / sizeof(R);
  constexpr int CH = LW / V;
  static_assert(LW % V == 0, "LDS rows hold whole 16-byte chunks");
  typedef R vec_t __attribute__((ext_vector_type(V)));
  for (int q = threadIdx.x; q < LR * CH; q += NT) {
    const int rr = q / CH, ch = q - rr * CH;
    const int jj = row0 + rr;
    const int ii = col0 + ch * V;
    R* dst = lds + rr * LW + ch * V;
    if (jj < 0 || jj >= ny) {
#pragma unroll
      for (int e = 0; e < V; ++e) dst[e] = R(0);
    } else if (vec && ii >= 0 && ii + V <= nx) {
      const vec_t v = *reinterpret_cast<const vec_t*>(a + jj * nx + ii);
#pragma unroll
      for (int e = 0; e < V; ++e) dst[e] = v[e];
    } else {
#pragma unroll
      for (int e = 0; e < V; ++e) {
        const int c = ii + e;
        dst[e] = (c >= 0 && c < nx) ? a[jj * nx + c] : R(0);
      }
    }
  }
}

// ------------------------------------------------------- block reductions
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

// Block sums of two values, each over the 256 threads in a fixed order.
__device__ inline void block_sum2(double& a, double& b) {
  a = block_sum(a);
  __syncthreads();  // block_sum's wave sums are reused
  b = block_sum(b);
}

// Gradients of the step constants, fused into the adjoint kernels: one
// adjoint step's share of dL/dp is the sum over points of g_t[c] times the
// step's partial dF_c/dp at x_{t-1} (a constant read by every point of every
// step is a multiply-read input whose gradient accumulates, Sec. II). The
// partials are the sub-expressions the forward step forms, in its order:
//   Jacobi               dF/dw  = (((x[c]+x[W])+x[E])+x[S])+x[N] on interior points
//   Allen-Cahn           dF/dD  = lap,   dF/dC = -((x[c]*x[c])*x[c])
//   variable coefficient dF/ddt = acc
// Products and sums are in double. Each workgroup (one tile of the adjoint
// launch, whose tiling depends only on the grid) sums its points in a fixed
// order and adds the result into its own slot, step after step in the
// adjoint order t = T..1 (first: the step t = T overwrites), so the result
// does not depend on the schedule. part holds nslots slots per constant.
struct DpOut {
  double* part;
  int nslots, first;
};

// All threads of the block call this (it synchronises).
__device__ inline void dp_commit(DpOut dp, int slot, double a0, double a1) {
  block_sum2(a0, a1);
  if (threadIdx.x == 0 && threadIdx.y == 0) {
    double* p0 = dp.part + slot;
    double* p1 = dp.part + dp.nslots + slot;
    *p0 = dp.first ? a0 : *p0 + a0;
    *p1 = dp.first ? a1 : *p1 + a1;
  }
}

// Point updates read from an LDS array with row stride LW; q is the flat
// index of the point, (i, j) its grid coordinates. Single-step and fused
// kernels call the same functions, so a fused launch is bit-identical to two
// single launches.

// w*((((v[c]+v[W])+v[E])+v[S])+v[N]): the forward step at an interior point.
template <class R, int LW>
__device__ inline R jacobi_avg_at(const R* s, int q, R w) {
  R sum = s[q];
  sum += s[q - 1];
  sum += s[q + 1];
  sum += s[q - LW];
  sum += s[q + LW];
  return w * sum;
}

// Jacobi forward: interior x'[c] = w*((((x[c]+x[W])+x[E])+x[S])+x[N]);
// the ring is copied.
template <class R, int LW>
__device__ inline R jacobi_fwd_at(const R* s, int q, int i, int j, int nx, int ny, R w) {
  if (i > 0 && i < nx - 1 && j > 0 && j < ny - 1) return jacobi_avg_at<R, LW>(s, q, w);
  return s[q];
}

// Jacobi adjoint (gather): with gi(p) = g[p] on interior p and 0 elsewhere,
//   interior m: g'[m] = w * (g[m] + sum_{p in nbr(m)} gi(p))
//   ring m:     g'[m] = g[m] + w * sum_{p in nbr(m)} gi(p)
// the neighbours summed in the order W, E, S, N. Points two or more cells
// from the edge see only interior neighbours: w*(g[m] + (((W+E)+S)+N)).
template <class R, int LW>
__device__ inline R jacobi_adj_inner_at(const R* s, int q, R w) {
  R sum = s[q - 1];
  sum += s[q + 1];
  sum += s[q - LW];
  sum += s[q + LW];
  return w * (s[q] + sum);
}

// The value of a point whose stencil reads only interior points: the
// forward's average, or the adjoint's inner form.
template <class R, int LW, bool ADJ>
__device__ inline R jacobi_inner_at(const R* s, int q, R w) {
  return ADJ ? jacobi_adj_inner_at<R, LW>(s, q, w) : jacobi_avg_at<R, LW>(s, q, w);
}

template <class R, int LW>
__device__ inline R jacobi_adj_at(const R* s, int q, int i, int j, int nx, int ny, R w) {
  if (i >= 2 && i <= nx - 3 && j >= 2 && j <= ny - 3) return jacobi_adj_inner_at<R, LW>(s, q, w);
  const R c = s[q];
  auto interior = [&](int a, int b) { return a > 0 && a < nx - 1 && b > 0 && b < ny - 1; };
  R sum = interior(i - 1, j) ? s[q - 1] : R(0);
  sum += interior(i + 1, j) ? s[q + 1] : R(0);
  sum += interior(i, j - 1) ? s[q - LW] : R(0);
  sum += interior(i, j + 1) ? s[q + LW] : R(0);
  return interior(i, j) ? w * (c + sum) : c + w * sum;
}

// Variable-coefficient diffusion. Neighbour order (-1,0),(+1,0),(0,-1),
// (0,+1),(-1,-1),(+1,-1),(-1,+1),(+1,+1); the first four carry weight ca
// (1/3), the last four cd (1/12).
constexpr int kNbrDx[8] = {-1, 1, 0, 0, -1, 1, -1, 1};
constexpr int kNbrDy[8] = {0, 0, -1, 1, -1, -1, 1, 1};

// Forward: acc = sum over in-grid n of (c_n*(K[c]+K[n]))*(x[n]-x[c]),
// x' = x[c] + dt*acc.
template <class R, int LW>
__device__ inline R vardiff_fwd_at(const R* sx, const R* sk, int q, int i, int j, int nx, int ny,
                                   R dt, R ca, R cd) {
  const R xc = sx[q], Kc = sk[q];
  R acc = R(0);
  if (i > 0 && i < nx - 1 && j > 0 && j < ny - 1) {
#pragma unroll
    for (int n = 0; n < 8; ++n) {
      const int m = q + kNbrDy[n] * LW + kNbrDx[n];
      acc += ((n < 4 ? ca : cd) * (Kc + sk[m])) * (sx[m] - xc);
    }
  } else {
#pragma unroll
    for (int n = 0; n < 8; ++n) {
      const int a = i + kNbrDx[n], b = j + kNbrDy[n];
      if (a < 0 || a >= nx || b < 0 || b >= ny) continue;
      const int m = q + kNbrDy[n] * LW + kNbrDx[n];
      acc += ((n < 4 ? ca : cd) * (Kc + sk[m])) * (sx[m] - xc);
    }
  }
  return xc + dt * acc;
}

// The limiter: a new value below lo becomes lo, above hi becomes hi (the
// branch the step takes at each point; NaN passes through unchanged).
template <class R>
struct Limit {
  R lo, hi;
};
template <class R>
__device__ inline R limited(R y, Limit<R> l) {
  return y < l.lo ? l.lo : (y > l.hi ? l.hi : y);
}

// Single-step tiles: TW columns x TR rows, halo one cell (staged as one
// 16-byte chunk on each side).
template <class R, int TW, int TR>
struct Tile2 {
  static constexpr int V = 16 / sizeof(R);
  static constexpr int LW = TW + 2 * V;  // LDS row length
  static constexpr int LR = TR + 2;      // LDS rows
};

// Fused-pair tiles: kX2TW output columns, TR rows, halo two cells. The first
// step is evaluated on kX2TW + 2 columns and TR + 2 rows, so 254 columns fit
// the 256 threads one each and no wavefront does double work.
constexpr int kX2TW = 252, kX2Threads = 256, kX2TR = 4;
template <class R, int TR>
struct Tile2x2 {
  static constexpr int V = 16 / sizeof(R);
  static constexpr int PADL = ((2 + V - 1) / V) * V;  // left halo, whole chunks
  static constexpr int LW = PADL + ((kX2TW + 2 + V - 1) / V) * V;
  static constexpr int LR = TR + 4;
};

// ------------------------------------------------------------- Jacobi 2-D
constexpr int kJacTW = 256, kJacTR = 8;

// Every point of rows [ja, jb] x columns [ia, ib] takes the plain average:
// interior for the forward, two cells from the edge for the adjoint.
template <bool ADJ>
__device__ inline bool jacobi_all_avg(int ia, int ib, int ja, int jb, int nx, int ny) {
  const int m = ADJ ? 2 : 1;
  return ia >= m && ib <= nx - 1 - m && ja >= m && jb <= ny - 1 - m;
}

// Forward (ADJ = false) or adjoint (ADJ = true) Jacobi step on one tile;
// LIM clamps the forward's new values.
template <class R, bool ADJ, bool LIM = false>
__device__ inline void jacobi_tile(const R* __restrict__ x, R* __restrict__ y, int nx, int ny,
                                   int tiles_x, int ntiles, int vec, R w, Limit<R> lim = {}) {
  auto out = [&](R v) { return LIM ? limited(v, lim) : v; };
  using G = Tile2<R, kJacTW, kJacTR>;
  __shared__ R s[G::LR * G::LW];
  const int b = xcd_tile(ntiles);
  if (b >= ntiles) return;
  const int i0 = (b % tiles_x) * kJacTW, j0 = (b / tiles_x) * kJacTR;
  stage_rows<R, kJacTW, G::LR, G::LW>(s, x, i0 - G::V, j0 - 1, nx, ny, vec);
  __syncthreads();
  const int i = i0 + (int)threadIdx.x;
  if (i >= nx) return;
  const int cx = G::V + (int)threadIdx.x;
  if (jacobi_all_avg<ADJ>(i0, i0 + kJacTW - 1, j0, j0 + kJacTR - 1, nx, ny)) {
#pragma unroll
    for (int r = 0; r < kJacTR; ++r)
      y[(j0 + r) * nx + i] = out(jacobi_inner_at<R, G::LW, ADJ>(s, (r + 1) * G::LW + cx, w));
    return;
  }
#pragma unroll
  for (int r = 0; r < kJacTR; ++r) {
    const int j = j0 + r;
    if (j >= ny) break;
    const int q = (r + 1) * G::LW + cx;
    y[j * nx + i] = ADJ ? jacobi_adj_at<R, G::LW>(s, q, i, j, nx, ny, w)
                        : out(jacobi_fwd_at<R, G::LW>(s, q, i, j, nx, ny, w));
  }
}

// Two Jacobi steps (forward or adjoint) on one tile in one launch.
template <class R, bool ADJ>
__device__ inline void jacobi_tile_x2(const R* __restrict__ x, R* __restrict__ y, int nx, int ny,
                                      int tiles_x, int ntiles, int vec, R w) {
  using G = Tile2x2<R, kX2TR>;
  __shared__ R s[G::LR * G::LW];
  const int b = xcd_tile(ntiles);
  if (b >= ntiles) return;
  const int i0 = (b % tiles_x) * kX2TW, j0 = (b / tiles_x) * kX2TR;
  stage_rows<R, kX2Threads, G::LR, G::LW>(s, x, i0 - G::PADL, j0 - 2, nx, ny, vec);
  // the first step covers the tile plus one cell; whole tiles away from the
  // edges take the plain average everywhere (workgroup-uniform)
  const bool avg = jacobi_all_avg<ADJ>(i0 - 1, i0 + kX2TW, j0 - 1, j0 + kX2TR, nx, ny);
  __syncthreads();
  const int t = threadIdx.x;
  // first step: LDS rows 1..TR+2, LDS columns PADL-1 .. PADL+kX2TW
  const int c = G::PADL - 1 + t;
  const bool act = t < kX2TW + 2;
  const int ic = i0 - 1 + t;
  R v[kX2TR + 2];
  if (act) {
    if (avg) {
#pragma unroll
      for (int r = 1; r <= kX2TR + 2; ++r)
        v[r - 1] = jacobi_inner_at<R, G::LW, ADJ>(s, r * G::LW + c, w);
    } else {
#pragma unroll
      for (int r = 1; r <= kX2TR + 2; ++r) {
        const int q = r * G::LW + c;
        const int j = j0 - 2 + r;
        v[r - 1] = ADJ ? jacobi_adj_at<R, G::LW>(s, q, ic, j, nx, ny, w)
                       : jacobi_fwd_at<R, G::LW>(s, q, ic, j, nx, ny, w);
      }
    }
  }
  __syncthreads();
  if (act) {
#pragma unroll
    for (int r = 1; r <= kX2TR + 2; ++r) s[r * G::LW + c] = v[r - 1];
  }
  __syncthreads();
  // second step on the output tile
  const int i = i0 + t;
  if (t >= kX2TW || i >= nx) return;
  const int cx = G::PADL + t;
  if (avg) {
#pragma unroll
    for (int r = 0; r < kX2TR; ++r)
      y[(j0 + r) * nx + i] = jacobi_inner_at<R, G::LW, ADJ>(s, (r + 2) * G::LW + cx, w);
    return;
  }
#pragma unroll
  for (int r = 0; r < kX2TR; ++r) {
    const int j = j0 + r;
    if (j >= ny) break;
    const int q = (r + 2) * G::LW + cx;
    y[j * nx + i] = ADJ ? jacobi_adj_at<R, G::LW>(s, q, i, j, nx, ny, w)
                        : jacobi_fwd_at<R, G::LW>(s, q, i, j, nx, ny, w);
  }
}

template <class R, bool LIM>
__global__ __launch_bounds__(kJacTW) void fwd_jacobi2d5(const R* __restrict__ x,
                                                        R* __restrict__ y, int nx, int ny,
                                                        int tiles_x, int ntiles, int vec, R w,
                                                        Limit<R> lim) {
  jacobi_tile<R, false, LIM>(x, y, nx, ny, tiles_x, ntiles, vec, w, lim);
}
template <class R>
__global__ __launch_bounds__(kJacTW) void adj_jacobi2d5(const R* __restrict__ g,
                                                        R* __restrict__ gp, int nx, int ny,
                                                        int tiles_x, int ntiles, int vec, R w) {
  jacobi_tile<R, true>(g, gp, nx, ny, tiles_x, ntiles, vec, w);
}
template <class R>
__global__ __launch_bounds__(kX2Threads) void fwd_jacobi2d5_x2(const R* __restrict__ x,
                                                               R* __restrict__ y, int nx, int ny,
                                                               int tiles_x, int ntiles, int vec,
                                                               R w) {
  jacobi_tile_x2<R, false>(x, y, nx, ny, tiles_x, ntiles, vec, w);
}
template <class R>
__global__ __launch_bounds__(kX2Threads) void adj_jacobi2d5_x2(const R* __restrict__ g,
                                                               R* __restrict__ gp, int nx, int ny,
                                                               int tiles_x, int ntiles, int vec,
                                                               R w) {
  jacobi_tile_x2<R, true>(g, gp, nx, ny, tiles_x, ntiles, vec, w);
}

// ------------------------------------------------------- Allen-Cahn 3-D
// 2.5-D blocking: a workgroup of 64 x 4 threads owns a 64 x 8 column of the
// grid over kAcZC planes (two rows per thread) and marches in z. The plane
// being updated is staged in LDS with a one-cell xy halo; the planes below
// and above live in registers, so every input plane is read from HBM once
// per tile.
constexpr int kAcTX = 64, kAcTY = 8, kAcZC = 32;

struct AcTile {
  int b, i, ja, jb, by, bx, z0, z1;
};

__device__ inline bool ac_tile(int nx, int ny, int nz, int tiles_x, int tiles_y, int ntiles,
                               AcTile* t) {
  int b = xcd_tile(ntiles);
  if (b >= ntiles) return false;
  t->b = b;
  t->bx = b % tiles_x;
  b /= tiles_x;
  t->by = b % tiles_y;
  const int bz = b / tiles_y;
  t->i = t->bx * kAcTX + (int)threadIdx.x;
  t->ja = t->by * kAcTY + (int)threadIdx.y;
  t->jb = t->ja + 4;
  t->z0 = bz * kAcZC;
  t->z1 = min(t->z0 + kAcZC, nz);
  return true;
}

// Halo cell this thread stages (at most one; 2*64 + 2*8 = 144 < 256).
__device__ inline void ac_halo_cell(int tid, int* ly, int* lx) {
  constexpr int LY = kAcTY + 2, LX = kAcTX + 2;
  const int h = tid;
  if (h < kAcTX) {
    *ly = 0;
    *lx = h + 1;
  } else if (h < 2 * kAcTX) {
    *ly = LY - 1;
    *lx = h - kAcTX + 1;
  } else if (h < 2 * kAcTX + kAcTY) {
    *ly = h - 2 * kAcTX + 1;
    *lx = 0;
  } else if (h < 2 * kAcTX + 2 * kAcTY) {
    *ly = h - 2 * kAcTX - kAcTY + 1;
    *lx = LX - 1;
  } else {
    *ly = -1;
    *lx = 0;
  }
}

// Forward, zero ghost values:
//   lap = (((((x[-x]+x[+x])+x[-y])+x[+y])+x[-z])+x[+z]) - 6*a
//   x'  = (a + D*lap) - C*((a*a)*a)
// Single-step and fused kernels evaluate every point through this function.
template <class R>
__device__ inline R allencahn_point(R a, R xm, R xp, R ym, R yp, R zm, R zp, R D, R C) {
  R lap = xm + xp;
  lap += ym;
  lap += yp;
  lap += zm;
  lap += zp;
  lap = lap - R(6) * a;
  return (a + D * lap) - C * ((a * a) * a);
}

template <class R, bool LIM, bool NT>
__global__ __launch_bounds__(kThreads) void fwd_allencahn3d7(const R* __restrict__ x,
                                                             R* __restrict__ y, int nx, int ny,
                                                             int nz, int tiles_x, int tiles_y,
                                                             int ntiles, R D, R C, Limit<R> lim) {
  auto out = [&](R v) { return LIM ? limited(v, lim) : v; };
  __shared__ R tile[kAcTY + 2][kAcTX + 2];
  AcTile t;
  if (!ac_tile(nx, ny, nz, tiles_x, tiles_y, ntiles, &t)) return;
  const int plane = nx * ny;
  auto ld = [&](int k, int j, int i) -> R {
    return (k >= 0 && k < nz && j >= 0 && j < ny && i >= 0 && i < nx) ? x[k * plane + j * nx + i]
                                                                      : R(0);
  };
  const int tx = threadIdx.x, ty = threadIdx.y, tid = ty * kBX + tx;
  int hly, hlx;
  ac_halo_cell(tid, &hly, &hlx);
  const int hj = t.by * kAcTY + hly - 1, hi = t.bx * kAcTX + hlx - 1;
  const bool va = t.i < nx && t.ja < ny, vb = t.i < nx && t.jb < ny;
  R belowA = ld(t.z0 - 1, t.ja, t.i), belowB = ld(t.z0 - 1, t.jb, t.i);
  R curA = ld(t.z0, t.ja, t.i), curB = ld(t.z0, t.jb, t.i);
  R halo = hly >= 0 ? ld(t.z0, hj, hi) : R(0);
  for (int k = t.z0; k < t.z1; ++k) {
    // the next plane's cells are requested before this plane is computed
    const R aboveA = ld(k + 1, t.ja, t.i), aboveB = ld(k + 1, t.jb, t.i);
    const R haloN = hly >= 0 ? ld(k + 1, hj, hi) : R(0);
    __syncthreads();
    tile[ty + 1][tx + 1] = curA;
    tile[ty + 5][tx + 1] = curB;
    if (hly >= 0) tile[hly][hlx] = halo;
    __syncthreads();
    if (va)
      put<NT>(&y[k * plane + t.ja * nx + t.i],
              out(allencahn_point(curA, tile[ty + 1][tx], tile[ty + 1][tx + 2], tile[ty][tx + 1],
                                  tile[ty + 2][tx + 1], belowA, aboveA, D, C)));
    if (vb)
      put<NT>(&y[k * plane + t.jb * nx + t.i],
              out(allencahn_point(curB, tile[ty + 5][tx], tile[ty + 5][tx + 2], tile[ty + 4][tx + 1],
                                  tile[ty + 6][tx + 1], belowB, aboveB, D, C)));
    belowA = curA;
    belowB = curB;
    curA = aboveA;
    curB = aboveB;
    halo = haloN;
  }
}

// K forward steps in one launch (temporal blocking in 2.5-D).
// A workgroup of 64 x 4 threads owns a region of 64 columns x SY = 4 RPT
// rows of each plane (RPT rows per thread, four apart) and marches in z. At
// iteration p it evaluates step 1 at plane p from x(p-1..p+1), and step l at
// plane p-l+1 from step l-1's planes p-l..p-l+2. Every step is evaluated on
// the whole region but is valid only on its inner (64 - 2(l-1)) x (SY -
// 2(l-1)) cells, because its xy neighbours come from the step before it on
// the same region; the last step's valid cells are the output tile. x(p)
// (with a one-cell ring) and each intermediate step's latest plane are
// staged in LDS for the xy neighbours, the planes below and above stay in
// registers. Intermediate values are 0 outside the grid, which is the zero
// ghost value the next step reads; every point evaluates the single-step
// expression, so any split of the steps into launches gives the same bits.
// Measured at 1024^3 f64, three steps per launch (64 x 16 regions, 64
// planes) beat two (the launches of a recomputation run drop by a third);
// four, with 24-row regions, needed 178 VGPRs and with 16-row regions
// evaluated 7 points per output point, and both were slower.
template <int K, int RPT, int NZ>
struct AcN {
  static constexpr int SX = kBX, SY = kBY * RPT;
  static constexpr int OX = SX - 2 * (K - 1), OY = SY - 2 * (K - 1);  // output tile
  static constexpr int ZC = NZ;                                     // output planes
};

// ST: the intermediate states are stored too, step l's into mid[l-1], each
// point by the workgroup whose output tile holds it (a run of steps whose
// every state is kept moves 8 + 8n bytes per point for n steps instead of
// 16n). They are stored without the non-temporal hint: the reverse sweep
// reads them back soon after (measured at 512^3: 58.9 -> 58.5 ms per call).
template <class R, int K, int RPT, int NZ, bool NT, bool ST>
__global__ __launch_bounds__(kThreads) void fwd_allencahn3d7_n(const R* __restrict__ x,
                                                               R* __restrict__ y,
                                                               R* __restrict__ mid0,
                                                               R* __restrict__ mid1, int nx,
                                                               int ny, int nz, int tiles_x,
                                                               int tiles_y, int ntiles, R D,
                                                               R C) {
  using A = AcN<K, RPT, NZ>;
  constexpr int SX = A::SX, SY = A::SY, LX = SX + 2, LY = SY + 2, H = K - 1;
  static_assert(K >= 2 && 2 * LX + 2 * SY <= kThreads, "ring cells: one per thread");
  static_assert(!ST || K <= 3, "intermediate states go to mid0 (step 1) and mid1 (step 2)");
  __shared__ R xt[LY][LX];
  __shared__ R yt[K - 1][SY][SX];  // steps 1 .. K-1
  int b = xcd_tile(ntiles);
  if (b >= ntiles) return;
  const int bx = b % tiles_x;
  b /= tiles_x;
  const int by = b % tiles_y;
  const int bz = b / tiles_y;
  const int i0 = bx * A::OX, j0 = by * A::OY;
  const int z0 = bz * A::ZC, z1 = min(z0 + A::ZC, nz);
  const int tx = threadIdx.x, ty = threadIdx.y, tid = ty * kBX + tx;
  const int ic = i0 - H + tx;  // column of this thread
  const int plane = nx * ny;
  auto inxy = [&](int j, int i) { return i >= 0 && i < nx && j >= 0 && j < ny; };
  auto ld = [&](int k, int j, int i) -> R {
    return (k >= 0 && k < nz && inxy(j, i)) ? x[k * plane + j * nx + i] : R(0);
  };
  auto row = [&](int q) { return ty + kBY * q; };  // region row of the thread's q-th cell
  // one cell of the LDS ring around the region
  int hly = -1, hlx = 0;
  if (tid < LX) {
    hly = 0;
    hlx = tid;
  } else if (tid < 2 * LX) {
    hly = LY - 1;
    hlx = tid - LX;
  } else if (tid < 2 * LX + SY) {
    hly = tid - 2 * LX + 1;
    hlx = 0;
  } else if (tid < 2 * LX + 2 * SY) {
    hly = tid - 2 * LX - SY + 1;
    hlx = LX - 1;
  }
  const int hj = j0 - H - 1 + hly, hi = i0 - H - 1 + hlx;
  // x at planes p-1, p, p+1; step l (index l-1) at planes p-l, p-l+1 and the
  // one evaluated in this iteration
  R xp[RPT], xc[RPT], xn[RPT];
  R sb[K - 1][RPT], sc[K - 1][RPT], sn[K - 1][RPT];
  const int pfirst = z0 - K + 1, plast = z1 + K - 2;
  // this thread's column lies in the output tile (rows are checked per cell)
  const bool tile_col = tx >= H && tx < SX - H;
#pragma unroll
  for (int q = 0; q < RPT; ++q) {
    const int j = j0 - H + row(q);
    xp[q] = ld(pfirst - 1, j, ic);
    xc[q] = ld(pfirst, j, ic);
#pragma unroll
    for (int l = 0; l < K - 1; ++l) sb[l][q] = sc[l][q] = R(0);
  }
  R hv = hly >= 0 ? ld(pfirst, hj, hi) : R(0);
  for (int p = pfirst; p <= plast; ++p) {
    // the next plane's cells are requested before this plane is computed
#pragma unroll
    for (int q = 0; q < RPT; ++q) xn[q] = ld(p + 1, j0 - H + row(q), ic);
    const R hvn = hly >= 0 ? ld(p + 1, hj, hi) : R(0);
    __syncthreads();
#pragma unroll
    for (int q = 0; q < RPT; ++q) xt[row(q) + 1][tx + 1] = xc[q];
    if (hly >= 0) xt[hly][hlx] = hv;
    __syncthreads();
    {  // step 1 at plane p, on every cell of the region
      const bool pin = p >= 0 && p < nz;
#pragma unroll
      for (int q = 0; q < RPT; ++q) {
        const int r = row(q);
        const bool cin = pin && inxy(j0 - H + r, ic);
        sn[0][q] = cin ? allencahn_point(xc[q], xt[r + 1][tx], xt[r + 1][tx + 2], xt[r][tx + 1],
                                         xt[r + 2][tx + 1], xp[q], xn[q], D, C)
                       : R(0);
        if constexpr (ST) {
          if (cin && tile_col && r >= H && r < SY - H && p >= z0 && p < z1)
            put<false>(&mid0[p * plane + (j0 - H + r) * nx + ic], sn[0][q]);
        }
      }
    }
#pragma unroll
    for (int l = 2; l <= K; ++l) {  // step l at plane p - l + 1
      const int pl = p - l + 1;
      const bool pin = pl >= 0 && pl < nz;
      const bool xin = tx >= l - 1 && tx <= SX - l;
#pragma unroll
      for (int q = 0; q < RPT; ++q) {
        const int r = row(q);
        const int j = j0 - H + r;
        const bool ok = pin && xin && r >= l - 1 && r <= SY - l && inxy(j, ic);
        const R(*t)[SX] = yt[l - 2];
        const R v = ok ? allencahn_point(sc[l - 2][q], t[r][tx - 1], t[r][tx + 1], t[r - 1][tx],
                                         t[r + 1][tx], sb[l - 2][q], sn[l - 2][q], D, C)
                       : R(0);
        if (l < K) {
          sn[l - 1][q] = v;
          if constexpr (ST) {
            if (ok && tile_col && r >= H && r < SY - H && pl >= z0 && pl < z1)
              put<false>(&(l == 2 ? mid1 : mid0)[pl * plane + j * nx + ic], v);
          }
        } else if (ok && pl >= z0 && pl < z1) {
          put<NT>(&y[pl * plane + j * nx + ic], v);
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int l = 0; l < K - 1; ++l)
#pragma unroll
      for (int q = 0; q < RPT; ++q) yt[l][row(q)][tx] = sn[l][q];
#pragma unroll
    for (int q = 0; q < RPT; ++q) {
      xp[q] = xc[q];
      xc[q] = xn[q];
#pragma unroll
      for (int l = 0; l < K - 1; ++l) {
        sb[l][q] = sc[l][q];
        sc[l][q] = sn[l][q];
      }
    }
    hv = hvn;
  }
}

// Adjoint: dx'[m]/dx[m] = (1 - 6D) - 3C x[m]^2 (the nonlinear term's adjoint,
// fused), dx'[c]/dx[m] = D for each in-grid face neighbour c of m. The
// Laplacian with zero ghosts is symmetric, so the gather reads g at m's own
// neighbours:  g'[m] = (k0 - k1*x[m]^2) * g[m] + D * sum_nbr g.
// DP: also this step's share of dL/dD and dL/dC (see DpOut), from x_{t-1}
// staged the same way as g (its plane in LDS, the planes below and above in
// registers).
template <class R, bool DP, bool NT>
__global__ __launch_bounds__(kThreads) void adj_allencahn3d7(const R* __restrict__ x,
                                                             const R* __restrict__ g,
                                                             R* __restrict__ gp, int nx, int ny,
                                                             int nz, int tiles_x, int tiles_y,
                                                             int ntiles, R D, R k0, R k1,
                                                             DpOut dp) {
  __shared__ R tile[kAcTY + 2][kAcTX + 2];
  __shared__ R tilex[DP ? kAcTY + 2 : 1][DP ? kAcTX + 2 : 1];
  AcTile t;
  if (!ac_tile(nx, ny, nz, tiles_x, tiles_y, ntiles, &t)) return;  // the whole block
  const int plane = nx * ny;
  auto ld = [&](const R* a, int k, int j, int i) -> R {
    return (k >= 0 && k < nz && j >= 0 && j < ny && i >= 0 && i < nx) ? a[k * plane + j * nx + i]
                                                                      : R(0);
  };
  // without the constants' gradients x is read once per point (streamed)
  auto ldnt = [&](const R* a, int k, int j, int i) -> R {
    return (k >= 0 && k < nz && j >= 0 && j < ny && i >= 0 && i < nx)
               ? take<NT>(&a[k * plane + j * nx + i])
               : R(0);
  };
  auto ldg = [&](int k, int j, int i) -> R { return ld(g, k, j, i); };
  const int tx = threadIdx.x, ty = threadIdx.y, tid = ty * kBX + tx;
  int hly, hlx;
  ac_halo_cell(tid, &hly, &hlx);
  const int hj = t.by * kAcTY + hly - 1, hi = t.bx * kAcTX + hlx - 1;
  const bool va = t.i < nx && t.ja < ny, vb = t.i < nx && t.jb < ny;
  // Every value a plane needs (g and x at the thread's cells, the halo cell)
  // is requested one plane ahead, before the current plane is computed.
  R belowA = ldg(t.z0 - 1, t.ja, t.i), belowB = ldg(t.z0 - 1, t.jb, t.i);
  R curA = ldg(t.z0, t.ja, t.i), curB = ldg(t.z0, t.jb, t.i);
  R halo = hly >= 0 ? ldg(t.z0, hj, hi) : R(0);
  R xbelowA = R(0), xbelowB = R(0);
  R xcurA = ld(x, t.z0, t.ja, t.i), xcurB = ld(x, t.z0, t.jb, t.i);
  R xhalo = R(0);
  if (DP) {
    xbelowA = ld(x, t.z0 - 1, t.ja, t.i);
    xbelowB = ld(x, t.z0 - 1, t.jb, t.i);
    xhalo = hly >= 0 ? ld(x, t.z0, hj, hi) : R(0);
  }
  double a0 = 0.0, a1 = 0.0;
  for (int k = t.z0; k < t.z1; ++k) {
    const R aboveA = ldg(k + 1, t.ja, t.i), aboveB = ldg(k + 1, t.jb, t.i);
    const R haloN = hly >= 0 ? ldg(k + 1, hj, hi) : R(0);
    const R xaboveA = DP ? ld(x, k + 1, t.ja, t.i) : ldnt(x, k + 1, t.ja, t.i);
    const R xaboveB = DP ? ld(x, k + 1, t.jb, t.i) : ldnt(x, k + 1, t.jb, t.i);
    const R xhaloN = DP && hly >= 0 ? ld(x, k + 1, hj, hi) : R(0);
    const R xa = xcurA, xb = xcurB;
    __syncthreads();
    tile[ty + 1][tx + 1] = curA;
    tile[ty + 5][tx + 1] = curB;
    if (hly >= 0) tile[hly][hlx] = halo;
    if (DP) {
      tilex[ty + 1][tx + 1] = xcurA;
      tilex[ty + 5][tx + 1] = xcurB;
      if (hly >= 0) tilex[hly][hlx] = xhalo;
    }
    __syncthreads();
    // lap of x at row r of this thread (r = 1: A, r = 5: B), the forward's order
    auto lapx = [&](int r, R xzm, R xzp, R a) {
      R lap = tilex[ty + r][tx] + tilex[ty + r][tx + 2];
      lap += tilex[ty + r - 1][tx + 1];
      lap += tilex[ty + r + 1][tx + 1];
      lap += xzm;
      lap += xzp;
      return lap - R(6) * a;
    };
    if (va) {
      R s = tile[ty + 1][tx] + tile[ty + 1][tx + 2];
      s += tile[ty][tx + 1];
      s += tile[ty + 2][tx + 1];
      s += belowA;
      s += aboveA;
      put<NT>(&gp[k * plane + t.ja * nx + t.i], (k0 - k1 * (xa * xa)) * curA + D * s);
      if (DP) {
        a0 += (double)curA * (double)lapx(1, xbelowA, xaboveA, xa);
        a1 += (double)curA * (double)(-((xa * xa) * xa));
      }
    }
    if (vb) {
      R s = tile[ty + 5][tx] + tile[ty + 5][tx + 2];
      s += tile[ty + 4][tx + 1];
      s += tile[ty + 6][tx + 1];
      s += belowB;
      s += aboveB;
      put<NT>(&gp[k * plane + t.jb * nx + t.i], (k0 - k1 * (xb * xb)) * curB + D * s);
      if (DP) {
        a0 += (double)curB * (double)lapx(5, xbelowB, xaboveB, xb);
        a1 += (double)curB * (double)(-((xb * xb) * xb));
      }
    }
    belowA = curA;
    belowB = curB;
    curA = aboveA;
    curB = aboveB;
    halo = haloN;
    xbelowA = xcurA;
    xbelowB = xcurB;
    xcurA = xaboveA;
    xcurB = xaboveB;
    xhalo = xhaloN;
  }
  if (DP) {
    __syncthreads();
    dp_commit(dp, t.b, a0, a1);
  }
}

// The limiter's adjoint, g'[m] = (k0 - k1*x[m]^2) * gm[m] + D * sum_nbr gm,
// with gm = g where the step's unlimited value (re-evaluated from x =
// x_{t-1} with the forward's expression) lies in [lo, hi] and 0 elsewhere.
// The masked plane k+1 is formed in iteration k: x(k+1) is staged in LDS
// with a two-cell ring (the masks of g's one-cell ring need their own xy
// neighbours), x(k) and x(k+2) at the thread's cells and ring cell stay in
// registers, so every mask is evaluated from on-chip values and x is read
// from HBM about once per point.
template <class R, bool NT>
__global__ __launch_bounds__(kThreads) void adj_allencahn3d7_lim(const R* __restrict__ x,
                                                                 const R* __restrict__ g,
                                                                 R* __restrict__ gp, int nx,
                                                                 int ny, int nz, int tiles_x,
                                                                 int tiles_y, int ntiles, R D,
                                                                 R k0, R k1, R C, Limit<R> lim) {
  constexpr int LY = kAcTY + 2, LX = kAcTX + 2;          // g: one-cell ring
  constexpr int XY = kAcTY + 4, XX = kAcTX + 4;          // x: two-cell ring
  __shared__ R tile[LY][LX];
  __shared__ R xt[XY][XX];
  AcTile t;
  if (!ac_tile(nx, ny, nz, tiles_x, tiles_y, ntiles, &t)) return;  // the whole block
  const int plane = nx * ny;
  auto in = [&](int k, int j, int i) {
    return k >= 0 && k < nz && j >= 0 && j < ny && i >= 0 && i < nx;
  };
  auto ld = [&](const R* a, int k, int j, int i) -> R {
    return in(k, j, i) ? a[k * plane + j * nx + i] : R(0);
  };
  auto keep = [&](R y) { return !(y < lim.lo || y > lim.hi); };
  // g at a cell masked from global memory (the first planes only)
  auto ldg = [&](int k, int j, int i) -> R {
    if (!in(k, j, i)) return R(0);
    const int q = k * plane + j * nx + i;
    const R y = allencahn_point(x[q], i > 0 ? x[q - 1] : R(0), i < nx - 1 ? x[q + 1] : R(0),
                                j > 0 ? x[q - nx] : R(0), j < ny - 1 ? x[q + nx] : R(0),
                                k > 0 ? x[q - plane] : R(0), k < nz - 1 ? x[q + plane] : R(0),
                                D, C);
    return keep(y) ? g[q] : R(0);
  };
  const int tx = threadIdx.x, ty = threadIdx.y, tid = ty * kBX + tx;
  const int i0 = t.bx * kAcTX, j0 = t.by * kAcTY;
  // this thread's cell of g's ring (tile coordinates hly-1, hlx-1), if any
  int hly, hlx;
  ac_halo_cell(tid, &hly, &hlx);
  const bool hr = hly >= 0;
  const int hj = j0 + hly - 1, hi = i0 + hlx - 1;
  // this thread's cell of x's outer ring, or one of the four corners of
  // g's ring (which g's ring cells need as x neighbours), in x-tile
  // coordinates, if any: 2*68 + 2*10 + 4 = 160 cells
  int oy = -1, ox = 0;
  if (tid < XX) {
    oy = 0;
    ox = tid;
  } else if (tid < 2 * XX) {
    oy = XY - 1;
    ox = tid - XX;
  } else if (tid < 2 * XX + LY) {
    oy = tid - 2 * XX + 1;
    ox = 0;
  } else if (tid < 2 * XX + 2 * LY) {
    oy = tid - 2 * XX - LY + 1;
    ox = XX - 1;
  } else if (tid < 2 * XX + 2 * LY + 4) {
    const int c = tid - 2 * XX - 2 * LY;
    oy = (c & 2) ? XY - 2 : 1;
    ox = (c & 1) ? XX - 2 : 1;
  }
  const bool orr = oy >= 0;
  const int oj = j0 + oy - 2, oi = i0 + ox - 2;
  const bool va = t.i < nx && t.ja < ny, vb = t.i < nx && t.jb < ny;
  // masked g: planes k-1, k at the thread's cells, plane k at its ring cell
  R belowA = ldg(t.z0 - 1, t.ja, t.i), belowB = ldg(t.z0 - 1, t.jb, t.i);
  R curA = ldg(t.z0, t.ja, t.i), curB = ldg(t.z0, t.jb, t.i);
  R halo = hr ? ldg(t.z0, hj, hi) : R(0);
  // x at planes k, k+1 (the thread's cells and ring cell), outer ring at k+1
  R xA0 = ld(x, t.z0, t.ja, t.i), xB0 = ld(x, t.z0, t.jb, t.i);
  R xA1 = ld(x, t.z0 + 1, t.ja, t.i), xB1 = ld(x, t.z0 + 1, t.jb, t.i);
  R xr0 = hr ? ld(x, t.z0, hj, hi) : R(0), xr1 = hr ? ld(x, t.z0 + 1, hj, hi) : R(0);
  R xo1 = orr ? ld(x, t.z0 + 1, oj, oi) : R(0);
  for (int k = t.z0; k < t.z1; ++k) {
    // plane k+1's g, plane k+2's x and the outer ring of plane k+2 (for the
    // next iteration) are requested before this plane is computed
    const R gA = ld(g, k + 1, t.ja, t.i), gB = ld(g, k + 1, t.jb, t.i);
    const R gr = hr ? ld(g, k + 1, hj, hi) : R(0);
    const R xA2 = ld(x, k + 2, t.ja, t.i), xB2 = ld(x, k + 2, t.jb, t.i);
    const R xr2 = hr ? ld(x, k + 2, hj, hi) : R(0);
    const R xo2 = orr ? ld(x, k + 2, oj, oi) : R(0);
    __syncthreads();
    tile[ty + 1][tx + 1] = curA;
    tile[ty + 5][tx + 1] = curB;
    if (hr) tile[hly][hlx] = halo;
    xt[ty + 2][tx + 2] = xA1;
    xt[ty + 6][tx + 2] = xB1;
    if (hr) xt[hly + 1][hlx + 1] = xr1;
    if (orr) xt[oy][ox] = xo1;
    __syncthreads();
    // the masks of plane k+1 (x-tile position r, c; x(k) and x(k+2) there)
    auto masked = [&](int r, int c, R xb, R xa, R gv) {
      const R y = allencahn_point(xt[r][c], xt[r][c - 1], xt[r][c + 1], xt[r - 1][c],
                                  xt[r + 1][c], xb, xa, D, C);
      return keep(y) ? gv : R(0);
    };
    const R aboveA = masked(ty + 2, tx + 2, xA0, xA2, gA);
    const R aboveB = masked(ty + 6, tx + 2, xB0, xB2, gB);
    const R halon = hr ? masked(hly + 1, hlx + 1, xr0, xr2, gr) : R(0);
    if (va) {
      R s = tile[ty + 1][tx] + tile[ty + 1][tx + 2];
      s += tile[ty][tx + 1];
      s += tile[ty + 2][tx + 1];
      s += belowA;
      s += aboveA;
      put<NT>(&gp[k * plane + t.ja * nx + t.i], (k0 - k1 * (xA0 * xA0)) * curA + D * s);
    }
    if (vb) {
      R s = tile[ty + 5][tx] + tile[ty + 5][tx + 2];
      s += tile[ty + 4][tx + 1];
      s += tile[ty + 6][tx + 1];
      s += belowB;
      s += aboveB;
      put<NT>(&gp[k * plane + t.jb * nx + t.i], (k0 - k1 * (xB0 * xB0)) * curB + D * s);
    }
    belowA = curA;
    belowB = curB;
    curA = aboveA;
    curB = aboveB;
    halo = halon;
    xA0 = xA1;
    xB0 = xB1;
    xA1 = xA2;
    xB1 = xB2;
    xr0 = xr1;
    xr1 = xr2;
    xo1 = xo2;
  }
}

// ------------------------------------------ variable-coefficient diffusion 2-D
constexpr int kVdTW = 256, kVdTR = 8, kVdAdjTR = 4;

template <class R, bool LIM, bool NT>
__global__ __launch_bounds__(kVdTW) void fwd_vardiff2d9(const R* __restrict__ x,
                                                        const R* __restrict__ K,
                                                        R* __restrict__ y, int nx, int ny,
                                                        int tiles_x, int ntiles, int vec, R dt,
                                                        R ca, R cd, Limit<R> lim) {
  using G = Tile2<R, kVdTW, kVdTR>;
  __shared__ R sx[G::LR * G::LW];
  __shared__ R sk[G::LR * G::LW];
  const int b = xcd_tile(ntiles);
  if (b >= ntiles) return;
  const int i0 = (b % tiles_x) * kVdTW, j0 = (b / tiles_x) * kVdTR;
  stage_rows<R, kVdTW, G::LR, G::LW>(sx, x, i0 - G::V, j0 - 1, nx, ny, vec);
  stage_rows<R, kVdTW, G::LR, G::LW>(sk, K, i0 - G::V, j0 - 1, nx, ny, vec);
  __syncthreads();
  const int i = i0 + (int)threadIdx.x;
  if (i >= nx) return;
  const int cx = G::V + (int)threadIdx.x;
  // A 3 x 3 window of x and K slides down the thread's column: each row
  // enters once (three LDS reads of each array) and serves three outputs.
  // Window rows 0, 1, 2 are grid rows j-1, j, j+1; columns i-1, i, i+1. The
  // neighbours are visited in the forward's order (kNbrDx, kNbrDy).
  R xw[3][3], kw[3][3];
  auto enter = [&](int slot, int lr) {
#pragma unroll
    for (int c = 0; c < 3; ++c) {
      xw[slot][c] = sx[lr * G::LW + cx - 1 + c];
      kw[slot][c] = sk[lr * G::LW + cx - 1 + c];
    }
  };
  enter(0, 0);
  enter(1, 1);
  // tiles whose points all have eight in-grid neighbours skip the bounds
  // tests (a workgroup-uniform branch)
  const bool all_in = i0 >= 1 && i0 + kVdTW <= nx - 1 && j0 >= 1 && j0 + kVdTR <= ny - 1;
  auto rows = [&](auto all_in_t) {
    constexpr bool ALL_IN = decltype(all_in_t)::value;
    const bool xin = i > 0 && i < nx - 1;
#pragma unroll
    for (int r = 0; r < kVdTR; ++r) {
      const int j = j0 + r;
      if (!ALL_IN && j >= ny) break;
      enter(2, r + 2);
      const R xc = xw[1][1], Kc = kw[1][1];
      R acc = R(0);
      const bool inner = ALL_IN || (xin && j > 0 && j < ny - 1);
#pragma unroll
      for (int n = 0; n < 8; ++n) {
        if (!ALL_IN && !inner) {
          const int a = i + kNbrDx[n], bb = j + kNbrDy[n];
          if (a < 0 || a >= nx || bb < 0 || bb >= ny) continue;
        }
        const int wr = 1 + kNbrDy[n], wc = 1 + kNbrDx[n];
        acc += ((n < 4 ? ca : cd) * (Kc + kw[wr][wc])) * (xw[wr][wc] - xc);
      }
      const R v = xc + dt * acc;
      put<NT>(&y[j * nx + i], LIM ? limited(v, lim) : v);
#pragma unroll
      for (int c = 0; c < 3; ++c) {
        xw[0][c] = xw[1][c];
        kw[0][c] = kw[1][c];
        xw[1][c] = xw[2][c];
        kw[1][c] = kw[2][c];
      }
    }
  };
  if (all_in)
    rows(std::true_type{});
  else
    rows(std::false_type{});
}

// Two forward steps in one launch. A workgroup owns kX2TW = 252 output
// columns and TR rows; x and K are staged with a two-cell halo, the first
// step is evaluated on the tile plus a one-cell ring (254 columns, one per
// thread, TR + 2 rows) and written back over the staged x, the second on
// the tile. Both slide the 3 x 3 windows of the single step down a column
// and evaluate its expression in its order, so the result is bit-identical
// to two single steps. Values of the first step outside the grid are never
// read: the second step drops out-of-grid neighbours as the single step
// does.
constexpr int kVdX2TR = 8;
// ST: the first step's state is stored too, into mid, on the tile's cells.
template <class R, int TR, bool NT, bool ST>
__global__ __launch_bounds__(kX2Threads) void fwd_vardiff2d9_x2(const R* __restrict__ x,
                                                                const R* __restrict__ K,
                                                                R* __restrict__ y,
                                                                R* __restrict__ mid, int nx,
                                                                int ny, int tiles_x, int ntiles,
                                                                int vec, R dt, R ca, R cd) {
  using G = Tile2x2<R, TR>;
  __shared__ R sx[G::LR * G::LW];
  __shared__ R sk[G::LR * G::LW];
  const int b = xcd_tile(ntiles);
  if (b >= ntiles) return;
  const int i0 = (b % tiles_x) * kX2TW, j0 = (b / tiles_x) * TR;
  // LDS row r is grid row j0 - 2 + r, LDS column c grid column i0 - PADL + c
  stage_rows<R, kX2Threads, G::LR, G::LW>(sx, x, i0 - G::PADL, j0 - 2, nx, ny, vec);
  stage_rows<R, kX2Threads, G::LR, G::LW>(sk, K, i0 - G::PADL, j0 - 2, nx, ny, vec);
  __syncthreads();
  const int t = threadIdx.x;
  R xw[3][3], kw[3][3];
  // one step on LDS rows r_first .. r_first + n - 1 at LDS column c (grid
  // column i), from the windows of sx and sk; out[k] = value at row r_first + k
  auto column = [&](auto all_in_t, int c, int i, int r_first, int n, R* out) {
    constexpr bool ALL_IN = decltype(all_in_t)::value;
    auto enter = [&](int slot, int lr) {
#pragma unroll
      for (int e = 0; e < 3; ++e) {
        xw[slot][e] = sx[lr * G::LW + c - 1 + e];
        kw[slot][e] = sk[lr * G::LW + c - 1 + e];
      }
    };
    enter(0, r_first - 1);
    enter(1, r_first);
    const bool xin = i > 0 && i < nx - 1;
#pragma unroll
    for (int k = 0; k < TR + 2; ++k) {
      if (k >= n) break;
      const int j = j0 - 2 + r_first + k;
      enter(2, r_first + k + 1);
      const R xc = xw[1][1], Kc = kw[1][1];
      R acc = R(0);
      const bool inner = ALL_IN || (xin && j > 0 && j < ny - 1);
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        if (!ALL_IN && !inner) {
          const int a = i + kNbrDx[q], bb = j + kNbrDy[q];
          if (a < 0 || a >= nx || bb < 0 || bb >= ny) continue;
        }
        const int wr = 1 + kNbrDy[q], wc = 1 + kNbrDx[q];
        acc += ((q < 4 ? ca : cd) * (Kc + kw[wr][wc])) * (xw[wr][wc] - xc);
      }
      out[k] = xc + dt * acc;
#pragma unroll
      for (int e = 0; e < 3; ++e) {
        xw[0][e] = xw[1][e];
        kw[0][e] = kw[1][e];
        xw[1][e] = xw[2][e];
        kw[1][e] = kw[2][e];
      }
    }
  };
  // every cell of the first step's region has eight in-grid neighbours
  // (workgroup-uniform)
  const bool all_in = i0 - 1 >= 1 && i0 + kX2TW <= nx - 2 && j0 - 1 >= 1 && j0 + TR <= ny - 2;
  // first step: LDS rows 1 .. TR + 2, LDS column PADL - 1 + t
  R v[TR + 2];
  const int c1 = G::PADL - 1 + t, i1 = i0 - 1 + t;
  const bool act = t < kX2TW + 2;
  if (act) {
    if (all_in)
      column(std::true_type{}, c1, i1, 1, TR + 2, v);
    else
      column(std::false_type{}, c1, i1, 1, TR + 2, v);
    if constexpr (ST) {  // v[r] is grid row j0 - 1 + r; the tile's rows are r = 1 .. TR
      if (t >= 1 && t <= kX2TW && i1 < nx) {
#pragma unroll
        for (int r = 1; r <= TR; ++r)
          if (j0 - 1 + r < ny) put<NT>(&mid[(j0 - 1 + r) * nx + i1], v[r]);
      }
    }
  }
  __syncthreads();
  if (act) {
#pragma unroll
    for (int r = 0; r < TR + 2; ++r) sx[(r + 1) * G::LW + c1] = v[r];
  }
  __syncthreads();
  // second step on the tile: LDS rows 2 .. TR + 1, LDS column PADL + t
  const int i = i0 + t;
  if (t >= kX2TW || i >= nx) return;
  const int rows = min(TR, ny - j0);
  if (all_in)
    column(std::true_type{}, G::PADL + t, i, 2, TR, v);
  else
    column(std::false_type{}, G::PADL + t, i, 2, rows, v);
#pragma unroll
  for (int r = 0; r < TR; ++r)
    if (r < rows) put<NT>(&y[(j0 + r) * nx + i], v[r]);
}

// Adjoint (the operator is symmetric in x):
//   g'[m] = g[m] + dt * sum_n (c_n*(K[m]+K[n]))*(g[n]-g[m])
//   dK[m] += dt * sum_n (c_n*(x[n]-x[m]))*(g[m]-g[n])      (x = x_{t-1})
// the second line being the coefficient-field gradient of step t, fused;
// DP adds this step's share of dL/ddt (see DpOut), sum_m g[m] * acc[m] with
// the forward's acc. Threads past the grid's last column take part in the
// block sum.
template <class R, bool WANT_DK, int TR, bool DP, bool NT>
__global__ __launch_bounds__(kVdTW) void adj_vardiff2d9(const R* __restrict__ x,
                                                        const R* __restrict__ K,
                                                        const R* __restrict__ g,
                                                        R* __restrict__ gp, R* __restrict__ dK,
                                                        int dk_first, int nx, int ny,
                                                        int tiles_x, int ntiles, int vec, R dt,
                                                        R ca, R cd, DpOut dp) {
  constexpr bool XS = WANT_DK || DP;  // x_{t-1} staged
  using G = Tile2<R, kVdTW, TR>;
  constexpr int LW = G::LW;
  __shared__ R sg[G::LR * LW];
  __shared__ R sk[G::LR * LW];
  __shared__ R sx[XS ? G::LR * LW : 1];
  const int b = xcd_tile(ntiles);
  if (b >= ntiles) return;  // the whole block
  const int i0 = (b % tiles_x) * kVdTW, j0 = (b / tiles_x) * TR;
  stage_rows<R, kVdTW, G::LR, LW>(sg, g, i0 - G::V, j0 - 1, nx, ny, vec);
  stage_rows<R, kVdTW, G::LR, LW>(sk, K, i0 - G::V, j0 - 1, nx, ny, vec);
  if (XS) stage_rows<R, kVdTW, G::LR, LW>(sx, x, i0 - G::V, j0 - 1, nx, ny, vec);
  const int i = i0 + (int)threadIdx.x;
  // the accumulated dK of the thread's cells, requested with the staged
  // rows (where the row loop is unrolled, so the registers stay static)
  constexpr bool PRE = WANT_DK && !DP;
  R dk0[PRE ? TR : 1];
  if (PRE) {
#pragma unroll
    for (int r = 0; r < TR; ++r) {
      const int j = j0 + r;
      dk0[PRE ? r : 0] = (!dk_first && i < nx && j < ny) ? dK[j * nx + i] : R(0);
    }
  }
  __syncthreads();
  const int cx = G::V + (int)threadIdx.x;
  const bool xin = i > 0 && i < nx - 1;
  double a0 = 0.0;
  if (i < nx) {
    // 3 x 3 windows of g, K (and x) slide down the thread's column, as in
    // the forward: rows j-1, j, j+1, columns i-1, i, i+1.
    R gw[3][3], kw[3][3], xw[XS ? 3 : 1][3];
    auto enter = [&](int slot, int lr) {
#pragma unroll
      for (int c = 0; c < 3; ++c) {
        gw[slot][c] = sg[lr * LW + cx - 1 + c];
        kw[slot][c] = sk[lr * LW + cx - 1 + c];
        if (XS) xw[XS ? slot : 0][c] = sx[lr * LW + cx - 1 + c];
      }
    };
    enter(0, 0);
    enter(1, 1);
    const bool all_in = i0 >= 1 && i0 + kVdTW <= nx - 1 && j0 >= 1 && j0 + TR <= ny - 1;
    auto rows = [&](auto all_in_t) {
    constexpr bool ALL_IN = decltype(all_in_t)::value;
    // rolled with both dK and the constants' sums, to keep four waves per SIMD
    constexpr int kRowUnroll = (WANT_DK && DP) ? 1 : TR;
#pragma unroll kRowUnroll
    for (int r = 0; r < TR; ++r) {
      const int j = j0 + r;
      if (!ALL_IN && j >= ny) break;
      enter(2, r + 2);
      const R gc = gw[1][1], Kc = kw[1][1];
      const R xc = XS ? xw[XS ? 1 : 0][1] : R(0);
      R ag = R(0), ak = R(0), acc = R(0);
      const bool inner = ALL_IN || (xin && j > 0 && j < ny - 1);
#pragma unroll
      for (int n = 0; n < 8; ++n) {
        if (!ALL_IN && !inner) {
          const int a = i + kNbrDx[n], bb = j + kNbrDy[n];
          if (a < 0 || a >= nx || bb < 0 || bb >= ny) continue;
        }
        const int wr = 1 + kNbrDy[n], wc = 1 + kNbrDx[n];
        const R cn = n < 4 ? ca : cd;
        const R gn = gw[wr][wc];
        ag += (cn * (Kc + kw[wr][wc])) * (gn - gc);
        if (WANT_DK) ak += (cn * (xw[XS ? wr : 0][wc] - xc)) * (gc - gn);
        if (DP) acc += (cn * (Kc + kw[wr][wc])) * (xw[XS ? wr : 0][wc] - xc);
      }
      const int o = j * nx + i;
      put<NT>(&gp[o], gc + dt * ag);
      if (WANT_DK)
        put<NT>(&dK[o], (PRE ? dk0[PRE ? r : 0] : (dk_first ? R(0) : dK[o])) + dt * ak);
      if (DP) a0 += (double)gc * (double)acc;
#pragma unroll
      for (int c = 0; c < 3; ++c) {
        gw[0][c] = gw[1][c];
        kw[0][c] = kw[1][c];
        gw[1][c] = gw[2][c];
        kw[1][c] = kw[2][c];
        if (XS) {
          xw[0][c] = xw[XS ? 1 : 0][c];
          xw[XS ? 1 : 0][c] = xw[XS ? 2 : 0][c];
        }
      }
    }
    };
    if (all_in)
      rows(std::true_type{});
    else
      rows(std::false_type{});
  }
  if (DP) dp_commit(dp, b, a0, 0.0);
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
    if (g) g[i] = gv;
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

// ------------------------------------------------------- limiter branches
// The limiter's derivative is that of the branch taken: a clamped value
// depends on nothing, so g_t is zeroed where the step's unlimited value y
// left [lo, hi]. y is re-evaluated from x_{t-1} (Sec. III-B: branch outcomes
// recomputed rather than stored) through the same per-point functions the
// forward kernels use, fed from a small local neighbourhood, so every
// branch is decided on the bits the forward step produced.
template <class R, int KIND>
__global__ __launch_bounds__(kThreads) void limit_mask(const R* __restrict__ x,
                                                       const R* __restrict__ K,
                                                       R* __restrict__ g, int nx, int ny, int nz,
                                                       R p0, R p1, R ca, R cd, Limit<R> lim) {
  const int tid = threadIdx.y * kBX + threadIdx.x;
  const int64_t plane = (int64_t)nx * ny, n = plane * nz;
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t q = (int64_t)blockIdx.x * kThreads + tid; q < n; q += stride) {
    const int i = (int)(q % nx);
    const int64_t r = q / nx;
    const int j = (int)(r % ny), k = (int)(r / ny);
    R y;
    if (KIND == ADST_ALLENCAHN3D7) {
      y = allencahn_point(x[q], i > 0 ? x[q - 1] : R(0), i < nx - 1 ? x[q + 1] : R(0),
                          j > 0 ? x[q - nx] : R(0), j < ny - 1 ? x[q + nx] : R(0),
                          k > 0 ? x[q - plane] : R(0), k < nz - 1 ? x[q + plane] : R(0), p0, p1);
    } else {
      // 3 x 3 neighbourhood, row stride 3, centre at 4; 0 outside the grid
      R sx[9], sk[9];
#pragma unroll
      for (int dy = -1; dy <= 1; ++dy)
#pragma unroll
        for (int dx = -1; dx <= 1; ++dx) {
          const bool in = i + dx >= 0 && i + dx < nx && j + dy >= 0 && j + dy < ny;
          const int64_t m = q + (int64_t)dy * nx + dx;
          sx[(dy + 1) * 3 + dx + 1] = in ? x[m] : R(0);
          if (KIND == ADST_VARDIFF2D9) sk[(dy + 1) * 3 + dx + 1] = in ? K[m] : R(0);
        }
      if (KIND == ADST_JACOBI2D5)
        y = jacobi_fwd_at<R, 3>(sx, 4, i, j, nx, ny, p0);
      else
        y = vardiff_fwd_at<R, 3>(sx, sk, 4, i, j, nx, ny, p0, ca, cd);
    }
    if (y < lim.lo || y > lim.hi) g[q] = R(0);
  }
}

// ------------------------------------------- gradients of the step constants
// dparams[k] = the sum of the nslots slots of constant k, in a fixed order.
__global__ __launch_bounds__(kThreads) void dparam_finalize(const double* __restrict__ part,
                                                            int nslots,
                                                            double* __restrict__ out) {
  const int tid = threadIdx.y * kBX + threadIdx.x;
  double a0 = 0.0, a1 = 0.0;
  for (int i = tid; i < nslots; i += kThreads) {
    a0 += part[i];
    a1 += part[nslots + i];
  }
  block_sum2(a0, a1);
  if (tid == 0) {
    out[0] = a0;
    out[1] = a1;
  }
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

// One-shot copy: every work-item moves one 16-byte vector and exits. With
// one-wave workgroups this is the fastest plain copy measured on the chip
// (6.1-6.4 TB/s read + write at 2 GiB), the ceiling stencil kernels are
// compared with.
constexpr int kCopyLanes = 64;
__global__ __launch_bounds__(kCopyLanes) void copy_once(uint4* __restrict__ d,
                                                        const uint4* __restrict__ s, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * kCopyLanes + threadIdx.x;
  if (i < n) d[i] = s[i];
}

int grid_for(int64_t n, int64_t per_block, int64_t cap) {
  int64_t b = (n + per_block - 1) / per_block;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return (int)b;
}

// 16-byte vector loads need every staged array 16-byte aligned and rows whose
// starts stay aligned (nx a multiple of the vector width).
template <class R>
int vec_ok(int nx, const void* a, const void* b = nullptr, const void* c = nullptr) {
  if (nx % (16 / (int)sizeof(R))) return 0;
  for (const void* p : {a, b, c})
    if (p && (reinterpret_cast<uintptr_t>(p) & 15u)) return 0;
  return 1;
}

inline int cdiv(int a, int b) { return (a + b - 1) / b; }

// 1 when the kernels of this shape stream their stores (see kStreamBytes)
inline int streams(const StepShape& s) {
  const int64_t bytes = int64_t(s.nx) * s.ny * s.nz * (s.dtype == ADST_F64 ? 8 : 4);
  return bytes >= kStreamBytes ? 1 : 0;
}

// mids (nullable): the intermediate states' buffers, step l's at mids[l-1].
template <class R, int K, int RPT, int NZ>
hipError_t ac_forward_n(const StepShape& s, const R* x, R* y, R* const* mids, hipStream_t st) {
  using A = AcN<K, RPT, NZ>;
  const int tx = cdiv(s.nx, A::OX), ty = cdiv(s.ny, A::OY);
  const int nt = tx * ty * cdiv(s.nz, A::ZC);
  const dim3 grid(xcd_grid(nt)), block(kBX, kBY);
  R* m0 = mids ? mids[0] : nullptr;
  R* m1 = (mids && K >= 3) ? mids[1] : nullptr;
  const bool str = streams(s) != 0;
  if (mids && str)
    fwd_allencahn3d7_n<R, K, RPT, NZ, true, true><<<grid, block, 0, st>>>(
        x, y, m0, m1, s.nx, s.ny, s.nz, tx, ty, nt, R(s.p0), R(s.p1));
  else if (mids)
    fwd_allencahn3d7_n<R, K, RPT, NZ, false, true><<<grid, block, 0, st>>>(
        x, y, m0, m1, s.nx, s.ny, s.nz, tx, ty, nt, R(s.p0), R(s.p1));
  else if (str)
    fwd_allencahn3d7_n<R, K, RPT, NZ, true, false><<<grid, block, 0, st>>>(
        x, y, m0, m1, s.nx, s.ny, s.nz, tx, ty, nt, R(s.p0), R(s.p1));
  else
    fwd_allencahn3d7_n<R, K, RPT, NZ, false, false><<<grid, block, 0, st>>>(
        x, y, m0, m1, s.nx, s.ny, s.nz, tx, ty, nt, R(s.p0), R(s.p1));
  return hipGetLastError();
}

// Allen-Cahn, n fused forward steps (2 <= n <= kAcMaxFuse); mids as above.
template <class R>
hipError_t ac_forward_steps(const StepShape& s, const void* xv, void* yv, void* const* mids,
                            int32_t n, hipStream_t st) {
  const R* x = static_cast<const R*>(xv);
  R* y = static_cast<R*>(yv);
  R* const* m = reinterpret_cast<R* const*>(mids);
  switch (n) {
    case 2:
      return ac_forward_n<R, 2, 4, 32>(s, x, y, m, st);
    case 3:
      return ac_forward_n<R, 3, 4, 64>(s, x, y, m, st);
  }
  return hipErrorInvalidValue;
}

template <class R>
hipError_t forward_t(const StepShape& s, const void* xv, const void* Kv, void* yv, bool two,
                     hipStream_t st, void* midv = nullptr) {
  R* mid = static_cast<R*>(midv);
  const R* x = static_cast<const R*>(xv);
  const R* K = static_cast<const R*>(Kv);
  R* y = static_cast<R*>(yv);
  const Limit<R> lim{R(s.lo), R(s.hi)};
  if (two && s.limit) return hipErrorInvalidValue;  // fused steps have no limiter
  switch (s.kind) {
    case ADST_JACOBI2D5: {
      if (two) {
        const int tx = cdiv(s.nx, kX2TW), nt = tx * cdiv(s.ny, kX2TR);
        fwd_jacobi2d5_x2<R><<<dim3(xcd_grid(nt)), dim3(kX2Threads), 0, st>>>(
            x, y, s.nx, s.ny, tx, nt, vec_ok<R>(s.nx, x), R(s.p0));
      } else {
        const int tx = cdiv(s.nx, kJacTW), nt = tx * cdiv(s.ny, kJacTR);
        if (s.limit)
          fwd_jacobi2d5<R, true><<<dim3(xcd_grid(nt)), dim3(kJacTW), 0, st>>>(
              x, y, s.nx, s.ny, tx, nt, vec_ok<R>(s.nx, x), R(s.p0), lim);
        else
          fwd_jacobi2d5<R, false><<<dim3(xcd_grid(nt)), dim3(kJacTW), 0, st>>>(
              x, y, s.nx, s.ny, tx, nt, vec_ok<R>(s.nx, x), R(s.p0), lim);
      }
      break;
    }
    case ADST_ALLENCAHN3D7: {
      if (two) {
        return ac_forward_n<R, 2, 4, 32>(s, x, y, nullptr, st);
      } else {
        const int tx = cdiv(s.nx, kAcTX), ty = cdiv(s.ny, kAcTY);
        const int nt = tx * ty * cdiv(s.nz, kAcZC);
        const dim3 grid(xcd_grid(nt)), block(kBX, kBY);
        const bool str = streams(s) != 0;
        if (s.limit && str)
          fwd_allencahn3d7<R, true, true><<<grid, block, 0, st>>>(
              x, y, s.nx, s.ny, s.nz, tx, ty, nt, R(s.p0), R(s.p1), lim);
        else if (s.limit)
          fwd_allencahn3d7<R, true, false><<<grid, block, 0, st>>>(
              x, y, s.nx, s.ny, s.nz, tx, ty, nt, R(s.p0), R(s.p1), lim);
        else if (str)
          fwd_allencahn3d7<R, false, true><<<grid, block, 0, st>>>(
              x, y, s.nx, s.ny, s.nz, tx, ty, nt, R(s.p0), R(s.p1), lim);
        else
          fwd_allencahn3d7<R, false, false><<<grid, block, 0, st>>>(
              x, y, s.nx, s.ny, s.nz, tx, ty, nt, R(s.p0), R(s.p1), lim);
      }
      break;
    }
    case ADST_VARDIFF2D9: {
      const bool str = streams(s) != 0;
      const int vec = vec_ok<R>(s.nx, x, K);
      const R dt = R(s.p0), ca = R(1) / R(3), cd = R(1) / R(12);
      if (two) {
        const int tx = cdiv(s.nx, kX2TW), nt = tx * cdiv(s.ny, kVdX2TR);
        const dim3 grid(xcd_grid(nt)), block(kX2Threads);
        if (mid && str)
          fwd_vardiff2d9_x2<R, kVdX2TR, true, true><<<grid, block, 0, st>>>(
              x, K, y, mid, s.nx, s.ny, tx, nt, vec, dt, ca, cd);
        else if (mid)
          fwd_vardiff2d9_x2<R, kVdX2TR, false, true><<<grid, block, 0, st>>>(
              x, K, y, mid, s.nx, s.ny, tx, nt, vec, dt, ca, cd);
        else if (str)
          fwd_vardiff2d9_x2<R, kVdX2TR, true, false><<<grid, block, 0, st>>>(
              x, K, y, mid, s.nx, s.ny, tx, nt, vec, dt, ca, cd);
        else
          fwd_vardiff2d9_x2<R, kVdX2TR, false, false><<<grid, block, 0, st>>>(
              x, K, y, mid, s.nx, s.ny, tx, nt, vec, dt, ca, cd);
        break;
      }
      const int tx = cdiv(s.nx, kVdTW), nt = tx * cdiv(s.ny, kVdTR);
      const dim3 grid(xcd_grid(nt)), block(kVdTW);
      if (s.limit && str)
        fwd_vardiff2d9<R, true, true><<<grid, block, 0, st>>>(x, K, y, s.nx, s.ny, tx, nt, vec,
                                                              dt, ca, cd, lim);
      else if (s.limit)
        fwd_vardiff2d9<R, true, false><<<grid, block, 0, st>>>(x, K, y, s.nx, s.ny, tx, nt, vec,
                                                               dt, ca, cd, lim);
      else if (str)
        fwd_vardiff2d9<R, false, true><<<grid, block, 0, st>>>(x, K, y, s.nx, s.ny, tx, nt, vec,
                                                               dt, ca, cd, lim);
      else
        fwd_vardiff2d9<R, false, false><<<grid, block, 0, st>>>(x, K, y, s.nx, s.ny, tx, nt, vec,
                                                                dt, ca, cd, lim);
      break;
    }
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// One variable-coefficient adjoint launch over ntiles tiles, streaming or not.
template <class R, bool WANT_DK, int TR, bool DP>
void vd_adjoint(bool str, int ntiles, hipStream_t st, const R* x, const R* K, const R* g, R* gp,
                R* dK, int dk_first, int nx, int ny, int tiles_x, int vec, R dt, R ca, R cd,
                DpOut dp) {
  const dim3 grid(xcd_grid(ntiles)), block(kVdTW);
  if (str)
    adj_vardiff2d9<R, WANT_DK, TR, DP, true><<<grid, block, 0, st>>>(
        x, K, g, gp, dK, dk_first, nx, ny, tiles_x, ntiles, vec, dt, ca, cd, dp);
  else
    adj_vardiff2d9<R, WANT_DK, TR, DP, false><<<grid, block, 0, st>>>(
        x, K, g, gp, dK, dk_first, nx, ny, tiles_x, ntiles, vec, dt, ca, cd, dp);
}

template <class R>
hipError_t adjoint_t(const StepShape& s, const void* xv, const void* Kv, const void* gv,
                     void* gpv, void* dKv, bool dk_first, double* dp_part, bool dp_first,
                     hipStream_t st) {
  const R* x = static_cast<const R*>(xv);
  const R* K = static_cast<const R*>(Kv);
  const R* g = static_cast<const R*>(gv);
  R* gp = static_cast<R*>(gpv);
  R* dK = static_cast<R*>(dKv);
  const DpOut dp{dp_part, (int)dparam_slots(s), dp_first ? 1 : 0};
  switch (s.kind) {
    case ADST_JACOBI2D5: {
      const int tx = cdiv(s.nx, kJacTW), nt = tx * cdiv(s.ny, kJacTR);
      if (dp_part) {
        // slot layout: nslots for w, then nslots for the unused second constant
        const int64_t n = dparam_slots(s);
        if (dp_first) {
          const hipError_t e = launch_fill_zero(dp_part + n, n * (int64_t)sizeof(double), st);
          if (e != hipSuccess) return e;
        }
        return launch_jacobi_dp_adjoint(s, xv, gv, gpv, dp_part, dp_first, st);
      }
      adj_jacobi2d5<R><<<dim3(xcd_grid(nt)), dim3(kJacTW), 0, st>>>(
          g, gp, s.nx, s.ny, tx, nt, vec_ok<R>(s.nx, g), R(s.p0));
      break;
    }
    case ADST_ALLENCAHN3D7: {
      const R D = R(s.p0), C = R(s.p1);
      const R k0 = R(1) + D * R(-6), k1 = R(3) * C;
      const int tx = cdiv(s.nx, kAcTX), ty = cdiv(s.ny, kAcTY);
      const int nt = tx * ty * cdiv(s.nz, kAcZC);
      const dim3 grid(xcd_grid(nt)), block(kBX, kBY);
      const bool str = streams(s) != 0, lm = adjoint_applies_limit(s, dp_part != nullptr);
      const Limit<R> lim{R(s.lo), R(s.hi)};
#define ADST_AC_ADJ(DPV, NTV)                                                        \
  adj_allencahn3d7<R, DPV, NTV><<<grid, block, 0, st>>>(x, g, gp, s.nx, s.ny, s.nz, tx, ty, nt, \
                                                         D, k0, k1, dp)
#define ADST_AC_LIM(NTV)                                                             \
  adj_allencahn3d7_lim<R, NTV><<<grid, block, 0, st>>>(x, g, gp, s.nx, s.ny, s.nz, tx, ty, nt, \
                                                        D, k0, k1, C, lim)
      if (dp_part && str)
        ADST_AC_ADJ(true, true);
      else if (dp_part)
        ADST_AC_ADJ(true, false);
      else if (lm && str)
        ADST_AC_LIM(true);
      else if (lm)
        ADST_AC_LIM(false);
      else if (str)
        ADST_AC_ADJ(false, true);
      else
        ADST_AC_ADJ(false, false);
#undef ADST_AC_ADJ
#undef ADST_AC_LIM
      break;
    }
    case ADST_VARDIFF2D9: {
      const int tx = cdiv(s.nx, kVdTW);
      const R dt = R(s.p0), ca = R(1) / R(3), cd = R(1) / R(12);
      const int nt4 = tx * cdiv(s.ny, kVdAdjTR);
      const bool str = streams(s) != 0;
      const int dkf = dk_first ? 1 : 0, vx = vec_ok<R>(s.nx, g, K, x);
      if (dK && dp_part)
        vd_adjoint<R, true, kVdAdjTR, true>(str, nt4, st, x, K, g, gp, dK, dkf, s.nx, s.ny, tx,
                                            vx, dt, ca, cd, dp);
      else if (dK)
        vd_adjoint<R, true, kVdAdjTR, false>(str, nt4, st, x, K, g, gp, dK, dkf, s.nx, s.ny, tx,
                                             vx, dt, ca, cd, dp);
      else if (dp_part)
        vd_adjoint<R, false, kVdAdjTR, true>(str, nt4, st, x, K, g, gp, nullptr, 0, s.nx, s.ny,
                                             tx, vx, dt, ca, cd, dp);
      else
        vd_adjoint<R, false, kVdTR, false>(str, tx * cdiv(s.ny, kVdTR), st, nullptr, K, g, gp,
                                           nullptr, 0, s.nx, s.ny, tx, vec_ok<R>(s.nx, g, K), dt,
                                           ca, cd, dp);
      break;
    }
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <class R>
hipError_t adjoint2_t(const StepShape& s, const void* gv, void* gpv, hipStream_t st) {
  const R* g = static_cast<const R*>(gv);
  R* gp = static_cast<R*>(gpv);
  if (s.kind != ADST_JACOBI2D5) return hipErrorInvalidValue;
  const int tx = cdiv(s.nx, kX2TW), nt = tx * cdiv(s.ny, kX2TR);
  adj_jacobi2d5_x2<R><<<dim3(xcd_grid(nt)), dim3(kX2Threads), 0, st>>>(
      g, gp, s.nx, s.ny, tx, nt, vec_ok<R>(s.nx, g), R(s.p0));
  return hipGetLastError();
}

template <class R>
hipError_t seed_t(int32_t loss, int64_t n, const void* xv, const void* auxv, void* gv,
                  void* xcopyv, double* partials, hipStream_t st) {
  const R* x = static_cast<const R*>(xv);
  const R* aux = static_cast<const R*>(auxv);
  // g_T = x_T for the half square: when x_T already sits in g_T's buffer,
  // only the loss is computed
  R* g = (loss == ADST_LOSS_HALF_SQ && gv == xv) ? nullptr : static_cast<R*>(gv);
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
  return s.dtype == ADST_F64 ? forward_t<double>(s, x, K, y, false, stream)
                             : forward_t<float>(s, x, K, y, false, stream);
}

int32_t max_stored_forward(int32_t kind) {
  switch (kind) {
    case ADST_ALLENCAHN3D7:
      return kAcMaxFuse;
    case ADST_VARDIFF2D9:
      return 2;
  }
  return 1;
}

hipError_t launch_forward_store(const StepShape& s, const void* x, const void* K, void* const* ys,
                                int32_t n, hipStream_t stream) {
  if (n < 2 || n > max_stored_forward(s.kind) || s.limit) return hipErrorInvalidValue;
  if (s.kind == ADST_ALLENCAHN3D7)
    return s.dtype == ADST_F64 ? ac_forward_steps<double>(s, x, ys[n - 1], ys, n, stream)
                               : ac_forward_steps<float>(s, x, ys[n - 1], ys, n, stream);
  return s.dtype == ADST_F64 ? forward_t<double>(s, x, K, ys[1], true, stream, ys[0])
                             : forward_t<float>(s, x, K, ys[1], true, stream, ys[0]);
}

int32_t max_fused_forward(int32_t kind) {
  switch (kind) {
    case ADST_JACOBI2D5:
      return kJacMaxFuse;
    case ADST_ALLENCAHN3D7:
      return kAcMaxFuse;
    case ADST_VARDIFF2D9:
      return 2;
  }
  return 1;
}
// The marching adjoint needs rows wider than one lane's 16 bytes; narrower
// grids take the fused pair.
int32_t max_fused_adjoint(int32_t kind, int64_t nx) {
  if (kind != ADST_JACOBI2D5) return 1;
  return nx > 4 ? kJacMaxFuse : 2;
}

hipError_t launch_forward_n(const StepShape& s, const void* x, const void* K, void* y, int32_t n,
                            hipStream_t stream) {
  if (n < 2 || n > max_fused_forward(s.kind)) return hipErrorInvalidValue;
  if (s.kind == ADST_ALLENCAHN3D7)
    return s.dtype == ADST_F64 ? ac_forward_steps<double>(s, x, y, nullptr, n, stream)
                               : ac_forward_steps<float>(s, x, y, nullptr, n, stream);
  if (n == 2)
    return s.dtype == ADST_F64 ? forward_t<double>(s, x, K, y, true, stream)
                               : forward_t<float>(s, x, K, y, true, stream);
  return launch_jacobi_march(s, x, y, n, false, stream);
}

hipError_t launch_adjoint_n(const StepShape& s, const void* g_next, void* g_prev, int32_t n,
                            hipStream_t stream) {
  if (n < 2 || n > max_fused_adjoint(s.kind, s.nx)) return hipErrorInvalidValue;
  if (n == 2)
    return s.dtype == ADST_F64 ? adjoint2_t<double>(s, g_next, g_prev, stream)
                               : adjoint2_t<float>(s, g_next, g_prev, stream);
  return launch_jacobi_march(s, g_next, g_prev, n, true, stream);
}

bool adjoint_applies_limit(const StepShape& s, bool dparams) {
  return s.limit && !dparams && (s.kind == ADST_JACOBI2D5 || s.kind == ADST_ALLENCAHN3D7);
}

hipError_t launch_adjoint(const StepShape& s, const void* x, const void* K, const void* g_next,
                          void* g_prev, void* dK, bool dk_first, double* dp_part, bool dp_first,
                          hipStream_t stream) {
  if (dp_part && (s.kind < ADST_JACOBI2D5 || s.kind > ADST_VARDIFF2D9 || !x))
    return hipErrorInvalidValue;
  if (s.kind == ADST_JACOBI2D5 && adjoint_applies_limit(s, dp_part != nullptr))
    return launch_jacobi_lim_adjoint(s, x, g_next, g_prev, stream);
  return s.dtype == ADST_F64
             ? adjoint_t<double>(s, x, K, g_next, g_prev, dK, dk_first, dp_part, dp_first, stream)
             : adjoint_t<float>(s, x, K, g_next, g_prev, dK, dk_first, dp_part, dp_first, stream);
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

template <class R>
hipError_t limit_mask_t(const StepShape& s, const void* xv, const void* Kv, void* gv,
                        hipStream_t st) {
  const R* x = static_cast<const R*>(xv);
  const R* K = static_cast<const R*>(Kv);
  R* g = static_cast<R*>(gv);
  const int64_t n = (int64_t)s.nx * s.ny * s.nz;
  const dim3 grid(grid_for(n, 4 * kThreads, 65536)), block(kBX, kBY);
  const Limit<R> lim{R(s.lo), R(s.hi)};
  switch (s.kind) {
    case ADST_JACOBI2D5:
      limit_mask<R, ADST_JACOBI2D5><<<grid, block, 0, st>>>(x, K, g, s.nx, s.ny, s.nz, R(s.p0),
                                                            R(s.p1), R(0), R(0), lim);
      break;
    case ADST_ALLENCAHN3D7:
      limit_mask<R, ADST_ALLENCAHN3D7><<<grid, block, 0, st>>>(x, K, g, s.nx, s.ny, s.nz,
                                                               R(s.p0), R(s.p1), R(0), R(0), lim);
      break;
    case ADST_VARDIFF2D9:
      limit_mask<R, ADST_VARDIFF2D9><<<grid, block, 0, st>>>(
          x, K, g, s.nx, s.ny, s.nz, R(s.p0), R(s.p1), R(1) / R(3), R(1) / R(12), lim);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_limit_mask(const StepShape& s, const void* x, const void* K, void* g,
                             hipStream_t stream) {
  return s.dtype == ADST_F64 ? limit_mask_t<double>(s, x, K, g, stream)
                             : limit_mask_t<float>(s, x, K, g, stream);
}

int64_t dparam_slots(const StepShape& s) {
  switch (s.kind) {
    case ADST_JACOBI2D5: return jacobi_x_adjoint_slots(s);
    case ADST_ALLENCAHN3D7:
      return int64_t(cdiv(s.nx, kAcTX)) * cdiv(s.ny, kAcTY) * cdiv(s.nz, kAcZC);
    case ADST_VARDIFF2D9: return int64_t(cdiv(s.nx, kVdTW)) * cdiv(s.ny, kVdAdjTR);
    default: return 0;
  }
}

int64_t dparam_partial_bytes(const StepShape& s) { return 2 * dparam_slots(s) * int64_t(sizeof(double)); }

hipError_t launch_dparam_finalize(const StepShape& s, const double* partials, double* dparams,
                                  hipStream_t stream) {
  dparam_finalize<<<dim3(1), dim3(kBX, kBY), 0, stream>>>(partials, (int)dparam_slots(s), dparams);
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
  if (bytes <= 0) return hipSuccess;
  const uintptr_t d = reinterpret_cast<uintptr_t>(dst), s = reinterpret_cast<uintptr_t>(src);
  if ((d | s | uintptr_t(bytes)) & 3u) return hipErrorInvalidValue;
  int64_t done = 0;
  if (((d | s) & 15u) == 0) {
    // at most 2^30 vectors (16 GiB) per launch keeps the work-item count in 32 bits
    const int64_t nvec = bytes / 16;
    for (int64_t v0 = 0; v0 < nvec; v0 += int64_t(1) << 30) {
      const int64_t n = std::min<int64_t>(nvec - v0, int64_t(1) << 30);
      copy_once<<<dim3((unsigned)((n + kCopyLanes - 1) / kCopyLanes)), dim3(kCopyLanes), 0,
                  stream>>>(static_cast<uint4*>(dst) + v0, static_cast<const uint4*>(src) + v0,
                            n);
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
    done = nvec * 16;
  }
  const int64_t n = (bytes - done) / 4;
  if (n == 0) return hipSuccess;
  copy_u32<<<dim3(grid_for(n, kThreads * 4, 65536)), dim3(kBX, kBY), 0, stream>>>(
      reinterpret_cast<uint32_t*>(static_cast<char*>(dst) + done),
      reinterpret_cast<const uint32_t*>(static_cast<const char*>(src) + done), n);
  return hipGetLastError();
}

}  // namespace adst
