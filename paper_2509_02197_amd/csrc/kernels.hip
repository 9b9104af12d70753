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
#include "device_common.h"
#include "kernels.h"

namespace adst {
namespace {

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
  DpPrev prev;
  if (DP) prev = dp_prev<1>(dp, b);
  stage_rows<R, kVdTW, G::LR, LW>(sg, g, i0 - G::V, j0 - 1, nx, ny, vec);
  stage_rows<R, kVdTW, G::LR, LW>(sk, K, i0 - G::V, j0 - 1, nx, ny, vec);
  if (XS) stage_rows<R, kVdTW, G::LR, LW>(sx, x, i0 - G::V, j0 - 1, nx, ny, vec);
  const int i = i0 + (int)threadIdx.x;
  // the accumulated dK of the thread's cells, requested with the staged
  // rows (the row loop is unrolled, so the registers stay static)
  constexpr bool PRE = WANT_DK;
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
    // unrolled also with both dK and the constants' sums: with the dK
    // requests moved ahead of the loop, 389 -> 377 us per 8192^2 f32 step
    // (a rolled loop had kept four waves per SIMD; unrolled without the
    // early requests it took 508 us)
#pragma unroll
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
  if (DP) dp_commit<1>(dp, b, prev, a0, 0.0);
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
    case ADST_ALLENCAHN3D7:
      return two ? ac_launch_forward_steps(s, x, y, nullptr, 2, st)
                 : ac_launch_forward(s, x, y, st);
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
    case ADST_ALLENCAHN3D7:
      return ac_launch_adjoint(s, x, g, gp, dp_part, dp_first, st);
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
  if (s.kind == ADST_ALLENCAHN3D7) return ac_launch_forward_steps(s, x, ys[n - 1], ys, n, stream);
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
  if (s.kind == ADST_ALLENCAHN3D7) return ac_launch_forward_steps(s, x, y, nullptr, n, stream);
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
    case ADST_ALLENCAHN3D7: return ac_dparam_slots(s);
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
