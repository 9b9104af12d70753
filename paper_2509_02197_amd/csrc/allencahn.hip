// gfx950 kernels of the Allen-Cahn kind (adst.h, ADST_ALLENCAHN3D7): the
// single forward step, up to three fused forward steps (also writing every
// intermediate state for store-through runs), and the gather adjoint with the
// cubic term's adjoint fused, the constants' gradients and the limiter's
// branch mask. Built with -ffp-contract=off: every point evaluates
// allencahn_point in the documented order, so fused and single steps, sweep
// and recomputation give the same bits.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <type_traits>

#include "adst.h"
#include "device_common.h"
#include "kernels.h"

namespace adst {
namespace {

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
// A workgroup of 64 x BY threads owns a region of 64 columns x SY = BY * RPT
// rows of each plane (RPT rows per thread, BY apart) and marches in z. At
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
// Measured at 1024^3 f64, three steps per launch (64-plane chunks) beat two
// (the launches of a recomputation run drop by a third); four, with 24-row
// regions, needed 178 VGPRs and with 16-row regions evaluated 7 points per
// output point, and both were slower. Three steps run on 64 x 32 regions of
// sixteen waves of two rows (a region point per output point and step
// 1.42 -> 1.22; 1024^3 launch 4.84 -> 4.49 ms, in one process; four waves
// of four rows had been the shape before, eight waves of three or four
// rows and sixteen of three or four were slower), two steps on 64 x 16
// regions of four waves of four rows (no other shape was faster).
// Output tiles narrower than the region allows: non-temporal stores into a
// 64-byte segment that two workgroups share were measured to cost a third
// of a single step's time (3.26 -> 4.48 ms for a 1024^3 step whose tiles
// were shifted by one column), so a fused launch's tile is a whole number of
// 64-byte segments wide where that pays: two steps on 56-column tiles,
// 4.93 -> 3.79 ms at 1024^3. Three steps keep 60 columns (56: no faster,
// and more of the region evaluated for nothing).
template <int K>
constexpr int ac_out_width() { return K == 2 ? 56 : kBX - 2 * (K - 1); }
template <int K, int RPT, int NZ, int BY>
struct AcN {
  static constexpr int SX = kBX, SY = BY * RPT;
  static constexpr int OX = ac_out_width<K>(), OY = SY - 2 * (K - 1);  // output tile
  static constexpr int ZC = NZ;                               // output planes
  static_assert(OX + 2 * (K - 1) <= SX, "the output tile and its halo fit the region");
};

// ST: the intermediate states are stored too, step l's into mid[l-1], each
// point by the workgroup whose output tile holds it (a run of steps whose
// every state is kept moves 8 + 8n bytes per point for n steps instead of
// 16n). They take the non-temporal hint with the output where states are
// large (1024^3 call 1890 -> 1875 ms, in one process; 512^3 unchanged): the
// reverse sweep reads them back, but only after many other launches.
template <class R, int K, int RPT, int NZ, bool NT, bool ST, int BY>
__global__ __launch_bounds__(kBX * BY) void fwd_allencahn3d7_n(const R* __restrict__ x,
                                                               R* __restrict__ y,
                                                               R* __restrict__ mid0,
                                                               R* __restrict__ mid1, int nx,
                                                               int ny, int nz, int tiles_x,
                                                               int tiles_y, int ntiles, R D,
                                                               R C) {
  using A = AcN<K, RPT, NZ, BY>;
  constexpr int SX = A::SX, SY = A::SY, LX = SX + 2, LY = SY + 2, H = K - 1;
  static_assert(K >= 2 && 2 * LX + 2 * SY <= kBX * BY, "ring cells: one per thread");
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
  auto row = [&](int q) { return ty + BY * q; };  // region row of the thread's q-th cell
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
  const bool tile_col = tx >= H && tx < H + A::OX;
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
            put<NT>(&mid0[p * plane + (j0 - H + r) * nx + ic], sn[0][q]);
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
              put<NT>(&(l == 2 ? mid1 : mid0)[pl * plane + j * nx + ic], v);
          }
        } else if (ok && tile_col && pl >= z0 && pl < z1) {
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
  DpPrev prev;
  if (DP) prev = dp_prev<2>(dp, t.b);
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
    dp_commit<2>(dp, t.b, prev, a0, a1);
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
template <class R, bool NT, int TW, int ZC>
__global__ __launch_bounds__(kBX * TW) void adj_allencahn3d7_lim(const R* __restrict__ x,
                                                                 const R* __restrict__ g,
                                                                 R* __restrict__ gp, int nx,
                                                                 int ny, int nz, int tiles_x,
                                                                 int tiles_y, int ntiles, R D,
                                                                 R k0, R k1, R C, Limit<R> lim) {
  constexpr int TY = 2 * TW;                             // tile rows: two per thread
  constexpr int LY = TY + 2, LX = kAcTX + 2;             // g: one-cell ring
  constexpr int XY = TY + 4, XX = kAcTX + 4;             // x: two-cell ring
  static_assert(2 * XX + 2 * LY + 4 <= kBX * TW, "ring cells: one per thread");
  __shared__ R tile[LY][LX];
  __shared__ R xt[XY][XX];
  AcTile t;
  {
    int b = xcd_tile(ntiles);
    if (b >= ntiles) return;  // the whole block
    t.bx = b % tiles_x;
    b /= tiles_x;
    t.by = b % tiles_y;
    t.i = t.bx * kAcTX + (int)threadIdx.x;
    t.ja = t.by * TY + (int)threadIdx.y;
    t.jb = t.ja + TW;
    t.z0 = (b / tiles_y) * ZC;
    t.z1 = min(t.z0 + ZC, nz);
  }
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
  const int i0 = t.bx * kAcTX, j0 = t.by * TY;
  // this thread's cell of g's ring (tile coordinates hly-1, hlx-1), if any
  int hly = -1, hlx = 0;
  if (tid < kAcTX) {
    hly = 0;
    hlx = tid + 1;
  } else if (tid < 2 * kAcTX) {
    hly = LY - 1;
    hlx = tid - kAcTX + 1;
  } else if (tid < 2 * kAcTX + TY) {
    hly = tid - 2 * kAcTX + 1;
    hlx = 0;
  } else if (tid < 2 * kAcTX + 2 * TY) {
    hly = tid - 2 * kAcTX - TY + 1;
    hlx = LX - 1;
  }
  const bool hr = hly >= 0;
  const int hj = j0 + hly - 1, hi = i0 + hlx - 1;
  // this thread's cell of x's outer ring, or one of the four corners of
  // g's ring (which g's ring cells need as x neighbours), in x-tile
  // coordinates, if any: 2*68 + 2*(TY+2) + 4 cells
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
    tile[ty + 1 + TW][tx + 1] = curB;
    if (hr) tile[hly][hlx] = halo;
    xt[ty + 2][tx + 2] = xA1;
    xt[ty + 2 + TW][tx + 2] = xB1;
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
    const R aboveB = masked(ty + 2 + TW, tx + 2, xB0, xB2, gB);
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
      R s = tile[ty + 1 + TW][tx] + tile[ty + 1 + TW][tx + 2];
      s += tile[ty + TW][tx + 1];
      s += tile[ty + 2 + TW][tx + 1];
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

// ------------------------------------------------------------- z-march
// Register z-march: a workgroup of kMW waves owns a region of 64 columns
// (one per lane) by kMW * RR rows (RR consecutive rows per wave) of every
// plane and marches in z. Each value's x-neighbours come from the adjacent
// lanes by DPP whole-wave shifts, its y-neighbours from the same lane's
// registers (the rows of its wave) or, for a wave's first and last row,
// from the neighbouring wave's row published in LDS, its z-neighbours from
// the registers of the planes below and above. A launch evaluates NF >= 0
// forward steps (level l = step l, level 0 the input state) and, with ADJ,
// one adjoint step at the end: g'(m) from g's stencil and x_{t-1} at m, where
// x_{t-1} is the last forward level (or, with NF = 0, the input state read
// at m). The adjoint's only use of x_{t-1} is pointwise, so a recomputed
// x_{t-1} is used where it is formed and never stored.
//
// At iteration p, level 1 is evaluated at plane p and level l at plane
// p-l+1; the adjoint at the plane of level NF (p with NF = 0). Level l is
// valid on the region less l-1 cells per side (the input state and g are
// read with a one-cell ring: lanes 0 and 63 read the columns beyond the
// region, the first and last wave the rows beyond it), so the output tile
// is the region less NF-1 cells per side. Values outside the grid are 0,
// the ghost value the next level reads. Every point evaluates the single
// step's expressions, so any split of the steps into launches, and the
// fused adjoint, give the bits of one launch per step.
//
// Memory goes through buffer instructions with one descriptor per plane:
// every lane's offset within a plane is fixed for the whole launch (an
// offset beyond the descriptor's range for cells outside the grid, and a
// range of 0 for planes outside it, so those reads return 0 without a
// branch). Stores are issued only by the lanes whose cell lies in the
// output tile (exec-masked), never to an out-of-range offset. Planes are
// held in rings of 4 slots, plane q in slot (q - pfirst) mod 4, and the
// iteration body is unrolled 4 times so every slot index is a compile-time
// constant. The input planes are requested DA planes ahead of the plane
// being evaluated (the side columns two). One barrier per iteration: rows
// published at iteration p (into LDS half (p - pfirst + 1) mod 2) are read
// at iteration p + 1.
constexpr int kMW = 4;
constexpr uint32_t kOob = 0xFFFFFF00u;  // a buffer offset beyond any plane

template <int NF, int RR, int ZC, int MW = kMW>
struct AcMarch {
  static constexpr int SX = kBX, SY = MW * RR;
  static constexpr int H = NF > 1 ? NF - 1 : 0;  // cells per side the last level loses
  // output tile: 64 columns (aligned) for the plain adjoint; 56 (a whole
  // number of 64-byte segments) with two forward levels (6.92 -> 6.84 ms
  // at 1024^3); 60 with three (56 was slower: 8.09 -> 8.50 ms)
  static constexpr int OX = H == 1 ? 56 : SX - 2 * H, OY = SY - 2 * H;
  static_assert(OX + 2 * H <= SX, "the output tile and its halo fit the region");
};

template <class R>
struct AcMarchArgs {
  const R* x;  // the input state (level 0)
  const R* g;  // ADJ: g_t
  R* y;        // forward: level NF; ADJ: g_{t-1}
  R* mid0;     // ST: level 1
  R* mid1;     // ST: level 2
  int nx, ny, nz, tiles_x, tiles_y, ntiles;
  R D, C, k0, k1;
};

// The buffer descriptor of plane q of an array (range 0 outside the grid).
template <class R>
__device__ inline __amdgpu_buffer_rsrc_t plane_rsrc(const R* base, int q, int nz, int plane) {
  const bool in = q >= 0 && q < nz;
  const R* p = base + (int64_t)(in ? q : 0) * plane;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<R*>(p), (short)0,
                                           in ? plane * (int)sizeof(R) : 0, 0x00020000);
}
template <class R, int AUX>
__device__ inline R bload(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  if constexpr (sizeof(R) == 8) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, AUX);
    return __longlong_as_double((long long)(((uint64_t)v[1] << 32) | v[0]));
  } else {
    return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, AUX));
  }
}
template <class R, int AUX>
__device__ inline void bstore(__amdgpu_buffer_rsrc_t r, uint32_t off, R v) {
  if constexpr (sizeof(R) == 8) {
    const uint64_t u = (uint64_t)__double_as_longlong(v);
    typedef unsigned int u2 __attribute__((ext_vector_type(2)));
    u2 d;
    d[0] = (unsigned)u;
    d[1] = (unsigned)(u >> 32);
    __builtin_amdgcn_raw_buffer_store_b64(d, r, (int)off, 0, AUX);
  } else {
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, (int)off, 0, AUX);
  }
}
constexpr int kAuxNT = 2;  // cache policy bit: non-temporal

// Lane i receives lane i-1's value (lane 0: `edge`, or 0 without one) or
// lane i+1's (lane 63: `edge`, or 0).
__device__ inline uint32_t dpp_shr(uint32_t v, uint32_t edge) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)edge, (int)v, 0x138, 0xf, 0xf, false);
}
__device__ inline uint32_t dpp_shl(uint32_t v, uint32_t edge) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)edge, (int)v, 0x130, 0xf, 0xf, false);
}
__device__ inline double from_left(double v, double edge) {
  const uint64_t a = __double_as_longlong(v), e = __double_as_longlong(edge);
  const uint32_t lo = dpp_shr((uint32_t)a, (uint32_t)e);
  const uint32_t hi = dpp_shr((uint32_t)(a >> 32), (uint32_t)(e >> 32));
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}
__device__ inline double from_right(double v, double edge) {
  const uint64_t a = __double_as_longlong(v), e = __double_as_longlong(edge);
  const uint32_t lo = dpp_shl((uint32_t)a, (uint32_t)e);
  const uint32_t hi = dpp_shl((uint32_t)(a >> 32), (uint32_t)(e >> 32));
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}
__device__ inline uint32_t dpp_shr0(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x138, 0xf, 0xf, true);
}
__device__ inline uint32_t dpp_shl0(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x130, 0xf, 0xf, true);
}
__device__ inline double from_left(double v) {
  const uint64_t a = __double_as_longlong(v);
  return __longlong_as_double(
      (long long)(((uint64_t)dpp_shr0((uint32_t)(a >> 32)) << 32) | dpp_shr0((uint32_t)a)));
}
__device__ inline double from_right(double v) {
  const uint64_t a = __double_as_longlong(v);
  return __longlong_as_double(
      (long long)(((uint64_t)dpp_shl0((uint32_t)(a >> 32)) << 32) | dpp_shl0((uint32_t)a)));
}
__device__ inline float from_left(float v) { return __uint_as_float(dpp_shr0(__float_as_uint(v))); }
__device__ inline float from_right(float v) {
  return __uint_as_float(dpp_shl0(__float_as_uint(v)));
}
__device__ inline float from_left(float v, float edge) {
  return __uint_as_float(dpp_shr(__float_as_uint(v), __float_as_uint(edge)));
}
__device__ inline float from_right(float v, float edge) {
  return __uint_as_float(dpp_shl(__float_as_uint(v), __float_as_uint(edge)));
}

// v in the lanes of mask m, 0 in the others (outside the grid, where a
// level holds the ghost value 0). Written as the select instruction itself:
// as a C++ select with a uniform mask the compiler turns it into a branch
// around the arithmetic, splitting the iteration into blocks it cannot
// schedule loads across.
__device__ inline double zero_outside(double v, uint64_t m) {
  const uint64_t u = (uint64_t)__double_as_longlong(v);
  uint32_t lo, hi;
  asm("v_cndmask_b32_e64 %0, 0, %1, %2" : "=v"(lo) : "v"((uint32_t)u), "s"(m));
  asm("v_cndmask_b32_e64 %0, 0, %1, %2" : "=v"(hi) : "v"((uint32_t)(u >> 32)), "s"(m));
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}
__device__ inline float zero_outside(float v, uint64_t m) {
  uint32_t r;
  asm("v_cndmask_b32_e64 %0, 0, %1, %2" : "=v"(r) : "v"(__float_as_uint(v)), "s"(m));
  return __uint_as_float(r);
}

template <int N>
using IC = std::integral_constant<int, N>;

template <class R, int NF, bool ADJ, int RR, int ZC, int DA, bool ST, bool NT, int MW>
__global__ __launch_bounds__(kBX * MW) void ac_march(AcMarchArgs<R> a) {
  using M = AcMarch<NF, RR, ZC, MW>;
  constexpr int H = M::H, SY = M::SY;
  constexpr int NL = NF > 0 ? NF : 1;   // levels kept in rings: 0 .. NL-1
  constexpr int NE = (NF > 0 ? NF : 0) + (ADJ ? 1 : 0);  // exchanged fields
  constexpr int GF = NE - 1;            // exchange field of g
  static_assert(NF >= 0 && NF <= 3 && (NF > 0 || ADJ), "levels");
  static_assert(!ST || (NF >= 2 && !ADJ), "store-through runs are forward runs");
  // rows published for the neighbours: [half][field][0: a wave's last row
  // (read by the wave below it), 1: its first row (read by the wave above)]
  __shared__ R pub[2][NE][2][MW][kBX];
  int b = xcd_tile(a.ntiles);
  if (b >= a.ntiles) return;
  const int bx = b % a.tiles_x;
  b /= a.tiles_x;
  const int by = b % a.tiles_y;
  const int bz = b / a.tiles_y;
  // the wave index is uniform across the wave: kept scalar, so the choices
  // between a wave's own rows and its neighbours' are branch-free
  const int lane = (int)threadIdx.x, w = __builtin_amdgcn_readfirstlane((int)threadIdx.y);
  const int c = bx * M::OX - H + lane;      // this lane's column
  const int jw = by * M::OY - H + w * RR;   // this wave's first row
  const int z0 = bz * ZC, z1 = min(z0 + ZC, a.nz);
  const int nx = a.nx, ny = a.ny, nz = a.nz, plane = nx * ny;
  const bool cin = c >= 0 && c < nx;
  // the lanes at the region's sides read the column beyond it (ring), the
  // first and last wave the row beyond it
  const int cr = lane == 0 ? c - 1 : c + 1;
  const bool crin = (lane == 0 || lane == kBX - 1) && cr >= 0 && cr < nx;
  const int jr = w == 0 ? jw - 1 : jw + RR;
  const bool jrin = (w == 0 || w == MW - 1) && jr >= 0 && jr < ny && cin;
  // byte offsets within a plane (kOob where the cell is not read or written)
  uint32_t off[RR], offx[RR], offo[RR];
  bool in[RR];
#pragma unroll
  for (int i = 0; i < RR; ++i) {
    const int j = jw + i, r = w * RR + i;
    in[i] = cin && j >= 0 && j < ny;
    off[i] = in[i] ? uint32_t(j * nx + c) * sizeof(R) : kOob;
    offx[i] = (crin && j >= 0 && j < ny) ? uint32_t(j * nx + cr) * sizeof(R) : kOob;
    // output tile: lanes H .. H+OX-1, region rows H .. SY-1-H
    offo[i] = (in[i] && lane >= H && lane < H + M::OX && r >= H && r < SY - H) ? off[i] : kOob;
  }
  const uint32_t offy = jrin ? uint32_t(jr * nx + c) * sizeof(R) : kOob;

  // lanes whose cell of row i lies in the grid
  uint64_t rowmask[RR];
#pragma unroll
  for (int i = 0; i < RR; ++i) rowmask[i] = __builtin_amdgcn_ballot_w64(in[i]);
  auto plane_in = [&](int q) { return q >= 0 && q < nz; };

  // Rings of planes: the inputs (level 0 and g, with their rows beyond the
  // region) in RA = 6 slots, requested DA planes ahead of their first use;
  // levels 1 .. NL-1, the inputs' side columns and the pointwise x of the
  // plain adjoint in RB = 3 slots. Plane q sits in slot (q - pfirst) mod RA
  // (or RB; g's planes are counted from pfirst + GD), and the iteration
  // body is unrolled 6 times so every slot index is a compile-time constant.
  // (with DA = 1, RA = RB = 4 and the body is unrolled 4 times: fewer
  // values live at once)
  constexpr int RA = DA == 1 ? 4 : 6, RB = DA == 1 ? 4 : 3, UN = DA == 1 ? 4 : 6;
  static_assert(DA >= 1 && DA + 2 <= RA && RB >= 3 && UN % RA == 0 && UN % RB == 0,
                "request distance and rings");
  R X[RA][RR], Xy[RA], Xs[RB][RR];  // level 0 (x pointwise with NF = 0), row beyond, side columns
  R L[NL][RB][RR];                  // levels 1 .. NL-1 (index 0 unused)
  R G[ADJ ? RA : 1][RR], Gy[ADJ ? RA : 1], Gs[ADJ ? RB : 1][RR];
#pragma unroll
  for (int s = 0; s < RB; ++s)
#pragma unroll
    for (int i = 0; i < RR; ++i)
#pragma unroll
      for (int l = 0; l < NL; ++l) L[l][s][i] = R(0);

  const int pfirst = NF > 0 ? z0 - NF + 1 : z0;
  const int plast = NF > 0 ? z1 + NF - 2 : z1 - 1;
  constexpr int GD = NF > 0 ? -(NF - 1) : 0;  // g's centre plane is p + GD

  // plane q of an input array: the region's cells and, for the first and
  // last wave, the row beyond it
  auto fetch = [&](const R* src, int q, R (&dst)[RR], R& dy) {
    const auto rs = plane_rsrc(src, q, nz, plane);
#pragma unroll
    for (int i = 0; i < RR; ++i) dst[i] = bload<R, 0>(rs, off[i]);
    dy = bload<R, 0>(rs, offy);
  };
  // the columns beyond the region's sides at plane q (lanes 0 and 63)
  auto fetch_side = [&](const R* src, int q, R (&dx)[RR]) {
    const auto rs = plane_rsrc(src, q, nz, plane);
#pragma unroll
    for (int i = 0; i < RR; ++i) dx[i] = bload<R, 0>(rs, offx[i]);
  };
  // x read pointwise by the plain adjoint, once: streamed
  auto fetch_point = [&](int q, R (&dst)[RR]) {
    const auto rs = plane_rsrc(a.x, q, nz, plane);
#pragma unroll
    for (int i = 0; i < RR; ++i) dst[i] = bload<R, NT ? kAuxNT : 0>(rs, off[i]);
  };
  // the requests iteration p (slot index U) makes: level 0 and g DA planes
  // ahead, side columns and pointwise x two planes ahead
  auto request = [&](int p, auto Uc) {
    constexpr int U = decltype(Uc)::value;
    if constexpr (NF > 0) {
      fetch(a.x, p + DA, X[(U + DA) % RA], Xy[(U + DA) % RA]);
      fetch_side(a.x, p + 2, Xs[(U + 2) % RB]);
    } else {
      fetch_point(p + 2, X[(U + 2) % RB]);
    }
    if constexpr (ADJ) {
      fetch(a.g, p + GD + DA, G[(U + DA) % RA], Gy[(U + DA) % RA]);
      fetch_side(a.g, p + GD + 2, Gs[(U + 2) % RB]);
    }
  };
  // LDS slots of a field: [0][w] holds wave w's last row (the row below the
  // last wave for w = 3), [1][w] wave w's first row (the row above the first
  // wave for w = 0). A wave's first row reads its y-1 neighbours from the
  // slot above it, its last row its y+1 neighbours from the slot below.
  const int up_slot = w > 0 ? w - 1 : MW;                 // [0][w-1], or [1][0]
  const int dn_slot = w < MW - 1 ? MW + w + 1 : MW - 1;   // [1][w+1], or [0][MW-1]
  auto lds = [&](int hh, int f, int slot) -> R& {
    return (&pub[hh][f][0][0][0])[slot * kBX + lane];
  };
  auto publish = [&](int hh, int f, const R (&v)[RR], R beyond) {
    lds(hh, f, w) = w == MW - 1 ? beyond : v[RR - 1];
    lds(hh, f, MW + w) = w == 0 ? beyond : v[0];
  };
  // the stencil's neighbour sum at row i, in the forward's order
  //   ((((x-1 + x+1) + y-1) + y+1) + z-1) + z+1
  // (side: the side-column values of an input field; levels computed here
  // read 0 beyond the region, where they are not valid anyway)
  auto nbr_sum = [&](int hh, int f, const R (&v)[RR], const R* side, int i, R zm, R zp) -> R {
    R s = side ? from_left(v[i], *side) + from_right(v[i], *side)
               : from_left(v[i]) + from_right(v[i]);
    s += i > 0 ? v[i - 1] : lds(hh, f, up_slot);
    s += i < RR - 1 ? v[i + 1] : lds(hh, f, dn_slot);
    s += zm;
    s += zp;
    return s;
  };
  auto point = [&](R cv, R s) {
    const R lap = s - R(6) * cv;
    return (cv + a.D * lap) - a.C * ((cv * cv) * cv);
  };

  // prologue: the planes the first iterations read before their own
  // requests arrive, and the rows the first iteration reads
  if constexpr (NF > 0) {
#pragma unroll
    for (int d = -1; d < DA; ++d) fetch(a.x, pfirst + d, X[(d + RA) % RA], Xy[(d + RA) % RA]);
    fetch_side(a.x, pfirst, Xs[0]);
    fetch_side(a.x, pfirst + 1, Xs[1]);
  } else {
    fetch_point(pfirst, X[0]);
    fetch_point(pfirst + 1, X[1]);
  }
  if constexpr (ADJ) {
#pragma unroll
    for (int d = -1; d < DA; ++d)
      fetch(a.g, pfirst + GD + d, G[(d + RA) % RA], Gy[(d + RA) % RA]);
    fetch_side(a.g, pfirst + GD, Gs[0]);
    fetch_side(a.g, pfirst + GD + 1, Gs[1]);
  }
  if constexpr (NF > 0) publish(0, 0, X[0], Xy[0]);
  if constexpr (ADJ) publish(0, GF, G[0], Gy[0]);
  __syncthreads();

  auto body = [&](auto Uc, int p) {
    constexpr int U = decltype(Uc)::value;
    constexpr int h = U & 1, hn = h ^ 1;
    constexpr int Am = (U + RA - 1) % RA, A0 = U % RA, Ap = (U + 1) % RA;  // input slots
    constexpr int B0 = U % RB;
    request(p, Uc);
    // nothing below may move above these requests: a wait hoisted above
    // them would wait for every request in flight, the last iteration's
    // included, and leave no request in flight across iterations
    __builtin_amdgcn_sched_barrier(0);
    R last[RR];  // level NF at plane p-NF+1 (x_{t-1} for the adjoint)
    if constexpr (NF > 0) {  // level 1 at plane p from level 0 at p-1, p, p+1
      const bool qin = plane_in(p);
      const auto rm = plane_rsrc(a.mid0, ST && p >= z0 && p < z1 ? p : -1, nz, plane);
#pragma unroll
      for (int i = 0; i < RR; ++i) {
        const R v = point(X[A0][i], nbr_sum(h, 0, X[A0], &Xs[B0][i], i, X[Am][i], X[Ap][i]));
        const R o = zero_outside(v, qin ? rowmask[i] : 0);
        if constexpr (NF > 1) L[1][B0][i] = o; else last[i] = o;
        if constexpr (ST) {
          if (offo[i] != kOob) bstore<R, 0>(rm, offo[i], o);
        }
      }
    }
    // level l at plane p-l+1 from level l-1 at planes p-l .. p-l+2
    auto level = [&](auto Lc) {
      constexpr int l = decltype(Lc)::value;
      constexpr int sm = (U - l + 3 * RB) % RB, sc = (U - l + 1 + 3 * RB) % RB,
                    sp = (U - l + 2 + 3 * RB) % RB;
      const int q = p - l + 1;
      const bool qin = plane_in(q);
      const auto rm =
          plane_rsrc(a.mid1, ST && l == 2 && q >= z0 && q < z1 ? q : -1, nz, plane);
#pragma unroll
      for (int i = 0; i < RR; ++i) {
        const R v = point(L[l - 1][sc][i], nbr_sum(h, l - 1, L[l - 1][sc], nullptr, i,
                                                    L[l - 1][sm][i], L[l - 1][sp][i]));
        const R o = zero_outside(v, qin ? rowmask[i] : 0);
        if constexpr (l < NF) L[l][sc][i] = o; else last[i] = o;
        if constexpr (ST && l == 2 && NF == 3) {
          if (offo[i] != kOob) bstore<R, 0>(rm, offo[i], o);
        }
      }
    };
    if constexpr (NF >= 2) level(IC<2>{});
    if constexpr (NF >= 3) level(IC<3>{});
    const int qo = NF > 0 ? p - NF + 1 : p;  // the output plane
    const auto ro = plane_rsrc(a.y, qo >= z0 && qo < z1 ? qo : -1, nz, plane);
    if constexpr (ADJ) {
      // g'(m) = (k0 - k1 x(m)^2) g(m) + D * (sum of g over m's neighbours)
#pragma unroll
      for (int i = 0; i < RR; ++i) {
        const R xa = NF > 0 ? last[i] : X[B0][i];
        const R s = nbr_sum(h, GF, G[A0], &Gs[B0][i], i, G[Am][i], G[Ap][i]);
        const R v = (a.k0 - a.k1 * (xa * xa)) * G[A0][i] + a.D * s;
        if (offo[i] != kOob) bstore<R, NT ? kAuxNT : 0>(ro, offo[i], v);
      }
    } else {
#pragma unroll
      for (int i = 0; i < RR; ++i)
        if (offo[i] != kOob) bstore<R, NT ? kAuxNT : 0>(ro, offo[i], last[i]);
    }
    // rows the next iteration reads: level 0 and g at their next centre
    // planes, levels 1 .. NF-1 as evaluated now
    if constexpr (NF > 0) publish(hn, 0, X[Ap], Xy[Ap]);
    if constexpr (NF >= 2) publish(hn, 1, L[1][B0], R(0));
    if constexpr (NF >= 3) publish(hn, 2, L[2][(U + RB - 1) % RB], R(0));
    if constexpr (ADJ) publish(hn, GF, G[Ap], Gy[Ap]);
    __syncthreads();
  };

  int p = pfirst;
  for (; p + UN - 1 <= plast; p += UN) {
    body(IC<0>{}, p);
    body(IC<1>{}, p + 1);
    body(IC<2>{}, p + 2);
    body(IC<3>{}, p + 3);
    if constexpr (UN == 6) {
      body(IC<4 % UN>{}, p + 4);
      body(IC<5 % UN>{}, p + 5);
    }
  }
  if (p <= plast) body(IC<0>{}, p);
  if (p + 1 <= plast) body(IC<1>{}, p + 1);
  if (p + 2 <= plast) body(IC<2>{}, p + 2);
  if constexpr (UN == 6) {
    if (p + 3 <= plast) body(IC<3>{}, p + 3);
    if (p + 4 <= plast) body(IC<4 % UN>{}, p + 4);
  }
}

inline int cdiv(int a, int b) { return (a + b - 1) / b; }

// 1 when the kernels of this shape stream their stores (see kStreamBytes)
inline int streams(const StepShape& s) {
  const int64_t bytes = int64_t(s.nx) * s.ny * s.nz * (s.dtype == ADST_F64 ? 8 : 4);
  return bytes >= kStreamBytes ? 1 : 0;
}

// The z-march kernels address a plane with 32-bit byte offsets.
inline bool march_fits(const StepShape& s) {
  return int64_t(s.nx) * s.ny * (s.dtype == ADST_F64 ? 8 : 4) < (int64_t(1) << 31);
}

// Rows per wave and planes per chunk of the z-march launches. The plain
// adjoint (no forward level: few values live per row) runs a 64 x 32 region,
// as eight waves of four rows, where a plane is kTallPlaneBytes or more: its
// row-beyond reads halve per point and eight waves hide more of the LDS
// exchange (1024^3 step 4.76 -> 4.68 ms and 4.67 -> 4.55 ms in the two
// buffer placements against a 64 x 16 region; four waves of eight rows:
// 4.62 ms in the faster placement, sixteen waves of two rows: 5.24 ms;
// 128-plane chunks no faster). At 512^3 (2 MiB planes) the 64 x 16 region
// stays faster (0.568 against 0.586 ms).
constexpr int kMarchRows = 4, kMarchPlanes = 64, kMarchAhead = 1, kTallAdjWaves = 8;
constexpr int64_t kTallPlaneBytes = int64_t(4) << 20;

template <class R, int NF, bool ADJ, bool ST, int RR = kMarchRows, int MW = kMW>
hipError_t march(const StepShape& s, const R* x, const R* g, R* y, R* m0, R* m1,
                 hipStream_t st) {
  if constexpr (NF == 0 && MW == kMW) {
    if (int64_t(s.nx) * s.ny * int64_t(sizeof(R)) >= kTallPlaneBytes)
      return march<R, NF, ADJ, ST, RR, kTallAdjWaves>(s, x, g, y, m0, m1, st);
  }
  using M = AcMarch<NF, RR, kMarchPlanes, MW>;
  const int tx = cdiv(s.nx, M::OX), ty = cdiv(s.ny, M::OY);
  const int nt = tx * ty * cdiv(s.nz, kMarchPlanes);
  const R D = R(s.p0), C = R(s.p1);
  const AcMarchArgs<R> a{x, g, y, m0, m1, s.nx, s.ny, s.nz, tx, ty, nt,
                         D, C, R(1) + D * R(-6), R(3) * C};
  const dim3 grid(xcd_grid(nt)), block(kBX, MW);
  if (streams(s))
    ac_march<R, NF, ADJ, RR, kMarchPlanes, kMarchAhead, ST, true, MW><<<grid, block, 0, st>>>(a);
  else
    ac_march<R, NF, ADJ, RR, kMarchPlanes, kMarchAhead, ST, false, MW><<<grid, block, 0, st>>>(a);
  return hipGetLastError();
}

// mids (nullable): the intermediate states' buffers, step l's at mids[l-1].
template <class R, int K, int RPT, int NZ, int BY>
hipError_t ac_forward_n(const StepShape& s, const R* x, R* y, R* const* mids, hipStream_t st) {
  using A = AcN<K, RPT, NZ, BY>;
  const int tx = cdiv(s.nx, A::OX), ty = cdiv(s.ny, A::OY);
  const int nt = tx * ty * cdiv(s.nz, A::ZC);
  const dim3 grid(xcd_grid(nt)), block(kBX, BY);
  R* m0 = mids ? mids[0] : nullptr;
  R* m1 = (mids && K >= 3) ? mids[1] : nullptr;
  const bool str = streams(s) != 0;
  if (mids && str)
    fwd_allencahn3d7_n<R, K, RPT, NZ, true, true, BY><<<grid, block, 0, st>>>(
        x, y, m0, m1, s.nx, s.ny, s.nz, tx, ty, nt, R(s.p0), R(s.p1));
  else if (mids)
    fwd_allencahn3d7_n<R, K, RPT, NZ, false, true, BY><<<grid, block, 0, st>>>(
        x, y, m0, m1, s.nx, s.ny, s.nz, tx, ty, nt, R(s.p0), R(s.p1));
  else if (str)
    fwd_allencahn3d7_n<R, K, RPT, NZ, true, false, BY><<<grid, block, 0, st>>>(
        x, y, m0, m1, s.nx, s.ny, s.nz, tx, ty, nt, R(s.p0), R(s.p1));
  else
    fwd_allencahn3d7_n<R, K, RPT, NZ, false, false, BY><<<grid, block, 0, st>>>(
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
      return ac_forward_n<R, 2, 4, 32, kBY>(s, x, y, m, st);
    case 3:
      return ac_forward_n<R, 3, 2, 64, 16>(s, x, y, m, st);
  }
  return hipErrorInvalidValue;
}

// One forward step (with the limiter when s.limit).
template <class R>
hipError_t forward1(const StepShape& s, const R* x, R* y, hipStream_t st) {
  const int tx = cdiv(s.nx, kAcTX), ty = cdiv(s.ny, kAcTY);
  const int nt = tx * ty * cdiv(s.nz, kAcZC);
  const dim3 grid(xcd_grid(nt)), block(kBX, kBY);
  const bool str = streams(s) != 0;
  const Limit<R> lim{R(s.lo), R(s.hi)};
  if (s.limit && str)
    fwd_allencahn3d7<R, true, true><<<grid, block, 0, st>>>(x, y, s.nx, s.ny, s.nz, tx, ty, nt,
                                                            R(s.p0), R(s.p1), lim);
  else if (s.limit)
    fwd_allencahn3d7<R, true, false><<<grid, block, 0, st>>>(x, y, s.nx, s.ny, s.nz, tx, ty, nt,
                                                             R(s.p0), R(s.p1), lim);
  else if (str)
    fwd_allencahn3d7<R, false, true><<<grid, block, 0, st>>>(x, y, s.nx, s.ny, s.nz, tx, ty, nt,
                                                             R(s.p0), R(s.p1), lim);
  else
    fwd_allencahn3d7<R, false, false><<<grid, block, 0, st>>>(x, y, s.nx, s.ny, s.nz, tx, ty,
                                                              nt, R(s.p0), R(s.p1), lim);
  return hipGetLastError();
}

template <class R>
hipError_t adjoint1(const StepShape& s, const R* x, const R* g, R* gp, double* dp_part,
                    bool dp_first, hipStream_t st) {
  const R D = R(s.p0), C = R(s.p1);
  const R k0 = R(1) + D * R(-6), k1 = R(3) * C;
  const int tx = cdiv(s.nx, kAcTX), ty = cdiv(s.ny, kAcTY);
  const int nt = tx * ty * cdiv(s.nz, kAcZC);
  const dim3 grid(xcd_grid(nt)), block(kBX, kBY);
  const bool str = streams(s) != 0, lm = adjoint_applies_limit(s, dp_part != nullptr);
  const Limit<R> lim{R(s.lo), R(s.hi)};
  const DpOut dp{dp_part, nt, dp_first ? 1 : 0};
  if (!dp_part && !lm && march_fits(s)) return march<R, 0, true, false>(s, x, g, gp, nullptr, nullptr, st);
#define ADST_AC_ADJ(DPV, NTV)                                                                   \
  adj_allencahn3d7<R, DPV, NTV><<<grid, block, 0, st>>>(x, g, gp, s.nx, s.ny, s.nz, tx, ty, nt, \
                                                         D, k0, k1, dp)
  // waves (and rows per half-tile) of the limiter's adjoint: 64 x 16 tiles
  // (0.703 -> 0.686 ms per 512^3 step against 64 x 8; 64 x 32 was slower),
  // marching over 256-plane chunks (0.686 -> 0.620 ms against 32 planes;
  // 128: 0.636). The other tiled kernels keep 32: at 128 the forward with
  // the limiter went from 0.409 to 0.436 ms and the adjoint with the
  // constants' partials from 0.629 to 0.653.
  constexpr int kLimTW = 8, kLimZC = 256;
  const int tyl = cdiv(s.ny, 2 * kLimTW), ntl = tx * tyl * cdiv(s.nz, kLimZC);
#define ADST_AC_LIM(NTV)                                                                          \
  adj_allencahn3d7_lim<R, NTV, kLimTW, kLimZC><<<dim3(xcd_grid(ntl)), dim3(kBX, kLimTW), 0, st>>>( \
      x, g, gp, s.nx, s.ny, s.nz, tx, tyl, ntl, D, k0, k1, C, lim)
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
  return hipGetLastError();
}

}  // namespace

hipError_t ac_launch_forward(const StepShape& s, const void* x, void* y, hipStream_t st) {
  return s.dtype == ADST_F64
             ? forward1<double>(s, static_cast<const double*>(x), static_cast<double*>(y), st)
             : forward1<float>(s, static_cast<const float*>(x), static_cast<float*>(y), st);
}

hipError_t ac_launch_forward_steps(const StepShape& s, const void* x, void* y, void* const* mids,
                                   int32_t n, hipStream_t st) {
  if (s.limit) return hipErrorInvalidValue;  // fused steps have no limiter
  return s.dtype == ADST_F64 ? ac_forward_steps<double>(s, x, y, mids, n, st)
                             : ac_forward_steps<float>(s, x, y, mids, n, st);
}

hipError_t ac_launch_adjoint(const StepShape& s, const void* x, const void* g, void* gp,
                             double* dp_part, bool dp_first, hipStream_t st) {
  return s.dtype == ADST_F64
             ? adjoint1<double>(s, static_cast<const double*>(x), static_cast<const double*>(g),
                                static_cast<double*>(gp), dp_part, dp_first, st)
             : adjoint1<float>(s, static_cast<const float*>(x), static_cast<const float*>(g),
                               static_cast<float*>(gp), dp_part, dp_first, st);
}

// Three recomputed levels take eight waves (a 64 x 32 region: 1.42 -> 1.22
// region points per output point and level; at 1024^3, 11.21 -> 10.93 ms
// for a launch that also wrote two intermediate states, in one process and
// one placement of the buffers); one or two keep four (eight measured no
// faster for two).
constexpr int kFused3Waves = 8;

template <class R>
hipError_t forward_adjoint(const StepShape& s, const R* x, const R* g, R* gp, int32_t n,
                           hipStream_t st) {
  switch (n) {
    case 1: return march<R, 1, true, false>(s, x, g, gp, nullptr, nullptr, st);
    case 2: return march<R, 2, true, false>(s, x, g, gp, nullptr, nullptr, st);
    case 3:
      return march<R, 3, true, false, kMarchRows, kFused3Waves>(s, x, g, gp, nullptr, nullptr,
                                                                st);
  }
  return hipErrorInvalidValue;
}

hipError_t ac_launch_forward_adjoint(const StepShape& s, const void* x, const void* g, void* gp,
                                     int32_t n, hipStream_t st) {
  if (s.limit || !march_fits(s)) return hipErrorInvalidValue;
  return s.dtype == ADST_F64
             ? forward_adjoint<double>(s, static_cast<const double*>(x),
                                       static_cast<const double*>(g), static_cast<double*>(gp), n,
                                       st)
             : forward_adjoint<float>(s, static_cast<const float*>(x),
                                      static_cast<const float*>(g), static_cast<float*>(gp), n, st);
}

bool ac_fuses_forward_adjoint(const StepShape& s) { return !s.limit && march_fits(s); }

int64_t ac_dparam_slots(const StepShape& s) {
  return int64_t(cdiv(s.nx, kAcTX)) * cdiv(s.ny, kAcTY) * cdiv(s.nz, kAcZC);
}

}  // namespace adst
