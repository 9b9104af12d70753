// Device helpers shared by the kernel sources: launch geometry, the
// XCD-aware tile order, streaming stores, the block reduction of the
// constants' gradients, the limiter, and the Allen-Cahn point update that
// every Allen-Cahn kernel (forward, fused, limiter mask) evaluates.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

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

// The slot's sums of the steps before, requested when the workgroup starts
// so that the read's latency passes while it works (none on the first step,
// which overwrites). NC: the constants of the kind (1 or 2).
struct DpPrev {
  double p0 = 0.0, p1 = 0.0;
};
template <int NC>
__device__ inline DpPrev dp_prev(DpOut dp, int slot) {
  DpPrev r;
  if (!dp.first && threadIdx.x == 0 && threadIdx.y == 0) {
    r.p0 = dp.part[slot];
    if (NC == 2) r.p1 = dp.part[dp.nslots + slot];
  }
  return r;
}

// All threads of the block call this (it synchronises). With one constant
// the second slots hold +0.
template <int NC>
__device__ inline void dp_commit(DpOut dp, int slot, DpPrev prev, double a0, double a1) {
  if (NC == 2)
    block_sum2(a0, a1);
  else
    a0 = block_sum(a0);
  if (threadIdx.x == 0 && threadIdx.y == 0) {
    dp.part[slot] = dp.first ? a0 : prev.p0 + a0;
    dp.part[dp.nslots + slot] = NC == 2 ? (dp.first ? a1 : prev.p1 + a1) : 0.0;
  }
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

}  // namespace
}  // namespace adst
