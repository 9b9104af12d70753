// In-place Gauss-Seidel sweeps and their reverse sweeps on gfx950.
//
// The step (adst.h, ADST_GAUSSSEIDEL2D5): interior points are overwritten
// one at a time in row-major order with
//     x[c] = w * ((((x[c] + x[E]) + x[N]) + x[S]) + x[W]),
// so S and W already hold the current sweep's values and c, E, N the
// previous sweep's (the paper's Seidel2d case study, Sec. V-B: an in-place
// stencil inside a time loop, where a loop-carried dependency runs through
// every sweep). Any order in which each point comes after its W and S
// neighbours and before its E and N neighbours gives bit-identical values,
// which is what lets a wavefront evaluate it in parallel.
//
// Reverse sweep. One sweep is the product U_n ... U_1 of point updates, so
// its transpose applies U_1^T ... U_n^T: the points in reverse order (the
// reversed loop of Sec. III-C; the overwritten value's gradient is cleared
// and replaced, Sec. II). With h[k] the gradient at point k when its update
// is reversed and h = 0 on the ring, this gives
//     h[k]     = g[k] + w * (h[E] + h[N])         (reverse order: E and N
//                                                   are reversed earlier)
//     g'[k]    = w * ((h[k] + h[W]) + h[S])        interior k
//     g'[ring] = g[ring] + w * h[its interior neighbour]
// The first line is again a sweep with a loop-carried dependency, the
// mirror image of the forward one; the last two are local. In place, h[k]
// overwrites g[k]; g'[k] needs h at k, W and S, which are still old when the
// next reverse sweep reaches k, so "finish sweep t, then start sweep t-1"
// fuses into one pass:
//     phase 0 (after the seed):  h = g + w*(h[N] + h[E])          (recur)
//     phase p (0 < p < P-1):     gin = w*((h[k] + h[W]) + h[S]);
//                                h' = (gin + w*h'[N]) + w*h'[E] (fused)
//     phase P-1:                 g' = gin                       (finish)
// with ring accumulators updated in every phase after the first. The
// arithmetic of a point is the same whether a phase runs alone or
// pipelined, so every schedule gives bit-identical gradients.
//
// Parallel layout. Both directions use "processing" coordinates: the
// forward pass walks rows upward and columns rightward, the reverse pass the
// mirror image (rows downward, columns leftward); in processing coordinates
// each point needs the new values of its previous row (PR) and previous
// element (PX) and the old values of itself (C), its next row (NR) and next
// element (NX). A workgroup is one wave of 64 lanes. Lane j owns a column
// block of V = 16 bytes (2 doubles or 4 floats) and walks kGsRows rows, the
// wave skewed by one row per lane: at step m lane j is on row
// rho = kGsRows*I + m - j. Its PR is its own result of step m-1, its PX the
// last new value of lane j-1 from step m-1 (a DPP lane shift), its NX the
// first old value of lane j+1's next row (another shift), so a tile needs no
// LDS except two halo columns. Each lane loads all its rows at once (every
// load in flight), computes kGsRows steps and stores each row as it goes.
//
// Tiles (I, J) of phase s run in launch tau = I + 3 J + 3 s. Lane 0 reads
// new values from lane 63 of tiles (I+1, J-1) and (I+2, J-1) (tau-2 and
// tau-1); lane 63 reads old values from lane 0 of (I-2, J+1) and (I-1, J+1)
// (tau+1 and tau+2, so still at the previous phase, whose own launches are
// at tau-2 and tau-1); the first row reads (I-1, J) of the same phase
// (tau-1) and the last row (I+1, J) of the previous phase (tau-2). Tiles that
// share a launch therefore never exchange data, a launch holds tiles of many
// phases at once (temporal pipelining), and the stream order of launches is
// the only synchronisation.

#include <hip/hip_runtime.h>

#include <algorithm>

#include "adst.h"
#include "kernels.h"

namespace adst {
namespace {

constexpr int kGsLanes = 64;  // one wave per tile
constexpr int kGsRows = 32;   // rows each lane walks per tile
constexpr int kGsLagJ = 3;    // tau = I + kGsLagJ * J + kGsLagS * s
constexpr int kGsLagS = 3;
constexpr int kGsChunk = 16;  // steps whose outputs are staged in LDS before a flush
static_assert(kGsLagJ == 2 + (kGsLanes - 2) / kGsRows, "lane 0 waits on tiles up to I+2");
static_assert(kGsLanes == 2 * kGsRows, "each lane holds one halo value");
static_assert(kGsRows % kGsChunk == 0, "the steps split into whole flush chunks");

enum : int { kGsRecur = 0, kGsFused = 1, kGsFinish = 2 };

// Whole-wave lane shifts (DPP wave_shr:1 / wave_shl:1). Lane 0 (resp. 63)
// has no source lane and receives `edge`.
__device__ inline uint32_t shr1_u32(uint32_t v, uint32_t edge) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)edge, (int)v, 0x138, 0xf, 0xf, false);
}
__device__ inline uint32_t shl1_u32(uint32_t v, uint32_t edge) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)edge, (int)v, 0x130, 0xf, 0xf, false);
}
__device__ inline float lane_from_prev(float v, float edge) {
  return __uint_as_float(shr1_u32(__float_as_uint(v), __float_as_uint(edge)));
}
__device__ inline float lane_from_next(float v, float edge) {
  return __uint_as_float(shl1_u32(__float_as_uint(v), __float_as_uint(edge)));
}
__device__ inline double lane_from_prev(double v, double edge) {
  const uint64_t a = __double_as_longlong(v), e = __double_as_longlong(edge);
  const uint32_t lo = shr1_u32((uint32_t)a, (uint32_t)e);
  const uint32_t hi = shr1_u32((uint32_t)(a >> 32), (uint32_t)(e >> 32));
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}
__device__ inline double lane_from_next(double v, double edge) {
  const uint64_t a = __double_as_longlong(v), e = __double_as_longlong(edge);
  const uint32_t lo = shl1_u32((uint32_t)a, (uint32_t)e);
  const uint32_t hi = shl1_u32((uint32_t)(a >> 32), (uint32_t)(e >> 32));
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

template <class R>
struct GsVec {
  static constexpr int V = 16 / (int)sizeof(R);
  R v[V];
};

// Value of lane `src` (a compile-time constant) in every lane.
__device__ inline float lane_value(float v, int src) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), src));
}
__device__ inline double lane_value(double v, int src) {
  const uint64_t a = __double_as_longlong(v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)a, src);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(a >> 32), src);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// Loads never branch: an address outside the grid is clamped into it and
// the value replaced by 0. Without divergent branches around them, the
// compiler waits for each load only where its value is first used, so a
// tile starts computing as soon as its first rows arrive.
template <class R>
__device__ inline R gs_load1(const R* a, int row, int col, int nx, int ny, bool ok) {
  const int r = min(max(row, 0), ny - 1);
  const int c = min(max(col, 0), nx - 1);
  const R v = a[(int64_t)r * nx + c];
  return ok ? v : R(0);
}

// The V elements of real row `row`, real columns [c0, c0 + V), 0 outside
// the grid or when !ok. VEC: nx is a multiple of V and rows are 16-byte
// aligned, so an in-grid block is whole.
template <class R, bool VEC>
__device__ inline GsVec<R> gs_load(const R* a, int row, int c0, int nx, int ny, bool ok) {
  constexpr int V = GsVec<R>::V;
  GsVec<R> r;
  if (VEC) {
    typedef R vec_t __attribute__((ext_vector_type(V)));
    const int rr = min(max(row, 0), ny - 1);
    const int cc = min(max(c0, 0), nx - V);
    const vec_t t = *reinterpret_cast<const vec_t*>(a + (int64_t)rr * nx + cc);
#pragma unroll
    for (int e = 0; e < V; ++e) r.v[e] = ok ? t[e] : R(0);
  } else {
#pragma unroll
    for (int e = 0; e < V; ++e) r.v[e] = gs_load1(a, row, c0 + e, nx, ny, ok && c0 + e < nx);
  }
  return r;
}

template <class R, bool VEC>
__device__ inline void gs_store(R* a, int row, int c0, int nx, const GsVec<R>& r) {
  constexpr int V = GsVec<R>::V;
  if (VEC) {
    typedef R vec_t __attribute__((ext_vector_type(V)));
    vec_t t;
#pragma unroll
    for (int e = 0; e < V; ++e) t[e] = r.v[e];
    *reinterpret_cast<vec_t*>(a + (int64_t)row * nx + c0) = t;
  } else {
#pragma unroll
    for (int e = 0; e < V; ++e)
      if (c0 + e < nx) a[(int64_t)row * nx + c0 + e] = r.v[e];
  }
}

// One tile of one phase. buf is updated in place; old_src is where the
// forward pass's first phase reads old values (the sweep's input; equal to
// buf when it runs in place). ADJ selects the reverse pass.
template <class R, bool ADJ, bool VEC>
__global__ __launch_bounds__(kGsLanes) void gs_wave(R* buf, const R* old_src, int nx, int ny,
                                                   int nb, int nti, int tau, int s_lo,
                                                   int nphase, R w) {
  constexpr int V = GsVec<R>::V;
  constexpr int B = kGsRows;
  const int s = s_lo + (int)blockIdx.y;
  const int J = (int)blockIdx.x;
  const int I = tau - kGsLagS * s - kGsLagJ * J;
  if (I < 0 || I >= nti) return;  // whole wave: no tile at this (s, J)

  const int j = (int)threadIdx.x;
  const int jj = kGsLanes * J + j;              // processing block
  const bool blk_ok = jj < nb;
  const int rb = ADJ ? nb - 1 - jj : jj;        // real block
  const int c0 = rb * V;                        // first real column of the block
  const int phase = !ADJ ? kGsFused : s == 0 ? kGsRecur : s == nphase - 1 ? kGsFinish : kGsFused;
  const bool recur = phase == kGsRecur, finish = phase == kGsFinish;
  const R* old_a = (!ADJ && s == 0) ? old_src : buf;
  const int rho0 = B * I - j;                   // processing row of step 0
  auto real_row = [&](int rho) { return ADJ ? ny - 1 - rho : rho; };
  auto row_ok = [&](int rho) { return rho >= 0 && rho < ny; };

  // Real column of the processing element just before processing block q
  // (its last element) and just after it (the first element of block q+1).
  auto col_before = [&](int q) { return ADJ ? (nb - q) * V : q * V - 1; };
  auto col_after = [&](int q) { return ADJ ? (nb - 2 - q) * V + V - 1 : (q + 1) * V; };

  // ---- halos, one value per lane, broadcast by readlane at each step:
  // lanes 0..B-1 hold lane 0's PX for step m = j (new values), lanes B..2B-1
  // lane 63's NX for step m = j - B (old values).
  R halo;
  {
    const bool px_half = j < B;
    const int m = j % B;
    const int qa = kGsLanes * J, qb = kGsLanes * J + kGsLanes - 1;
    const int rho = px_half ? B * I + m : B * I + m - (kGsLanes - 1);
    const int col = px_half ? col_before(qa) : col_after(qb);
    const bool okh = row_ok(rho) && (px_half ? qa >= 1 : qb + 1 < nb);
    halo = gs_load1(px_half ? static_cast<const R*>(buf) : old_a, real_row(rho), col, nx, ny, okh);
  }
  // PX of step 0: the new value before the block on this lane's first row.
  const R px0 = gs_load1(buf, real_row(rho0), col_before(jj), nx, ny,
                         blk_ok && jj >= 1 && row_ok(rho0));
  // ---- this lane's rows: L[0] is the previous row (new values), L[1..B]
  // the rows it updates and L[B+1] the row after (old values).
  GsVec<R> L[B + 2];
#pragma unroll
  for (int k = 0; k < B + 2; ++k) {
    const int rho = rho0 - 1 + k;
    L[k] = gs_load<R, VEC>(k == 0 ? buf : old_a, real_row(rho), c0, nx, ny,
                           blk_ok && row_ok(rho));
  }

  // Outputs of the current chunk of steps, by (step within chunk, lane). A
  // lane's rows are skewed against its neighbours', so storing each step
  // directly would touch 64 rows with 16 bytes each; flushing the chunk by
  // grid row instead stores up to kGsChunk neighbouring blocks (contiguous
  // bytes) per instruction.
  __shared__ GsVec<R> stage[kGsChunk][kGsLanes];
  auto flush = [&](int m0) {
    __syncthreads();
    // The chunk covers grid rows rho = B*I + m0 - 63 + i, i < kGsChunk + 63;
    // row i holds the outputs of lanes 63 - i + d at step m0 + d. Each
    // store instruction takes four rows, sixteen lanes (d) per row.
    constexpr int kRows = kGsChunk + kGsLanes - 1;
    constexpr int kPer = kGsLanes / kGsChunk;
#pragma unroll
    for (int q = 0; q < (kRows + kPer - 1) / kPer; ++q) {
      const int i = q * kPer + j / kGsChunk;
      const int d = j % kGsChunk;
      const int src = (kGsLanes - 1) - i + d;  // lane that produced it
      const int srcc = min(max(src, 0), kGsLanes - 1);
      const GsVec<R> v = stage[d][srcc];
      const int rho = B * I + m0 - (kGsLanes - 1) + i;
      const int jjs = kGsLanes * J + srcc;
      if (i < kRows && src == srcc && jjs < nb && row_ok(rho))
        gs_store<R, VEC>(buf, real_row(rho), (ADJ ? nb - 1 - jjs : jjs) * V, nx, v);
    }
    __syncthreads();
  };

  GsVec<R> prev_new = L[0];
  R last_new = R(0);  // new value of this lane's last processing element, previous step
#pragma unroll
  for (int m = 0; m < B; ++m) {
    const int rho = rho0 + m;
    const int row = real_row(rho);
    const bool ok = blk_ok && row_ok(rho);
    const bool row_in = row >= 1 && row <= ny - 2;
    // processing order element e sits at real offset ix(e) of the block
    auto ix = [&](int e) { return ADJ ? V - 1 - e : e; };
    const R px_first = m == 0 ? px0 : lane_from_prev(last_new, lane_value(halo, m));
    const R nx_last = lane_from_next(L[m + 2].v[ix(0)], lane_value(halo, B + m));
    const GsVec<R> C = L[m + 1];
    const GsVec<R> NR = L[m + 2];
    GsVec<R> out;
    R px = px_first;
#pragma unroll
    for (int e = 0; e < V; ++e) {
      const int col = c0 + ix(e);
      const R c = C.v[ix(e)];
      const R nxv = e + 1 < V ? C.v[ix(e + 1)] : nx_last;
      const R nr = NR.v[ix(e)];
      const R pr = prev_new.v[ix(e)];
      const bool col_in = col >= 1 && col <= nx - 2;
      R y;
      if (!ADJ) {
        const R yi = w * ((((c + nxv) + nr) + pr) + px);
        y = (row_in && col_in) ? yi : c;
      } else {
        const R hW = col - 1 == 0 ? R(0) : nxv;      // real W: next element, old
        const R hS = row - 1 == 0 ? R(0) : nr;       // real S: next row, old
        const R hE = col + 1 == nx - 1 ? R(0) : px;  // real E: previous element, new
        const R hN = row + 1 == ny - 1 ? R(0) : pr;  // real N: previous row, new
        const R gin = recur ? c : w * ((c + hW) + hS);
        const R yi = finish ? gin : (gin + w * hN) + w * hE;
        // Ring columns collect w * h of their interior neighbour: (row, 1) is
        // the previous element, (row, nx-2) the next; the top ring row's
        // neighbour row ny-2 is the next row, still old.
        const R prev_old = e > 0 ? C.v[ix(e > 0 ? e - 1 : 0)] : c;
        const R yc = c + w * (col == 0 ? prev_old : nxv);
        const R yt = c + w * nr;
        const bool ring_col = !recur && row_in && nx >= 3 && (col == 0 || col == nx - 1);
        const bool ring_top = !recur && row == ny - 1 && col_in && ny >= 3;
        y = (row_in && col_in) ? yi : ring_col ? yc : ring_top ? yt : c;
      }
      out.v[ix(e)] = y;
      px = y;
    }
    if (ADJ) {
      // The bottom ring row is reversed after row 1, whose old h it needs:
      // push w * h(1, col) into the register copy of row 0 (the next row).
      const bool push = !recur && row == 1 && ny >= 3;
#pragma unroll
      for (int e = 0; e < V; ++e) {
        const int col = c0 + e;
        const R pushed = L[m + 2].v[e] + w * C.v[e];
        L[m + 2].v[e] = (push && col >= 1 && col <= nx - 2) ? pushed : L[m + 2].v[e];
      }
      if (m == B - 1 && push && ok) gs_store<R, VEC>(buf, 0, c0, nx, L[m + 2]);
    }
    stage[m % kGsChunk][j] = out;
    if (m % kGsChunk == kGsChunk - 1) flush(m - (kGsChunk - 1));
    prev_new = out;
    last_new = px;
  }
}

struct GsGeom {
  int V, nb, nti, ntj;
};

GsGeom gs_geom(const StepShape& s) {
  GsGeom g;
  g.V = s.dtype == ADST_F64 ? 2 : 4;
  g.nb = (s.nx + g.V - 1) / g.V;
  g.nti = (s.ny + kGsLanes - 1 + kGsRows - 1) / kGsRows;
  g.ntj = (g.nb + kGsLanes - 1) / kGsLanes;
  return g;
}

int64_t gs_levels(const GsGeom& g, int nphase) {
  return (int64_t)(g.nti - 1) + (int64_t)kGsLagJ * (g.ntj - 1) + (int64_t)kGsLagS * (nphase - 1) + 1;
}

template <class R>
int gs_vec_ok(int nx, const void* a, const void* b) {
  if (nx % (16 / (int)sizeof(R))) return 0;
  for (const void* p : {a, b})
    if (p && (reinterpret_cast<uintptr_t>(p) & 15u)) return 0;
  return 1;
}

template <class R, bool ADJ>
hipError_t gs_run(const StepShape& sh, R* buf, const R* old_src, int nphase, hipStream_t st) {
  const GsGeom g = gs_geom(sh);
  const int64_t dmax = (int64_t)(g.nti - 1) + (int64_t)kGsLagJ * (g.ntj - 1);
  const int64_t levels = gs_levels(g, nphase);
  const bool vec = gs_vec_ok<R>(sh.nx, buf, old_src) != 0;
  for (int64_t tau = 0; tau < levels; ++tau) {
    const int64_t s_lo = std::max<int64_t>(0, (tau - dmax + kGsLagS - 1) / kGsLagS);
    const int64_t s_hi = std::min<int64_t>(nphase - 1, tau / kGsLagS);
    if (s_hi < s_lo) continue;
    const dim3 grid((unsigned)g.ntj, (unsigned)(s_hi - s_lo + 1));
    if (vec)
      gs_wave<R, ADJ, true><<<grid, dim3(kGsLanes), 0, st>>>(
          buf, old_src, sh.nx, sh.ny, g.nb, g.nti, (int)tau, (int)s_lo, nphase, R(sh.p0));
    else
      gs_wave<R, ADJ, false><<<grid, dim3(kGsLanes), 0, st>>>(
          buf, old_src, sh.nx, sh.ny, g.nb, g.nti, (int)tau, (int)s_lo, nphase, R(sh.p0));
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace

int64_t gs_kernel_launches(const StepShape& s, bool adjoint, int32_t sweeps) {
  if (sweeps <= 0) return 0;
  return gs_levels(gs_geom(s), adjoint ? sweeps + 1 : sweeps);
}

hipError_t launch_gs_forward(const StepShape& s, const void* src, void* dst, int32_t sweeps,
                             hipStream_t stream) {
  if (sweeps <= 0) return hipErrorInvalidValue;
  if (s.dtype == ADST_F64)
    return gs_run<double, false>(s, static_cast<double*>(dst), static_cast<const double*>(src),
                                 sweeps, stream);
  return gs_run<float, false>(s, static_cast<float*>(dst), static_cast<const float*>(src),
                              sweeps, stream);
}

hipError_t launch_gs_adjoint(const StepShape& s, void* g, int32_t sweeps, hipStream_t stream) {
  if (sweeps <= 0) return hipErrorInvalidValue;
  if (s.dtype == ADST_F64)
    return gs_run<double, true>(s, static_cast<double*>(g), static_cast<const double*>(g),
                                sweeps + 1, stream);
  return gs_run<float, true>(s, static_cast<float*>(g), static_cast<const float*>(g), sweeps + 1,
                             stream);
}

}  // namespace adst
