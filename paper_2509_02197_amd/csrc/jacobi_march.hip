// Temporal blocking of the Jacobi kind on gfx950: n = 3..kJacMaxFuse steps,
// forward or gather adjoint, in one launch with the intermediate time levels
// in registers.
//
// The step (adst.h, ADST_JACOBI2D5): interior points take
//     x'[c] = w * ((((x[c] + x[W]) + x[E]) + x[S]) + x[N]),
// the ring is copied; the adjoint is its transpose in gather form,
//     interior m: g'[m] = w * (g[m] + (((gi[W] + gi[E]) + gi[S]) + gi[N]))
//     ring m:     g'[m] = g[m] + w * (((gi[W] + gi[E]) + gi[S]) + gi[N])
// with gi = g on interior points and 0 on the ring (and outside the grid).
// A point two or more cells from the edge sees only interior neighbours, so
// there both take their unmasked form. The step is linear in the carried
// state, so its adjoint reads no forward state (Sec. IV) and n steps of
// either compose without any stored value in between.
//
// Layout. A workgroup is one wave of 64 lanes owning a strip of 64 * V
// columns (V elements, 16 bytes, per lane) and a chunk of rows. It marches
// along the rows carrying the last three rows of each of the n time levels:
// when input row q arrives, level k evaluates row q - k from level k - 1's
// rows q - k - 1, q - k, q - k + 1. East/west neighbours of a lane's first
// and last element come from the adjacent lanes by DPP whole-wave shifts.
// Each level is valid on one column fewer at each side of the strip and one
// row fewer at each end of the chunk, so strips overlap by H >= n columns
// (whole vectors) and a chunk reads n rows beyond each of its ends. Every
// point evaluates the single-step expressions above, so any split of the
// steps into launches gives the same bits.
//
// Memory. Each input row is loaded kAhead rows before it enters the
// pipeline, into registers that nothing touches until then (its validity
// mask is applied on entry), so the loads stay in flight behind the
// arithmetic. Rows beyond the ones a chunk needs are never fetched from new
// addresses. Odd chunks march downward, so the rows two neighbouring chunks
// share are read by both at about the same time and the second read can hit
// the L2 cache they share (their blocks go to the same XCD); measured, this
// cut the fetched bytes from 1.46x to 1.24x the state's size.
//
// Boundary. Blocks of kUnroll consecutive input rows whose evaluated rows all
// lie two or more cells from the top and bottom edge, in a strip two or more
// cells from the side edges, take the unmasked forms; the others evaluate the
// ring logic. A strip's first and last chunk are short, so the slower blocks
// near the top and bottom edge do not make their waves the launch's tail;
// the first and last strip (the side edges) take short chunks throughout,
// and every XCD gets an equal share of them.
//
// The same layout carries the limiter's one-step adjoint (jacobi_lim_adjoint
// below), which masks g by the branch outcome and transposes it in one pass.

#include <hip/hip_runtime.h>

#include <type_traits>

#include "adst.h"
#include "kernels.h"

namespace adst {
namespace {

constexpr int kLanes = 64;
constexpr int kRows = 48;      // rows per chunk of an interior strip (42 for the
                               // adjoint measured the same: 56.3 against 56.1 us
                               // per 6-step launch at 4096^2, one rocprofv3 job)
constexpr int kLimRows = 128;  // rows per chunk of the limiter's one-step adjoint:
                               // with x and g read non-temporally, 64 / 96 /
                               // 128 / 160 / 192 / 256 / 384 rows took 82.0 /
                               // 82.3 / 81.5 / 86.5 / 83.4 / 97.2 / 115.0 us
                               // per launch at 4096^2 f64 (before the hint,
                               // 192 was best: 90.4 against 92.7 us at 128)
constexpr int kEdgeRows = 12;  // rows per chunk of the first and last strip
constexpr int kEndRows = 6;    // rows of a strip's first and last chunk, whose
                               // blocks near the grid's top and bottom edge
                               // take the slower general path
constexpr int kAhead = 3;      // input rows loaded ahead of the pipeline
constexpr int kUnroll = 6;     // input rows per straight-line block
constexpr int kXcds = 8;       // workgroup i runs on XCD i mod 8
static_assert(kUnroll % kAhead == 0 && kUnroll % 3 == 0, "register slots must stay static");
static_assert(2 * kEndRows <= kRows && kEdgeRows <= kRows && kRows <= 64, "chunk sizes");

// Whole-wave lane shifts: lane i receives lane i-1's value (lane 0: 0) or
// lane i+1's (lane 63: 0).
__device__ inline uint32_t shr1(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x138, 0xf, 0xf, true);
}
__device__ inline uint32_t shl1(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x130, 0xf, 0xf, true);
}
__device__ inline float from_prev(float v) { return __uint_as_float(shr1(__float_as_uint(v))); }
__device__ inline float from_next(float v) { return __uint_as_float(shl1(__float_as_uint(v))); }
__device__ inline double from_prev(double v) {
  const uint64_t a = __double_as_longlong(v);
  return __longlong_as_double(
      (long long)(((uint64_t)shr1((uint32_t)(a >> 32)) << 32) | shr1((uint32_t)a)));
}
__device__ inline double from_next(double v) {
  const uint64_t a = __double_as_longlong(v);
  return __longlong_as_double(
      (long long)(((uint64_t)shl1((uint32_t)(a >> 32)) << 32) | shl1((uint32_t)a)));
}

template <class R, int K>
struct Geom {
  static constexpr int V = 16 / sizeof(R);
  static constexpr int H = ((K + V - 1) / V) * V;  // column overlap, whole vectors
  static constexpr int OW = kLanes * V - 2 * H;    // output columns per strip
};

// Work list: the chunks of the first and last strip (E of them) and of the
// interior strips (I). XCD x takes edge chunks [x*pe, (x+1)*pe) and interior
// chunks [x*pi, (x+1)*pi), edge chunks first.
struct MarchGrid {
  int ns, nedge, ce, ci, pe, pi;
  int rows;  // rows per chunk of an interior strip (at most kRows)
};

// This workgroup's strip and chunk of rows [r0, r1); false when the
// workgroup has no work (the grid is rounded up to whole XCD shares).
// item (optional): the work item's index, edge items first, unique in
// [0, nedge*ce + (ns-nedge)*ci).
__device__ inline bool march_item(const MarchGrid& g, int ny, int* strip, int* chunk, int* r0,
                                  int* r1, int* item = nullptr) {
  const int xcd = (int)blockIdx.x % kXcds, slot = (int)blockIdx.x / kXcds;
  int nch, mid;
  if (slot < g.pe) {
    const int t = xcd * g.pe + slot;
    if (t >= g.nedge * g.ce) return false;
    *strip = (t / g.ce == 0) ? 0 : g.ns - 1;
    *chunk = t % g.ce;
    nch = g.ce;
    mid = kEdgeRows;
    if (item) *item = t;
  } else {
    const int t = xcd * g.pi + (slot - g.pe);
    if (t >= (g.ns - g.nedge) * g.ci) return false;
    *strip = 1 + t / g.ci;
    *chunk = t % g.ci;
    nch = g.ci;
    mid = g.rows;
    if (item) *item = g.nedge * g.ce + t;
  }
  // kEndRows at each end of the strip, mid rows between
  const int c = *chunk;
  if (nch == 1) {
    *r0 = 0;
    *r1 = ny;
  } else if (c == 0) {
    *r0 = 0;
    *r1 = kEndRows;
  } else if (c == nch - 1) {
    *r0 = ny - kEndRows;
    *r1 = ny;
  } else {
    *r0 = kEndRows + (c - 1) * mid;
    *r1 = min(*r0 + mid, ny - kEndRows);
  }
  return true;
}

// The work list for strips of ow output columns; false if it is too long.
inline bool make_grid(int nx, int ny, int ow, MarchGrid* g, int64_t* blocks, int rows = kRows) {
  g->rows = rows;
  g->ns = (nx + ow - 1) / ow;
  g->nedge = g->ns >= 2 ? 2 : 1;
  auto chunks = [&](int mid) {
    return ny > 2 * kEndRows ? 2 + (ny - 2 * kEndRows + mid - 1) / mid : 1;
  };
  g->ce = chunks(kEdgeRows);
  g->ci = chunks(rows);
  const int64_t E = int64_t(g->nedge) * g->ce, I = int64_t(g->ns - g->nedge) * g->ci;
  g->pe = (int)((E + kXcds - 1) / kXcds);
  g->pi = (int)((I + kXcds - 1) / kXcds);
  *blocks = int64_t(kXcds) * (g->pe + g->pi);
  return *blocks > 0 && *blocks <= INT32_MAX;
}

template <class R, int K, bool ADJ, bool VEC>
__global__ __launch_bounds__(kLanes) void jacobi_march(const R* __restrict__ x, R* __restrict__ y,
                                                       int nx, int ny, MarchGrid g, R w) {
  using G = Geom<R, K>;
  constexpr int V = G::V, H = G::H, OW = G::OW, P = kAhead, U = kUnroll;
  typedef R vec_t __attribute__((ext_vector_type(V)));
  int strip, chunk, r0, r1;
  if (!march_item(g, ny, &strip, &chunk, &r0, &r1)) return;
  const int lane = threadIdx.x;
  const int s0 = strip * OW;
  const int c0 = s0 - H + lane * V;  // first column of this lane
  const int nit = (r1 - r0) + 2 * K;  // input rows through the pipeline
  const int lo_need = max(r0 - K, 0), hi_need = min(r1 + K - 1, ny - 1);

  // Per-lane column facts of the V columns.
  auto cin = [&](int c) { return c >= 1 && c <= nx - 2; };
  bool cok[V], cI[V];
  int side[V];  // 0: column 0, 1: column nx-1, -1: neither
#pragma unroll
  for (int e = 0; e < V; ++e) {
    const int c = c0 + e;
    cok[e] = c >= 0 && c < nx;
    cI[e] = cin(c);
    side[e] = c == 0 ? 0 : (c == nx - 1 ? 1 : -1);
  }
  const bool strip_in = s0 - H >= 2 && s0 - H + kLanes * V <= nx - 2;
  const bool st_lane = lane * V >= H && lane * V < H + OW;
  // This lane's ring column, if any (a lane holds at most one: nx > V), and
  // its element; with 16-byte rows, column 0 is a lane's first element and
  // column nx-1 its last.
  int rside = -1, relem = 0;
#pragma unroll
  for (int e = 0; e < V; ++e)
    if (side[e] >= 0) {
      rside = side[e];
      relem = e;
    }

  // Raw load of input row `row` (clamped to the rows the chunk needs, and
  // to the grid, so every address is in bounds); masked on entry.
  auto load = [&](int row, R* out) {
    const int rr = min(max(row, lo_need), hi_need);
    const R* src = x + (int64_t)rr * nx;
    if constexpr (VEC) {
      const int cc = min(max(c0, 0), nx - V);
      const vec_t t = *reinterpret_cast<const vec_t*>(src + cc);
#pragma unroll
      for (int e = 0; e < V; ++e) out[e] = t[e];
    } else {
#pragma unroll
      for (int e = 0; e < V; ++e) out[e] = src[min(max(c0 + e, 0), nx - 1)];
    }
  };

  // The adjoint's pipeline holds gi: every ring cell and every cell outside
  // the grid holds +0 there, so each interior point's masked neighbour sum
  // is the plain sum of the pipeline's values (the terms a mask would drop
  // are +0 already). The ring's own values, g + w*sum, read no other ring
  // value and are kept beside the pipeline: ring_lo and ring_hi hold the
  // bottom and top ring rows at the highest level that has evaluated them
  // (one level reaches a given row per input row), and the one interior
  // neighbour a ring-column cell has is recorded at every level in LDS, from
  // which the ring columns of the chunk's rows are summed after the march.
  // Rows of the record: every row a level may evaluate, [r0 - K - U, r1 + K + U).
  constexpr int NR = kRows + 2 * (K + U);
  __shared__ R nbr[ADJ ? 2 * K * NR + kLanes : 1];
  // LDS index of row j's record at level k: nbr_lane + (k-1)*NR + j, or the
  // lane's scratch cell when it has no ring column
  const bool has_ring = rside >= 0;
  const int nbr_lane = rside * K * NR + (K + U) - r0;
  enum { kFast = 0, kCols = 1, kGeneral = 2 };
  // mid_t: the mode of the blocks away from the top and bottom edge.
  auto march = [&](auto dir_t, auto mid_t) {
    constexpr int DIR = decltype(dir_t)::value;  // +1 upward, -1 downward
    const int ifirst = DIR > 0 ? r0 - K : r1 - 1 + K;  // row of input index 0
    // Level k's row of pipeline index p (row ifirst + DIR*p) sits in slot p mod 3.
    R lv[K][3][V];
    R pf[P][V];
    R ring_lo[V], ring_hi[V];
#pragma unroll
    for (int e = 0; e < V; ++e) ring_lo[e] = ring_hi[e] = R(0);
#pragma unroll
    for (int k = 0; k < K; ++k)
#pragma unroll
      for (int s3 = 0; s3 < 3; ++s3)
#pragma unroll
        for (int e = 0; e < V; ++e) lv[k][s3][e] = R(0);
#pragma unroll
    for (int u = 0; u < P; ++u) load(ifirst + DIR * u, pf[u]);

    // kFast: rows in [2, ny-3], strip in columns [2, nx-3]: unmasked forms.
    // kCols: rows in [2, ny-3], strip touching the side edges.
    // kGeneral: anything (rows near or beyond the top and bottom edge).
    auto block = [&](int base, auto mode_t) {
      constexpr int MODE = decltype(mode_t)::value;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int rr = base + u;
        {  // input row rr enters level 0; the row P ahead is requested
          const int row = ifirst + DIR * rr;
          if constexpr (MODE == kFast) {
#pragma unroll
            for (int e = 0; e < V; ++e) lv[0][u % 3][e] = pf[u % P][e];
          } else if constexpr (!ADJ) {
            const bool rok = row >= 0 && row < ny;
#pragma unroll
            for (int e = 0; e < V; ++e)
              lv[0][u % 3][e] = (rok && cok[e]) ? pf[u % P][e] : R(0);
          } else {
            if constexpr (MODE == kGeneral) {
#pragma unroll
              for (int e = 0; e < V; ++e) {
                const R v = cok[e] ? pf[u % P][e] : R(0);
                ring_lo[e] = row == 0 ? v : ring_lo[e];
                ring_hi[e] = row == ny - 1 ? v : ring_hi[e];
              }
            }
            const bool rin = MODE == kCols || (row >= 1 && row <= ny - 2);
#pragma unroll
            for (int e = 0; e < V; ++e) lv[0][u % 3][e] = (rin && cI[e]) ? pf[u % P][e] : R(0);
          }
          load(row + DIR * P, pf[u % P]);
        }
#pragma unroll
        for (int k = 1; k <= K; ++k) {
          const int j = ifirst + DIR * (rr - k);  // row level k evaluates now
          constexpr int off = 3 * (K + 2);
          const int sOld = (u - k - 1 + off) % 3, sc = (u - k + off) % 3,
                    sNew = (u - k + 1 + off) % 3;
          const R* a = lv[k - 1][sc];
          const R* S = lv[k - 1][DIR > 0 ? sOld : sNew];
          const R* N = lv[k - 1][DIR > 0 ? sNew : sOld];
          const R wl = from_prev(a[V - 1]), er = from_next(a[0]);
          const bool rj = MODE != kGeneral || (j >= 1 && j <= ny - 2);  // uniform
          R o[V];
          if constexpr (!ADJ) {
#pragma unroll
            for (int e = 0; e < V; ++e) {
              const R Wn = e > 0 ? a[e > 0 ? e - 1 : 0] : wl;
              const R En = e < V - 1 ? a[e < V - 1 ? e + 1 : 0] : er;
              const R f = w * ((((a[e] + Wn) + En) + S[e]) + N[e]);
              if constexpr (MODE == kFast)
                o[e] = f;
              else
                o[e] = (cI[e] && rj) ? f : a[e];
            }
          } else {
            R sum[V], Ws[V], Es[V];
#pragma unroll
            for (int e = 0; e < V; ++e) {
              Ws[e] = e > 0 ? a[e > 0 ? e - 1 : 0] : wl;
              Es[e] = e < V - 1 ? a[e < V - 1 ? e + 1 : 0] : er;
              sum[e] = ((Ws[e] + Es[e]) + S[e]) + N[e];
            }
#pragma unroll
            for (int e = 0; e < V; ++e) {
              if constexpr (MODE == kFast)
                o[e] = w * (a[e] + sum[e]);
              else
                o[e] = (cI[e] && rj) ? w * (a[e] + sum[e]) : R(0);
            }
            if constexpr (MODE != kFast) {
              // record the ring cell's interior neighbour (E of column 0, W
              // of column nx-1) for rows of this chunk; other lanes write
              // their own scratch cell
              R nb;
              if constexpr (VEC) {
                nb = rside == 0 ? Es[0] : Ws[V - 1];
              } else {
                nb = R(0);
#pragma unroll
                for (int e = 0; e < V; ++e) nb = relem == e ? (rside == 0 ? Es[e] : Ws[e]) : nb;
              }
              nbr[has_ring ? nbr_lane + (k - 1) * NR + j : 2 * K * NR + lane] = nb;
            }
            if constexpr (MODE == kGeneral) {
#pragma unroll
              for (int e = 0; e < V; ++e) {
                ring_lo[e] = j == 0 ? (cok[e] ? ring_lo[e] + w * sum[e] : R(0)) : ring_lo[e];
                ring_hi[e] = j == ny - 1 ? (cok[e] ? ring_hi[e] + w * sum[e] : R(0)) : ring_hi[e];
              }
            }
          }
          if (k < K) {
#pragma unroll
            for (int e = 0; e < V; ++e) lv[k][sc][e] = o[e];
          } else if (j >= r0 && j < r1 && st_lane) {
            if constexpr (ADJ && MODE == kGeneral) {  // ring rows
#pragma unroll
              for (int e = 0; e < V; ++e)
                o[e] = j == 0 ? ring_lo[e] : (j == ny - 1 ? ring_hi[e] : o[e]);
            }
            R* dst = y + (int64_t)j * nx;
            if constexpr (VEC) {
              if (c0 + V <= nx) {
                vec_t t;
#pragma unroll
                for (int e = 0; e < V; ++e) t[e] = o[e];
                *reinterpret_cast<vec_t*>(dst + c0) = t;
              }
            } else {
#pragma unroll
              for (int e = 0; e < V; ++e)
                if (c0 + e < nx) dst[c0 + e] = o[e];
            }
          }
        }
      }
    };

    // A block of U input rows evaluates rows ifirst + DIR*[base - K, base + U - 1];
    // blocks [fa, fb) have all of them in [2, ny - 3].
    int fa, fb;
    if (DIR > 0) {
      fa = 2 + K - ifirst;
      fb = ny - 1 - ifirst - U;
    } else {
      fa = ifirst + K - (ny - 3);
      fb = ifirst - U;
    }
    fa = ((max(fa, 0) + U - 1) / U) * U;
    using General = std::integral_constant<int, kGeneral>;
    int base = 0;
    for (; base < nit && base < fa; base += U) block(base, General{});
    for (; base < nit && base < fb; base += U) block(base, mid_t);
    for (; base < nit; base += U) block(base, General{});
  };
  // Each combination gets its own straight code path, chosen before any
  // state is live.
  using Up = std::integral_constant<int, 1>;
  using Down = std::integral_constant<int, -1>;
  using Fast = std::integral_constant<int, kFast>;
  using Cols = std::integral_constant<int, ADJ ? kCols : kGeneral>;
  if (strip_in) {
    if (chunk & 1)
      march(Down{}, Fast{});
    else
      march(Up{}, Fast{});
    return;
  }
  if (chunk & 1)
    march(Down{}, Cols{});
  else
    march(Up{}, Cols{});
  if constexpr (ADJ) {
    // The ring columns of this chunk's interior rows, one row per lane:
    // g_n = g_0 + w*(((0 + E) + 0) + 0) level by level on the left,
    // g_0 + w*(((W + 0) + 0) + 0) on the right, E and W the recorded
    // neighbours. All earlier stores and LDS writes complete first.
    __builtin_amdgcn_s_waitcnt(0);
    asm volatile("" ::: "memory");
    const int jr = r0 + lane;
    if (lane < kRows && jr < r1 && jr >= 1 && jr <= ny - 2) {
#pragma unroll
      for (int sd = 0; sd < 2; ++sd) {
        const int col = sd == 0 ? 0 : nx - 1;
        if (col < s0 || col >= s0 + OW) continue;  // not this strip's output column
        const int64_t q = (int64_t)jr * nx + col;
        R g = x[q];
#pragma unroll
        for (int k = 0; k < K; ++k) {
          const R v = nbr[(sd * K + k) * NR + (K + U) + lane];
          const R sum = sd == 0 ? ((R(0) + v) + R(0)) + R(0) : ((v + R(0)) + R(0)) + R(0);
          g = g + w * sum;
        }
        y[q] = g;
      }
    }
  }
}

template <class R, int K, bool ADJ>
hipError_t march_launch(const StepShape& s, const R* x, R* y, hipStream_t st) {
  using G = Geom<R, K>;
  if (ADJ && s.nx <= G::V) return hipErrorInvalidValue;  // a lane would hold both ring columns
  MarchGrid g;
  int64_t blocks;
  if (!make_grid(s.nx, s.ny, G::OW, &g, &blocks))
    return hipErrorInvalidValue;
  const bool vec = s.nx % G::V == 0 && (reinterpret_cast<uintptr_t>(x) & 15u) == 0 &&
                   (reinterpret_cast<uintptr_t>(y) & 15u) == 0;
  if (vec)
    jacobi_march<R, K, ADJ, true><<<dim3((unsigned)blocks), dim3(kLanes), 0, st>>>(
        x, y, s.nx, s.ny, g, R(s.p0));
  else
    jacobi_march<R, K, ADJ, false><<<dim3((unsigned)blocks), dim3(kLanes), 0, st>>>(
        x, y, s.nx, s.ny, g, R(s.p0));
  return hipGetLastError();
}

// ------------------------------------------- the limiter's adjoint, fused
// One Jacobi adjoint step under the limiter: g_t is masked by the branch
// each point took at step t (its unlimited value re-evaluated from x_{t-1}
// with the forward's expression; 0 where it left [lo, hi]) and the masked g
// is transposed with the single-step adjoint's expressions, in one pass
// that reads x and g once and writes g' once. A wave marches down a strip
// carrying three rows of x, the g rows waiting for their mask and three
// masked g rows: when input row p arrives, row p-1 is masked (its x
// neighbourhood is complete) and row p-2 transposed. The mask reads x one
// column beyond the masked g, so strips overlap by V >= 2 columns.
// DP (instead of the mask): g passes unmasked and the pass adds this step's
// share of dL/dw, sum over interior points of g[c] * ((((x[c]+x[W])+x[E])
// +x[S])+x[N]) (the forward's sum, in double), over the work item's output
// points; a wave butterfly then adds it into the item's slot
// (dp_part[item], or overwrites it on the step t = T).
template <class R, bool VEC, bool DP>
__global__ __launch_bounds__(kLanes) void jacobi_lim_adjoint(const R* __restrict__ x,
                                                             const R* __restrict__ g,
                                                             R* __restrict__ gp, int nx, int ny,
                                                             MarchGrid grid, R w, R lo, R hi,
                                                             double* dp_part, int dp_first) {
  // six rows of each array in flight: the pass is lighter than the n-step
  // march and registers allow it
  constexpr int V = 16 / sizeof(R), H = V, OW = kLanes * V - 2 * H, P = 6, U = kUnroll;
  static_assert(H >= 2, "the mask reaches two columns beyond an output");
  static_assert(U % P == 0, "register slots must stay static");
  typedef R vec_t __attribute__((ext_vector_type(V)));
  int strip, chunk, r0, r1, item;
  if (!march_item(grid, ny, &strip, &chunk, &r0, &r1, &item)) return;
  const int lane = threadIdx.x;
  const int s0 = strip * OW;
  const int c0 = s0 - H + lane * V;
  const int nit = (r1 - r0) + 4;  // input rows r0-2 .. r1+1
  double a0 = 0.0;
  const int lo_need = max(r0 - 2, 0), hi_need = min(r1 + 1, ny - 1);
  auto cin = [&](int c) { return c >= 1 && c <= nx - 2; };
  bool cok[V], cI[V], cW[V], cE[V];
#pragma unroll
  for (int e = 0; e < V; ++e) {
    const int c = c0 + e;
    cok[e] = c >= 0 && c < nx;
    cI[e] = cin(c);
    cW[e] = cin(c - 1);
    cE[e] = cin(c + 1);
  }
  const bool strip_in = s0 - H >= 2 && s0 - H + kLanes * V <= nx - 2;
  const bool st_lane = lane * V >= H && lane * V < H + OW;
  // x and g are read once per step, with the non-temporal hint (4096^2
  // f64: 90.5 -> 83.5 us per step; the hint on x alone did nothing)
  auto load = [&](const R* a, int row, R* out) {
    const int rr = min(max(row, lo_need), hi_need);
    const R* src = a + (int64_t)rr * nx;
    if constexpr (VEC) {
      const int cc = min(max(c0, 0), nx - V);
      const vec_t t = __builtin_nontemporal_load(reinterpret_cast<const vec_t*>(src + cc));
#pragma unroll
      for (int e = 0; e < V; ++e) out[e] = t[e];
    } else {
#pragma unroll
      for (int e = 0; e < V; ++e) out[e] = src[min(max(c0 + e, 0), nx - 1)];
    }
  };
  enum { kFast = 0, kGeneral = 2 };
  auto march = [&](auto dir_t, auto mid_t) {
    constexpr int DIR = decltype(dir_t)::value;
    const int ifirst = DIR > 0 ? r0 - 2 : r1 + 1;  // row of input index 0
    // slot p mod 3 holds pipeline index p (row ifirst + DIR*p)
    R xw[3][V], gr[3][V], mg[3][V];
    R px[P][V], pg[P][V];
#pragma unroll
    for (int s3 = 0; s3 < 3; ++s3)
#pragma unroll
      for (int e = 0; e < V; ++e) xw[s3][e] = gr[s3][e] = mg[s3][e] = R(0);
#pragma unroll
    for (int u = 0; u < P; ++u) {
      load(x, ifirst + DIR * u, px[u]);
      load(g, ifirst + DIR * u, pg[u]);
    }
    auto block = [&](int base, auto mode_t) {
      constexpr int MODE = decltype(mode_t)::value;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int rr = base + u;
        {  // input row rr enters; the rows P ahead are requested
          const int row = ifirst + DIR * rr;
          const bool rok = row >= 0 && row < ny;
#pragma unroll
          for (int e = 0; e < V; ++e) {
            const bool ok = MODE == kFast || (rok && cok[e]);
            xw[u % 3][e] = ok ? px[u % P][e] : R(0);
            gr[u % 3][e] = ok ? pg[u % P][e] : R(0);
          }
          load(x, row + DIR * P, px[u % P]);
          load(g, row + DIR * P, pg[u % P]);
        }
        {  // mask row index rr-1 from x rows rr-2 .. rr
          const int m = ifirst + DIR * (rr - 1);
          constexpr int off = 6;
          const int sOld = (u - 2 + off) % 3, sc = (u - 1 + off) % 3, sNew = u % 3;
          const R* a = xw[sc];
          const R* S = xw[DIR > 0 ? sOld : sNew];
          const R* N = xw[DIR > 0 ? sNew : sOld];
          const R wl = from_prev(a[V - 1]), er = from_next(a[0]);
          const bool rm = m >= 1 && m <= ny - 2;
          const bool own = m >= r0 && m < r1 && st_lane;  // this item's output row
#pragma unroll
          for (int e = 0; e < V; ++e) {
            const R Wn = e > 0 ? a[e > 0 ? e - 1 : 0] : wl;
            const R En = e < V - 1 ? a[e < V - 1 ? e + 1 : 0] : er;
            const R sum = (((a[e] + Wn) + En) + S[e]) + N[e];
            if constexpr (DP) {
              mg[sc][e] = gr[sc][e];
              if ((MODE == kFast || (cI[e] && rm)) && own)
                a0 += (double)gr[sc][e] * (double)sum;
            } else {
              const R yv = (MODE == kFast || (cI[e] && rm)) ? w * sum : a[e];
              mg[sc][e] = (yv < lo || yv > hi) ? R(0) : gr[sc][e];
            }
          }
        }
        {  // transpose row index rr-2 from masked rows rr-3 .. rr-1
          const int j = ifirst + DIR * (rr - 2);
          constexpr int off = 6;
          const int sOld = (u - 3 + off) % 3, sc = (u - 2 + off) % 3, sNew = (u - 1 + off) % 3;
          const R* a = mg[sc];
          const R* S = mg[DIR > 0 ? sOld : sNew];
          const R* N = mg[DIR > 0 ? sNew : sOld];
          const R wl = from_prev(a[V - 1]), er = from_next(a[0]);
          const bool rj = j >= 1 && j <= ny - 2, rS = j >= 2 && j <= ny - 1,
                     rN = j >= 0 && j <= ny - 3;
          R o[V];
#pragma unroll
          for (int e = 0; e < V; ++e) {
            const R Wn = e > 0 ? a[e > 0 ? e - 1 : 0] : wl;
            const R En = e < V - 1 ? a[e < V - 1 ? e + 1 : 0] : er;
            if constexpr (MODE == kFast) {
              o[e] = w * (a[e] + (((Wn + En) + S[e]) + N[e]));
            } else {
              R sum = (cW[e] && rj) ? Wn : R(0);
              sum += (cE[e] && rj) ? En : R(0);
              sum += (cI[e] && rS) ? S[e] : R(0);
              sum += (cI[e] && rN) ? N[e] : R(0);
              o[e] = (cI[e] && rj) ? w * (a[e] + sum) : a[e] + w * sum;
            }
          }
          if (j >= r0 && j < r1 && st_lane) {
            R* dst = gp + (int64_t)j * nx;
            if constexpr (VEC) {
              if (c0 + V <= nx) {
                vec_t t;
#pragma unroll
                for (int e = 0; e < V; ++e) t[e] = o[e];
                *reinterpret_cast<vec_t*>(dst + c0) = t;
              }
            } else {
#pragma unroll
              for (int e = 0; e < V; ++e)
                if (c0 + e < nx) dst[c0 + e] = o[e];
            }
          }
        }
      }
    };
    // A block of U input rows touches rows ifirst + DIR*[base - 4, base + U - 1];
    // blocks [fa, fb) have all of them in [2, ny - 3].
    constexpr int R4 = 4;
    int fa, fb;
    if (DIR > 0) {
      fa = 2 + R4 - ifirst;
      fb = ny - 1 - ifirst - U;
    } else {
      fa = ifirst + R4 - (ny - 3);
      fb = ifirst - U;
    }
    fa = ((max(fa, 0) + U - 1) / U) * U;
    using General = std::integral_constant<int, kGeneral>;
    int base = 0;
    for (; base < nit && base < fa; base += U) block(base, General{});
    for (; base < nit && base < fb; base += U) block(base, mid_t);
    for (; base < nit; base += U) block(base, General{});
  };
  using Up = std::integral_constant<int, 1>;
  using Down = std::integral_constant<int, -1>;
  using Fast = std::integral_constant<int, kFast>;
  using General = std::integral_constant<int, kGeneral>;
  if (strip_in) {
    if (chunk & 1)
      march(Down{}, Fast{});
    else
      march(Up{}, Fast{});
  } else {
    if (chunk & 1)
      march(Down{}, General{});
    else
      march(Up{}, General{});
  }
  if constexpr (DP) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) a0 += __shfl_xor(a0, off, kLanes);
    if (lane == 0) dp_part[item] = dp_first ? a0 : dp_part[item] + a0;
  }
}

// One pass reading x and g: the limiter's masked adjoint (dp_part null) or
// the adjoint with dL/dw's share (dp_part: jacobi_x_adjoint_slots doubles).
template <class R>
hipError_t lim_adjoint_launch(const StepShape& s, const R* x, const R* g, R* gp,
                              double* dp_part, bool dp_first, hipStream_t st) {
  constexpr int V = 16 / sizeof(R), OW = kLanes * V - 2 * V;
  MarchGrid grid;
  int64_t blocks;
  if (!make_grid(s.nx, s.ny, OW, &grid, &blocks, kLimRows)) return hipErrorInvalidValue;
  const bool vec = s.nx % V == 0 && (reinterpret_cast<uintptr_t>(x) & 15u) == 0 &&
                   (reinterpret_cast<uintptr_t>(g) & 15u) == 0 &&
                   (reinterpret_cast<uintptr_t>(gp) & 15u) == 0;
  const dim3 gr((unsigned)blocks), bl(kLanes);
  const R w = R(s.p0), lo = R(s.lo), hi = R(s.hi);
  const int first = dp_first ? 1 : 0;
  if (dp_part && vec)
    jacobi_lim_adjoint<R, true, true><<<gr, bl, 0, st>>>(x, g, gp, s.nx, s.ny, grid, w, lo, hi,
                                                         dp_part, first);
  else if (dp_part)
    jacobi_lim_adjoint<R, false, true><<<gr, bl, 0, st>>>(x, g, gp, s.nx, s.ny, grid, w, lo, hi,
                                                          dp_part, first);
  else if (vec)
    jacobi_lim_adjoint<R, true, false><<<gr, bl, 0, st>>>(x, g, gp, s.nx, s.ny, grid, w, lo, hi,
                                                          nullptr, 0);
  else
    jacobi_lim_adjoint<R, false, false><<<gr, bl, 0, st>>>(x, g, gp, s.nx, s.ny, grid, w, lo,
                                                           hi, nullptr, 0);
  return hipGetLastError();
}

template <class R, bool ADJ>
hipError_t march_n(const StepShape& s, const void* xv, void* yv, int n, hipStream_t st) {
  const R* x = static_cast<const R*>(xv);
  R* y = static_cast<R*>(yv);
  switch (n) {
    case 3: return march_launch<R, 3, ADJ>(s, x, y, st);
    case 4: return march_launch<R, 4, ADJ>(s, x, y, st);
    case 5: return march_launch<R, 5, ADJ>(s, x, y, st);
    case 6: return march_launch<R, 6, ADJ>(s, x, y, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_jacobi_lim_adjoint(const StepShape& s, const void* x, const void* g, void* gp,
                                     hipStream_t stream) {
  if (s.kind != ADST_JACOBI2D5 || !s.limit || !x) return hipErrorInvalidValue;
  if (s.dtype == ADST_F64)
    return lim_adjoint_launch<double>(s, static_cast<const double*>(x),
                                      static_cast<const double*>(g), static_cast<double*>(gp),
                                      nullptr, false, stream);
  return lim_adjoint_launch<float>(s, static_cast<const float*>(x), static_cast<const float*>(g),
                                   static_cast<float*>(gp), nullptr, false, stream);
}

hipError_t launch_jacobi_dp_adjoint(const StepShape& s, const void* x, const void* g, void* gp,
                                    double* dp_part, bool dp_first, hipStream_t stream) {
  if (s.kind != ADST_JACOBI2D5 || !x || !dp_part) return hipErrorInvalidValue;
  if (s.dtype == ADST_F64)
    return lim_adjoint_launch<double>(s, static_cast<const double*>(x),
                                      static_cast<const double*>(g), static_cast<double*>(gp),
                                      dp_part, dp_first, stream);
  return lim_adjoint_launch<float>(s, static_cast<const float*>(x), static_cast<const float*>(g),
                                   static_cast<float*>(gp), dp_part, dp_first, stream);
}

int64_t jacobi_x_adjoint_slots(const StepShape& s) {
  const int V = s.dtype == ADST_F64 ? 2 : 4, OW = kLanes * V - 2 * V;  // as lim_adjoint_launch
  MarchGrid g;
  int64_t blocks;
  if (!make_grid(s.nx, s.ny, OW, &g, &blocks, kLimRows)) return 0;
  return int64_t(g.nedge) * g.ce + int64_t(g.ns - g.nedge) * g.ci;
}

hipError_t launch_jacobi_march(const StepShape& s, const void* x, void* y, int32_t n, bool adjoint,
                               hipStream_t stream) {
  if (s.kind != ADST_JACOBI2D5 || n < 3 || n > kJacMaxFuse) return hipErrorInvalidValue;
  if (s.dtype == ADST_F64)
    return adjoint ? march_n<double, true>(s, x, y, n, stream)
                   : march_n<double, false>(s, x, y, n, stream);
  return adjoint ? march_n<float, true>(s, x, y, n, stream)
                 : march_n<float, false>(s, x, y, n, stream);
}

}  // namespace adst
