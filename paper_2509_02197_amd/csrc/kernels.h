// Launchers of the gfx950 kernels. Plain host signatures: device pointers,
// sizes, the caller's stream. Every launcher only enqueues and returns the
// launch status (hipGetLastError after the launch).
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstdint>

namespace adst {

struct StepShape {
  int32_t kind;   // adst_kind
  int32_t dtype;  // adst_dtype
  int32_t nx, ny, nz;
  double p0, p1;
  int32_t limit;  // 1: every new value is clamped to [lo, hi] (a per-point branch)
  double lo, hi;
};

// x_t = F(x_{t-1}; K): x -> y. K only for the variable-coefficient kind.
hipError_t launch_forward(const StepShape& s, const void* x, const void* K, void* y,
                          hipStream_t stream);

// Allen-Cahn launchers (allencahn.hip): one forward step; n = 2..kAcMaxFuse
// fused forward steps (mids: the intermediate states' buffers for a
// store-through run, else null); one adjoint step with the constants'
// gradients (dp_part, per-workgroup slots) or the limiter's mask.
hipError_t ac_launch_forward(const StepShape& s, const void* x, void* y, hipStream_t st);
hipError_t ac_launch_forward_steps(const StepShape& s, const void* x, void* y, void* const* mids,
                                   int32_t n, hipStream_t st);
hipError_t ac_launch_adjoint(const StepShape& s, const void* x, const void* g, void* gp,
                             double* dp_part, bool dp_first, hipStream_t st);
int64_t ac_dparam_slots(const StepShape& s);
// n = 1 .. kAcMaxFuse recomputed forward steps and the adjoint step that
// reads their result, in one launch: g_prev = J_t^T g_next with x_{t-1} =
// F^n(x) formed on chip and never stored (x = x_{t-1-n}); no limiter and no
// constants' gradients. ac_fuses_forward_adjoint tells whether the shape
// takes it.
hipError_t ac_launch_forward_adjoint(const StepShape& s, const void* x, const void* g, void* gp,
                                     int32_t n, hipStream_t st);
bool ac_fuses_forward_adjoint(const StepShape& s);

// Temporal blocking: the most steps one launch may take (1 = none). The
// fused adjoint is for state-free adjoints only.
constexpr int32_t kJacMaxFuse = 6;
constexpr int32_t kAcMaxFuse = 3;
int32_t max_fused_forward(int32_t kind);
int32_t max_fused_adjoint(int32_t kind, int64_t nx);

// x_t = F^n(x_{t-n}) in one launch (2 <= n <= max_fused_forward), the
// intermediate states kept on chip.
hipError_t launch_forward_n(const StepShape& s, const void* x, const void* K, void* y, int32_t n,
                            hipStream_t stream);

// A run of n single steps whose every state is kept (2 <= n <=
// max_stored_forward): x_{t-n+1+k} = F^{k+1}(x_{t-n}) into ys[k] for
// k = 0 .. n-1, in one launch that reads x once and writes each state once.
// The ys are distinct and none overlaps x. Allen-Cahn and the
// variable-coefficient kind only, without the limiter.
constexpr int32_t kMaxStoredRun = kAcMaxFuse;
int32_t max_stored_forward(int32_t kind);
hipError_t launch_forward_store(const StepShape& s, const void* x, const void* K, void* const* ys,
                                int32_t n, hipStream_t stream);

// g_{t-n} = J_{t-n+1}^T ... J_t^T g_t in one launch, state-free adjoints.
hipError_t launch_adjoint_n(const StepShape& s, const void* g_next, void* g_prev, int32_t n,
                            hipStream_t stream);

// Jacobi only, 3 <= n <= kJacMaxFuse: n forward steps (adjoint = false) or
// n adjoint steps in one launch (jacobi_march.hip).
hipError_t launch_jacobi_march(const StepShape& s, const void* x, void* y, int32_t n, bool adjoint,
                               hipStream_t stream);

// Jacobi under the limiter: one adjoint step with the branch mask of step t
// (from x = x_{t-1}) applied on the fly, g_prev = J_t^T (mask_t * g_next),
// in one pass (jacobi_march.hip).
hipError_t launch_jacobi_lim_adjoint(const StepShape& s, const void* x, const void* g_next,
                                     void* g_prev, hipStream_t stream);

// Jacobi: one adjoint step and its share of dL/dw in the same one-pass
// layout, into jacobi_x_adjoint_slots(s) per-work-item slots of dp_part
// (overwritten when dp_first, else added to).
hipError_t launch_jacobi_dp_adjoint(const StepShape& s, const void* x, const void* g_next,
                                    void* g_prev, double* dp_part, bool dp_first,
                                    hipStream_t stream);
int64_t jacobi_x_adjoint_slots(const StepShape& s);

// g_prev = J_t^T g_next with x = x_{t-1} (may be null when the kind's adjoint
// reads no state and neither dK nor the constants' gradients are asked for).
// dK (nullable) is accumulated: dK = (dk_first ? 0 : dK) + contribution of
// step t. dp_part (nullable; dparam_partial_bytes(s) bytes) receives step
// t's share of the constants' gradients: sum_c g_t[c] dF_c/dp (x = x_{t-1}),
// added per workgroup into its slot (dp_first = the step t = T, which
// overwrites the slots).
hipError_t launch_adjoint(const StepShape& s, const void* x, const void* K, const void* g_next,
                          void* g_prev, void* dK, bool dk_first, double* dp_part, bool dp_first,
                          hipStream_t stream);

// With the limiter on, whether launch_adjoint applies the branch mask itself
// (reading x = x_{t-1}; Jacobi and Allen-Cahn without the constants'
// gradients); otherwise launch_limit_mask must run first.
bool adjoint_applies_limit(const StepShape& s, bool dparams);

// Number of per-block loss partials launch_seed writes for n points.
int32_t seed_partials(int64_t n);
constexpr int32_t kMaxSeedPartials = 1024;

// Loss partials and seed g from x_T (x and g may be the same buffer: the
// kernel reads each point before writing it). xcopy (nullable) receives x.
hipError_t launch_seed(int32_t dtype, int32_t loss, int64_t n, const void* x, const void* aux,
                       void* g, void* xcopy, double* partials, hipStream_t stream);

// Sum the partials in a fixed order into *loss (one block).
hipError_t launch_finalize(const double* partials, int32_t nparts, double* loss,
                           hipStream_t stream);

// In-place Gauss-Seidel kind: `sweeps` forward sweeps from src into dst
// (src may equal dst), and `sweeps` reverse sweeps applied to g in place.
// Each call is a sequence of wavefront launches (gs_kernel_launches of them)
// that pipelines the sweeps.
hipError_t launch_gs_forward(const StepShape& s, const void* src, void* dst, int32_t sweeps,
                             hipStream_t stream);
hipError_t launch_gs_adjoint(const StepShape& s, void* g, int32_t sweeps, hipStream_t stream);
int64_t gs_kernel_launches(const StepShape& s, bool adjoint, int32_t sweeps);

// The limiter's branch outcome at step t: g[c] = 0 wherever the step's
// unlimited value at c (re-evaluated from x = x_{t-1} with the forward's own
// expressions) lies outside [lo, hi]; g is updated in place.
hipError_t launch_limit_mask(const StepShape& s, const void* x, const void* K, void* g,
                             hipStream_t stream);

// Gradients of the step constants: the adjoint launches add their steps'
// shares into per-workgroup slots (launch_adjoint's dp_part; one slot per
// adjoint tile and constant); finalize sums the slots in a fixed order into
// dparams[0..1] (device doubles).
int64_t dparam_slots(const StepShape& s);
int64_t dparam_partial_bytes(const StepShape& s);
hipError_t launch_dparam_finalize(const StepShape& s, const double* partials, double* dparams,
                                  hipStream_t stream);

hipError_t launch_fill_zero(void* p, int64_t bytes, hipStream_t stream);
hipError_t launch_copy(void* dst, const void* src, int64_t bytes, hipStream_t stream);

// The static workspace of adst_vjp_static_ws: kStaticWsBytes of device memory
// per GPU, held from the library's first use on that GPU to the end of the
// process. static_workspace() returns the current device's address of it
// (looked up once per device; no allocation).
constexpr uint64_t kStaticWsBytes = uint64_t(64) << 20;
hipError_t static_workspace(void** ptr);

}  // namespace adst
