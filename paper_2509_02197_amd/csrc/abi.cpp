// C-ABI of adst: argument validation, workspace layout, and the executor that
// interprets a plan's action list by enqueueing kernels on the caller's
// stream. All arguments are checked before the first HIP call, so every
// argument error is reported without touching the GPU.

#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <string>
#include <utility>
#include <vector>

#include <rocprofiler-sdk-roctx/roctx.h>

#include "adst.h"
#include "kernels.h"
#include "ilp.h"
#include "planner.h"

namespace adst {


namespace {

thread_local std::string g_last_error;

adst_status fail(adst_status st, const std::string& msg) {
  g_last_error = msg;
  return st;
}

constexpr uint64_t kAlign = 4096;
constexpr uint64_t kHeaderBytes = 16384;  // loss partials (8 KiB) + loss scalar
constexpr uint64_t kLossOffset = 8192;

uint64_t align_up(uint64_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

int itemsize(int32_t dtype) { return dtype == ADST_F64 ? 8 : 4; }

struct Checked {
  StepShape shape;
  int64_t npoints = 0;
  uint64_t state_bytes = 0;
  bool needs_state = false;
  bool trace = false;
  int32_t fuse_fwd = 1, fuse_adj = 1;  // most steps per launch
  int32_t store_fwd = 1;  // most single steps per launch that stores every state
  bool fuse_adj_fwd = false;  // a recomputed step may share the adjoint's launch
  bool pair_tail = false;     // build_plan's pair_tail
  bool in_place = false;  // the Gauss-Seidel kind: pipelined sweeps, adjoint in place
  bool want_dk = false, want_dp = false;
};

adst_status check_problem(const adst_problem* p, int32_t grads, Checked* out) {
  if (!p) return fail(ADST_ERR_ARG, "problem is NULL");
  if (p->kind < ADST_JACOBI2D5 || p->kind > ADST_GAUSSSEIDEL2D5)
    return fail(ADST_ERR_ARG, "unknown kind " + std::to_string(p->kind));
  if (p->dtype != ADST_F64 && p->dtype != ADST_F32)
    return fail(ADST_ERR_ARG, "unknown dtype " + std::to_string(p->dtype));
  if (p->flags & ~(ADST_FORCE_TAPE | ADST_TRACE | ADST_NO_FUSE | ADST_LIMIT))
    return fail(ADST_ERR_ARG, "unknown flag bits");
  const bool limit = (p->flags & ADST_LIMIT) != 0;
  if (limit && !(p->lim[0] <= p->lim[1]))
    return fail(ADST_ERR_ARG, "limiter bounds must satisfy lim[0] <= lim[1]");
  if (limit && p->kind == ADST_GAUSSSEIDEL2D5)
    return fail(ADST_ERR_UNSUPPORTED, "the limiter is not built for the in-place kind");
  for (int d = 0; d < 3; ++d)
    if (p->n[d] < 1) return fail(ADST_ERR_ARG, "every extent n[i] must be >= 1");
  if (p->n[0] > INT32_MAX || p->n[1] > INT32_MAX || p->n[2] > INT32_MAX)
    return fail(ADST_ERR_ARG, "extent too large");
  const int64_t n = p->n[0] * p->n[1] * p->n[2];
  if (n >= (int64_t(1) << 31)) return fail(ADST_ERR_ARG, "grid must have fewer than 2^31 points");
  if (p->kind != ADST_ALLENCAHN3D7 && p->n[2] != 1)
    return fail(ADST_ERR_UNSUPPORTED, "this kind is 2-D: n[2] must be 1");
  // Every launch covers the grid with workgroups of 256 work-items: tiles of
  // 240 to 256 columns by 4 or 8 rows for the 2-D kinds, columns of 56 to 64
  // by 8 to 16 points over 32 to 256 planes for the 3-D kind. The work-item
  // count of the smallest tiles must fit the 32-bit dispatch grid.
  const int64_t tiles =
      p->kind == ADST_ALLENCAHN3D7
          ? ((p->n[0] + 55) / 56) * ((p->n[1] + 7) / 8) * ((p->n[2] + 31) / 32)
          : ((p->n[0] + 239) / 240) * ((p->n[1] + 3) / 4);
  if ((tiles + 8) * 256 >= (int64_t(1) << 32))
    return fail(ADST_ERR_UNSUPPORTED, "grid too thin in x/y for the tile shape");
  if (grads & ~(ADST_GRAD_COEFF | ADST_GRAD_PARAMS))
    return fail(ADST_ERR_ARG, "unknown gradient bits");
  const bool want_dk = (grads & ADST_GRAD_COEFF) != 0;
  const bool want_dp = (grads & ADST_GRAD_PARAMS) != 0;
  if (want_dk && p->kind != ADST_VARDIFF2D9)
    return fail(ADST_ERR_UNSUPPORTED, "only the variable-coefficient kind has a coefficient field");
  if (want_dp && p->kind == ADST_GAUSSSEIDEL2D5)
    return fail(ADST_ERR_UNSUPPORTED,
                "the constants' gradients are not built for the in-place kind");
  out->shape = {p->kind, p->dtype, (int32_t)p->n[0], (int32_t)p->n[1], (int32_t)p->n[2],
                p->p[0], p->p[1], limit ? 1 : 0, p->lim[0], p->lim[1]};
  out->npoints = n;
  out->state_bytes = uint64_t(n) * itemsize(p->dtype);
  const bool kind_reads_state = p->kind == ADST_ALLENCAHN3D7 ||
                                (p->kind == ADST_VARDIFF2D9 && want_dk) || want_dp || limit;
  out->needs_state = kind_reads_state || (p->flags & ADST_FORCE_TAPE);
  out->want_dk = want_dk;
  out->want_dp = want_dp;
  out->trace = (p->flags & ADST_TRACE) != 0;
  const bool fuse = (p->flags & ADST_NO_FUSE) == 0;
  out->fuse_fwd = (fuse && !limit) ? max_fused_forward(p->kind) : 1;
  out->fuse_adj = fuse ? max_fused_adjoint(p->kind, p->n[0]) : 1;
  out->in_place = p->kind == ADST_GAUSSSEIDEL2D5;
  out->store_fwd = (fuse && !limit) ? max_stored_forward(p->kind) : 1;
  out->fuse_adj_fwd = fuse && p->kind == ADST_ALLENCAHN3D7 && ac_fuses_forward_adjoint(out->shape);
  // Allen-Cahn: two 2-step launches take less time than a 3-step launch and
  // a single step (at 1024^3 f64: 3.7 + 3.7 against 4.5 + 3.3 ms).
  out->pair_tail = out->fuse_fwd == 3 && p->kind == ADST_ALLENCAHN3D7;
  return ADST_OK;
}

// A forward action (one step, or a fused run of up to three) whose result
// only the next action, the adjoint step that reads it as x_{t-1}, uses: the
// two run as one launch (ac_launch_forward_adjoint), x_{t-1} formed on chip
// and never written. True when acts[i] is that forward action: the kind's adjoint reads x_{t-1} only pointwise
// (Allen-Cahn without the limiter or the constants' gradients), and no later
// action reads the buffer before it is written again.
bool fused_fwd_adj(const Checked& c, const std::vector<adst_action>& acts, size_t i) {
  if (c.shape.kind != ADST_ALLENCAHN3D7 || c.want_dp || c.shape.limit || !c.fuse_adj_fwd)
    return false;
  if (i + 1 >= acts.size()) return false;
  const adst_action& f = acts[i];
  const adst_action& g = acts[i + 1];
  const bool fwd = (f.op == ADST_OP_FWD && f.n == 1) ||
                   (f.op == ADST_OP_FWD2 && f.n >= 2 && f.n <= kAcMaxFuse);
  if (!fwd || g.op != ADST_OP_ADJ || g.src != f.dst || g.t != f.t + 1 || f.dst == f.src)
    return false;
  for (size_t k = i + 2; k < acts.size(); ++k) {
    const adst_action& a = acts[k];
    const bool reads = (a.op == ADST_OP_FWD || a.op == ADST_OP_FWD2 || a.op == ADST_OP_FWDW ||
                        a.op == ADST_OP_ADJ || a.op == ADST_OP_SEED) && a.src == f.dst;
    if (reads) return false;
    const bool writes = (a.op == ADST_OP_FWD || a.op == ADST_OP_FWD2 || a.op == ADST_OP_FWDW) &&
                        a.dst == f.dst;
    if (writes) break;
  }
  return true;
}

// Length of the run of single forward steps starting at acts[i] that one
// store-through launch takes (1: none): each action reads the state the one
// before it wrote, and the states go to buffers that differ from each other
// and from the run's input (which the launch reads while it writes them).
// A step fused with the adjoint after it ends the run before it.
int32_t stored_run(const Checked& c, const std::vector<adst_action>& acts, size_t i) {
  const int32_t depth = c.store_fwd;
  if (depth < 2 || acts[i].op != ADST_OP_FWD || fused_fwd_adj(c, acts, i)) return 1;
  int32_t n = 1;
  while (n < depth && i + n < acts.size()) {
    const adst_action& a = acts[i + n];
    const adst_action& p = acts[i + n - 1];
    if (a.op != ADST_OP_FWD || a.src != p.dst || a.t != p.t + 1) break;
    if (fused_fwd_adj(c, acts, i + n)) break;
    bool clash = a.dst == acts[i].src;
    for (int32_t k = 0; k < n; ++k) clash = clash || acts[i + k].dst == a.dst;
    if (clash) break;
    ++n;
  }
  return n;
}

struct Layout {
  uint64_t state_stride = 0;  // aligned bytes per state buffer
  uint64_t w0 = 0, w1 = 0, g = 0, slot0 = 0, dp = 0, total = 0;
};

// Header, two work states, the second adjoint buffer G, then the slots. The
// in-place kind keeps its gradient in dx0 (no G) and needs the work states
// only for a forced tape: its pipelined plan runs x0 -> x_T directly.
Layout layout_for(const Checked& c, const Plan& plan) {
  Layout L;
  L.state_stride = align_up(c.state_bytes);
  if (plan.steps == 0) {
    L.total = kHeaderBytes;
    return L;
  }
  const uint64_t nwork = (c.in_place && !plan.needs_state) ? 0 : 2;
  L.w0 = kHeaderBytes;
  L.w1 = L.w0 + (nwork ? L.state_stride : 0);
  L.g = L.w1 + (nwork ? L.state_stride : 0);
  L.slot0 = L.g + (c.in_place ? 0 : L.state_stride);
  L.total = L.slot0 + uint64_t(plan.slots) * L.state_stride;
  if (c.want_dp) {  // per-block slots of the constants' gradients
    L.dp = L.total;
    L.total += align_up(uint64_t(dparam_partial_bytes(c.shape)));
  }
  return L;
}

// Algorithmic HBM bytes per point of one forward / adjoint step and of the
// seed: what the step must read and write at least once.
struct PerPoint {
  uint64_t fwd = 0, adj = 0, adj_first = 0, seed = 0;
  uint64_t adj_extra = 0;  // reads the adjoint launch adds for the constants or the limiter
  uint64_t mask = 0;       // the limiter's separate mask pass, where the adjoint does not apply it
};

PerPoint per_point_bytes(const Checked& c, bool want_dk, int32_t loss) {
  PerPoint b;
  const uint64_t s = itemsize(c.shape.dtype);
  switch (c.shape.kind) {
    case ADST_JACOBI2D5:
    case ADST_GAUSSSEIDEL2D5:  // in place: read and write each point once per step
      b.fwd = 2 * s;
      b.adj = b.adj_first = 2 * s;
      break;
    case ADST_ALLENCAHN3D7:
      b.fwd = 2 * s;
      b.adj = b.adj_first = 3 * s;  // g, x, g'
      break;
    default:                        // VARDIFF2D9
      b.fwd = 3 * s;                // x, K, x'
      b.adj = want_dk ? 6 * s : 3 * s;  // g, x, K, dK read+write, g'  |  g, K, g'
      b.adj_first = want_dk ? 5 * s : 3 * s;
      break;
  }
  b.seed = (loss == ADST_LOSS_HALF_SQ ? 2 : 3) * s;
  // the constants' gradients, fused into the adjoint, add the reads of
  // x_{t-1} the adjoint does not already make
  if (c.want_dp && (c.shape.kind == ADST_JACOBI2D5 || (c.shape.kind == ADST_VARDIFF2D9 && !want_dk)))
    b.adj_extra = s;
  // the limiter's branch mask reads x_{t-1} (and K) and updates g_t in place
  // in a pass of its own; where the adjoint applies it, it only adds the
  // read of x_{t-1} an adjoint without state does not make
  if (c.shape.limit) {
    if (!adjoint_applies_limit(c.shape, c.want_dp))
      b.mask = (c.shape.kind == ADST_VARDIFF2D9 ? 4 : 3) * s;
    else if (c.shape.kind == ADST_JACOBI2D5)
      b.adj_extra += s;
  }
  return b;
}

// Short name of the kernel an action launches, as a profiler reports its
// base name (template arguments that select the kernel's variant are
// written out where the variants differ in the bytes they move).
std::string kernel_label(const Checked& c, const adst_action& a, int32_t stored, bool dparams) {
  const int32_t k = c.shape.kind;
  const bool adj = a.op == ADST_OP_ADJ || a.op == ADST_OP_ADJ2 || a.op == ADST_OP_ADJW;
  if (k == ADST_GAUSSSEIDEL2D5) return adj ? "gs_wave<adj>" : "gs_wave<fwd>";
  static const char* const kFwd[3] = {"fwd_jacobi2d5", "fwd_allencahn3d7", "fwd_vardiff2d9"};
  static const char* const kAdj[3] = {"adj_jacobi2d5", "adj_allencahn3d7", "adj_vardiff2d9"};
  const bool march = k == ADST_ALLENCAHN3D7 && !c.shape.limit && ac_fuses_forward_adjoint(c.shape);
  if (march && adj && a.n == 1 && !dparams) return "ac_march<adj>";
  if (!adj) {
    if (stored >= 2)
      return k == ADST_ALLENCAHN3D7
                 ? "fwd_allencahn3d7_n<" + std::to_string(stored) + ",store>"
                 : std::string(kFwd[k]) + "_x2<store>";
    if (a.n <= 1) return c.shape.limit ? std::string(kFwd[k]) + "<lim>" : std::string(kFwd[k]);
    if (k == ADST_ALLENCAHN3D7) return "fwd_allencahn3d7_n<" + std::to_string(a.n) + ">";
    if (a.n == 2) return std::string(kFwd[k]) + "_x2";
    return "jacobi_march<fwd," + std::to_string(a.n) + ">";
  }
  if (a.n >= 3) return "jacobi_march<adj," + std::to_string(a.n) + ">";
  if (a.n == 2) return std::string(kAdj[k]) + "_x2";
  if (k == ADST_JACOBI2D5 && dparams) return "jacobi_lim_adjoint<dp>";
  if (k == ADST_JACOBI2D5 && adjoint_applies_limit(c.shape, dparams)) return "jacobi_lim_adjoint";
  if (k == ADST_ALLENCAHN3D7 && adjoint_applies_limit(c.shape, dparams))
    return "adj_allencahn3d7_lim";
  std::string n = kAdj[k];
  if (k == ADST_VARDIFF2D9 && c.want_dk) n += dparams ? "<dK,dp>" : "<dK>";
  else if (dparams) n += "<dp>";
  return n;
}

// For the dot-product and explicit-seed losses g_T is loss_aux itself: the
// first adjoint launch reads it there, and the loss pass reads x_T and
// loss_aux and writes no g_T. The in-place kind reverses in dx0 itself and
// the limiter's separate mask pass rewrites g_t in place, so both keep the
// copy, as does a call of zero steps (dx0 = g_T).
bool seed_in_aux(const Checked& c, int32_t loss, int32_t steps) {
  return (loss == ADST_LOSS_DOT_W || loss == ADST_LOSS_SEED) && steps > 0 && !c.in_place &&
         !(c.shape.limit && !adjoint_applies_limit(c.shape, c.want_dp));
}

void fill_info(const Checked& c, const Plan& plan, uint64_t budget, bool want_dk, int32_t loss,
               adst_plan_info* info) {
  const Layout L = layout_for(c, plan);
  const PerPoint pp = per_point_bytes(c, want_dk, loss);
  const uint64_t sb = seed_in_aux(c, loss, plan.steps) ? 2 * itemsize(c.shape.dtype) : pp.seed;
  const uint64_t fb = pp.fwd, ab = pp.adj, ab1 = pp.adj_first, db = pp.adj_extra + pp.mask;
  *info = adst_plan_info{};
  info->steps = plan.steps;
  info->sched = plan.sched;
  info->slots = plan.slots;
  info->needs_state = plan.needs_state ? 1 : 0;
  info->fwd_steps_total = plan.fwd_total;
  info->recompute_steps = plan.fwd_total - plan.steps;
  info->adj_steps = plan.adj_total;
  info->n_actions = (int64_t)plan.acts.size();
  info->fwd_launches = plan.fwd_launches;
  info->adj_launches = plan.adj_launches;
  for (size_t i = 0; i < plan.acts.size(); ++i) {
    const adst_action& a = plan.acts[i];
    const bool fwd_op = a.op == ADST_OP_FWD || a.op == ADST_OP_FWD2 || a.op == ADST_OP_FWDW;
    const bool adj_op = a.op == ADST_OP_ADJ || a.op == ADST_OP_ADJ2 || a.op == ADST_OP_ADJW;
    if (!fwd_op && !adj_op) continue;
    if (fused_fwd_adj(c, plan.acts, i)) continue;  // counted with its adjoint
    const int64_t k = c.in_place ? gs_kernel_launches(c.shape, adj_op, a.n) : 1;
    (fwd_op ? info->fwd_kernels : info->adj_kernels) += k;
    i += stored_run(c, plan.acts, i) - 1;
  }
  info->state_bytes = c.state_bytes;
  info->budget_bytes = budget;
  info->slot_bytes_peak = uint64_t(plan.slots) * c.state_bytes;
  info->workspace_bytes = L.total;
  info->fwd_workspace_bytes = (plan.steps >= 2 && !c.in_place) ? c.state_bytes : 0;
  // A fused launch moves its inputs and outputs once for its n steps (a
  // store-through run writes each of its n states); a pipelined run of the
  // in-place kind is counted as its n steps.
  const uint64_t n = uint64_t(c.npoints);
  uint64_t per_point = sb, fwd_per_point = 0;
  bool first_adj = true;
  for (size_t i = 0; i < plan.acts.size(); ++i) {
    const adst_action& a = plan.acts[i];
    switch (a.op) {
      case ADST_OP_FWD: {
        if (fused_fwd_adj(c, plan.acts, i)) break;  // moves the adjoint's bytes only
        const int32_t r = stored_run(c, plan.acts, i);
        fwd_per_point += fb + uint64_t(r - 1) * itemsize(c.shape.dtype);
        i += r - 1;
        break;
      }
      case ADST_OP_FWD2:
        if (fused_fwd_adj(c, plan.acts, i)) break;  // moves the adjoint's bytes only
        fwd_per_point += fb;
        break;
      case ADST_OP_FWDW:
        fwd_per_point += uint64_t(a.n) * fb;
        break;
      case ADST_OP_ADJ:
      case ADST_OP_ADJ2:
        per_point += (first_adj ? ab1 : ab) + db;
        first_adj = false;
        break;
      case ADST_OP_ADJW:
        per_point += uint64_t(a.n) * ab;
        first_adj = false;
        break;
      default:
        break;
    }
  }
  info->alg_bytes = n * (per_point + fwd_per_point);
  info->fwd_alg_bytes = n * fwd_per_point;
}

// ADST_LOG=1 in the environment prints each adst_vjp call's plan to
// stderr before anything is enqueued; ADST_LOG=2 also its action list.
int log_level() {
  static const int level = [] {
    const char* v = std::getenv("ADST_LOG");
    return v ? std::atoi(v) : 0;
  }();
  return level;
}

void log_plan(const Checked& c, const Plan& plan, uint64_t budget, bool want_dk, int32_t loss) {
  static const char* const kSched[4] = {"auto", "store_all", "uniform", "binomial"};
  static const char* const kKind[4] = {"jacobi2d5", "allencahn3d7", "vardiff2d9",
                                       "gaussseidel2d5"};
  adst_plan_info info;
  fill_info(c, plan, budget, want_dk, loss, &info);
  std::fprintf(stderr,
               "adst plan: %s %s %dx%dx%d T=%d budget=%llu B sched=%s slots=%d (c=%d) "
               "needs_state=%d fwd_steps=%lld (recompute %lld) adj_steps=%lld "
               "actions=%lld kernels fwd=%lld adj=%lld workspace=%llu B alg_bytes=%llu\n",
               kKind[c.shape.kind], c.shape.dtype == ADST_F64 ? "f64" : "f32", c.shape.nx,
               c.shape.ny, c.shape.nz, plan.steps, (unsigned long long)budget,
               kSched[plan.sched & 3], plan.slots, plan.slots + 1, plan.needs_state ? 1 : 0,
               (long long)info.fwd_steps_total, (long long)info.recompute_steps,
               (long long)info.adj_steps, (long long)info.n_actions, (long long)info.fwd_kernels,
               (long long)info.adj_kernels, (unsigned long long)info.workspace_bytes,
               (unsigned long long)info.alg_bytes);
  if (log_level() >= 2) {
    static const char* const kOp[7] = {"FWD", "SEED", "ADJ", "FWD2", "ADJ2", "FWDW", "ADJW"};
    for (size_t i = 0; i < plan.acts.size(); ++i) {
      const adst_action& a = plan.acts[i];
      std::fprintf(stderr, "  %5zu %-4s t=%-6d src=%-3d dst=%-3d n=%d\n", i,
                   (a.op >= 0 && a.op < 7) ? kOp[a.op] : "?", a.t, a.src, a.dst, a.n);
    }
  }
}

adst_status make_plan(const adst_problem* prob, int32_t steps, uint64_t budget, int32_t sched,
                      int32_t grads, Checked* c, Plan* plan) {
  adst_status st = check_problem(prob, grads, c);
  if (st != ADST_OK) return st;
  if (steps < 0) return fail(ADST_ERR_ARG, "steps must be >= 0");
  const int64_t slots_avail = (int64_t)std::min<uint64_t>(budget / c->state_bytes, INT32_MAX);
  std::string err;
  st = build_plan(steps, slots_avail, sched, c->needs_state, c->fuse_fwd, c->fuse_adj,
                  c->pair_tail, c->in_place, plan, &err);
  if (st != ADST_OK) return fail(st, err);
  return ADST_OK;
}

struct Range {
  const char* name;
  uintptr_t lo, hi;  // [lo, hi)
};

bool overlaps(const Range& a, const Range& b) {
  return a.lo < b.hi && b.lo < a.hi && a.lo != a.hi && b.lo != b.hi;
}

Range range_of(const char* name, const void* p, uint64_t bytes) {
  const uintptr_t lo = reinterpret_cast<uintptr_t>(p);
  return {name, lo, p ? lo + bytes : lo};
}

// Every output range must be disjoint from every other output and from the
// inputs (inputs may overlap each other: they are only read).
adst_status check_disjoint(const std::vector<Range>& outs, const std::vector<Range>& ins) {
  for (size_t a = 0; a < outs.size(); ++a) {
    for (size_t b = a + 1; b < outs.size(); ++b)
      if (overlaps(outs[a], outs[b]))
        return fail(ADST_ERR_ARG, std::string(outs[a].name) + " overlaps " + outs[b].name);
    for (const Range& r : ins)
      if (overlaps(outs[a], r))
        return fail(ADST_ERR_ARG, std::string(outs[a].name) + " overlaps input " + r.name);
  }
  return ADST_OK;
}

// Per-launch statistics of the last traced call on this thread.
struct KernelStat {
  std::string name;
  int32_t phase = 0;
  int64_t launches = 0;
  double ms_sum = 0, ms_min = 0, ms_max = 0, alg_bytes = 0;
};
thread_local std::vector<KernelStat> g_kernel_stats;

// HIP event timing for ADST_TRACE: an event pair brackets every launch (or
// every pipelined sequence of launches), so the per-kernel averages are
// kernel durations, comparable with a profiler's. Phases (forward sweep,
// recomputation, adjoint, seed, the constants' final sum) are also marked
// as roctx ranges whether or not the call is traced, for rocprofv3's marker
// trace.
class Tracer {
 public:
  enum Cat { SWEEP = 0, RECOMPUTE, ADJ, SEED, DPARAM, NCAT };
  explicit Tracer(bool on) : on_(on) {}
  ~Tracer() {
    if (phase_open_) roctxRangePop();
    for (auto& g : segs_) {
      if (g.start) (void)hipEventDestroy(g.start);
      if (g.stop) (void)hipEventDestroy(g.stop);
    }
  }
  // Call before enqueueing a launch (or a pipelined sequence of `launches`
  // kernels) of category cat; alg_bytes are the algorithmic bytes it moves.
  hipError_t begin(hipStream_t s, Cat cat, std::string label, double alg_bytes,
                   int64_t launches = 1) {
    if (!phase_open_ || cat != phase_) {
      static const char* const kPhase[NCAT] = {"adst forward sweep", "adst recomputation",
                                               "adst adjoint", "adst loss and seed",
                                               "adst constants' gradients"};
      if (phase_open_) roctxRangePop();
      roctxRangePushA(kPhase[cat]);
      phase_open_ = true;
      phase_ = cat;
    }
    if (!on_) return hipSuccess;
    Seg g{nullptr, nullptr, cat, std::move(label), alg_bytes, launches};
    hipError_t r = hipEventCreate(&g.start);
    if (r != hipSuccess) return r;
    segs_.push_back(g);
    if ((r = hipEventCreate(&segs_.back().stop)) != hipSuccess) return r;
    return hipEventRecord(segs_.back().start, s);
  }
  // Call after enqueueing what begin() announced.
  hipError_t end(hipStream_t s) {
    if (!on_ || segs_.empty()) return hipSuccess;
    return hipEventRecord(segs_.back().stop, s);
  }
  // Waits for the last marker, fills the ms_* fields and the per-kernel
  // statistics adst_trace_kernels returns.
  hipError_t finish(hipStream_t s, adst_plan_info* info) {
    (void)s;
    if (phase_open_) {
      roctxRangePop();
      phase_open_ = false;
    }
    if (!on_) return hipSuccess;
    g_kernel_stats.clear();
    if (segs_.empty()) return hipSuccess;
    hipError_t r = hipEventSynchronize(segs_.back().stop);
    if (r != hipSuccess) return r;
    float ms[NCAT] = {0, 0, 0, 0, 0};
    for (const Seg& g : segs_) {
      float dt = 0.f;
      if ((r = hipEventElapsedTime(&dt, g.start, g.stop)) != hipSuccess) return r;
      ms[g.cat] += dt;
      KernelStat* k = nullptr;
      for (KernelStat& e : g_kernel_stats)
        if (e.name == g.label) k = &e;
      if (!k) {
        g_kernel_stats.push_back(KernelStat{});
        k = &g_kernel_stats.back();
        k->name = g.label;
        k->phase = g.cat;
        k->ms_min = 1e30;
      }
      const double per = double(dt) / double(g.launches);
      k->launches += g.launches;
      k->ms_sum += dt;
      k->ms_min = std::min(k->ms_min, per);
      k->ms_max = std::max(k->ms_max, per);
      k->alg_bytes += g.alg_bytes;
    }
    float total = 0.f;
    if ((r = hipEventElapsedTime(&total, segs_.front().start, segs_.back().stop)) != hipSuccess)
      return r;
    if (info) {
      info->ms_fwd_sweep = ms[SWEEP];
      info->ms_fwd_recompute = ms[RECOMPUTE];
      info->ms_adj = ms[ADJ];
      info->ms_seed = ms[SEED];
      info->ms_dparams = ms[DPARAM];
      info->ms_total = total;
    }
    return hipSuccess;
  }

 private:
  struct Seg {
    hipEvent_t start, stop;
    Cat cat;
    std::string label;
    double alg_bytes;
    int64_t launches;
  };
  bool on_;
  bool phase_open_ = false;
  Cat phase_ = SWEEP;
  std::vector<Seg> segs_;
};

adst_status hip_fail(hipError_t e, const char* what) {
  return fail(ADST_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

}  // namespace
}  // namespace adst

namespace adst {
namespace {

// adst_vjp, with the workspace either the caller's (ws, ws_bytes) or, with
// static_ws, this device's static workspace.
adst_status vjp_impl(const adst_problem* prob, const void* x0, const void* coeff, int32_t steps,
                     int32_t loss, const void* loss_aux, uint64_t mem_budget_bytes, int32_t sched,
                     void* dx0, void* dcoeff, void* xT, double* loss_dev, double* dparams,
                     void* ws, uint64_t ws_bytes, bool static_ws, hipStream_t stream,
                     adst_plan_info* info) {
  const int32_t grads = (dcoeff ? ADST_GRAD_COEFF : 0) | (dparams ? ADST_GRAD_PARAMS : 0);
  const bool want_dk = dcoeff != nullptr;
  Checked c;
  Plan plan;
  adst_status st = make_plan(prob, steps, mem_budget_bytes, sched, grads, &c, &plan);
  if (st != ADST_OK) return st;
  if (!x0 || !dx0) return fail(ADST_ERR_ARG, "x0 and dx0 are required");
  if (prob->kind == ADST_VARDIFF2D9 && !coeff)
    return fail(ADST_ERR_ARG, "the variable-coefficient kind needs coeff (K)");
  if (loss < ADST_LOSS_HALF_SQ || loss > ADST_LOSS_SEED)
    return fail(ADST_ERR_ARG, "unknown loss " + std::to_string(loss));
  if (loss != ADST_LOSS_HALF_SQ && !loss_aux)
    return fail(ADST_ERR_ARG, "this loss needs loss_aux");
  const Layout L = layout_for(c, plan);
  if (static_ws) {
    if (c.trace)
      return fail(ADST_ERR_ARG, "ADST_TRACE creates HIP events: use adst_vjp to trace");
    if (L.total > kStaticWsBytes)
      return fail(ADST_ERR_WORKSPACE,
                  "adst_vjp_static_ws: this plan needs " + std::to_string(L.total) +
                      " workspace bytes; the static workspace holds " +
                      std::to_string(kStaticWsBytes) + " (use adst_vjp with a caller buffer)");
    const hipError_t e = static_workspace(&ws);
    if (e != hipSuccess) return hip_fail(e, "static workspace");
    ws_bytes = kStaticWsBytes;
  }
  if (ws_bytes < L.total || !ws)
    return fail(ADST_ERR_WORKSPACE, "adst_vjp needs " + std::to_string(L.total) +
                                        " workspace bytes, got " + std::to_string(ws_bytes));
  const uint64_t S = c.state_bytes;
  std::vector<Range> outs = {range_of("dx0", dx0, S), range_of("ws", ws, L.total)};
  if (dcoeff) outs.push_back(range_of("dcoeff", dcoeff, S));
  if (xT) outs.push_back(range_of("xT", xT, S));
  if (loss_dev) outs.push_back(range_of("loss_dev", loss_dev, sizeof(double)));
  if (dparams) outs.push_back(range_of("dparams", dparams, 2 * sizeof(double)));
  std::vector<Range> ins = {range_of("x0", x0, S)};
  if (prob->kind == ADST_VARDIFF2D9) ins.push_back(range_of("coeff", coeff, S));
  if (loss != ADST_LOSS_HALF_SQ) ins.push_back(range_of("loss_aux", loss_aux, S));
  st = check_disjoint(outs, ins);
  if (st != ADST_OK) return st;
  if (info) fill_info(c, plan, mem_budget_bytes, want_dk, loss, info);
  if (log_level() > 0) log_plan(c, plan, mem_budget_bytes, want_dk, loss);

  // ---- interpret the plan
  // The adjoint ping-pongs between dx0 and the workspace buffer G, one swap
  // per adjoint launch; g_T starts where the last launch leaves g_0 in dx0.
  // The in-place kind reverses its sweeps in dx0 itself.
  char* wsb = static_cast<char*>(ws);
  double* partials = reinterpret_cast<double*>(wsb);
  double* loss_out = loss_dev ? loss_dev : reinterpret_cast<double*>(wsb + kLossOffset);
  void* gws = wsb + L.g;
  void* gcur = (c.in_place || plan.adj_launches % 2 == 0) ? dx0 : gws;
  void* gnext = (gcur == dx0) ? gws : dx0;
  void* const g_T = gcur;
  const bool g_T_is_aux = seed_in_aux(c, loss, steps);
  double* dp_part = reinterpret_cast<double*>(wsb + L.dp);
  auto buffer = [&](int32_t id) -> void* {
    switch (id) {
      case ADST_BUF_X0: return const_cast<void*>(x0);
      case ADST_BUF_W0: return wsb + L.w0;
      case ADST_BUF_W1: return wsb + L.w1;
      case ADST_BUF_XT: return xT ? xT : g_T;
      default: return wsb + L.slot0 + uint64_t(id - ADST_BUF_SLOT0) * L.state_stride;
    }
  };

  Tracer tr(c.trace);
  const PerPoint pp = per_point_bytes(c, want_dk, loss);
  const double npts = double(c.npoints);
  bool seeded = false, first_adj = true;
  // the gradient the next adjoint launch reads
  auto g_in = [&]() -> const void* { return first_adj && g_T_is_aux ? loss_aux : gcur; };
  hipError_t e = hipSuccess;
  auto traced = [&](Tracer::Cat cat, std::string label, double bytes, auto&& launch,
                    int64_t launches = 1) -> hipError_t {
    hipError_t r = tr.begin(stream, cat, std::move(label), bytes, launches);
    if (r == hipSuccess) r = launch();
    if (r == hipSuccess) r = tr.end(stream);
    return r;
  };
  // a recomputed forward action and the adjoint step after it, in one launch
  auto fused_launch = [&](const adst_action& f) -> hipError_t {
    const double bytes = npts * double((first_adj ? pp.adj_first : pp.adj) + pp.adj_extra);
    const hipError_t r = traced(Tracer::ADJ, "ac_march<fwd" + std::to_string(f.n) + "+adj>",
                                bytes, [&] {
                                  return ac_launch_forward_adjoint(c.shape, buffer(f.src), g_in(),
                                                                   gnext, f.n, stream);
                                });
    std::swap(gcur, gnext);
    first_adj = false;
    return r;
  };
  for (size_t ai = 0; ai < plan.acts.size(); ++ai) {
    const adst_action& a = plan.acts[ai];
    const bool fwd_op = a.op == ADST_OP_FWD || a.op == ADST_OP_FWD2 || a.op == ADST_OP_FWDW;
    const Tracer::Cat cat = fwd_op               ? (seeded ? Tracer::RECOMPUTE : Tracer::SWEEP)
                            : a.op == ADST_OP_SEED ? Tracer::SEED
                                                   : Tracer::ADJ;
    if (c.in_place && a.op != ADST_OP_SEED) {
      const bool adj = a.op == ADST_OP_ADJ || a.op == ADST_OP_ADJW;
      if (!adj && a.op != ADST_OP_FWD && a.op != ADST_OP_FWDW) return hip_fail(hipErrorInvalidValue, "plan");
      e = traced(cat, kernel_label(c, a, 1, false),
                 npts * double(a.n) * double(adj ? pp.adj : pp.fwd),
                 [&] {
                   return adj ? launch_gs_adjoint(c.shape, dx0, a.n, stream)
                              : launch_gs_forward(c.shape, buffer(a.src), buffer(a.dst), a.n,
                                                  stream);
                 },
                 gs_kernel_launches(c.shape, adj, a.n));
      if (e != hipSuccess) return hip_fail(e, "kernel launch");
      continue;
    }
    switch (a.op) {
      case ADST_OP_FWD: {
        if (fused_fwd_adj(c, plan.acts, ai)) {
          e = fused_launch(a);
          ++ai;
          break;
        }
        const int32_t r = stored_run(c, plan.acts, ai);
        const double bytes = npts * double(pp.fwd + uint64_t(r - 1) * itemsize(c.shape.dtype));
        if (r >= 2) {  // one launch writes the run's r states
          void* ys[kMaxStoredRun];
          for (int32_t k = 0; k < r; ++k) ys[k] = buffer(plan.acts[ai + k].dst);
          e = traced(cat, kernel_label(c, a, r, false), bytes, [&] {
            return launch_forward_store(c.shape, buffer(a.src), coeff, ys, r, stream);
          });
          ai += r - 1;
        } else {
          e = traced(cat, kernel_label(c, a, 1, false), bytes, [&] {
            return launch_forward(c.shape, buffer(a.src), coeff, buffer(a.dst), stream);
          });
        }
        break;
      }
      case ADST_OP_FWD2:
        if (fused_fwd_adj(c, plan.acts, ai)) {
          e = fused_launch(a);
          ++ai;
          break;
        }
        e = traced(cat, kernel_label(c, a, 1, false), npts * double(pp.fwd), [&] {
          return launch_forward_n(c.shape, buffer(a.src), coeff, buffer(a.dst), a.n, stream);
        });
        break;
      case ADST_OP_SEED: {
        const void* xsrc = buffer(a.src);
        void* xcopy = (steps == 0 && xT) ? xT : nullptr;
        // the half square with x_T already in g_T's buffer only reads it;
        // with g_T read from loss_aux the pass reads x_T and loss_aux only
        const double isz = double(itemsize(c.shape.dtype));
        const double seed_bytes =
            (loss == ADST_LOSS_HALF_SQ && xsrc == g_T ? isz
             : g_T_is_aux                             ? 2.0 * isz
                                                      : double(pp.seed)) +
            (xcopy ? isz : 0.0);
        e = traced(cat, "seed_loss", npts * seed_bytes, [&] {
          return launch_seed(c.shape.dtype, loss, c.npoints, xsrc, loss_aux,
                             g_T_is_aux ? nullptr : g_T, xcopy, partials, stream);
        });
        if (e == hipSuccess)
          e = traced(cat, "finalize_loss", 8.0 * seed_partials(c.npoints), [&] {
            return launch_finalize(partials, seed_partials(c.npoints), loss_out, stream);
          });
        if (e == hipSuccess && steps == 0 && dcoeff)
          e = traced(cat, "fill_zero", double(S), [&] {
            return launch_fill_zero(dcoeff, (int64_t)S, stream);
          });
        if (e == hipSuccess && steps == 0 && dparams)
          e = traced(cat, "fill_zero", 16.0, [&] {
            return launch_fill_zero(dparams, 2 * sizeof(double), stream);
          });
        seeded = true;
        break;
      }
      case ADST_OP_ADJ: {
        const void* xs = a.src == ADST_BUF_NONE ? nullptr : buffer(a.src);
        if (c.shape.limit && !adjoint_applies_limit(c.shape, dparams != nullptr)) {
          // the branch each point took at step t (otherwise applied by the
          // adjoint launch itself)
          e = traced(cat, "limit_mask", npts * double(pp.mask), [&] {
            return launch_limit_mask(c.shape, xs, coeff, gcur, stream);
          });
          if (e != hipSuccess) return hip_fail(e, "kernel launch");
        }
        // with dparams, the launch also adds this step's share of the
        // constants' gradients, from g_t and x_{t-1}
        const double bytes = npts * double((first_adj ? pp.adj_first : pp.adj) + pp.adj_extra);
        e = traced(cat, kernel_label(c, a, 1, dparams != nullptr), bytes, [&] {
          return launch_adjoint(c.shape, xs, coeff, g_in(), gnext, dcoeff, a.t == steps,
                                dparams ? dp_part : nullptr, a.t == steps, stream);
        });
        std::swap(gcur, gnext);
        first_adj = false;
        break;
      }
      case ADST_OP_ADJ2:
        e = traced(cat, kernel_label(c, a, 1, false), npts * double(pp.adj), [&] {
          return launch_adjoint_n(c.shape, g_in(), gnext, a.n, stream);
        });
        std::swap(gcur, gnext);
        first_adj = false;
        break;
      default:
        e = hipErrorInvalidValue;
    }
    if (e != hipSuccess) return hip_fail(e, "kernel launch");
  }
  if (dparams && steps > 0) {
    e = traced(Tracer::DPARAM, "dparam_finalize", 16.0 * dparam_slots(c.shape), [&] {
      return launch_dparam_finalize(c.shape, dp_part, dparams, stream);
    });
    if (e != hipSuccess) return hip_fail(e, "kernel launch");
  }
  if ((e = tr.finish(stream, info)) != hipSuccess) return hip_fail(e, "trace");
  g_last_error.clear();
  return ADST_OK;
}

}  // namespace
}  // namespace adst

using namespace adst;

extern "C" {

adst_status adst_plan(const adst_problem* prob, int32_t steps, uint64_t mem_budget_bytes,
                      int32_t sched, int32_t grads, adst_plan_info* out) {
  if (!out) return fail(ADST_ERR_ARG, "out is NULL");
  Checked c;
  Plan plan;
  adst_status st = make_plan(prob, steps, mem_budget_bytes, sched, grads, &c, &plan);
  if (st != ADST_OK) return st;
  fill_info(c, plan, mem_budget_bytes, c.want_dk, ADST_LOSS_HALF_SQ, out);
  g_last_error.clear();
  return ADST_OK;
}

adst_status adst_plan_actions(const adst_problem* prob, int32_t steps, uint64_t mem_budget_bytes,
                              int32_t sched, int32_t grads, adst_action* out, int64_t cap,
                              int64_t* n_out) {
  if (!n_out) return fail(ADST_ERR_ARG, "n_out is NULL");
  if (cap < 0 || (cap > 0 && !out)) return fail(ADST_ERR_ARG, "bad output capacity");
  Checked c;
  Plan plan;
  adst_status st = make_plan(prob, steps, mem_budget_bytes, sched, grads, &c, &plan);
  if (st != ADST_OK) return st;
  const int64_t n = (int64_t)plan.acts.size();
  std::copy(plan.acts.begin(), plan.acts.begin() + std::min(n, cap), out);
  *n_out = n;
  g_last_error.clear();
  return ADST_OK;
}

adst_status adst_forward(const adst_problem* prob, const void* x0, const void* coeff,
                         int32_t steps, void* xT, void* ws, uint64_t ws_bytes,
                         hipStream_t stream) {
  Checked c;
  adst_status st = check_problem(prob, 0, &c);
  if (st != ADST_OK) return st;
  if (steps < 0) return fail(ADST_ERR_ARG, "steps must be >= 0");
  if (!x0 || !xT) return fail(ADST_ERR_ARG, "x0 and xT are required");
  if (prob->kind == ADST_VARDIFF2D9 && !coeff)
    return fail(ADST_ERR_ARG, "the variable-coefficient kind needs coeff (K)");
  const uint64_t S = c.state_bytes;
  const uint64_t need = (steps >= 2 && !c.in_place) ? S : 0;
  if (ws_bytes < need || (need && !ws))
    return fail(ADST_ERR_WORKSPACE, "adst_forward needs " + std::to_string(need) + " workspace bytes");
  std::vector<Range> outs = {range_of("xT", xT, S)};
  if (need) outs.push_back(range_of("ws", ws, need));
  std::vector<Range> ins = {range_of("x0", x0, S)};
  if (prob->kind == ADST_VARDIFF2D9) ins.push_back(range_of("coeff", coeff, S));
  st = check_disjoint(outs, ins);
  if (st != ADST_OK) return st;

  hipError_t e;
  if (steps == 0) {
    e = launch_copy(xT, x0, (int64_t)S, stream);
    if (e != hipSuccess) return hip_fail(e, "copy");
    g_last_error.clear();
    return ADST_OK;
  }
  if (c.in_place) {  // pipelined sweeps from x0 straight into xT
    e = launch_gs_forward(c.shape, x0, xT, steps, stream);
    if (e != hipSuccess) return hip_fail(e, "forward sweeps");
    g_last_error.clear();
    return ADST_OK;
  }
  // Launches of up to fuse_fwd steps each, the shorter remainder first;
  // they alternate between xT and ws so that the last one writes xT.
  const int32_t d = c.fuse_fwd;
  const int32_t n_launch = (steps + d - 1) / d;
  const void* cur = x0;
  int32_t done = 0;
  for (int32_t k = 0; k < n_launch; ++k) {
    void* dst = ((n_launch - 1 - k) % 2 == 0) ? xT : ws;
    const int32_t n = (k == 0 && steps % d != 0) ? steps % d : d;
    e = n >= 2 ? launch_forward_n(c.shape, cur, coeff, dst, n, stream)
               : launch_forward(c.shape, cur, coeff, dst, stream);
    if (e != hipSuccess) return hip_fail(e, "forward step");
    done += n;
    cur = dst;
  }
  if (done != steps) return fail(ADST_ERR_ARG, "internal: forward launch count");
  g_last_error.clear();
  return ADST_OK;
}

adst_status adst_vjp(const adst_problem* prob, const void* x0, const void* coeff, int32_t steps,
                     int32_t loss, const void* loss_aux, uint64_t mem_budget_bytes, int32_t sched,
                     void* dx0, void* dcoeff, void* xT, double* loss_dev, double* dparams,
                     void* ws, uint64_t ws_bytes, hipStream_t stream, adst_plan_info* info) {
  return vjp_impl(prob, x0, coeff, steps, loss, loss_aux, mem_budget_bytes, sched, dx0, dcoeff,
                  xT, loss_dev, dparams, ws, ws_bytes, false, stream, info);
}

adst_status adst_vjp_static_ws(const adst_problem* prob, const void* x0, const void* coeff,
                               int32_t steps, int32_t loss, const void* loss_aux,
                               uint64_t mem_budget_bytes, int32_t sched, void* dx0, void* dcoeff,
                               void* xT, double* loss_dev, double* dparams, hipStream_t stream,
                               adst_plan_info* info) {
  return vjp_impl(prob, x0, coeff, steps, loss, loss_aux, mem_budget_bytes, sched, dx0, dcoeff,
                  xT, loss_dev, dparams, nullptr, 0, true, stream, info);
}

adst_status adst_ilp_solve(const adst_ilp_array* arrays, int32_t n_arrays,
                           const adst_ilp_event* events, int64_t n_events, double limit,
                           int32_t* store_out, adst_ilp_info* info) {
  if (n_arrays < 0 || n_arrays > 48) return fail(ADST_ERR_ARG, "n_arrays must be in [0, 48]");
  if (n_events < 0) return fail(ADST_ERR_ARG, "n_events must be >= 0");
  if ((n_arrays > 0 && (!arrays || !store_out)) || (n_events > 0 && !events))
    return fail(ADST_ERR_ARG, "NULL arrays, events or store_out");
  if (!std::isfinite(limit) || limit < 0) return fail(ADST_ERR_ARG, "limit must be finite and >= 0");
  for (int32_t i = 0; i < n_arrays; ++i) {
    const adst_ilp_array& a = arrays[i];
    if (!std::isfinite(a.size) || !std::isfinite(a.overhead) || !std::isfinite(a.cost) ||
        a.size < 0 || a.overhead < 0 || a.cost < 0)
      return fail(ADST_ERR_ARG, "array " + std::to_string(i) + ": values must be finite and >= 0");
  }
  IlpResult r;
  std::string err;
  const adst_status st = ilp_solve(arrays, n_arrays, events, n_events, limit, &r, &err);
  if (info) {
    *info = adst_ilp_info{};
    info->measurements = r.measurements;
    info->nodes = r.nodes;
    info->paths = r.paths;
  }
  if (st != ADST_OK) return fail(st, err);
  for (int32_t i = 0; i < n_arrays; ++i) store_out[i] = r.v[i];
  if (info) {
    info->objective = r.objective;
    info->peak = r.peak;
  }
  g_last_error.clear();
  return ADST_OK;
}

adst_status adst_copy(void* dst, const void* src, uint64_t bytes, hipStream_t stream) {
  if (bytes == 0) {
    g_last_error.clear();
    return ADST_OK;
  }
  if (!dst || !src) return fail(ADST_ERR_ARG, "dst and src are required");
  if ((reinterpret_cast<uintptr_t>(dst) | reinterpret_cast<uintptr_t>(src) | bytes) & 3u)
    return fail(ADST_ERR_ARG, "dst, src and bytes must be multiples of 4");
  if (bytes > (uint64_t(1) << 62)) return fail(ADST_ERR_ARG, "bytes too large");
  const adst_status st = check_disjoint({range_of("dst", dst, bytes)}, {range_of("src", src, bytes)});
  if (st != ADST_OK) return st;
  const hipError_t e = launch_copy(dst, src, (int64_t)bytes, stream);
  if (e != hipSuccess) return hip_fail(e, "copy");
  g_last_error.clear();
  return ADST_OK;
}

adst_status adst_trace_kernels(adst_kernel_stat* out, int32_t cap, int32_t* n_out) {
  if (!n_out) return fail(ADST_ERR_ARG, "n_out is NULL");
  if (cap < 0 || (cap > 0 && !out)) return fail(ADST_ERR_ARG, "bad output capacity");
  const int32_t n = (int32_t)g_kernel_stats.size();
  for (int32_t i = 0; i < std::min(n, cap); ++i) {
    const KernelStat& k = g_kernel_stats[i];
    adst_kernel_stat& o = out[i];
    o = adst_kernel_stat{};
    std::snprintf(o.name, sizeof(o.name), "%s", k.name.c_str());
    o.phase = k.phase;
    o.launches = k.launches;
    o.ms_sum = k.ms_sum;
    o.ms_min = k.ms_min;
    o.ms_max = k.ms_max;
    o.alg_bytes_sum = k.alg_bytes;
  }
  *n_out = n;
  g_last_error.clear();
  return ADST_OK;
}

const char* adst_status_str(adst_status s) {
  switch (s) {
    case ADST_OK: return "ok";
    case ADST_ERR_ARG: return "invalid argument";
    case ADST_ERR_BUDGET: return "memory budget too small for the requested schedule";
    case ADST_ERR_WORKSPACE: return "workspace too small";
    case ADST_ERR_UNSUPPORTED: return "unsupported problem";
    case ADST_ERR_HIP: return "HIP error";
  }
  return "unknown status";
}

const char* adst_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
