/* adst.h — reverse-mode gradients of time-iterated stencil programs under a
 * checkpoint-memory budget, on AMD MI355X (gfx950).
 *
 * The operation (DaCe AD, arXiv 2509.02197): given an unmodified time loop
 *     x_t = F(x_{t-1}; K),  t = 1..T,
 * and one scalar output L(x_T), return the vector-Jacobian products
 *     dx0 = dL/dx_0   and   dK = dL/dK
 * (Sec. II: the backward pass computes gradients of one dependent variable
 * with respect to a set of independent inputs; Sec. III-A limitations: a
 * single scalar output per gradient). The forward values the reverse sweep
 * needs are either stored or recomputed from checkpoints so that storage stays
 * within a caller-given byte budget (Sec. IV: store/recompute trade-off under
 * a user memory constraint, store-all as the default and a manual choice
 * available). Recomputation changes where x_{t-1} comes from, never the
 * gradient: results are bit-identical across every budget and schedule.
 *
 * Step kinds (F), arrays row-major [nz][ny][nx] with x fastest, unpadded:
 *   ADST_JACOBI2D5    2-D, 5-point average on interior points, outer ring held
 *                     fixed.  x'[c] = w*((((x[c]+x[W])+x[E])+x[S])+x[N]);
 *                     p[0] = w (0.2).
 *   ADST_ALLENCAHN3D7 3-D (nz >= 1), every point updated, out-of-grid
 *                     neighbours read 0.  lap = (((((x[-x]+x[+x])+x[-y])+x[+y])
 *                     +x[-z])+x[+z]) - 6*x[c];  x' = (x[c] + D*lap) - C*((x[c]*x[c])*x[c]);
 *                     p[0] = D (0.1), p[1] = C (0.1).
 *   ADST_VARDIFF2D9   2-D, x' = x[c] + dt*acc with acc the left-to-right sum
 *                     over the in-grid neighbours n in the order
 *                     (-1,0),(+1,0),(0,-1),(0,+1),(-1,-1),(+1,-1),(-1,+1),(+1,+1)
 *                     of (c_n*(K[c]+K[n]))*(x[n]-x[c]); c_n = 1/3 on the axes
 *                     and 1/12 on the diagonals (rounded to the working
 *                     precision); edges leaving the grid are dropped (no flux).
 *                     p[0] = dt (0.1). The per-point field K is the
 *                     coefficient ("coeff") whose gradient dK may be asked for.
 *   ADST_GAUSSSEIDEL2D5  2-D, in place: interior points are overwritten one
 *                     at a time in row-major order (x fastest) with
 *                     x[c] = w*((((x[c]+x[E])+x[N])+x[S])+x[W]), so x[S] and x[W]
 *                     already hold the current step's values; the outer ring
 *                     is held fixed. p[0] = w (0.2). The paper's Seidel2d case
 *                     study (Sec. V-B) is an in-place stencil of this kind: a
 *                     dependency carried through every sweep, whose reverse
 *                     visits the points in reverse order and clears each
 *                     overwritten value's gradient (Sec. II, Sec. III-C).
 * Each forward formula is evaluated in the order written, in the working
 * precision, without fused multiply-add contraction.
 *
 * Conventions for every call:
 *   - All device memory is caller-owned; adst never allocates or frees device
 *     memory. Pointers are device addresses on the current HIP device.
 *   - Inputs (x0, coeff, loss_aux) are read-only and must stay untouched
 *     until the call's work on the stream has run: x0 serves as the free
 *     base checkpoint, and for DOT_W and SEED the first adjoint step reads
 *     g_T from loss_aux itself.
 *   - Outputs are overwritten (=, never +=).
 *   - Calls that take a stream only enqueue work on it and never synchronise,
 *     except with ADST_TRACE set (see below). Argument errors are detected
 *     before anything is enqueued.
 *   - On failure the call returns a non-zero adst_status and
 *     adst_last_error() holds a thread-local description.
 *   - ADST_LOG=1 in the environment prints each adst_vjp plan to stderr
 *     (ADST_LOG=2 also its actions); the phases of a call are marked as
 *     roctx ranges for rocprofv3's marker trace.
 */
#ifndef ADST_H
#define ADST_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  ADST_OK = 0,
  ADST_ERR_ARG = 1,         /* NULL required pointer, bad shape/steps/enum, overlapping ranges */
  ADST_ERR_BUDGET = 2,      /* STORE_ALL asked for but the budget cannot hold its slots */
  ADST_ERR_WORKSPACE = 3,   /* ws_bytes below what the plan needs */
  ADST_ERR_UNSUPPORTED = 4, /* kind/dtype/dimension combination not built */
  ADST_ERR_HIP = 5          /* a HIP launch or runtime call failed */
} adst_status;

typedef enum {
  ADST_JACOBI2D5 = 0,
  ADST_ALLENCAHN3D7 = 1,
  ADST_VARDIFF2D9 = 2,
  ADST_GAUSSSEIDEL2D5 = 3
} adst_kind;
typedef enum { ADST_F64 = 0, ADST_F32 = 1 } adst_dtype;

/* Checkpoint schedules (Sec. IV: store-all default, a manual choice, or an
 * automatic one within the memory limit).
 *   STORE_ALL  keep every state the reverse sweep reads; no recomputation.
 *   UNIFORM    checkpoints every k = ceil(T/c) steps, one-level recompute.
 *   BINOMIAL   optimal for a single time loop with uniform step cost
 *              (Revolve, cited in the related work): minimal forward steps
 *              for the c checkpoints the budget allows.
 *   AUTO       STORE_ALL if it fits the budget, else BINOMIAL. */
typedef enum {
  ADST_SCHED_AUTO = 0,
  ADST_SCHED_STORE_ALL = 1,
  ADST_SCHED_UNIFORM = 2,
  ADST_SCHED_BINOMIAL = 3
} adst_sched;

/* The scalar output L. Its value is accumulated in double whatever the
 * working precision; the seed g_T = dL/dx_T is in the working precision.
 *   HALF_SQ       L = sum 0.5*x_T^2,            g_T = x_T        (aux unused)
 *   DOT_W         L = sum aux*x_T,              g_T = aux
 *   HALF_SQ_DIFF  d = x_T - aux, L = sum 0.5*d^2, g_T = d
 *   SEED          g_T = aux (explicit cotangent), L = sum aux*x_T */
typedef enum {
  ADST_LOSS_HALF_SQ = 0,
  ADST_LOSS_DOT_W = 1,
  ADST_LOSS_HALF_SQ_DIFF = 2,
  ADST_LOSS_SEED = 3
} adst_loss;

/* Problem flags. */
#define ADST_FORCE_TAPE 0x1u /* treat every step as reading x_{t-1} in its adjoint, even when
                                the kind is linear, so store/recompute runs at any shape */
#define ADST_TRACE 0x2u      /* time every launch with a HIP event pair, synchronise the
                                stream at the end of the call, fill the ms_* fields of
                                adst_plan_info and the per-kernel statistics that
                                adst_trace_kernels returns */
#define ADST_NO_FUSE 0x4u    /* run every step as its own launch (no temporal blocking:
                                otherwise up to 6 Jacobi steps, 3 Allen-Cahn forward steps
                                or 2 variable-coefficient forward steps share one launch);
                                results are bit-identical either way */
#define ADST_LIMIT 0x8u      /* a limiter on every step: each new value y (ring included)
                                becomes lim[0] if y < lim[0], lim[1] if y > lim[1], else stays
                                y. A data-dependent branch at every point of every step
                                (Sec. III-B): its derivative is that of the branch taken (1
                                where y was kept, 0 where clamped), and the reverse sweep
                                recomputes each branch outcome from x_{t-1} with the
                                forward's own expressions, so every adjoint reads state. Not
                                built for the in-place kind (ADST_ERR_UNSUPPORTED); steps
                                are then not fused. */

/* Which gradients besides dx0 a plan is for (the `grads` argument).
 *   ADST_GRAD_COEFF   dK, the per-point coefficient field (VARDIFF2D9 only)
 *   ADST_GRAD_PARAMS  dL/dp[0] and dL/dp[1], the scalar step constants:
 *                     Jacobi (dL/dw, 0), Allen-Cahn (dL/dD, dL/dC), variable
 *                     coefficients (dL/ddt, 0), each the derivative with
 *                     respect to the constant as rounded to the working
 *                     precision. A constant every point of every step reads
 *                     accumulates its gradient over all those uses (Sec. II);
 *                     its partials read x_{t-1}, so asking for it makes every
 *                     kind's adjoint read state. Not built for the in-place
 *                     kind (ADST_ERR_UNSUPPORTED). */
#define ADST_GRAD_COEFF 0x1
#define ADST_GRAD_PARAMS 0x2

typedef struct {
  int32_t kind;   /* adst_kind */
  int32_t dtype;  /* adst_dtype */
  int64_t n[3];   /* n[0] = nx (fastest), n[1] = ny, n[2] = nz (1 for the 2-D kinds);
                     every n[i] >= 1 and n[0]*n[1]*n[2] < 2^31 */
  double p[2];    /* step constants, see the kinds above; rounded to the working precision */
  double lim[2];  /* limiter bounds lo <= hi (with ADST_LIMIT; rounded likewise) */
  uint32_t flags; /* ADST_FORCE_TAPE | ADST_TRACE | ADST_NO_FUSE | ADST_LIMIT */
} adst_problem;

/* One action of a reverse-sweep plan. Buffers are named by small integers:
 * ADST_BUF_X0 the caller's x0, ADST_BUF_W0/W1 two work states, ADST_BUF_XT
 * the buffer that receives x_T, and ADST_BUF_SLOT0 + k checkpoint slot k.
 *   ADST_OP_FWD   x_t = F(state in src), written to dst
 *   ADST_OP_SEED  loss and seed g_T from x_T held in src (t = T)
 *   ADST_OP_ADJ   g_{t-1} = J_t^T g_t, reading x_{t-1} from src
 *                 (src = ADST_BUF_NONE when the step's adjoint reads no state)
 *   ADST_OP_FWD2  x_t = F^n(state in src), n >= 2 (steps t-n+1..t in one launch,
 *                 the intermediate states kept on chip; emitted only where
 *                 nothing else reads them), written to dst
 *   ADST_OP_ADJ2  g_{t-n} = J_{t-n+1}^T ... J_t^T g_t, n >= 2, in one launch
 *                 (state-free adjoints only; src = ADST_BUF_NONE)
 *   ADST_OP_FWDW  x_t from x_{t-n} in src by n steps of the in-place kind,
 *                 pipelined in one sequence of wavefront launches (tiles of
 *                 several steps share a launch), written to dst
 *   ADST_OP_ADJW  g_{t-n} = J_{t-n+1}^T ... J_t^T g_t for the in-place kind,
 *                 pipelined the same way (its adjoint reads no state)
 * Fused and pipelined actions evaluate every point with the same expression
 * as the single steps, so results are bit-identical. `n` is the number of
 * steps an action covers (1 for FWD/ADJ, 0 for SEED).
 * Consecutive FWD actions that form a chain (each reads the state the one
 * before it wrote, into buffers all different from each other and from the
 * chain's input) are run by adst_vjp as one launch per up to 3 (Allen-Cahn)
 * or 2 (variable coefficients) of them, which writes every state of the run
 * (a store-all run of the binomial schedule); fwd_kernels counts those
 * launches. Not with ADST_NO_FUSE or ADST_LIMIT. */
typedef enum {
  ADST_OP_FWD = 0,
  ADST_OP_SEED = 1,
  ADST_OP_ADJ = 2,
  ADST_OP_FWD2 = 3,
  ADST_OP_ADJ2 = 4,
  ADST_OP_FWDW = 5,
  ADST_OP_ADJW = 6
} adst_op;
enum {
  ADST_BUF_NONE = -1,
  ADST_BUF_X0 = 0,
  ADST_BUF_W0 = 1,
  ADST_BUF_W1 = 2,
  ADST_BUF_XT = 3,
  ADST_BUF_SLOT0 = 4
};
typedef struct {
  int32_t op;
  int32_t t;   /* the step the action ends at (forward) or starts from (adjoint) */
  int32_t src;
  int32_t dst;
  int32_t n;   /* steps covered */
} adst_action;

typedef struct {
  int32_t steps;            /* T */
  int32_t sched;            /* schedule actually used (never AUTO) */
  int32_t slots;            /* checkpoint slots used, x0 excluded (c = slots + 1) */
  int32_t needs_state;      /* 1 if the adjoint reads x_{t-1} */
  int64_t fwd_steps_total;  /* forward-step launches: sweep (T) + recompute */
  int64_t recompute_steps;  /* fwd_steps_total - T */
  int64_t adj_steps;        /* T */
  int64_t n_actions;        /* length of the action list */
  int64_t fwd_launches;     /* forward actions (a fused or a pipelined run counts once) */
  int64_t adj_launches;     /* adjoint actions (likewise) */
  int64_t fwd_kernels;      /* forward kernel dispatches the actions enqueue */
  int64_t adj_kernels;      /* adjoint kernel dispatches the actions enqueue */
  uint64_t state_bytes;     /* bytes of one state */
  uint64_t budget_bytes;    /* the budget passed in */
  uint64_t slot_bytes_peak; /* slots * state_bytes: checkpoint storage actually used */
  uint64_t workspace_bytes; /* ws bytes adst_vjp needs for this plan */
  uint64_t fwd_workspace_bytes; /* ws bytes adst_forward needs */
  uint64_t alg_bytes;       /* algorithmic HBM bytes of one adst_vjp call */
  float ms_fwd_sweep;       /* ADST_TRACE only: summed kernel time of the first T forward steps */
  float ms_fwd_recompute;   /*   ... of the recomputed forward steps */
  float ms_adj;             /*   ... of the adjoint steps */
  float ms_seed;            /*   ... of the loss/seed and its final reduction */
  float ms_total;           /*   first launch start to last launch end */
  float ms_dparams;         /*   ... of the constants' gradient sum (the final reduction; the
                               per-step shares run inside the adjoint launches) */
  uint64_t fwd_alg_bytes;   /* algorithmic HBM bytes of the forward launches (sweep and
                               recomputation; part of alg_bytes) */
} adst_plan_info;

/* Plan a forward+VJP call without touching the GPU (host only).
 * Defined by Sec. IV (the store/recompute trade-off for the forwarded
 * values the backward pass reads, made within a user memory limit, with
 * store-all as the default and a manual choice available) and Sec. III-B
 * (the loop is reversed as one compact loop of the same range, so the
 * reverse sweep needs x_{t-1} in the order t = T..1).
 * The budget counts checkpoint-slot storage only: slots = floor(budget /
 * state_bytes); x0 is the caller's and is the free base checkpoint, so the
 * schedule has c = slots + 1 checkpoints. grads is a mask of ADST_GRAD_COEFF
 * (dK, VARDIFF2D9 only, which makes its adjoint read x_{t-1}) and
 * ADST_GRAD_PARAMS (the constants' gradients; every adjoint then reads
 * x_{t-1}). For the in-place
 * kind (GAUSSSEIDEL2D5, linear) nothing is stored: the plan is one pipelined
 * forward run, the seed and one pipelined reverse run (FWDW, SEED, ADJW);
 * with ADST_FORCE_TAPE it is a per-step checkpointed plan like the others.
 * Errors: ADST_ERR_ARG (NULL prob/out, steps < 0, bad kind/dtype/sched, bad
 * shape), ADST_ERR_UNSUPPORTED (shape not valid for the kind, or dK asked for
 * a kind without a coefficient field), ADST_ERR_BUDGET (STORE_ALL does not fit). */
adst_status adst_plan(const adst_problem* prob, int32_t steps, uint64_t mem_budget_bytes,
                      int32_t sched, int32_t grads, adst_plan_info* out);

/* The same plan as its action list (host only; for tests and inspection).
 * Sec. IV: which forward values are stored and which are recomputed from
 * the nearest checkpoint, written out step by step.
 * Writes min(cap, n) actions to out (out may be NULL when cap == 0) and the
 * full length to *n_out. Same errors as adst_plan. */
adst_status adst_plan_actions(const adst_problem* prob, int32_t steps, uint64_t mem_budget_bytes,
                              int32_t sched, int32_t grads, adst_action* out, int64_t cap,
                              int64_t* n_out);

/* x_T after `steps` forward steps: the unmodified program whose gradient
 * adst_vjp computes (Sec. I: the user's program is differentiated without
 * modification; the step kinds are defined at the top of this file).
 * x0 and xT are [nz][ny][nx] arrays of the working precision; coeff is K for
 * VARDIFF2D9 and must be NULL-or-ignored otherwise. ws must hold
 * adst_plan_info.fwd_workspace_bytes (one state when steps >= 2, else 0;
 * always 0 for the in-place kind, which runs in xT).
 * Errors: as adst_plan, plus ADST_ERR_WORKSPACE and ADST_ERR_HIP. */
adst_status adst_forward(const adst_problem* prob, const void* x0, const void* coeff,
                         int32_t steps, void* xT, void* ws, uint64_t ws_bytes,
                         hipStream_t stream);

/* Forward sweep, loss, and reverse sweep under the budget, enqueued on
 * `stream`: the vector-Jacobian product of one scalar output with respect to
 * the inputs (Sec. II: gradients of one dependent variable, accumulated over
 * every read of an input and cleared where a value is overwritten; Sec.
 * III-B: the time loop reversed as one compact loop; Sec. III-C: each
 * parallel map of a step reversed into a map of the same range, here in
 * gather form; Sec. IV: forwarded values stored or recomputed within
 * mem_budget_bytes). Arrays are [nz][ny][nx] of the working precision,
 * device memory owned by the caller. Outputs: dx0 (required), dcoeff (dK, VARDIFF2D9 only, NULL = not
 * requested), xT (optional), loss_dev (optional device double), dparams
 * (optional device double[2]: the constants' gradients, see
 * ADST_GRAD_PARAMS; NULL = not requested). The plan is the one adst_plan
 * gives for grads = (dcoeff ? ADST_GRAD_COEFF : 0) | (dparams ?
 * ADST_GRAD_PARAMS : 0). ws must hold
 * adst_plan_info.workspace_bytes and is clobbered. dx0 doubles as one of the
 * two adjoint buffers (for the in-place kind, the only one: the reverse
 * sweeps run in place in dx0). steps = 0 is valid: dx0 = seed, dK = 0.
 * info (optional, host) receives the plan; with ADST_TRACE it also receives
 * the per-phase kernel times, and the call synchronises the stream.
 * Errors: as adst_plan, plus ADST_ERR_ARG for overlapping input/output ranges
 * or a missing loss_aux, ADST_ERR_WORKSPACE, ADST_ERR_HIP. */
adst_status adst_vjp(const adst_problem* prob, const void* x0, const void* coeff, int32_t steps,
                     int32_t loss, const void* loss_aux, uint64_t mem_budget_bytes, int32_t sched,
                     void* dx0, void* dcoeff, void* xT, double* loss_dev, double* dparams,
                     void* ws, uint64_t ws_bytes, hipStream_t stream, adst_plan_info* info);

/* ---- Without allocation -------------------------------------------------
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): adst_vjp
 * with its workspace in a static device array of ADST_STATIC_WS_BYTES
 * (64 MiB) per GPU instead of a caller buffer. The array is part of the
 * library's code object: each GPU the library runs on holds its own copy
 * until the process ends; its address is looked up on the call's first use
 * of a device, with no allocation. Arguments, outputs, plan and results are
 * those of adst_vjp with the same arguments (bit for bit: the same kernels
 * run). No part of the workspace needs to start at zero: every value the
 * call reads from it was written earlier in the same call. Every call on a
 * GPU shares that GPU's array, so calls that overlap on one GPU (on
 * different streams, or from several host threads) race and must be
 * serialised by the caller. Calls no hipMalloc, hipFree or allocating
 * library routine.
 * Errors: as adst_vjp; ADST_ERR_WORKSPACE when the plan's workspace_bytes
 * (adst_plan) exceed ADST_STATIC_WS_BYTES; ADST_ERR_ARG with ADST_TRACE
 * (tracing creates HIP events). */
#define ADST_STATIC_WS_BYTES (64ull << 20)
adst_status adst_vjp_static_ws(const adst_problem* prob, const void* x0, const void* coeff,
                               int32_t steps, int32_t loss, const void* loss_aux,
                               uint64_t mem_budget_bytes, int32_t sched, void* dx0, void* dcoeff,
                               void* xT, double* loss_dev, double* dparams, hipStream_t stream,
                               adst_plan_info* info);

/* ---- Store/recompute selection for a general program (Sec. IV) --------
 * The integer program of Sec. IV-A: one binary per forwarded array (store or
 * recompute), objective sum_i cost_i * (1 - store_i), and every memory
 * measurement of the program's allocation timeline at or below the limit;
 * with control flow every path contributes its own timeline (Sec. IV-B).
 * The timeline is a list of events; each changes the running total of the
 * current path by an affine amount and records one measurement:
 *   ALLOC / FREE      +amount / -amount
 *   PRODUCE i         +size_i                     the forward pass creates A_i
 *   DROP i            -size_i * (1 - store_i)     after its forward use
 *   RECOMPUTE i       +(overhead_i + size_i) * (1 - store_i)   backward rebuild
 *   RECOMPUTE_DONE i  -overhead_i * (1 - store_i) rebuild temporaries freed
 *   RELEASE i         -size_i                     backward use is over
 *   PATH              starts the next path's timeline at 0
 * Units are the caller's (e.g. MiB and FLOP). Solved exactly by branch and
 * bound (exponential in the worst case; n_arrays <= 48). Among optimal
 * choices the lower peak wins, then storing lower-numbered arrays. */
typedef struct {
  double size;     /* memory of the array */
  double overhead; /* peak extra memory while recomputing it */
  double cost;     /* cost of recomputing it (e.g. FLOP) */
} adst_ilp_array;

typedef enum {
  ADST_ILP_ALLOC = 0,
  ADST_ILP_FREE = 1,
  ADST_ILP_PRODUCE = 2,
  ADST_ILP_DROP = 3,
  ADST_ILP_RECOMPUTE = 4,
  ADST_ILP_RECOMPUTE_DONE = 5,
  ADST_ILP_RELEASE = 6,
  ADST_ILP_PATH = 7
} adst_ilp_kind;

typedef struct {
  int32_t kind;  /* adst_ilp_kind */
  int32_t array; /* array index for PRODUCE .. RELEASE */
  double amount; /* for ALLOC / FREE, >= 0 */
} adst_ilp_event;

typedef struct {
  double objective;     /* recompute cost of the choice */
  double peak;          /* largest measurement under the choice */
  int64_t measurements; /* measurements over all paths */
  int64_t nodes;        /* search nodes visited */
  int32_t paths;
  int32_t reserved;
} adst_ilp_info;

/* Host only. store_out[i] receives 1 (store) or 0 (recompute); info
 * (optional) the objective and peak. Errors: ADST_ERR_ARG (NULL arrays or
 * events with a positive count, n_arrays outside [0, 48], a bad event kind
 * or index, a negative or non-finite amount or limit), ADST_ERR_BUDGET (no
 * choice fits the limit). */
adst_status adst_ilp_solve(const adst_ilp_array* arrays, int32_t n_arrays,
                           const adst_ilp_event* events, int64_t n_events, double limit,
                           int32_t* store_out, adst_ilp_info* info);

/* ---- Measurement and observability ------------------------------------
 * Per-kernel launch statistics of the last adst_vjp call on this thread
 * that ran with ADST_TRACE (host only, no GPU call). With ADST_TRACE every
 * launch (every pipelined sequence of launches for the in-place kind) is
 * bracketed by a HIP event pair on the call's stream, so ms_sum / launches
 * is the kernel's average duration; alg_bytes_sum is the algorithmic HBM
 * bytes of those launches (each input read once and each output written
 * once per launch: a launch of n fused steps moves one step's bytes). name
 * is the kernel's base name as a profiler reports it, with the variant in
 * angle brackets (e.g. "fwd_allencahn3d7_n<3,store>", "jacobi_march<adj,6>").
 * Writes min(cap, n) entries to out (out may be NULL when cap == 0) and the
 * count to *n_out. Errors: ADST_ERR_ARG (NULL n_out, bad cap). */
typedef struct {
  char name[56];
  int32_t phase;          /* 0 forward sweep, 1 recomputation, 2 adjoint, 3 loss and seed,
                             4 the constants' final sum (the phase of its first launch) */
  int32_t reserved;
  int64_t launches;       /* kernel dispatches */
  double ms_sum;          /* summed duration (ms) */
  double ms_min, ms_max;  /* per dispatch (a pipelined sequence: its average dispatch) */
  double alg_bytes_sum;   /* algorithmic bytes of all those dispatches */
} adst_kernel_stat;

adst_status adst_trace_kernels(adst_kernel_stat* out, int32_t cap, int32_t* n_out);

/* Device-to-device copy of `bytes` (a multiple of 4) from src to dst on
 * `stream`, one 16-byte vector per work-item when both pointers are 16-byte
 * aligned. adst_forward uses it for steps = 0; the benchmark times it as the
 * plain-copy bandwidth ceiling the stencil kernels are compared with.
 * Errors: ADST_ERR_ARG (NULL pointer with bytes > 0, misaligned pointer or
 * size, overlapping ranges), ADST_ERR_HIP. */
adst_status adst_copy(void* dst, const void* src, uint64_t bytes, hipStream_t stream);

/* Static description of a status code. */
const char* adst_status_str(adst_status status);

/* Thread-local detail of the last failure on this thread ("" if none). */
const char* adst_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* ADST_H */
