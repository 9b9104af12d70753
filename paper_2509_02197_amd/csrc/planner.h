// Host-side checkpoint planner: turns (steps, usable slots, schedule,
// whether the adjoint reads state) into an explicit action list over named
// buffers. No GPU code; adst_plan and adst_plan_actions run on any host.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "adst.h"

namespace adst {

struct Plan {
  int32_t steps = 0;
  int32_t sched = ADST_SCHED_STORE_ALL;  // resolved
  int32_t slots = 0;                     // slots the actions use (x0 excluded)
  bool needs_state = false;
  int64_t fwd_total = 0;     // forward steps (a fused launch counts its n)
  int64_t adj_total = 0;     // adjoint steps
  int64_t fwd_launches = 0;  // forward actions (a fused launch counts 1)
  int64_t adj_launches = 0;  // adjoint actions
  std::vector<adst_action> acts;
};

// Minimal forward steps to make the inputs of l consecutive steps available
// in reverse order from one checkpoint, with c checkpoints in total
// (Griewank's closed form). Requires l >= 1, c >= 1.
int64_t binomial_cost(int64_t l, int64_t c);

// Slots the store-all schedule needs for T steps: x_1 .. x_{T-2}.
inline int64_t store_all_slots(int64_t T) { return T > 2 ? T - 2 : 0; }

// Build the action list. slots_avail is the number of checkpoint slots the
// budget allows (x0 excluded). sched may be AUTO. fuse_fwd lets up to that
// many forward steps whose intermediate states nothing reads share one launch
// (FWD2 with n steps; 1 = no fusion); fuse_adj does the same for state-free
// adjoint steps (ADJ2). pair_tail: a run into a checkpoint slot that would
// end with one step after a launch of fuse_fwd steps ends with two launches
// of about half that depth instead, for kinds where those cost less (the
// step count, the launch count and the stored states stay the same).
// pipelined (the in-place kind) turns a state-free plan into one pipelined
// forward run and one pipelined reverse run (FWDW, ADJW). Returns ADST_OK or
// ADST_ERR_BUDGET / ADST_ERR_ARG / ADST_ERR_UNSUPPORTED with *err filled.
adst_status build_plan(int32_t steps, int64_t slots_avail, int32_t sched, bool needs_state,
                       int32_t fuse_fwd, int32_t fuse_adj, bool pair_tail, bool pipelined,
                       Plan* out, std::string* err);

}  // namespace adst
