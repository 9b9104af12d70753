// Exact store/recompute selection for a general program (host only).
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "adst.h"

namespace adst {

struct IlpResult {
  bool feasible = false;
  std::vector<int32_t> v;  // 1 = store, 0 = recompute
  double objective = 0.0, peak = 0.0;
  int64_t nodes = 0, measurements = 0;
  int32_t paths = 0;
};

// Builds the measurement rows of every path from the event list and solves
// the integer program exactly. ADST_ERR_ARG for malformed events,
// ADST_ERR_BUDGET when no choice fits the limit.
adst_status ilp_solve(const adst_ilp_array* arrays, int32_t n, const adst_ilp_event* events,
                      int64_t n_events, double limit, IlpResult* out, std::string* err);

}  // namespace adst
