// Exact store/recompute selection: the integer program of the paper's
// Sec. IV-A (with the per-path constraints of Sec. IV-B), solved by
// depth-first branch and bound without an external solver.
//
// Variables: v_i in {0, 1} per forwarded array (1 = store). Objective:
// minimise sum_i c_i (1 - v_i). Constraints: every memory measurement m_j,
// an affine function a_j + sum_i b_ji v_i built from the allocation timeline
// of its control-flow path, stays at or below the limit.
//
// Search: variables are fixed in index order, "store" first. A node is cut
// when some measurement cannot reach the limit even with the most favourable
// completion (each open variable at the value that minimises that row), or
// when its recompute cost already exceeds the best found. Among assignments
// of equal cost the lower peak wins, then the one storing lower-numbered
// arrays, so the result is unique.

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <string>
#include <vector>

#include "ilp.h"

namespace adst {


namespace {

struct Rows {
  int n = 0;
  std::vector<double> a;  // constant of each measurement
  std::vector<double> b;  // coefficients, row-major [rows][n]
  int rows() const { return (int)a.size(); }
};

class Search {
 public:
  Search(const Rows& r, const std::vector<double>& cost, double limit)
      : R(r), cost_(cost), limit_(limit), n_(r.n) {
    const int m = R.rows();
    cur_.assign(m, 0.0);
    open_min_.assign(m, 0.0);
    for (int j = 0; j < m; ++j) {
      cur_[j] = R.a[j];
      for (int i = 0; i < n_; ++i) open_min_[j] += std::min(0.0, R.b[j * n_ + i]);
    }
    v_.assign(n_, 0);
  }

  void run(IlpResult* out) {
    dfs(0, 0.0);
    out->feasible = found_;
    out->v = best_v_;
    out->objective = best_cost_;
    out->peak = best_peak_;
    out->nodes = nodes_;
  }

 private:
  const Rows& R;
  const std::vector<double>& cost_;
  double limit_;
  int n_;
  std::vector<double> cur_, open_min_;
  std::vector<int32_t> v_, best_v_;
  bool found_ = false;
  double best_cost_ = 0.0, best_peak_ = 0.0;
  int64_t nodes_ = 0;

  // Tolerance for sums of sizes given in floating point.
  bool over(double x) const { return x > limit_ + 1e-9 * std::max(1.0, std::fabs(limit_)); }

  bool can_fit() const {
    for (int j = 0; j < R.rows(); ++j)
      if (over(cur_[j] + open_min_[j])) return false;
    return true;
  }

  void assign(int i, int val, double sign) {
    for (int j = 0; j < R.rows(); ++j) {
      const double bji = R.b[j * n_ + i];
      open_min_[j] -= sign * std::min(0.0, bji);
      cur_[j] += sign * bji * val;
    }
  }

  bool better(double c, double pk) const {
    if (!found_) return true;
    if (c != best_cost_) return c < best_cost_;
    if (pk != best_peak_) return pk < best_peak_;
    return false;  // equal: the earlier leaf stores lower-numbered arrays
  }

  void dfs(int i, double c) {
    ++nodes_;
    if (found_ && c > best_cost_) return;
    if (!can_fit()) return;
    if (i == n_) {
      double pk = -INFINITY;
      for (double x : cur_) pk = std::max(pk, x);
      if (better(c, pk)) {
        found_ = true;
        best_cost_ = c;
        best_peak_ = pk;
        best_v_ = v_;
      }
      return;
    }
    for (int val = 1; val >= 0; --val) {
      v_[i] = val;
      assign(i, val, +1.0);
      dfs(i + 1, c + (val ? 0.0 : cost_[i]));
      assign(i, val, -1.0);
    }
  }
};

}  // namespace

// Build the measurement rows from the event list, then search.
adst_status ilp_solve(const adst_ilp_array* arrays, int32_t n, const adst_ilp_event* events,
                      int64_t n_events, double limit, IlpResult* out, std::string* err) {
  Rows R;
  R.n = n;
  double a = 0.0;
  std::vector<double> b(n, 0.0);
  int32_t paths = 0;
  bool open_path = false;
  auto record = [&]() {
    R.a.push_back(a);
    R.b.insert(R.b.end(), b.begin(), b.end());
    open_path = true;
  };
  for (int64_t k = 0; k < n_events; ++k) {
    const adst_ilp_event& e = events[k];
    if (e.kind == ADST_ILP_PATH) {
      if (open_path) ++paths;
      a = 0.0;
      std::fill(b.begin(), b.end(), 0.0);
      open_path = false;
      continue;
    }
    if (e.kind == ADST_ILP_ALLOC || e.kind == ADST_ILP_FREE) {
      if (!std::isfinite(e.amount) || e.amount < 0) {
        *err = "event " + std::to_string(k) + ": amount must be finite and >= 0";
        return ADST_ERR_ARG;
      }
      a += e.kind == ADST_ILP_ALLOC ? e.amount : -e.amount;
      record();
      continue;
    }
    if (e.array < 0 || e.array >= n) {
      *err = "event " + std::to_string(k) + ": array index out of range";
      return ADST_ERR_ARG;
    }
    const adst_ilp_array& A = arrays[e.array];
    const int i = e.array;
    switch (e.kind) {
      case ADST_ILP_PRODUCE:  // +S
        a += A.size;
        break;
      case ADST_ILP_DROP:  // -S (1 - v)
        a -= A.size;
        b[i] += A.size;
        break;
      case ADST_ILP_RECOMPUTE:  // +(R + S)(1 - v)
        a += A.overhead + A.size;
        b[i] -= A.overhead + A.size;
        break;
      case ADST_ILP_RECOMPUTE_DONE:  // -R (1 - v)
        a -= A.overhead;
        b[i] += A.overhead;
        break;
      case ADST_ILP_RELEASE:  // -S
        a -= A.size;
        break;
      default:
        *err = "event " + std::to_string(k) + ": unknown kind";
        return ADST_ERR_ARG;
    }
    record();
  }
  if (open_path) ++paths;
  std::vector<double> cost(n);
  for (int i = 0; i < n; ++i) cost[i] = arrays[i].cost;
  Search s(R, cost, limit);
  s.run(out);
  out->measurements = R.rows();
  out->paths = paths;
  if (!out->feasible) {
    *err = "no store/recompute choice keeps every measurement within the limit";
    return ADST_ERR_BUDGET;
  }
  return ADST_OK;
}

}  // namespace adst
