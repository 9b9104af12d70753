// Checkpoint planner (host only).
//
// The store/recompute decision of the paper's Sec. IV, specialised to one
// time loop whose steps all cost the same and whose length T is known before
// the sweep starts (Sec. III-A: structured loops with static bounds). For this
// case the optimum is the binomial schedule of Revolve (cited in the related
// work), which the BINOMIAL plan realises; STORE_ALL is the paper's default
// and UNIFORM a simple manual choice. When the adjoint of a step reads no
// forwarded value (a linear step: only nonlinear uses need forwarded data,
// Sec. IV), nothing is stored or recomputed at any budget.
//
// A plan is an explicit action list over named buffers (adst.h): the planner
// decides which buffer every forward step writes, so checkpoints are written
// in place by the producing step and restores are pointer choices; the
// executor only interprets the list.

#include "planner.h"

#include <algorithm>

namespace adst {

int64_t binomial_cost(int64_t l, int64_t c) {
  // Griewank: with beta(c, r) = C(c + r, c) and r minimal with
  // beta(c, r) >= l, the cost is r*l - beta(c + 1, r - 1).
  if (l <= 1) return 0;
  c = std::min(c, l);
  int64_t r = 0, beta = 1, beta_prev = 1;  // beta = beta(c, r)
  while (beta < l) {
    beta_prev = beta;
    ++r;
    beta = beta * (c + r) / r;  // exact: C(c+r, r) = C(c+r-1, r-1) (c+r)/r
  }
  // beta(c + 1, r - 1) = C(c + r, r - 1) = beta(c, r - 1) (c + r) / (c + 1)
  return r * l - beta_prev * (c + r) / (c + 1);
}

namespace {

// Smallest m in [1, l-1] minimising m + G(l-m, c-1) + G(m, c). Each term is
// a convex function of m (G(., c) has non-decreasing increments), so the
// first m whose forward difference is non-negative is the smallest minimiser.
int64_t best_split(int64_t l, int64_t c) {
  auto f = [&](int64_t m) { return m + binomial_cost(l - m, c - 1) + binomial_cost(m, c); };
  int64_t lo = 1, hi = l - 1;
  while (lo < hi) {
    int64_t mid = lo + (hi - lo) / 2;
    if (f(mid + 1) - f(mid) >= 0)
      hi = mid;
    else
      lo = mid + 1;
  }
  return lo;
}

class Builder {
 public:
  Builder(int32_t T, bool needs_state, int32_t fuse_fwd, int32_t fuse_adj, bool pair_tail)
      : T_(T), needs_state_(needs_state), fuse_fwd_(std::max(fuse_fwd, 1)),
        fuse_adj_(std::max(fuse_adj, 1)), pair_tail_(pair_tail && fuse_fwd > 2) {}

  std::vector<adst_action> acts;
  int32_t slots_used = 0;
  int64_t nfwd = 0, fwd_launches = 0, adj_launches = 0;

  int32_t alloc_slot() {
    if (!free_.empty()) {
      int32_t s = free_.back();
      free_.pop_back();
      return s;
    }
    return ADST_BUF_SLOT0 + slots_used++;
  }
  void release_slot(int32_t b) { free_.push_back(b); }

  void fwd(int32_t t, int32_t src, int32_t dst) {
    acts.push_back({ADST_OP_FWD, t, src, dst, 1});
    ++nfwd;
    ++fwd_launches;
  }
  // Steps t-n+1..t in one launch; x_{t-n+1}..x_{t-1} are never materialised.
  void fwdn(int32_t t, int32_t n, int32_t src, int32_t dst) {
    acts.push_back({ADST_OP_FWD2, t, src, dst, n});
    nfwd += n;
    ++fwd_launches;
  }

  static int32_t other_work(int32_t cur) {
    return cur == ADST_BUF_W0 ? ADST_BUF_W1 : ADST_BUF_W0;
  }

  // From buffer b holding x_i, compute x_{i+1}..x_j through the work buffers;
  // the last step writes final_dst instead when one is given. Returns the
  // buffer holding x_j. The intermediate states are read by nothing else, so
  // with fusion on they are computed up to fuse_fwd_ steps per launch. With
  // pair_tail_, a run into a slot whose last fuse_fwd_ + 1 steps would be a
  // full launch and a single step takes them as two launches of about half
  // depth. Runs into a work buffer keep the single step last: the adjoint
  // step that reads the result may take it into its own launch, or a
  // store-through launch the steps after it.
  int32_t advance(int32_t b, int32_t i, int32_t j, int32_t final_dst) {
    int32_t cur = b;
    int32_t t = i;
    while (t < j) {
      int32_t n = std::min(fuse_fwd_, j - t);
      if (pair_tail_ && final_dst >= ADST_BUF_SLOT0 && j - t == fuse_fwd_ + 1)
        n = (fuse_fwd_ + 2) / 2;
      t += n;
      const int32_t dst = (t == j && final_dst != ADST_BUF_NONE) ? final_dst : other_work(cur);
      if (n >= 2)
        fwdn(t, n, cur, dst);
      else
        fwd(t, cur, dst);
      cur = dst;
    }
    return cur;
  }

  // Adjoint of step t with x_{t-1} in xbuf. The first adjoint step (t = T)
  // is preceded by the last forward step, which only now leaves x_{T-1} in
  // hand, and by the loss and seed.
  void adjoint(int32_t t, int32_t xbuf) {
    if (!seeded_) {
      fwd(T_, xbuf, ADST_BUF_XT);
      seed();
    }
    acts.push_back({ADST_OP_ADJ, t, needs_state_ ? xbuf : ADST_BUF_NONE, ADST_BUF_NONE, 1});
    ++adj_launches;
  }

  void seed() {
    acts.push_back({ADST_OP_SEED, T_, ADST_BUF_XT, ADST_BUF_NONE, 0});
    seeded_ = true;
  }

  // Reverse steps i+1..i+l from x_i in `base` keeping every state but the
  // last in its own slot (l - 2 slots; optimal whenever c >= l - 1).
  void reverse_store_all(int32_t i, int32_t l, int32_t base) {
    std::vector<int32_t> where(l);
    std::vector<int32_t> taken;
    where[0] = base;
    int32_t cur = base;
    for (int32_t j = 1; j <= l - 1; ++j) {
      int32_t dst;
      if (j <= l - 2) {
        dst = alloc_slot();
        taken.push_back(dst);
      } else {
        dst = other_work(cur);
      }
      fwd(i + j, cur, dst);
      where[j] = dst;
      cur = dst;
    }
    for (int32_t j = l; j >= 1; --j) adjoint(i + j, where[j - 1]);
    for (auto it = taken.rbegin(); it != taken.rend(); ++it) release_slot(*it);
  }

  // Binomial reversal of steps i+1..i+l from x_i in `base` with c checkpoints
  // (base included). Iterative, with an explicit stack of pending left parts.
  void reverse_binomial(int32_t i, int32_t l, int32_t c, int32_t base) {
    struct Pending { int32_t i, l, c, base, slot; };
    std::vector<Pending> stack;
    for (;;) {
      bool leaf = true;
      if (l == 1) {
        adjoint(i + 1, base);
      } else if (c >= l - 1) {
        reverse_store_all(i, l, base);
      } else if (c == 1) {
        for (int32_t t = i + l; t >= i + 1; --t) adjoint(t, advance(base, i, t - 1, ADST_BUF_NONE));
      } else {
        leaf = false;
        const int32_t m = static_cast<int32_t>(best_split(l, c));
        const int32_t s = alloc_slot();
        advance(base, i, i + m, s);
        stack.push_back({i, m, c, base, s});
        i += m;
        l -= m;
        c -= 1;
        base = s;
      }
      if (leaf) {
        if (stack.empty()) return;
        Pending p = stack.back();
        stack.pop_back();
        release_slot(p.slot);
        i = p.i;
        l = p.l;
        c = p.c;
        base = p.base;
      }
    }
  }

  void reverse_uniform(int32_t c) {
    const int32_t T = T_;
    const int32_t k = (T + c - 1) / c;
    std::vector<int32_t> where(T, ADST_BUF_NONE);  // checkpoint buffers by state
    where[0] = ADST_BUF_X0;
    // Sweep: the checkpoints at the multiples of k below T-1 are written in
    // place by the step producing them; the states between are transient.
    int32_t cur = ADST_BUF_X0, at = 0;
    for (int32_t cp = k; cp <= T - 2; cp += k) {
      const int32_t s = alloc_slot();
      cur = advance(cur, at, cp, s);
      where[cp] = s;
      at = cp;
    }
    cur = advance(cur, at, T - 1, ADST_BUF_NONE);
    adjoint(T, cur);
    for (int32_t t = T - 1; t >= 1; --t) {
      const int32_t s = t - 1;
      const int32_t b = (s / k) * k;
      adjoint(t, advance(where[b], b, s, ADST_BUF_NONE));
    }
  }

  // No adjoint step reads state: one sweep straight to x_T, the seed, then
  // the adjoint steps, up to fuse_adj_ per launch.
  void elided() {
    advance(ADST_BUF_X0, 0, T_, ADST_BUF_XT);
    seed();
    int32_t t = T_;
    while (t >= 1) {
      const int32_t n = std::min(fuse_adj_, t);
      if (n >= 2) {
        acts.push_back({ADST_OP_ADJ2, t, ADST_BUF_NONE, ADST_BUF_NONE, n});
        t -= n;
      } else {
        acts.push_back({ADST_OP_ADJ, t, ADST_BUF_NONE, ADST_BUF_NONE, 1});
        t -= 1;
      }
      ++adj_launches;
    }
  }

  // The in-place kind without a tape: its T steps run as one pipelined
  // forward sequence straight into x_T, then the seed, then one pipelined
  // reverse sequence.
  void pipelined() {
    acts.push_back({ADST_OP_FWDW, T_, ADST_BUF_X0, ADST_BUF_XT, T_});
    nfwd += T_;
    ++fwd_launches;
    seed();
    acts.push_back({ADST_OP_ADJW, T_, ADST_BUF_NONE, ADST_BUF_NONE, T_});
    ++adj_launches;
  }

  void zero_steps() { acts.push_back({ADST_OP_SEED, 0, ADST_BUF_X0, ADST_BUF_NONE, 0}); }

 private:
  int32_t T_;
  bool needs_state_;
  int32_t fuse_fwd_, fuse_adj_;  // most steps per launch (1 = no fusion)
  bool pair_tail_;               // see advance()
  bool seeded_ = false;
  std::vector<int32_t> free_;
};

// Forward steps a schedule will take, from its definition, so that absurdly
// long plans are refused before any list is built.
int64_t predicted_fwd(int32_t T, int32_t sched, int64_t c, bool needs_state) {
  if (T == 0) return 0;
  if (!needs_state || sched == ADST_SCHED_STORE_ALL) return T;
  if (sched == ADST_SCHED_BINOMIAL) return binomial_cost(T, c) + 1;
  // UNIFORM: every x_s, s <= T-2, is recomputed from the checkpoint below it.
  const int64_t k = (T + c - 1) / c;
  int64_t total = T;
  for (int64_t s = 0; s <= T - 2; ++s) total += s % k;
  return total;
}

constexpr int64_t kMaxActions = int64_t(1) << 24;

}  // namespace

adst_status build_plan(int32_t steps, int64_t slots_avail, int32_t sched, bool needs_state,
                       int32_t fuse_fwd, int32_t fuse_adj, bool pair_tail, bool pipelined,
                       Plan* out, std::string* err) {
  if (steps < 0) {
    *err = "steps must be >= 0";
    return ADST_ERR_ARG;
  }
  if (sched < ADST_SCHED_AUTO || sched > ADST_SCHED_BINOMIAL) {
    *err = "unknown schedule";
    return ADST_ERR_ARG;
  }
  if (slots_avail < 0) slots_avail = 0;
  const int64_t need_all = store_all_slots(steps);
  int32_t resolved = sched;
  if (sched == ADST_SCHED_AUTO)
    resolved = (!needs_state || slots_avail >= need_all) ? ADST_SCHED_STORE_ALL
                                                         : ADST_SCHED_BINOMIAL;
  if (needs_state && resolved == ADST_SCHED_STORE_ALL && slots_avail < need_all) {
    *err = "store-all needs " + std::to_string(need_all) + " checkpoint slots, the budget holds " +
           std::to_string(slots_avail);
    return ADST_ERR_BUDGET;
  }
  // c = checkpoints including x0; more than T - 1 cannot help.
  const int64_t c = std::min<int64_t>(slots_avail, need_all) + 1;
  const int64_t nf = predicted_fwd(steps, resolved, c, needs_state);
  if (nf + 2 * int64_t(steps) + 2 > kMaxActions) {
    *err = "plan would need " + std::to_string(nf) +
           " forward steps; raise the budget or lower the step count";
    return ADST_ERR_UNSUPPORTED;
  }

  Builder b(steps, needs_state, fuse_fwd, needs_state ? 1 : fuse_adj, pair_tail);
  if (steps == 0) {
    b.zero_steps();
  } else if (!needs_state && pipelined) {
    b.pipelined();
  } else if (!needs_state) {
    b.elided();
  } else if (resolved == ADST_SCHED_STORE_ALL) {
    b.reverse_store_all(0, steps, ADST_BUF_X0);
  } else if (resolved == ADST_SCHED_UNIFORM) {
    b.reverse_uniform(static_cast<int32_t>(c));
  } else {
    b.reverse_binomial(0, steps, static_cast<int32_t>(c), ADST_BUF_X0);
  }

  out->steps = steps;
  out->sched = resolved;
  out->slots = b.slots_used;
  out->needs_state = needs_state;
  out->fwd_total = b.nfwd;
  out->adj_total = steps;
  out->fwd_launches = b.fwd_launches;
  out->adj_launches = b.adj_launches;
  out->acts = std::move(b.acts);
  return ADST_OK;
}

}  // namespace adst
