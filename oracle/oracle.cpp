// Plain CPU oracle for the reverse-mode gradient of a time-iterated stencil.
//
// TEST INFRASTRUCTURE ONLY. Nothing in the product library links, loads or
// calls this file: only the tests, the smoke check and the benchmark's CPU
// baseline leg use it. It shares no source, header, constant or helper with
// the HIP path.
//
// What it computes (paper, Sec. IV: checkpointing only changes *where* a
// forwarded value comes from, never the gradient itself): the plain
// store-all reverse-mode gradient.
//   1. tape[0] = x0, tape[t] = F(tape[t-1]; K) for t = 1..T       (forward)
//   2. loss L(x_T) and its seed g_T = dL/dx_T                       (Sec. V-A:
//      a sum reduction scalarises the output)
//   3. for t = T..1: g_{t-1} = J_t^T g_t, in *scatter* form: every output
//      point c pushes g_t[c] * d x_t[c] / d x_{t-1}[n] into g_{t-1}[n] for
//      each n it read (Sec. III-C, reversed maps write into input gradients;
//      Sec. II "Gradient Accumulation": gradients start at zero and
//      accumulate, and an overwritten array's gradient is cleared, which is
//      why g_{t-1} is a fresh zeroed array each step).
//      The coefficient-field gradient dK accumulates the same way over all
//      steps (a multiply-read array, Sec. II).
//   4. dx0 = g_0.
// Optionally the gradients of the two scalar step constants p[0], p[1]
// (Sec. II: a value every point of every step reads is a multiply-read
// input whose gradient accumulates over all its uses): for each step t and
// point c, g_t[c] times the step's partial dF_c/dp at x_{t-1}, summed in
// double; for the in-place kind each point update's own partial times the
// gradient its output holds when the update is reversed.
// A tangent-linear (forward-mode) sweep is included so that tests can check
// the adjoint dot-product identity <J v, w> = <v, J^T w>, also along the
// constants.
//
// The four step kinds (the stencil programs the gradient is taken of):
//   JACOBI2D5  x'[c] = w * (x[c] + x[W] + x[E] + x[S] + x[N]) on interior
//              points, x'[c] = x[c] on the outer ring (boundary held fixed);
//              p[0] = w.
//   ALLENCAHN3D7  every point is updated, out-of-grid neighbours read 0:
//              lap = sum of the 6 face neighbours - 6 x[c]
//              x'  = (x[c] + D*lap) - C*x[c]^3;            p[0] = D, p[1] = C.
//   GAUSSSEIDEL2D5  the in-place counterpart of JACOBI2D5: interior points
//              are overwritten one at a time in row-major order (x fastest)
//              with x[c] = w * ((((x[c] + x[E]) + x[N]) + x[S]) + x[W]), so
//              x[S] and x[W] already hold this sweep's values while x[c],
//              x[E] and x[N] still hold the previous sweep's; the ring stays
//              fixed; p[0] = w. (The paper's Seidel2d case study, Sec. V-B,
//              names an in-place two-dimensional stencil in a time loop
//              without printing it; this is the five-point reading.)
//   VARDIFF2D9 conservative edge form of div(K grad x) on the isotropic
//              9-point stencil with no-flux boundary (edges leaving the grid
//              are dropped): x' = x[c] + dt * sum_n c_n (K[c]+K[n]) (x[n]-x[c]),
//              c_n = 1/3 for axis neighbours, 1/12 for diagonal ones;
//              p[0] = dt.
// Optional limiter (a branch in every step, Sec. III-B's data-dependent
// control flow): with bounds lim = {lo, hi} every point's new value y is
// replaced by lo if y < lo, by hi if y > hi, and kept otherwise (the ring of
// the 2-D kinds included). Its derivative is that of the branch taken: 1
// where lo <= y <= hi, 0 elsewhere. The reverse sweep recovers each branch
// outcome by re-evaluating y from the stored x_{t-1} (recomputation instead
// of a stored branch record, which the forward's fixed evaluation order
// makes exact). Not defined for the in-place kind.
// Evaluation order and rounding: each forward formula is evaluated exactly in
// the order written above, left to right, in the working precision R, with no
// contraction into fused multiply-adds (built with -ffp-contract=off).
// Arrays are row-major [nz][ny][nx], x fastest.
//
// The loss is accumulated in double whatever R is:
//   HALF_SQ       L = sum 0.5 x_T^2,           seed = x_T
//   DOT_W         L = sum aux * x_T,           seed = aux
//   HALF_SQ_DIFF  d = x_T - aux (in R), L = sum 0.5 d^2, seed = d
//   SEED          L = sum aux * x_T,           seed = aux (explicit cotangent)

#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <vector>

namespace {

enum Kind { JACOBI2D5 = 0, ALLENCAHN3D7 = 1, VARDIFF2D9 = 2, GAUSSSEIDEL2D5 = 3 };
enum Loss { HALF_SQ = 0, DOT_W = 1, HALF_SQ_DIFF = 2, SEED = 3 };

struct Grid {
  int64_t nx, ny, nz;
  int64_t size() const { return nx * ny * nz; }
  int64_t at(int64_t x, int64_t y, int64_t z) const { return (z * ny + y) * nx + x; }
  bool inside(int64_t x, int64_t y, int64_t z) const {
    return x >= 0 && x < nx && y >= 0 && y < ny && z >= 0 && z < nz;
  }
};

// The 8 neighbours of the 9-point stencil, in the summation order.
const int kNine[8][2] = {{-1, 0}, {1, 0}, {0, -1}, {0, 1},
                         {-1, -1}, {1, -1}, {-1, 1}, {1, 1}};
// The 6 face neighbours of the 7-point stencil, in the summation order.
const int kSeven[6][3] = {{-1, 0, 0}, {1, 0, 0}, {0, -1, 0},
                          {0, 1, 0}, {0, 0, -1}, {0, 0, 1}};

template <class R> R nine_weight(int n) {
  // Axis neighbours carry 1/3, diagonal ones 1/12, rounded to R.
  return n < 4 ? R(1) / R(3) : R(1) / R(12);
}

// ---------------------------------------------------------------- forward
// One in-place Gauss-Seidel sweep over the interior in row-major order.
template <class R>
void gauss_seidel_sweep(const Grid& g, const double* p, R* x) {
  const R w = R(p[0]);
  for (int64_t y = 1; y < g.ny - 1; ++y)
    for (int64_t i = 1; i < g.nx - 1; ++i) {
      const int64_t c = g.at(i, y, 0);
      R s = x[c];
      s += x[g.at(i + 1, y, 0)];  // E: previous sweep's value
      s += x[g.at(i, y + 1, 0)];  // N: previous sweep's value
      s += x[g.at(i, y - 1, 0)];  // S: this sweep's value
      s += x[g.at(i - 1, y, 0)];  // W: this sweep's value
      x[c] = w * s;
    }
}

template <class R>
void step_forward(int kind, const Grid& g, const double* p, const R* x,
                  const R* K, R* out) {
  if (kind == GAUSSSEIDEL2D5) {
    std::memcpy(out, x, sizeof(R) * g.size());
    gauss_seidel_sweep<R>(g, p, out);
    return;
  }
  for (int64_t z = 0; z < g.nz; ++z)
    for (int64_t y = 0; y < g.ny; ++y)
      for (int64_t i = 0; i < g.nx; ++i) {
        const int64_t c = g.at(i, y, z);
        if (kind == JACOBI2D5) {
          const R w = R(p[0]);
          bool interior = i > 0 && i < g.nx - 1 && y > 0 && y < g.ny - 1;
          if (interior) {
            R s = x[c];
            s += x[g.at(i - 1, y, z)];
            s += x[g.at(i + 1, y, z)];
            s += x[g.at(i, y - 1, z)];
            s += x[g.at(i, y + 1, z)];
            out[c] = w * s;
          } else {
            out[c] = x[c];
          }
        } else if (kind == ALLENCAHN3D7) {
          const R D = R(p[0]), C = R(p[1]);
          R nb[6];
          for (int n = 0; n < 6; ++n) {
            int64_t a = i + kSeven[n][0], b = y + kSeven[n][1], d = z + kSeven[n][2];
            nb[n] = g.inside(a, b, d) ? x[g.at(a, b, d)] : R(0);
          }
          const R a = x[c];
          R lap = nb[0] + nb[1];
          lap += nb[2];
          lap += nb[3];
          lap += nb[4];
          lap += nb[5];
          lap = lap - R(6) * a;
          out[c] = (a + D * lap) - C * ((a * a) * a);
        } else {  // VARDIFF2D9
          const R dt = R(p[0]);
          R acc = R(0);
          for (int n = 0; n < 8; ++n) {
            int64_t a = i + kNine[n][0], b = y + kNine[n][1];
            if (!g.inside(a, b, z)) continue;
            const int64_t m = g.at(a, b, z);
            acc += (nine_weight<R>(n) * (K[c] + K[m])) * (x[m] - x[c]);
          }
          out[c] = x[c] + dt * acc;
        }
      }
}

// The step followed by the limiter (lim = {lo, hi}, or null for none).
template <class R>
void step_forward_lim(int kind, const Grid& g, const double* p, const double* lim, const R* x,
                      const R* K, R* out) {
  step_forward<R>(kind, g, p, x, K, out);
  if (!lim) return;
  const R lo = R(lim[0]), hi = R(lim[1]);
  for (int64_t c = 0; c < g.size(); ++c) {
    if (out[c] < lo)
      out[c] = lo;
    else if (out[c] > hi)
      out[c] = hi;
  }
}

// The branch outcome of the limiter at every point: 1 where the step's
// unlimited value y satisfies lo <= y <= hi (the value is kept), else 0.
template <class R>
void limiter_mask(int kind, const Grid& g, const double* p, const double* lim, const R* x,
                  const R* K, std::vector<R>& y, std::vector<unsigned char>& keep) {
  y.resize(g.size());
  keep.resize(g.size());
  step_forward<R>(kind, g, p, x, K, y.data());
  const R lo = R(lim[0]), hi = R(lim[1]);
  for (int64_t c = 0; c < g.size(); ++c) keep[c] = !(y[c] < lo) && !(y[c] > hi);
}

// -------------------------------------------------------- reverse (scatter)
// gin receives g_{t-1} (must be zeroed by the caller), dK (if non-null)
// accumulates; x is the step's input state x_{t-1}; gout is g_t.
// Reverse of one in-place sweep: the sweep is the product of point updates
// U_1 ... U_n (row-major), so its transpose applies U_n^T ... U_1^T, i.e. the
// points in reverse order; U_k^T moves g[k] into the adjoints of the values
// the update read: g[k] <- w*g[k] (its old value) and w*g[k] added to each
// neighbour (whatever sweep's value it was). The gradient of the overwritten
// value is cleared by the assignment, as for any overwrite.
// With s (the sum each update formed, recorded in forward order) and dw
// given, dw accumulates gc * s[c], the update's partial in w times the
// gradient of its output.
template <class R>
void gauss_seidel_reverse(const Grid& g, const double* p, R* gr, const R* s = nullptr,
                          double* dw = nullptr) {
  const R w = R(p[0]);
  for (int64_t y = g.ny - 2; y >= 1; --y)
    for (int64_t i = g.nx - 2; i >= 1; --i) {
      const int64_t c = g.at(i, y, 0);
      const R gc = gr[c];
      if (dw) *dw += double(gc) * double(s[c]);
      gr[c] = w * gc;
      gr[g.at(i - 1, y, 0)] += w * gc;
      gr[g.at(i + 1, y, 0)] += w * gc;
      gr[g.at(i, y - 1, 0)] += w * gc;
      gr[g.at(i, y + 1, 0)] += w * gc;
    }
}

template <class R>
void step_adjoint_scatter(int kind, const Grid& g, const double* p, const R* x,
                          const R* K, const R* gout, R* gin, R* dK) {
  if (kind == GAUSSSEIDEL2D5) {
    for (int64_t c = 0; c < g.size(); ++c) gin[c] += gout[c];
    gauss_seidel_reverse<R>(g, p, gin);
    return;
  }
  for (int64_t z = 0; z < g.nz; ++z)
    for (int64_t y = 0; y < g.ny; ++y)
      for (int64_t i = 0; i < g.nx; ++i) {
        const int64_t c = g.at(i, y, z);
        const R gc = gout[c];
        if (kind == JACOBI2D5) {
          const R w = R(p[0]);
          bool interior = i > 0 && i < g.nx - 1 && y > 0 && y < g.ny - 1;
          if (interior) {
            // x'[c] = w*(x[c]+x[W]+x[E]+x[S]+x[N]): each read gets w*g[c].
            gin[c] += w * gc;
            gin[g.at(i - 1, y, z)] += w * gc;
            gin[g.at(i + 1, y, z)] += w * gc;
            gin[g.at(i, y - 1, z)] += w * gc;
            gin[g.at(i, y + 1, z)] += w * gc;
          } else {
            gin[c] += gc;  // x'[c] = x[c]
          }
        } else if (kind == ALLENCAHN3D7) {
          const R D = R(p[0]), C = R(p[1]);
          const R a = x[c];
          // d x'[c] / d x[c] = 1 + D*(-6) - C*3a^2
          gin[c] += gc * ((R(1) + D * R(-6)) - C * (R(3) * (a * a)));
          // d x'[c] / d x[n] = D for every in-grid face neighbour n
          for (int n = 0; n < 6; ++n) {
            int64_t a2 = i + kSeven[n][0], b = y + kSeven[n][1], d = z + kSeven[n][2];
            if (g.inside(a2, b, d)) gin[g.at(a2, b, d)] += gc * D;
          }
        } else {  // VARDIFF2D9
          const R dt = R(p[0]);
          gin[c] += gc;  // the x[c] term outside the sum
          for (int n = 0; n < 8; ++n) {
            int64_t a = i + kNine[n][0], b = y + kNine[n][1];
            if (!g.inside(a, b, z)) continue;
            const int64_t m = g.at(a, b, z);
            const R cn = nine_weight<R>(n);
            // term = dt * cn * (K[c]+K[m]) * (x[m]-x[c])
            const R dterm_dx = dt * (cn * (K[c] + K[m]));
            gin[m] += gc * dterm_dx;
            gin[c] -= gc * dterm_dx;
            if (dK) {
              const R dterm_dK = dt * (cn * (x[m] - x[c]));
              dK[c] += gc * dterm_dK;
              dK[m] += gc * dterm_dK;
            }
          }
        }
      }
}

// ------------------------------------------------ scalar-constant partials
// d0[c] = dF_c/dp[0], d1[c] = dF_c/dp[1] of one step at its input x, the
// sub-expressions the forward step forms, in its order:
//   JACOBI2D5     dF/dw  = (((x[c]+x[W])+x[E])+x[S])+x[N] on interior points, 0 on the ring
//   ALLENCAHN3D7  dF/dD  = lap,  dF/dC = -((x[c]*x[c])*x[c])
//   VARDIFF2D9    dF/ddt = acc
// (The in-place kind's partials depend on the order of the sweep; see
// gauss_seidel_sums.)
template <class R>
void step_param_partials(int kind, const Grid& g, const R* x, const R* K, R* d0, R* d1) {
  for (int64_t z = 0; z < g.nz; ++z)
    for (int64_t y = 0; y < g.ny; ++y)
      for (int64_t i = 0; i < g.nx; ++i) {
        const int64_t c = g.at(i, y, z);
        d0[c] = R(0);
        d1[c] = R(0);
        if (kind == JACOBI2D5) {
          if (i > 0 && i < g.nx - 1 && y > 0 && y < g.ny - 1) {
            R s = x[c];
            s += x[g.at(i - 1, y, z)];
            s += x[g.at(i + 1, y, z)];
            s += x[g.at(i, y - 1, z)];
            s += x[g.at(i, y + 1, z)];
            d0[c] = s;
          }
        } else if (kind == ALLENCAHN3D7) {
          R nb[6];
          for (int n = 0; n < 6; ++n) {
            int64_t a = i + kSeven[n][0], b = y + kSeven[n][1], d = z + kSeven[n][2];
            nb[n] = g.inside(a, b, d) ? x[g.at(a, b, d)] : R(0);
          }
          const R a = x[c];
          R lap = nb[0] + nb[1];
          lap += nb[2];
          lap += nb[3];
          lap += nb[4];
          lap += nb[5];
          d0[c] = lap - R(6) * a;
          d1[c] = -((a * a) * a);
        } else if (kind == VARDIFF2D9) {
          R acc = R(0);
          for (int n = 0; n < 8; ++n) {
            int64_t a = i + kNine[n][0], b = y + kNine[n][1];
            if (!g.inside(a, b, z)) continue;
            const int64_t m = g.at(a, b, z);
            acc += (nine_weight<R>(n) * (K[c] + K[m])) * (x[m] - x[c]);
          }
          d0[c] = acc;
        }
      }
}

// The in-place sweep from x, recording at each interior point the sum the
// update multiplies by w (its partial in w, formed from the values the
// point reads at that moment).
template <class R>
void gauss_seidel_sums(const Grid& g, const double* p, const R* x, R* s_out) {
  const R w = R(p[0]);
  std::vector<R> a(x, x + g.size());
  std::fill(s_out, s_out + g.size(), R(0));
  for (int64_t y = 1; y < g.ny - 1; ++y)
    for (int64_t i = 1; i < g.nx - 1; ++i) {
      const int64_t c = g.at(i, y, 0);
      R s = a[c];
      s += a[g.at(i + 1, y, 0)];
      s += a[g.at(i, y + 1, 0)];
      s += a[g.at(i, y - 1, 0)];
      s += a[g.at(i - 1, y, 0)];
      s_out[c] = s;
      a[c] = w * s;
    }
}

// ---------------------------------------------------- forward mode (JVP)
// xd_out = J_x xd + J_K kd at the step input x.
template <class R>
void step_tangent(int kind, const Grid& g, const double* p, const R* x,
                  const R* K, const R* xd, const R* kd, R* xd_out) {
  if (kind == GAUSSSEIDEL2D5) {  // linear: the tangent takes the same sweep
    std::memcpy(xd_out, xd, sizeof(R) * g.size());
    gauss_seidel_sweep<R>(g, p, xd_out);
    return;
  }
  for (int64_t z = 0; z < g.nz; ++z)
    for (int64_t y = 0; y < g.ny; ++y)
      for (int64_t i = 0; i < g.nx; ++i) {
        const int64_t c = g.at(i, y, z);
        if (kind == JACOBI2D5) {
          const R w = R(p[0]);
          bool interior = i > 0 && i < g.nx - 1 && y > 0 && y < g.ny - 1;
          if (interior)
            xd_out[c] = w * (xd[c] + xd[g.at(i - 1, y, z)] + xd[g.at(i + 1, y, z)] +
                             xd[g.at(i, y - 1, z)] + xd[g.at(i, y + 1, z)]);
          else
            xd_out[c] = xd[c];
        } else if (kind == ALLENCAHN3D7) {
          const R D = R(p[0]), C = R(p[1]);
          R s = R(0);
          for (int n = 0; n < 6; ++n) {
            int64_t a = i + kSeven[n][0], b = y + kSeven[n][1], d = z + kSeven[n][2];
            if (g.inside(a, b, d)) s += xd[g.at(a, b, d)];
          }
          const R a = x[c];
          xd_out[c] = xd[c] + D * (s - R(6) * xd[c]) - C * (R(3) * a * a * xd[c]);
        } else {  // VARDIFF2D9
          const R dt = R(p[0]);
          R acc = R(0);
          for (int n = 0; n < 8; ++n) {
            int64_t a = i + kNine[n][0], b = y + kNine[n][1];
            if (!g.inside(a, b, z)) continue;
            const int64_t m = g.at(a, b, z);
            const R cn = nine_weight<R>(n);
            R kdsum = kd ? (kd[c] + kd[m]) : R(0);
            acc += cn * (kdsum * (x[m] - x[c]) + (K[c] + K[m]) * (xd[m] - xd[c]));
          }
          xd_out[c] = xd[c] + dt * acc;
        }
      }
}

template <class R>
int check_problem(int kind, const Grid& g, const R* K) {
  if (g.nx < 1 || g.ny < 1 || g.nz < 1) return -1;
  if (kind == JACOBI2D5 || kind == VARDIFF2D9 || kind == GAUSSSEIDEL2D5) {
    if (g.nz != 1) return -1;
  } else if (kind != ALLENCAHN3D7) {
    return -1;
  }
  if (kind == VARDIFF2D9 && !K) return -1;
  return 0;
}

template <class R>
int forward(int kind, const int64_t* n, const double* p, const double* lim, const R* x0,
            const R* K, int steps, R* xT) {
  Grid g{n[0], n[1], n[2]};
  if (check_problem(kind, g, K) || steps < 0) return -1;
  if (lim && kind == GAUSSSEIDEL2D5) return -1;
  std::vector<R> a(x0, x0 + g.size()), b(g.size());
  for (int t = 1; t <= steps; ++t) {
    step_forward_lim<R>(kind, g, p, lim, a.data(), K, b.data());
    a.swap(b);
  }
  std::memcpy(xT, a.data(), sizeof(R) * g.size());
  return 0;
}

template <class R>
int vjp(int kind, const int64_t* n, const double* p, const double* lim, const R* x0, const R* K,
        int steps, int loss, const R* aux, R* dx0, R* dK, R* xT, double* loss_out,
        double* dp_out) {
  Grid g{n[0], n[1], n[2]};
  if (check_problem(kind, g, K) || steps < 0) return -1;
  if (lim && kind == GAUSSSEIDEL2D5) return -1;
  if (loss < HALF_SQ || loss > SEED) return -1;
  if (loss != HALF_SQ && !aux) return -1;
  const int64_t N = g.size();

  // 1. store-all tape
  std::vector<std::vector<R>> tape(steps + 1, std::vector<R>(N));
  std::memcpy(tape[0].data(), x0, sizeof(R) * N);
  for (int t = 1; t <= steps; ++t)
    step_forward_lim<R>(kind, g, p, lim, tape[t - 1].data(), K, tape[t].data());
  const std::vector<R>& xt = tape[steps];

  // 2. loss and seed
  std::vector<R> gcur(N);
  double L = 0.0;
  for (int64_t i = 0; i < N; ++i) {
    if (loss == HALF_SQ) {
      L += 0.5 * (double(xt[i]) * double(xt[i]));
      gcur[i] = xt[i];
    } else if (loss == HALF_SQ_DIFF) {
      const R d = xt[i] - aux[i];
      L += 0.5 * (double(d) * double(d));
      gcur[i] = d;
    } else {  // DOT_W and SEED
      L += double(aux[i]) * double(xt[i]);
      gcur[i] = aux[i];
    }
  }

  // 3. reverse sweep, scatter form
  std::vector<R> gprev(N);
  std::vector<R> dk_acc;
  if (dK) dk_acc.assign(N, R(0));
  std::vector<R> d0, d1;
  double dp[2] = {0.0, 0.0};
  if (dp_out) {
    d0.resize(N);
    d1.resize(N);
  }
  std::vector<R> yv;
  std::vector<unsigned char> keep;
  for (int t = steps; t >= 1; --t) {
    if (lim) {  // the branch taken at each point: a clamped value has no dependence
      limiter_mask<R>(kind, g, p, lim, tape[t - 1].data(), K, yv, keep);
      for (int64_t i = 0; i < N; ++i)
        if (!keep[i]) gcur[i] = R(0);
    }
    if (dp_out && kind == GAUSSSEIDEL2D5) {
      // the sweep's own reverse carries the partials (see gauss_seidel_reverse)
      gauss_seidel_sums<R>(g, p, tape[t - 1].data(), d0.data());
      gprev = gcur;
      gauss_seidel_reverse<R>(g, p, gprev.data(), d0.data(), &dp[0]);
      gcur.swap(gprev);
      continue;
    }
    if (dp_out) {
      step_param_partials<R>(kind, g, tape[t - 1].data(), K, d0.data(), d1.data());
      for (int64_t i = 0; i < N; ++i) {
        dp[0] += double(gcur[i]) * double(d0[i]);
        dp[1] += double(gcur[i]) * double(d1[i]);
      }
    }
    std::fill(gprev.begin(), gprev.end(), R(0));  // clearing on overwrite
    step_adjoint_scatter<R>(kind, g, p, tape[t - 1].data(), K, gcur.data(),
                            gprev.data(), dK ? dk_acc.data() : nullptr);
    gcur.swap(gprev);
  }
  if (dp_out) {
    dp_out[0] = dp[0];
    dp_out[1] = dp[1];
  }

  // 4. outputs
  std::memcpy(dx0, gcur.data(), sizeof(R) * N);
  if (dK) std::memcpy(dK, dk_acc.data(), sizeof(R) * N);
  if (xT) std::memcpy(xT, xt.data(), sizeof(R) * N);
  if (loss_out) *loss_out = L;
  return 0;
}

template <class R>
int jvp(int kind, const int64_t* n, const double* p, const double* lim, const R* x0, const R* K,
        const R* v, const R* kappa, const double* pdot, int steps, R* xT, R* xdT) {
  Grid g{n[0], n[1], n[2]};
  if (check_problem(kind, g, K) || steps < 0 || !v) return -1;
  if (lim && kind == GAUSSSEIDEL2D5) return -1;
  std::vector<R> yv;
  std::vector<unsigned char> keep;
  const int64_t N = g.size();
  std::vector<R> x(x0, x0 + N), xn(N), xd(v, v + N), xdn(N), d0(N), d1(N);
  for (int t = 1; t <= steps; ++t) {
    if (kind == GAUSSSEIDEL2D5 && pdot) {
      // tangent of the in-place sweep along (v, pdot): each update
      // x[c] = w*s becomes xd[c] = w*sd + pdot*s, in the sweep's order
      const R w = R(p[0]), wd = R(pdot[0]);
      std::vector<R> a = x, ad = xd;
      for (int64_t y = 1; y < g.ny - 1; ++y)
        for (int64_t i = 1; i < g.nx - 1; ++i) {
          const int64_t c = g.at(i, y, 0);
          const int64_t nb[4] = {g.at(i + 1, y, 0), g.at(i, y + 1, 0), g.at(i, y - 1, 0),
                                 g.at(i - 1, y, 0)};
          R sv = a[c], sd = ad[c];
          for (int k = 0; k < 4; ++k) {
            sv += a[nb[k]];
            sd += ad[nb[k]];
          }
          a[c] = w * sv;
          ad[c] = w * sd + wd * sv;
        }
      x.swap(a);
      xd.swap(ad);
      continue;
    }
    step_tangent<R>(kind, g, p, x.data(), K, xd.data(), kappa, xdn.data());
    if (pdot) {
      step_param_partials<R>(kind, g, x.data(), K, d0.data(), d1.data());
      for (int64_t i = 0; i < N; ++i)
        xdn[i] = (xdn[i] + R(pdot[0]) * d0[i]) + R(pdot[1]) * d1[i];
    }
    if (lim) {
      limiter_mask<R>(kind, g, p, lim, x.data(), K, yv, keep);
      for (int64_t i = 0; i < N; ++i)
        if (!keep[i]) xdn[i] = R(0);
    }
    step_forward_lim<R>(kind, g, p, lim, x.data(), K, xn.data());
    x.swap(xn);
    xd.swap(xdn);
  }
  if (xT) std::memcpy(xT, x.data(), sizeof(R) * N);
  std::memcpy(xdT, xd.data(), sizeof(R) * N);
  return 0;
}

}  // namespace

extern "C" {

// lim: {lo, hi} of the limiter, or null for none.
int oracle_forward_f64(int kind, const int64_t* n, const double* p, const double* lim,
                       const double* x0, const double* K, int steps, double* xT) {
  return forward<double>(kind, n, p, lim, x0, K, steps, xT);
}
int oracle_forward_f32(int kind, const int64_t* n, const double* p, const double* lim,
                       const float* x0, const float* K, int steps, float* xT) {
  return forward<float>(kind, n, p, lim, x0, K, steps, xT);
}
int oracle_vjp_f64(int kind, const int64_t* n, const double* p, const double* lim,
                   const double* x0, const double* K, int steps, int loss, const double* aux,
                   double* dx0, double* dK, double* xT, double* loss_out, double* dp_out) {
  return vjp<double>(kind, n, p, lim, x0, K, steps, loss, aux, dx0, dK, xT, loss_out, dp_out);
}
int oracle_vjp_f32(int kind, const int64_t* n, const double* p, const double* lim,
                   const float* x0, const float* K, int steps, int loss, const float* aux,
                   float* dx0, float* dK, float* xT, double* loss_out, double* dp_out) {
  return vjp<float>(kind, n, p, lim, x0, K, steps, loss, aux, dx0, dK, xT, loss_out, dp_out);
}
int oracle_jvp_f64(int kind, const int64_t* n, const double* p, const double* lim,
                   const double* x0, const double* K, const double* v, const double* kappa,
                   const double* pdot, int steps, double* xT, double* xdT) {
  return jvp<double>(kind, n, p, lim, x0, K, v, kappa, pdot, steps, xT, xdT);
}
int oracle_jvp_f32(int kind, const int64_t* n, const double* p, const double* lim,
                   const float* x0, const float* K, const float* v, const float* kappa,
                   const double* pdot, int steps, float* xT, float* xdT) {
  return jvp<float>(kind, n, p, lim, x0, K, v, kappa, pdot, steps, xT, xdT);
}

}  // extern "C"
