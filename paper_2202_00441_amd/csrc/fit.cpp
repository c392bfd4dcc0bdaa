// fit.cpp -- host-side optimal piecewise-constant fit of f' (Sec. 3).
//
// Builds the table consumed by the forward/backward kernels.  The problem is
// Eq. (3): minimise the w-weighted L2 distance between f' and a K-interval
// piecewise-constant q.  For fixed boundaries the best values are Eq. (4);
// the boundaries come from the dynamic programme over a grid (Eqs. (6)-(7))
// whose interval costs are O(1) differences of three prefix integrals
// (Eqs. (8)-(9)).  Run once per (activation, bits, weight); not on the
// device.
//
// Choices where the paper leaves room (same as documented in fewbit.h):
//   * uniform grid of n cells over [A, B] (over [max(A,0), B] for the
//     symmetric fit of an even f', whose loss is then doubled);
//   * each cell integral by 8-point Gauss-Legendre quadrature, with nodes
//     computed here by Newton's method on the Legendre polynomial;
//   * an interval with no weight costs 0 and takes f' at its midpoint; a
//     negative cost from cancellation is clamped to 0;
//   * every interval spans at least one cell; ties keep the leftmost cut;
//   * FEWBIT_FLAG_REFINE: the DP result is then refined by steepest descent
//     with the analytic gradient of Sec. 3 and backtracking, integrals at
//     off-grid boundaries taken as grid prefix plus partial cell.
#include <cmath>
#include <cstdint>
#include <cstring>
#include <new>
#include <vector>

#include "../../include/fewbit.h"

namespace {

constexpr double kPi = 3.141592653589793238462643383279502884;

// --- derivatives of the activations, in double ----------------------------
double logistic(double x) {
  // evaluated on the side where exp() cannot overflow
  if (x < 0.0) {
    const double e = std::exp(x);
    return e / (1.0 + e);
  }
  return 1.0 / (1.0 + std::exp(-x));
}

double activation_derivative(int act, double x) {
  switch (act) {
    case FEWBIT_GELU: {
      // d/dx [x Phi(x)] = Phi(x) + x phi(x)
      const double cdf = 0.5 * std::erfc(-x * 0.70710678118654752440);
      const double pdf = 0.39894228040143267794 * std::exp(-0.5 * x * x);
      return cdf + x * pdf;
    }
    case FEWBIT_SILU: {
      const double sg = logistic(x);
      return sg + x * sg * (1.0 - sg);
    }
    case FEWBIT_SIGMOID: {
      const double sg = logistic(x);
      return sg * (1.0 - sg);
    }
    case FEWBIT_TANH: {
      const double th = std::tanh(x);
      return (1.0 - th) * (1.0 + th);
    }
    case FEWBIT_RELU:
      return x > 0.0 ? 1.0 : 0.0;
    case FEWBIT_SELU: {
      // Klambauer et al. (2017): lambda and lambda * alpha
      constexpr double kLambda = 1.0507009873554804934;
      constexpr double kLambdaAlpha = 1.7580993408473768600;
      return x > 0.0 ? kLambda : kLambdaAlpha * std::exp(x);
    }
    case FEWBIT_SOFTPLUS:
      return logistic(x);
  }
  return 0.0;
}

// --- weight -------------------------------------------------------------------
struct Weight {
  int kind;
  double a, b, mu, sigma, p, sigma2;

  double gauss(double x, double s) const {
    const double z = (x - mu) / s;
    return std::exp(-0.5 * z * z) / (s * std::sqrt(2.0 * kPi));
  }
  double operator()(double x) const {
    if (x < a || x > b) return 0.0;
    if (kind == FEWBIT_W_UNIFORM) return 1.0;
    if (kind == FEWBIT_W_NORMAL) return gauss(x, sigma);
    return (1.0 - p) * gauss(x, sigma) + p * gauss(x, sigma2);
  }
};

// --- Gauss-Legendre nodes on [-1, 1] by Newton iteration -----------------------
struct Rule {
  double node[8];
  double weight[8];
};

Rule legendre_rule8() {
  Rule r{};
  const int n = 8;
  for (int k = 0; k < n; ++k) {
    double x = std::cos(kPi * (k + 0.75) / (n + 0.5));  // Tricomi start
    double dp = 1.0;
    for (int it = 0; it < 100; ++it) {
      // three-term recurrence for P_n and its derivative
      double p0 = 1.0, p1 = x;
      for (int m = 2; m <= n; ++m) {
        const double p2 = ((2.0 * m - 1.0) * x * p1 - (m - 1.0) * p0) / m;
        p0 = p1;
        p1 = p2;
      }
      dp = n * (x * p1 - p0) / (x * x - 1.0);
      const double step = p1 / dp;
      x -= step;
      if (std::fabs(step) < 1e-17) break;
    }
    r.node[k] = x;
    r.weight[k] = 2.0 / ((1.0 - x * x) * dp * dp);
  }
  return r;
}

bool is_finite_value(double v) { return std::isfinite(v); }

// Upper bound on accepted descent steps of the refinement (it stops earlier
// once no step lowers L).
constexpr int kRefineMaxSteps = 20000;

}  // namespace

extern "C" int fewbit_fit_table(int32_t act, int32_t bits, const fewbit_weight* w,
                                int64_t n_grid, int32_t flags, fewbit_table* out) {
  if (!w || !out) return FEWBIT_E_NULL;
  if (bits < 1 || bits > 4) return FEWBIT_E_BITS;
  if (act < FEWBIT_GELU || act > FEWBIT_SOFTPLUS) return FEWBIT_E_INVALID;
  if (flags & ~(FEWBIT_FLAG_SYMMETRIC | FEWBIT_FLAG_REFINE)) return FEWBIT_E_INVALID;
  if (w->reserved != 0) return FEWBIT_E_INVALID;
  if (w->kind < FEWBIT_W_UNIFORM || w->kind > FEWBIT_W_MIXTURE) return FEWBIT_E_INVALID;
  if (!is_finite_value(w->A) || !is_finite_value(w->B) || !(w->A < w->B)) return FEWBIT_E_INVALID;
  if (w->kind != FEWBIT_W_UNIFORM) {
    if (!is_finite_value(w->mu) || !(w->sigma > 0.0) || !is_finite_value(w->sigma)) return FEWBIT_E_INVALID;
    if (w->kind == FEWBIT_W_MIXTURE &&
        (!(w->p >= 0.0 && w->p <= 1.0) || !(w->sigma2 > 0.0) || !is_finite_value(w->sigma2)))
      return FEWBIT_E_INVALID;
  }
  const int K = 1 << bits;
  if (n_grid < K || n_grid > (int64_t(1) << 20)) return FEWBIT_E_INVALID;
  const bool sym = (flags & FEWBIT_FLAG_SYMMETRIC) != 0;

  Weight wt{w->kind, w->A, w->B, w->mu, w->sigma, w->p, w->sigma2};
  if (sym && wt.a < 0.0) wt.a = 0.0;
  if (!(wt.a < wt.b)) return FEWBIT_E_INVALID;
  const int64_t n = n_grid;
  const double lo = wt.a, hi = wt.b;
  auto grid = [&](int64_t i) { return lo + static_cast<double>(i) * (hi - lo) / static_cast<double>(n); };

  std::vector<double> W, FW, F2, cost_prev, cost_cur;
  std::vector<int32_t> back;
  try {
    W.assign(n + 1, 0.0);
    FW.assign(n + 1, 0.0);
    F2.assign(n + 1, 0.0);
    cost_prev.assign(n + 1, 0.0);
    cost_cur.assign(n + 1, 0.0);
    back.assign(static_cast<size_t>(n + 1) * (K + 1), 0);
  } catch (const std::bad_alloc&) {
    return FEWBIT_E_NOMEM;
  }

  // integrals of w, f' w, f'^2 w over [a, b] by the 8-point rule
  const Rule rule = legendre_rule8();
  auto quad = [&](double a, double b, double& s0, double& s1, double& s2) {
    const double mid = 0.5 * (a + b), half = 0.5 * (b - a);
    s0 = s1 = s2 = 0.0;
    for (int k = 0; k < 8; ++k) {
      const double x = mid + half * rule.node[k];
      const double wx = wt(x);
      const double d = activation_derivative(act, x);
      s0 += rule.weight[k] * wx;
      s1 += rule.weight[k] * d * wx;
      s2 += rule.weight[k] * d * d * wx;
    }
    s0 *= half;
    s1 *= half;
    s2 *= half;
  };
  // prefix integrals over the cells (Eqs. (8)-(9))
  for (int64_t i = 0; i < n; ++i) {
    double c0, c1, c2;
    quad(grid(i), grid(i + 1), c0, c1, c2);
    W[i + 1] = W[i] + c0;
    FW[i + 1] = FW[i] + c1;
    F2[i + 1] = F2[i] + c2;
  }

  // cost of one interval [t_j, t_i]: F2 diff minus y^2 times W diff (Eq. (8))
  auto interval_cost = [&](int64_t j, int64_t i) -> double {
    const double dw = W[i] - W[j];
    if (!(dw > 0.0)) return 0.0;
    const double y = (FW[i] - FW[j]) / dw;
    const double c = (F2[i] - F2[j]) - y * y * dw;
    return c > 0.0 ? c : 0.0;
  };
  auto interval_value = [&](int64_t j, int64_t i) -> double {
    const double dw = W[i] - W[j];
    if (!(dw > 0.0)) return activation_derivative(act, 0.5 * (grid(j) + grid(i)));
    return (FW[i] - FW[j]) / dw;
  };

  // layer 1: a single interval [t_0, t_i]
  for (int64_t i = 1; i <= n; ++i) cost_prev[i] = interval_cost(0, i);
  // layers 2..K: best split of [t_0, t_i] into k intervals (Eq. (7))
  for (int k = 2; k <= K; ++k) {
    int32_t* bk = back.data() + static_cast<size_t>(k) * (n + 1);
    for (int64_t i = k; i <= n; ++i) {
      const double w_i = W[i], fw_i = FW[i], f2_i = F2[i];
      double best = INFINITY;
      int64_t arg = k - 1;
      for (int64_t j = k - 1; j < i; ++j) {
        const double dw = w_i - W[j];
        double c = 0.0;
        if (dw > 0.0) {
          const double y = (fw_i - FW[j]) / dw;
          c = (f2_i - F2[j]) - y * y * dw;
          c = c > 0.0 ? c : 0.0;
        }
        const double total = cost_prev[j] + c;
        if (total < best) {
          best = total;
          arg = j;
        }
      }
      cost_cur[i] = best;
      bk[i] = static_cast<int32_t>(arg);
    }
    for (int64_t i = 0; i < k; ++i) cost_cur[i] = INFINITY;
    cost_prev.swap(cost_cur);
  }

  // walk the cut points back from t_n
  int64_t cut[17];
  cut[K] = n;
  for (int k = K; k >= 2; --k)
    cut[k - 1] = back[static_cast<size_t>(k) * (n + 1) + static_cast<size_t>(cut[k])];
  cut[0] = 0;

  // boundaries and values of the DP result
  double bnd[17], val[16];
  bnd[0] = lo;
  bnd[K] = hi;
  for (int m = 1; m < K; ++m) bnd[m] = grid(cut[m]);
  for (int m = 0; m < K; ++m) val[m] = interval_value(cut[m], cut[m + 1]);
  double loss = cost_prev[n];

  if (flags & FEWBIT_FLAG_REFINE) {
    // L(s, y(s)) at off-grid boundaries: each integral over [lo, x] is the
    // grid prefix up to the cell holding x plus the part of that cell below
    // x, by the same rule.  Values by Eq. (4); gradient of Sec. 3,
    //   dL/ds_m = (2 f'(s_m) - y_m - y_{m-1}) (y_m - y_{m-1}) w(s_m).
    auto upto = [&](double x, double& p0, double& p1, double& p2) {
      int64_t j = static_cast<int64_t>(std::floor((x - lo) / (hi - lo) * static_cast<double>(n)));
      j = j < 0 ? 0 : (j > n ? n : j);
      if (j > 0 && grid(j) > x) --j;
      p0 = W[j];
      p1 = FW[j];
      p2 = F2[j];
      if (j < n && x > grid(j)) {
        double c0, c1, c2;
        quad(grid(j), x, c0, c1, c2);
        p0 += c0;
        p1 += c1;
        p2 += c2;
      }
    };
    auto evaluate = [&](const double* e, double* y, double* grad) {
      double P0[17], P1[17], P2[17];
      for (int m = 0; m <= K; ++m) upto(e[m], P0[m], P1[m], P2[m]);
      double L = 0.0;
      for (int m = 0; m < K; ++m) {
        const double dw = P0[m + 1] - P0[m];
        if (!(dw > 0.0)) {
          y[m] = activation_derivative(act, 0.5 * (e[m] + e[m + 1]));
          continue;
        }
        y[m] = (P1[m + 1] - P1[m]) / dw;
        const double c = (P2[m + 1] - P2[m]) - y[m] * y[m] * dw;
        L += c > 0.0 ? c : 0.0;
      }
      if (grad)
        for (int m = 1; m < K; ++m)
          grad[m] = (2.0 * activation_derivative(act, e[m]) - y[m] - y[m - 1]) *
                    (y[m] - y[m - 1]) * wt(e[m]);
      return L;
    };
    // steepest descent with backtracking: a step must keep the boundaries
    // strictly increasing inside (lo, hi) and lower L by 1e-4 t |g|^2; the
    // first step moves a boundary by at most one cell, and each accepted
    // step doubles the next trial step
    double g[17], y[16], trial[17], ytrial[16];
    double L = evaluate(bnd, y, g);
    auto max_abs = [&](const double* v) {
      double r = 0.0;
      for (int m = 1; m < K; ++m) r = std::fmax(r, std::fabs(v[m]));
      return r;
    };
    double step = max_abs(g) > 0.0 ? (hi - lo) / static_cast<double>(n) / max_abs(g) : 0.0;
    for (int iter = 0; iter < kRefineMaxSteps && max_abs(g) > 0.0; ++iter) {
      double g2 = 0.0;
      for (int m = 1; m < K; ++m) g2 += g[m] * g[m];
      bool accepted = false;
      for (int halvings = 0; halvings < 80 && !accepted; ++halvings) {
        bool sorted = true;
        trial[0] = lo;
        trial[K] = hi;
        for (int m = 1; m < K; ++m) {
          trial[m] = bnd[m] - step * g[m];
          sorted = sorted && trial[m] > trial[m - 1];
        }
        sorted = sorted && trial[K - 1] < hi;
        if (sorted) {
          const double Lt = evaluate(trial, ytrial, nullptr);
          accepted = Lt < L && Lt <= L - 1e-4 * step * g2;
        }
        if (!accepted) step *= 0.5;
      }
      if (!accepted) break;
      for (int m = 1; m < K; ++m) bnd[m] = trial[m];
      L = evaluate(bnd, y, g);
      step *= 2.0;
    }
    for (int m = 0; m < K; ++m) val[m] = y[m];
    loss = L;
  }

  fewbit_table t;
  std::memset(&t, 0, sizeof t);
  t.act = act;
  t.bits = bits;
  t.flags = flags & FEWBIT_FLAG_SYMMETRIC;
  for (int m = 0; m < 15; ++m) t.s[m] = INFINITY;
  for (int m = 1; m < K; ++m) t.s[m - 1] = static_cast<float>(bnd[m]);
  for (int m = 0; m < K; ++m) t.v[m] = static_cast<float>(val[m]);
  t.loss = (sym ? 2.0 : 1.0) * loss;
  for (int m = 1; m + 1 < K; ++m)
    if (!(t.s[m - 1] < t.s[m])) return FEWBIT_E_NUMERIC;
  for (int m = 0; m < K; ++m)
    if (!std::isfinite(t.v[m])) return FEWBIT_E_NUMERIC;
  *out = t;
  return FEWBIT_OK;
}

extern "C" int64_t fewbit_packed_words(int64_t n, int32_t bits) {
  if (n < 0 || bits < 1 || bits > 4) return -1;
  // ceil(n * bits / 32) without forming n * bits, which overflows near 2^63
  return (n / 32) * bits + ((n % 32) * bits + 31) / 32;
}
