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
//   * every interval spans at least one cell; ties keep the leftmost cut.
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

}  // namespace

extern "C" int fewbit_fit_table(int32_t act, int32_t bits, const fewbit_weight* w,
                                int64_t n_grid, int32_t flags, fewbit_table* out) {
  if (!w || !out) return FEWBIT_E_NULL;
  if (bits < 1 || bits > 4) return FEWBIT_E_BITS;
  if (act < FEWBIT_GELU || act > FEWBIT_SOFTPLUS) return FEWBIT_E_INVALID;
  if (flags & ~FEWBIT_FLAG_SYMMETRIC) return FEWBIT_E_INVALID;
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

  // prefix integrals of w, f' w, f'^2 w over the cells (Eqs. (8)-(9))
  const Rule rule = legendre_rule8();
  for (int64_t i = 0; i < n; ++i) {
    const double a = grid(i), b = grid(i + 1);
    const double mid = 0.5 * (a + b), half = 0.5 * (b - a);
    double s0 = 0.0, s1 = 0.0, s2 = 0.0;
    for (int k = 0; k < 8; ++k) {
      const double x = mid + half * rule.node[k];
      const double wx = wt(x);
      const double d = activation_derivative(act, x);
      s0 += rule.weight[k] * wx;
      s1 += rule.weight[k] * d * wx;
      s2 += rule.weight[k] * d * d * wx;
    }
    W[i + 1] = W[i] + half * s0;
    FW[i + 1] = FW[i] + half * s1;
    F2[i + 1] = F2[i] + half * s2;
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

  fewbit_table t;
  std::memset(&t, 0, sizeof t);
  t.act = act;
  t.bits = bits;
  t.flags = flags;
  for (int m = 0; m < 15; ++m) t.s[m] = INFINITY;
  for (int m = 1; m < K; ++m) t.s[m - 1] = static_cast<float>(grid(cut[m]));
  for (int m = 0; m < K; ++m) t.v[m] = static_cast<float>(interval_value(cut[m], cut[m + 1]));
  t.loss = (sym ? 2.0 : 1.0) * cost_prev[n];
  for (int m = 1; m + 1 < K; ++m)
    if (!(t.s[m - 1] < t.s[m])) return FEWBIT_E_NUMERIC;
  for (int m = 0; m < K; ++m)
    if (!std::isfinite(t.v[m])) return FEWBIT_E_NUMERIC;
  *out = t;
  return FEWBIT_OK;
}

extern "C" int64_t fewbit_packed_words(int64_t n, int32_t bits) {
  if (n < 0 || bits < 1 || bits > 4) return -1;
  return (n * bits + 31) / 32;
}
