// rk_layer_budgets: the allocation half of Algorithm 1 (Section 4.4), host only.
//   1. min-max normalisation (Eq. sensitivity-normalization; a constant profile
//      maps to all zeros, an optional eps guards the denominator as Algorithm 1 does),
//   2. exponential mapping w~ = exp(log r * s_hat) = r^s_hat (Eq. sensitivity-mapping),
//   3. ClipNormalize: clip once to [1/gamma, gamma], rescale to mean one
//      (Eq. weight-normalization),
//   4. integer budgets from B/|A| * w (Eq. layer-budget).  Independent rounding
//      can miss sum(b) = B (Eq. global-budget), so the default apportions by
//      largest remainder after snapping the real shares to multiples of 2^-20
//      (which keeps one-ulp libm differences from moving a unit); ties go to the
//      larger sensitivity, then the lower index.
#include <math.h>

#include <algorithm>
#include <vector>

#include "rk.h"

namespace rk {
void set_error(const char* fmt, ...);
}

extern "C" rk_status rk_layer_budgets(const double* s, int32_t n, int64_t B, double r, double gamma, double eps,
                                      rk_rounding mode, double* w_out, int64_t* b_out) {
  using rk::set_error;
  if (!s || !b_out) { set_error("rk_layer_budgets: null pointer"); return RK_ERR_ARG; }
  if (n <= 0) { set_error("rk_layer_budgets: n must be > 0"); return RK_ERR_ARG; }
  if (B < 0) { set_error("rk_layer_budgets: B must be >= 0"); return RK_ERR_ARG; }
  if (!(r >= 1.0) || !isfinite(r)) { set_error("rk_layer_budgets: r must be finite and >= 1"); return RK_ERR_ARG; }
  if (gamma > 0.0 && isfinite(gamma) && gamma < 1.0) { set_error("rk_layer_budgets: gamma must be >= 1"); return RK_ERR_ARG; }
  if (isnan(gamma)) { set_error("rk_layer_budgets: gamma is NaN"); return RK_ERR_ARG; }
  if (!(eps >= 0.0) || !isfinite(eps)) { set_error("rk_layer_budgets: eps must be finite and >= 0"); return RK_ERR_ARG; }
  if (mode != RK_ROUND_LARGEST_REMAINDER && mode != RK_ROUND_NEAREST_EVEN) {
    set_error("rk_layer_budgets: unknown rounding mode");
    return RK_ERR_ARG;
  }
  for (int32_t i = 0; i < n; ++i)
    if (!isfinite(s[i])) { set_error("rk_layer_budgets: sensitivity %d is not finite", i); return RK_ERR_ARG; }

  double s_min = s[0], s_max = s[0];
  for (int32_t i = 1; i < n; ++i) { s_min = std::min(s_min, s[i]); s_max = std::max(s_max, s[i]); }
  const double lr = log(r);
  const bool clip = gamma > 0.0 && isfinite(gamma);
  std::vector<double> w(n);
  double sum = 0.0;
  for (int32_t i = 0; i < n; ++i) {
    const double sh = (s_max == s_min) ? 0.0 : (s[i] - s_min) / (s_max - s_min + eps);
    double x = exp(lr * sh);
    if (clip) x = std::min(std::max(x, 1.0 / gamma), gamma);
    w[i] = x;
    sum += x;
  }
  const double mean = sum / n;
  for (int32_t i = 0; i < n; ++i) w[i] = w[i] / mean;

  std::vector<int64_t> b(n);
  if (mode == RK_ROUND_NEAREST_EVEN) {
    for (int32_t i = 0; i < n; ++i) b[i] = (int64_t)nearbyint((double)B * w[i] / n);
  } else {
    const double snap = 1048576.0;  // 2^20
    std::vector<double> q(n), frac(n);
    int64_t used = 0;
    for (int32_t i = 0; i < n; ++i) {
      q[i] = floor(((double)B * w[i] / n) * snap + 0.5) / snap;
      b[i] = (int64_t)floor(q[i]);
      frac[i] = q[i] - (double)b[i];
      used += b[i];
    }
    int64_t left = B - used;
    std::vector<int32_t> order(n);
    for (int32_t i = 0; i < n; ++i) order[i] = i;
    std::sort(order.begin(), order.end(), [&](int32_t x, int32_t y) {
      if (frac[x] != frac[y]) return frac[x] > frac[y];
      if (s[x] != s[y]) return s[x] > s[y];
      return x < y;
    });
    for (int64_t k = 0; k < left; ++k) b[order[k % n]] += 1;
  }
  for (int32_t i = 0; i < n; ++i) {
    b_out[i] = b[i];
    if (w_out) w_out[i] = w[i];
  }
  return RK_OK;
}

// Spearman's rho of two profiles (Section 2, Table sensitivity-correlation): the
// Pearson correlation of their ranks, tied values sharing the mean of their
// ranks; NaN when either side is constant.  Host only, float64.
extern "C" rk_status rk_spearman(const double* x, const double* y, int32_t n, double* rho) {
  using rk::set_error;
  if (!x || !y || !rho) { set_error("rk_spearman: null pointer"); return RK_ERR_ARG; }
  if (n < 2) { set_error("rk_spearman: n must be >= 2"); return RK_ERR_ARG; }
  for (int32_t i = 0; i < n; ++i)
    if (!isfinite(x[i]) || !isfinite(y[i])) { set_error("rk_spearman: values must be finite"); return RK_ERR_ARG; }
  auto ranks = [n](const double* v) {
    std::vector<int32_t> idx(n);
    for (int32_t i = 0; i < n; ++i) idx[i] = i;
    std::stable_sort(idx.begin(), idx.end(), [v](int32_t a, int32_t b) { return v[a] < v[b]; });
    std::vector<double> r(n);
    for (int32_t i = 0; i < n;) {
      int32_t j = i;
      while (j + 1 < n && v[idx[j + 1]] == v[idx[i]]) ++j;
      for (int32_t k = i; k <= j; ++k) r[idx[k]] = 0.5 * (i + j) + 1.0;
      i = j + 1;
    }
    return r;
  };
  const std::vector<double> rx = ranks(x), ry = ranks(y);
  double mx = 0.0, my = 0.0;
  for (int32_t i = 0; i < n; ++i) { mx += rx[i]; my += ry[i]; }
  mx /= n;
  my /= n;
  double sxy = 0.0, sxx = 0.0, syy = 0.0;
  for (int32_t i = 0; i < n; ++i) {
    const double a = rx[i] - mx, b = ry[i] - my;
    sxy += a * b;
    sxx += a * a;
    syy += b * b;
  }
  *rho = (sxx > 0.0 && syy > 0.0) ? sxy / sqrt(sxx * syy) : NAN;
  return RK_OK;
}
