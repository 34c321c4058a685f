// Host-side calibration of the geometry-aware FP8 scale (arXiv 2602.18851).
//
// * gamma / alpha_min selection, Sec. 3.2 (Eqs. "gamma_selection",
//   "alpha_selection"), from the union bound N (T1 + T2) <= delta* with the
//   equal split N T1, N T2 <= delta*/2 of Prop. "Rank-aware overflow
//   probability bound".
// * auto-alpha, Sec. 3.5 and App. M, Algorithm "Auto-alpha Calibration":
//   alpha_final = Quantile_q({r_t}) * kappa over burn-in slack ratios
//   r_t = max|S| / B_max, B_max = sigma * d / sqrt(d_h).
// No device code: these run on the CPU and need no GPU.

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <vector>

#include "spectral.h"

void sn_set_last_error(const char* msg);  // spectral.hip: the text spectral_last_error returns

namespace {
int cal_fail(const char* m) {
  sn_set_last_error(m);
  return SN_EINVAL;
}
double h_gamma(double g) { return g - 1.0 - std::log(g); }
}  // namespace

extern "C" {

SN_API int spectral_alpha_select(int32_t d_model, int32_t head_dim, int64_t n_heads_total, int64_t seq_len,
                                 double delta, double* gamma, double* alpha_min) {
  if (!gamma || !alpha_min) return (sn_set_last_error("gamma and alpha_min must not be NULL"), SN_ENULL);
  if (d_model < 1 || head_dim < 1 || n_heads_total < 1 || seq_len < 1 || !(delta > 0.0 && delta < 1.0))
    return cal_fail("d_model, head_dim, n_heads_total, seq_len >= 1 and 0 < delta < 1 required");
  const double N = (double)n_heads_total, L = (double)seq_len;
  // smallest gamma > 1 with h(gamma) >= (2 / d_h) ln(2 N L / delta); h increases on (1, inf)
  const double rhs = 2.0 / head_dim * std::log(2.0 * N * L / delta);
  double lo = 1.0, hi = 2.0;
  while (h_gamma(hi) < rhs) hi *= 2.0;
  for (int it = 0; it < 200; ++it) {
    const double mid = 0.5 * (lo + hi);
    (h_gamma(mid) >= rhs ? hi : lo) = mid;
  }
  *gamma = hi;
  *alpha_min = std::sqrt(2.0 * hi * head_dim) / d_model * std::sqrt(std::log(4.0 * N * L * L / delta));
  return SN_OK;
}

SN_API int spectral_overflow_terms(int32_t d_model, int32_t head_dim, int64_t seq_len, double alpha, double gamma,
                                   double* t1, double* t2) {
  if (!t1 || !t2) return (sn_set_last_error("t1 and t2 must not be NULL"), SN_ENULL);
  if (d_model < 1 || head_dim < 1 || seq_len < 1 || !(alpha > 0.0) || !(gamma > 1.0))
    return cal_fail("d_model, head_dim, seq_len >= 1, alpha > 0 and gamma > 1 required");
  const double L = (double)seq_len, d = d_model;
  *t1 = L * std::exp(-0.5 * head_dim * h_gamma(gamma));
  *t2 = 2.0 * L * L * std::exp(-(d * d * alpha * alpha) / (2.0 * gamma * head_dim));
  return SN_OK;
}

SN_API int spectral_auto_alpha(const double* slack, int64_t n, double quantile, double kappa, double* alpha) {
  if (!slack || !alpha) return (sn_set_last_error("slack and alpha must not be NULL"), SN_ENULL);
  if (n < 1 || !(quantile >= 0.0 && quantile <= 1.0) || !(kappa >= 1.0))
    return cal_fail("n >= 1, 0 <= quantile <= 1 and kappa >= 1 required");
  std::vector<double> r(slack, slack + n);
  for (double x : r)
    if (!std::isfinite(x) || x < 0.0) return cal_fail("slack ratios must be finite and >= 0");
  std::sort(r.begin(), r.end());
  // linear interpolation between order statistics at position q (n - 1)
  const double pos = quantile * (double)(n - 1);
  const int64_t i = (int64_t)std::floor(pos);
  const double f = pos - (double)i;
  const double qv = (i + 1 < n) ? r[i] + f * (r[i + 1] - r[i]) : r[n - 1];
  *alpha = qv * kappa;
  return SN_OK;
}

SN_API double spectral_slack_ratio(double max_abs_logit, double sigma_layer, int32_t d_model, int32_t head_dim) {
  return max_abs_logit / (sigma_layer * (double)d_model / std::sqrt((double)head_dim));
}

}  // extern "C"
