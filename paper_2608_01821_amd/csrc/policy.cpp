// Allocation policy of DAVET (Sec. 4.2, Eqs. 6-9; Appendix A), host-side.
// Built with -ffp-contract=off: every product and sum below is a separately
// rounded IEEE double operation, evaluated in the order the equations print,
// so budgets and levels are reproducible bit for bit.

#include <algorithm>
#include <cmath>
#include <numeric>
#include <string>
#include <vector>

#include "davet.h"

namespace davet {
int set_error(int status, const std::string& msg);
}

namespace {

// Phase family (Sec. 4.2): early grounding 1 - (t - 0.5)/T, late verification
// (t - 0.5)/T, for t = 1..T.
void phase_profile(int T, bool early, double* p) {
  for (int t = 1; t <= T; ++t) {
    const double x = ((double)t - 0.5) / (double)T;
    p[t - 1] = early ? 1.0 - x : x;
  }
}

// N(p; beta): scale the profile and clip to [0, 1] so the mean is beta.  The
// scale is solved exactly: entries saturate from the largest p downwards
// (equal p: lower index first); with j saturated entries the scale is
// (T*beta - j) / (sum of the other p, ascending t), accepted once the largest
// unsaturated entry stays <= 1 under it.
void normalize(const double* p, int T, double beta, double* out) {
  if (beta >= 1.0) { std::fill(out, out + T, 1.0); return; }
  if (beta <= 0.0) { std::fill(out, out + T, 0.0); return; }
  std::vector<int> order(T);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(),
                   [&](int a, int b) { return p[a] > p[b]; });
  std::vector<char> sat(T, 0);
  const double target = (double)T * beta;
  double scale = 0.0;
  bool found = false;
  for (int j = 0; j < T; ++j) {
    double denom = 0.0;
    for (int t = 0; t < T; ++t)
      if (!sat[t]) denom = denom + p[t];
    const double sj = (target - (double)j) / denom;
    if (sj * p[order[j]] <= 1.0) { scale = sj; found = true; break; }
    sat[order[j]] = 1;
  }
  if (!found) { std::fill(out, out + T, 1.0); return; }
  for (int t = 0; t < T; ++t) out[t] = sat[t] ? 1.0 : scale * p[t];
}

bool is_fin(double x) { return std::isfinite(x); }

}  // namespace

extern "C" double davet_demand_prior(int32_t category) {
  // Appendix A, Table A.
  static const double prior[5] = {1.000, 0.941, 0.824, 0.647, 0.529};
  if (category < 0 || category > 4) return -1.0;
  return prior[category];
}

extern "C" int davet_policy_envelope(const davet_policy* pol, int32_t T,
                                     double* lower, double* upper) {
  using davet::set_error;
  if (!pol || !lower || !upper)
    return set_error(DAVET_EINVAL, "davet_policy_envelope: null argument");
  if (T < 1) return set_error(DAVET_EINVAL, "davet_policy_envelope: T < 1");
  if (!is_fin(pol->B) || !is_fin(pol->rho) || !is_fin(pol->demand) || !is_fin(pol->alpha))
    return set_error(DAVET_EINVAL, "davet_policy_envelope: non-finite parameter");
  std::vector<double> p(T);
  phase_profile(T, pol->early != 0, p.data());
  // Eq. (6)
  const double beta_lo = (1.0 - pol->rho) * pol->B;
  const double beta_up = ((1.0 - pol->rho) + pol->rho * pol->demand) * pol->B;
  normalize(p.data(), T, beta_lo, lower);
  normalize(p.data(), T, beta_up, upper);
  return DAVET_OK;
}

extern "C" int davet_policy_step(const davet_policy* pol, int32_t t, int32_t T,
                                 const double* lower, const double* upper,
                                 double cbar_prev, double churn_prev,
                                 double* b_t, int32_t* level, double* r_t) {
  using davet::set_error;
  if (!pol || !lower || !upper || !b_t || !level)
    return set_error(DAVET_EINVAL, "davet_policy_step: null argument");
  if (t < 1 || t > T) return set_error(DAVET_EINVAL, "davet_policy_step: t out of [1, T]");
  if (pol->K < 1 || pol->K > DAVET_MAX_LEVELS)
    return set_error(DAVET_EINVAL, "davet_policy_step: K out of range");
  // Eq. (7); r_1 = 1 before any prediction exists
  const double r = (t == 1) ? 1.0
                            : 1.0 - ((pol->alpha * cbar_prev) * (1.0 - churn_prev));
  // Eq. (8)
  const double b = lower[t - 1] + r * (upper[t - 1] - lower[t - 1]);
  // Eq. (9), K levels: count the thresholds j/K that b reaches
  int lv = 0;
  for (int j = 1; j < pol->K; ++j)
    if ((double)j / (double)pol->K <= b) ++lv;
  *b_t = b;
  *level = lv;
  if (r_t) *r_t = r;
  return DAVET_OK;
}

extern "C" int davet_step_stats(int32_t L, const float* conf,
                                const int32_t* argmax,
                                const int32_t* argmax_prev,
                                const uint8_t* masked_after, double* cbar,
                                double* churn) {
  using davet::set_error;
  if (L < 0 || !conf || !argmax || !masked_after || !cbar || !churn)
    return set_error(DAVET_EINVAL, "davet_step_stats: bad argument");
  double s = 0.0;
  int n = 0, changed = 0;
  for (int i = 0; i < L; ++i) {
    if (!masked_after[i]) continue;
    s = s + (double)conf[i];
    ++n;
    if (argmax_prev && argmax[i] != argmax_prev[i]) ++changed;
  }
  *cbar = n ? s / (double)n : 0.0;
  *churn = (n && argmax_prev) ? (double)changed / (double)n : 0.0;
  return DAVET_OK;
}
