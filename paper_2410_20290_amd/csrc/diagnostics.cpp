// Evaluation diagnostics on host arrays: the improvement score of section 5
// and the Pearson / Kendall correlations of Appendix B.  Host code only;
// double precision throughout.
#include <cmath>
#include <cstdint>

#include "specrej.h"

namespace sr {
// the calling thread's message for sr_last_error (empty clears it)
void set_last_error(const char* msg);
}

namespace {
bool finite_all(const float* v, int32_t n) {
  for (int32_t i = 0; i < n; ++i)
    if (!std::isfinite(v[i])) return false;
  return true;
}

sr_status fail(sr_status st, const char* msg) {
  sr::set_last_error(msg);
  return st;
}
}  // namespace

extern "C" {

sr_status sr_correlation(const float* x, const float* y, int32_t n, double* pearson, double* kendall) {
  if (!x || !y || !pearson || !kendall) return fail(SR_ERR_INVALID_ARG, "NULL argument");
  if (n < 2) return fail(SR_ERR_INVALID_ARG, "n must be >= 2");
  if (!finite_all(x, n) || !finite_all(y, n)) return fail(SR_ERR_INVALID_ARG, "values must be finite");
  // Pearson: centred sums around the sample means
  double mx = 0.0, my = 0.0;
  for (int32_t i = 0; i < n; ++i) {
    mx += x[i];
    my += y[i];
  }
  mx /= n;
  my /= n;
  double sxy = 0.0, sxx = 0.0, syy = 0.0;
  for (int32_t i = 0; i < n; ++i) {
    const double a = x[i] - mx, b = y[i] - my;
    sxy += a * b;
    sxx += a * a;
    syy += b * b;
  }
  const double den = std::sqrt(sxx * syy);
  *pearson = den > 0.0 ? sxy / den : NAN;
  // Kendall: concordant minus discordant pairs, tied pairs count zero
  int64_t s = 0;
  for (int32_t i = 0; i < n; ++i) {
    const float xi = x[i], yi = y[i];
    for (int32_t j = i + 1; j < n; ++j) {
      const int sx = (xi > x[j]) - (xi < x[j]);
      const int sy = (yi > y[j]) - (yi < y[j]);
      s += sx * sy;
    }
  }
  *kendall = 2.0 * (double)s / ((double)n * (double)(n - 1));
  sr::set_last_error("");
  return SR_OK;
}

sr_status sr_improvement_score(const float* bon_rewards, int32_t n, float sr_reward, double* score) {
  if (!bon_rewards || !score) return fail(SR_ERR_INVALID_ARG, "NULL argument");
  if (n < 1) return fail(SR_ERR_INVALID_ARG, "n must be >= 1");
  if (!finite_all(bon_rewards, n) || !std::isfinite(sr_reward)) return fail(SR_ERR_INVALID_ARG, "values must be finite");
  double hi = bon_rewards[0], lo = bon_rewards[0];
  for (int32_t i = 1; i < n; ++i) {
    hi = std::fmax(hi, (double)bon_rewards[i]);
    lo = std::fmin(lo, (double)bon_rewards[i]);
  }
  *score = hi > lo ? (1.0 - (hi - (double)sr_reward) / (hi - lo)) * 100.0 : NAN;
  sr::set_last_error("");
  return SR_OK;
}

}  // extern "C"
