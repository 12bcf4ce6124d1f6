// Appendix-A summary of a mode spectrum (section 3): dynamic range sigma_1 / sigma_min and
// the smallest ranks whose truncation error, the relative Frobenius error of keeping the
// top r singular values, is within each threshold.  Host-only arithmetic on a spectrum the
// device computed.
#include <cmath>
#include <limits>
#include <vector>

#include "host_util.h"
#include "jolt_internal.h"

namespace {

int rank_for(const std::vector<double> &tail, double total, double err) {
  // tail[r] = sum_{i >= r} lam[i], r = 0..n (summed from the smallest value up)
  const int n = (int)tail.size() - 1;
  if (total <= 0.0) return 0;
  for (int r = 0; r <= n; ++r)
    if (std::sqrt(tail[r] / total) <= err) return r;
  return n;
}

}  // namespace

extern "C" int jolt_mode_summary(const double *lam, int n, double err_a, double err_b, double *sigma_range,
                                 int32_t *rank_a, int32_t *rank_b) {
  if (!lam || n < 1 || !sigma_range || !rank_a || !rank_b)
    return jolt_fail(JOLT_E_INVAL, "jolt_mode_summary: null argument or n < 1");
  if (!(err_a >= 0.0 && err_a <= 1.0) || !(err_b >= 0.0 && err_b <= 1.0))
    return jolt_fail(JOLT_E_INVAL, "jolt_mode_summary: thresholds must lie in [0, 1]");
  for (int i = 0; i < n; ++i) {
    if (!(lam[i] >= 0.0) || !std::isfinite(lam[i]))
      return jolt_fail(JOLT_E_INVAL, "jolt_mode_summary: lam[%d] is negative or not finite", i);
    if (i > 0 && lam[i] > lam[i - 1]) return jolt_fail(JOLT_E_INVAL, "jolt_mode_summary: lam not descending");
  }
  std::vector<double> tail((size_t)n + 1, 0.0);
  for (int r = n - 1; r >= 0; --r) tail[r] = tail[r + 1] + lam[r];
  const double total = tail[0];
  *sigma_range = lam[n - 1] > 0.0 ? std::sqrt(lam[0] / lam[n - 1]) : std::numeric_limits<double>::infinity();
  *rank_a = rank_for(tail, total, err_a);
  *rank_b = rank_for(tail, total, err_b);
  return JOLT_OK;
}
