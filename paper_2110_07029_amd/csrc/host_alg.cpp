// Host-side parts of Adaptive SGD that decide, between mega-batches, how the
// replicas are weighted and how big their batches are:
//   asgd_merge_weights  - Alg. 2 normalization weights (+ optional perturbation)
//   asgd_scale_batches  - Alg. 1 batch-size scaling with the linear LR rule
#include <math.h>

#include "../../include/asgd.h"

namespace asgd {
asgd_status set_error(asgd_status s, const char* msg);  // the library's error channel
}

namespace {
asgd_status alg_fail(asgd_status s, const char* msg) { return asgd::set_error(s, msg); }
}  // namespace

extern "C" {

asgd_status asgd_merge_weights(int32_t n, const int32_t* u, const int32_t* b,
                               const int64_t* samples, int32_t mode, const double* l2_per_param,
                               double pert_thr, double delta, float* alpha_out) {
  if (n < 1 || !u || !b || !alpha_out) return alg_fail(ASGD_EINVAL, "invalid arguments");
  double alpha[64];
  if (n > 64) return alg_fail(ASGD_EINVAL, "n must be <= 64");
  if (mode == ASGD_WEIGHTS_ALG2) {
    bool equal = true;
    for (int i = 1; i < n; ++i) equal = equal && (u[i] == u[0]);
    double tot = 0.0;
    for (int i = 0; i < n; ++i) tot += equal ? (double)b[i] : (double)u[i];
    if (!(tot > 0.0)) return alg_fail(ASGD_EINVAL, "weights sum to zero");
    for (int i = 0; i < n; ++i) alpha[i] = (equal ? (double)b[i] : (double)u[i]) / tot;
  } else if (mode == ASGD_WEIGHTS_UNIFORM) {
    for (int i = 0; i < n; ++i) alpha[i] = 1.0 / (double)n;
  } else if (mode == ASGD_WEIGHTS_SAMPLES) {
    if (!samples) return alg_fail(ASGD_EINVAL, "samples is NULL");
    double tot = 0.0;
    for (int i = 0; i < n; ++i) tot += (double)samples[i];
    if (!(tot > 0.0)) return alg_fail(ASGD_EINVAL, "samples sum to zero");
    for (int i = 0; i < n; ++i) alpha[i] = (double)samples[i] / tot;
  } else {
    return alg_fail(ASGD_EINVAL, "unknown weight mode");
  }
  if (l2_per_param && n > 1) {
    bool regular = true;
    for (int i = 0; i < n; ++i) regular = regular && (l2_per_param[i] < pert_thr);
    if (regular) {
      // r: most updates, then larger batch, then lower index; s: fewest updates,
      // then smaller batch, then higher index.
      int r = 0, s = n - 1;
      for (int i = 1; i < n; ++i)
        if (u[i] > u[r] || (u[i] == u[r] && b[i] > b[r])) r = i;
      for (int i = n - 2; i >= 0; --i)
        if (u[i] < u[s] || (u[i] == u[s] && b[i] < b[s])) s = i;
      alpha[r] *= 1.0 + delta;
      alpha[s] *= 1.0 - delta;
    }
  }
  for (int i = 0; i < n; ++i) alpha_out[i] = (float)alpha[i];
  return ASGD_OK;
}

asgd_status asgd_scale_batches(int32_t n, const int32_t* u, int32_t* b, float* lr, int32_t b_min,
                               int32_t b_max, double beta) {
  if (n < 1 || !u || !b || !lr) return alg_fail(ASGD_EINVAL, "invalid arguments");
  if (b_min < 1 || b_max < b_min) return alg_fail(ASGD_EINVAL, "need 1 <= b_min <= b_max");
  double total = 0.0;
  for (int i = 0; i < n; ++i) total += (double)u[i];
  const double mu = total / (double)n;
  for (int i = 0; i < n; ++i) {
    if (b[i] < 1) return alg_fail(ASGD_EINVAL, "batch sizes must be >= 1");
    const double grow = (double)b[i] + beta * ((double)u[i] - mu);
    const double shrink = (double)b[i] - beta * (mu - (double)u[i]);
    double target;
    if ((double)u[i] > mu && grow <= (double)b_max)
      target = grow;
    else if ((double)u[i] < mu && shrink >= (double)b_min)
      target = shrink;
    else
      continue;
    const int32_t nb = (int32_t)(target >= 0 ? floor(target + 0.5) : -floor(-target + 0.5));
    lr[i] = (float)((double)lr[i] * (double)nb / (double)b[i]);
    b[i] = nb;
  }
  return ASGD_OK;
}

}  // extern "C"
