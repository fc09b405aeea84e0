// costmodel.cpp -- the speculative-decoding cost model (Sec. 3.1 Eq. 1-2,
// Sec. 4.1 Eq. 3-4) as host arithmetic behind the C ABI, so a serving loop
// can pick the speculation length from measured layer times.
#include <math.h>

#include "magicdec.h"

namespace {

bool valid_alpha(double a) { return a >= 0.0 && a <= 1.0; }

// Omega as the finite geometric series, Horner's rule: no cancellation as
// alpha -> 1, where the closed form divides two vanishing differences.
double omega(int gamma, double alpha) {
  double s = 1.0;
  for (int k = 0; k < gamma; ++k) s = 1.0 + alpha * s;
  return s;
}

bool valid_times(double t_target, double t_draft, double t_select) {
  return t_target > 0.0 && t_draft >= 0.0 && t_select >= 0.0 && isfinite(t_target) &&
         isfinite(t_draft) && isfinite(t_select);
}

}  // namespace

extern "C" {

double md_sd_expected_tokens(int32_t gamma, double alpha) {
  if (gamma < 0 || !valid_alpha(alpha)) return NAN;
  return omega(gamma, alpha);
}

double md_sd_latency_ratio(int32_t gamma, double alpha, double t_target, double t_draft,
                           double t_select, double t_verify) {
  if (gamma < 0 || !valid_alpha(alpha) || !valid_times(t_target, t_draft, t_select) ||
      !(t_verify >= 0.0) || !isfinite(t_verify))
    return NAN;
  return (gamma * (t_draft + t_select) + t_verify) / (omega(gamma, alpha) * t_target);
}

int md_sd_best_gamma(int32_t max_gamma, double alpha, double t_target, double t_draft,
                     double t_select, const double* t_verify, int32_t* gamma_out,
                     double* ratio_out) {
  if (max_gamma < 1 || !t_verify || !gamma_out || !ratio_out || !valid_alpha(alpha) ||
      !valid_times(t_target, t_draft, t_select))
    return MD_ERR_INVALID_ARG;
  int best_g = 0;
  double best_r = INFINITY;
  for (int g = 1; g <= max_gamma; ++g) {
    const double r = md_sd_latency_ratio(g, alpha, t_target, t_draft, t_select, t_verify[g - 1]);
    if (isnan(r)) return MD_ERR_INVALID_ARG;
    if (r < best_r) {
      best_r = r;
      best_g = g;
    }
  }
  *gamma_out = best_g;
  *ratio_out = best_r;
  return MD_OK;
}

double md_sd_alpha_from_omega(int32_t gamma, double om) {
  if (gamma < 0 || !(om >= 1.0) || om > gamma + 1.0) return NAN;
  if (gamma == 0) return om == 1.0 ? 0.0 : NAN;
  double lo = 0.0, hi = 1.0;  // Omega increases strictly in alpha for gamma >= 1
  for (int it = 0; it < 64 && hi - lo > 0.0; ++it) {
    const double mid = 0.5 * (lo + hi);
    if (mid <= lo || mid >= hi) break;
    if (omega(gamma, mid) < om)
      lo = mid;
    else
      hi = mid;
  }
  return 0.5 * (lo + hi);
}

}  // extern "C"
