// Draft window size and the speedup model of parallel decoding: host-only
// arithmetic (no device code), used by a scheduler to size the draft window
// from measured forward times.
//
// Times are per generated token in units of t = T_q, the draft's forward time;
// the target's verification forward is T_p = c t.  The accepted length of one
// window is the accepted prefix, TruncGeo(tau, gamma), whose mean is the sum
// of P(X >= k) = tau^k over k = 1..gamma (Suppl. Lemma 1); it is summed
// directly, which is exact at tau = 1 and free of the closed form's
// cancellation near it.
#include <cmath>

#include "pvlm.h"

namespace {

constexpr int kMaxGamma = 1 << 20;
constexpr double kSnapRel = 1e-9;

// sum_{k=1..gamma} tau^k, by Horner's rule from the innermost power out
double accepted_mean(double tau, int gamma) {
  double acc = 0.0;
  for (int k = 0; k < gamma; ++k) acc = tau * (1.0 + acc);
  return acc;
}

double ratio_of(double time) { return time == HUGE_VAL ? 0.0 : 1.0 / time; }

// c, or the integer it lies within kSnapRel (relative) of
double snap(double c) {
  const double r = std::nearbyint(c);
  return std::fabs(c - r) <= kSnapRel * std::fabs(c) ? r : c;
}

// T_p / T_PSD_r: the speedup of parallel decoding with rollback
double rollback_speedup(double c, double tau, int gamma) {
  const double total = (1.0 + std::pow(tau, gamma)) * accepted_mean(tau, gamma);
  if (total == 0.0) return 0.0;
  return c * total / (2.0 * std::fmax(static_cast<double>(gamma), c));
}

bool finite_pos(double x) { return std::isfinite(x) && x > 0.0; }

}  // namespace

extern "C" pvlm_status pvlm_speedup(double c, double tau, int gamma, pvlm_speedup_model* out) {
  if (!out) return PVLM_ERR_NULL;
  if (!finite_pos(c) || !(tau >= 0.0 && tau <= 1.0) || gamma < 1 || gamma > kMaxGamma)
    return PVLM_ERR_SHAPE;
  const double g = gamma;
  const double busy = std::fmax(g, c);  // one pipelined round: max(gamma t, c t)
  const double ex = accepted_mean(tau, gamma);
  const double tot = (1.0 + std::pow(tau, gamma)) * ex;
  pvlm_speedup_model m;
  m.expected_accepted = ex;
  m.expected_total = tot;
  m.t_sd_ideal = (g + c) / (g + 1.0);
  m.t_psd_ideal = busy / g;
  m.t_sd = (g + c) / (tau * g + 1.0);
  m.t_psd = tau > 0.0 ? busy / (tau * g) : HUGE_VAL;
  m.t_psd_rollback = tot > 0.0 ? 2.0 * busy / tot : HUGE_VAL;
  m.v_sd_ideal = c * ratio_of(m.t_sd_ideal);
  m.v_psd_ideal = c * ratio_of(m.t_psd_ideal);
  m.v_sd = c * ratio_of(m.t_sd);
  m.v_psd = c * ratio_of(m.t_psd);
  m.v_psd_rollback = c * ratio_of(m.t_psd_rollback);
  *out = m;
  return PVLM_OK;
}

extern "C" pvlm_status pvlm_window_size(double t_p, double t_q, pvlm_round rounding, double tau,
                                        int gamma_max, int* gamma, double* c_out) {
  if (!gamma) return PVLM_ERR_NULL;
  if (!finite_pos(t_p) || !finite_pos(t_q) || gamma_max < 1 || gamma_max > kMaxGamma)
    return PVLM_ERR_SHAPE;
  const double c = t_p / t_q;
  if (!finite_pos(c)) return PVLM_ERR_SHAPE;
  const double cs = snap(c);
  const auto clamp = [gamma_max](double v) {
    return v < 1.0 ? 1 : (v > gamma_max ? gamma_max : static_cast<int>(v));
  };
  int g;
  switch (rounding) {
    case PVLM_ROUND_DOWN: g = clamp(std::floor(cs)); break;
    case PVLM_ROUND_UP: g = clamp(std::ceil(cs)); break;
    case PVLM_ROUND_NEAREST: g = clamp(std::floor(cs + 0.5)); break;
    case PVLM_ROUND_BEST: {
      if (!(tau > 0.0 && tau <= 1.0)) return PVLM_ERR_SHAPE;
      // Below c the speedup grows with gamma, from c on it does not: the best
      // integer window is the rounded-down or the rounded-up ratio.
      const int lo = clamp(std::floor(cs)), hi = clamp(std::ceil(cs));
      g = (hi != lo && rollback_speedup(cs, tau, hi) > rollback_speedup(cs, tau, lo)) ? hi : lo;
      break;
    }
    default: return PVLM_ERR_SHAPE;
  }
  *gamma = g;
  if (c_out) *c_out = c;
  return PVLM_OK;
}
