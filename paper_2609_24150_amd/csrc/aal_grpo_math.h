// Group arithmetic of the GRPO loss on the debiased greedy acceptance length
// (Section "GRPO Loss on Acceptance Length": Eq. debiased_reward, the policy
// ratio, Eq. advantage and the clipped surrogate) for one group of windows.
// fp64 throughout.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace aal {

// Per-row inputs of the group arithmetic.
struct GrpoRowIn {
  int32_t s_theta, s_ref, xstar;
  float lp_theta, lp_ref;  // log pi_theta(s_theta), log pi_ref(s_theta), natural log
};

constexpr int kGrpoMaxM = 64;

// One group of m windows of K rows; row_at(i, k) gives row k of window i.
// Writes dloss/dlog rho of every window to coef[m] (the loss being the mean of
// the group losses over n_groups groups) and, when non-null, the accepted
// lengths, advantages and clipped log ratios; returns the group's loss.
// Derivatives at kinks: a clip passes 1 strictly inside its interval; min(u,
// v) takes u's derivative when u <= v.
template <class RowAt>
__device__ double grpo_group(int m, int K, RowAt row_at, double eps, double adv_clip, double eps_clip,
                             double rho_min, double rho_max, double inv_nm, float* coef, int32_t* tau_theta,
                             int32_t* tau_ref, float* advantage, float* log_rho) {
  double R[kGrpoMaxM], lr[kGrpoMaxM];
  double mean = 0.0;
  for (int i = 0; i < m; ++i) {
    int tth = 0, trf = 0;
    bool mth = true, mrf = true;
    double acc = 0.0;
    for (int k = 0; k < K; ++k) {
      const GrpoRowIn w = row_at(i, k);
      mth = mth && w.s_theta == w.xstar;
      mrf = mrf && w.s_ref == w.xstar;
      tth += mth ? 1 : 0;
      trf += mrf ? 1 : 0;
      acc += double(w.lp_theta) - double(w.lp_ref);
    }
    R[i] = double(tth - trf);
    lr[i] = acc / K;
    mean += R[i];
    if (tau_theta) tau_theta[i] = tth;
    if (tau_ref) tau_ref[i] = trf;
  }
  mean /= m;
  double var = 0.0;
  for (int i = 0; i < m; ++i) var += (R[i] - mean) * (R[i] - mean);
  const double sd = sqrt(var / m);
  double loss = 0.0;
  for (int i = 0; i < m; ++i) {
    double A = (R[i] - mean) / (sd + eps);
    if (adv_clip > 0.0) A = fmin(fmax(A, -adv_clip), adv_clip);
    const double lrc = fmin(fmax(lr[i], -10.0), 10.0);
    const double rho_e = exp(lrc);
    const double rho = fmin(fmax(rho_e, rho_min), rho_max);
    const double lo = 1.0 - eps_clip, hi = 1.0 + eps_clip;
    const double u = rho * A, v = fmin(fmax(rho, lo), hi) * A;
    loss += fmin(u, v);
    const double dclip = (rho > lo && rho < hi) ? 1.0 : 0.0;
    const double dsur = (u <= v) ? A : A * dclip;
    const bool inner = rho_e > rho_min && rho_e < rho_max && lr[i] > -10.0 && lr[i] < 10.0;
    coef[i] = float(-inv_nm * dsur * (inner ? rho_e : 0.0));
    if (advantage) advantage[i] = float(A);
    if (log_rho) log_rho[i] = float(lrc);
  }
  return -loss / m;
}

}  // namespace aal
