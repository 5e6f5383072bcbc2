// Per-token arithmetic of the GRPO loss (training recipe of Appendix F; the
// ratio, advantage and reference-KL terms of Propositions "rl_tree" /
// "rl_4d"; the drift of Eq. "logdiff"), shared by the stand-alone loss pass
// and the LM head's combine pass that fuses it, so that both take the same
// operations in the same order and agree bit for bit on every per-token
// output.
#pragma once
#include "mv_device.h"

namespace mv {

// Per-token terms summed into the statistics: loss-token count, loss,
// |drift|, clip active on the low side, on the high side, k3, ratio.
constexpr int kGrpoParts = 7;

// The last trajectory whose first token is <= t (traj_ptr non-decreasing,
// traj_ptr[0] = 0 <= t): binary search.
__device__ __forceinline__ int grpo_traj_of(const int32_t* traj_ptr, int n_traj, int t) {
  int lo = 0, hi = n_traj - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (traj_ptr[mid] <= t)
      lo = mid;
    else
      hi = mid - 1;
  }
  return lo;
}

// The same index found by one wave (all 64 lanes call it with the same t):
// each round the lanes test the first offsets of 64 equal sub-ranges and a
// ballot keeps the last sub-range that starts at or before t (one load per
// lane and round; one round for up to 64 trajectories).  Indices stay in
// [0, n_traj) whatever traj_ptr holds.
__device__ __forceinline__ int grpo_traj_of_wave(const int32_t* traj_ptr, int n_traj, int t,
                                                 int lane) {
  int lo = 0, n = n_traj;   // the answer lies in [lo, lo + n); traj_ptr[lo] <= t
  while (n > 1) {
    const int step = (n + 63) / 64;
    const bool le = lane * step < n && traj_ptr[lo + lane * step] <= t;
    const uint64_t m = __ballot(le) | 1ull;   // lane 0 starts at lo
    const int k = 63 - __clzll(m);
    lo += k * step;
    n = min(step, n - k * step);
  }
  return lo;
}

// Group-normalised advantage of trajectory i: its group is the run of G
// trajectories that holds it; mean and sample standard deviation (n - 1; 0
// for a group of one) in fp64, summed in trajectory order.
__device__ __forceinline__ float grpo_advantage(const float* reward, int G, int i,
                                                float adv_eps) {
  const float* r = reward + size_t(i / G) * G;
  double mean = 0.0;
  for (int k = 0; k < G; ++k) mean += r[k];
  mean /= G;
  double var = 0.0;
  for (int k = 0; k < G; ++k) var += (r[k] - mean) * (r[k] - mean);
  const double sd = G > 1 ? sqrt(var / (G - 1)) : 0.0;
  return float((reward[i] - mean) / (sd + adv_eps));
}

// One loss token: returns d(-surr + beta k3)/d logp (not yet divided by the
// number of loss tokens) and fills its statistics terms v.
__device__ __forceinline__ float grpo_token_terms(float lp, float old, const float* ref_t,
                                                  float A, float eps_lo, float eps_hi,
                                                  float beta, float (&v)[kGrpoParts]) {
  const float rho = expf(lp - old);
  const float lo_e = 1.f - eps_lo, hi_e = 1.f + eps_hi;
  const float clipped = fminf(fmaxf(rho, lo_e), hi_e);
  const float u = rho * A, c = clipped * A;
  const bool clip_active = c < u;
  float k3 = 0.f, dk3 = 0.f;
  if (ref_t != nullptr) {
    const float x = *ref_t - lp;
    const float em1 = expm1f(x);   // exp(x) - 1 without cancellation near x = 0
    k3 = em1 - x;
    dk3 = -em1;
  }
  v[0] = 1.f;
  v[1] = -fminf(u, c) + beta * k3;
  v[2] = fabsf(lp - old);
  v[3] = (clip_active && rho < lo_e) ? 1.f : 0.f;
  v[4] = (clip_active && rho > hi_e) ? 1.f : 0.f;
  v[5] = k3;
  v[6] = rho;
  return (clip_active ? 0.f : -u) + beta * dk3;
}

}  // namespace mv
