// GRPO token loss, its gradient into the per-token log-probs, and the drift
// diagnostics, on the outputs of the fused LM head.
//
// Four small launches (all HBM-trivial next to the LM-head GEMMs):
//   1. group-normalised advantage per trajectory (one thread per group);
//   2. per token: the trajectory by binary search of the packed offsets, the
//      ratio, the clipped surrogate and its gradient, the k3 reference KL and
//      the drift |logp - logp_old|; unnormalised gradient out, per-block
//      partial sums to the workspace (fixed-order tree in LDS);
//   3. one block sums the partials in block order (fp64) into the statistics;
//   4. the gradient is scaled by 1 / (number of loss tokens).
// Every reduction has a fixed order, so results are bitwise reproducible.
#include "mv_device.h"

namespace mv {

namespace {
constexpr int kTok = 256;          // threads (= tokens) per block of the token pass
// per-block partials: count, loss, |drift|, clip low, clip high, k3, ratio
constexpr int kRatioPart = 6;
constexpr int kNP = 7;
size_t al256(size_t x) { return (x + 255) & ~size_t(255); }
}  // namespace

struct GrpoArgs {
  const int32_t* traj_ptr;   // [n_traj + 1]
  const float* reward;       // [n_traj]
  const float* logp;
  const float* logp_old;
  const float* logp_ref;     // null when beta == 0
  const uint8_t* mask;       // null: every token carries loss
  float* adv;                // [n_traj]
  float* dlogp;              // [T]
  float* part;               // [n_blocks][kNP]
  float* stats;              // 8 floats
  int T, n_traj, G;
  float eps_lo, eps_hi, beta, adv_eps;
};

__global__ __launch_bounds__(256) void grpo_adv_kernel(GrpoArgs a) {
  const int grp = blockIdx.x * 256 + threadIdx.x;
  if (grp * a.G >= a.n_traj) return;
  const float* r = a.reward + size_t(grp) * a.G;
  double mean = 0.0;
  for (int i = 0; i < a.G; ++i) mean += r[i];
  mean /= a.G;
  double var = 0.0;
  for (int i = 0; i < a.G; ++i) var += (r[i] - mean) * (r[i] - mean);
  const double sd = a.G > 1 ? sqrt(var / (a.G - 1)) : 0.0;
  for (int i = 0; i < a.G; ++i)
    a.adv[size_t(grp) * a.G + i] = float((r[i] - mean) / (sd + a.adv_eps));
}

__global__ __launch_bounds__(kTok) void grpo_token_kernel(GrpoArgs a) {
  __shared__ float red[kNP][kTok];
  const int t = blockIdx.x * kTok + threadIdx.x;
  float v[kNP] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (t < a.T) {
    // last trajectory whose first token is <= t
    int lo = 0, hi = a.n_traj - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (a.traj_ptr[mid] <= t)
        lo = mid;
      else
        hi = mid - 1;
    }
    const bool on = a.mask == nullptr || a.mask[t] != 0;
    float g = 0.f;
    if (on) {
      const float A = a.adv[lo];
      const float lp = a.logp[t], old = a.logp_old[t];
      const float rho = expf(lp - old);
      const float lo_e = 1.f - a.eps_lo, hi_e = 1.f + a.eps_hi;
      const float clipped = fminf(fmaxf(rho, lo_e), hi_e);
      const float u = rho * A, c = clipped * A;
      const bool clip_active = c < u;
      float k3 = 0.f, dk3 = 0.f;
      if (a.logp_ref != nullptr) {
        const float x = a.logp_ref[t] - lp;
        const float em1 = expm1f(x);   // exp(x) - 1 without cancellation near x = 0
        k3 = em1 - x;
        dk3 = -em1;
      }
      g = (clip_active ? 0.f : -u) + a.beta * dk3;
      v[0] = 1.f;
      v[1] = -fminf(u, c) + a.beta * k3;
      v[2] = fabsf(lp - old);
      v[3] = (clip_active && rho < lo_e) ? 1.f : 0.f;
      v[4] = (clip_active && rho > hi_e) ? 1.f : 0.f;
      v[5] = k3;
      v[kRatioPart] = rho;
    }
    a.dlogp[t] = g;
  }
#pragma unroll
  for (int k = 0; k < kNP; ++k) red[k][threadIdx.x] = v[k];
  __syncthreads();
  for (int s = kTok / 2; s > 0; s >>= 1) {
    if (threadIdx.x < s) {
#pragma unroll
      for (int k = 0; k < kNP; ++k) red[k][threadIdx.x] += red[k][threadIdx.x + s];
    }
    __syncthreads();
  }
  if (threadIdx.x < kNP) a.part[size_t(blockIdx.x) * kNP + threadIdx.x] = red[threadIdx.x][0];
}

__global__ __launch_bounds__(256) void grpo_finish_kernel(GrpoArgs a, int n_blocks) {
  __shared__ double red[kNP + 1][256];
  double v[kNP + 1] = {0, 0, 0, 0, 0, 0, 0, 0};
  for (int b = threadIdx.x; b < n_blocks; b += 256)
#pragma unroll
    for (int k = 0; k < kNP; ++k) v[k] += a.part[size_t(b) * kNP + k];
  for (int i = threadIdx.x; i < a.n_traj; i += 256) v[kNP] += fabs(double(a.adv[i]));
#pragma unroll
  for (int k = 0; k <= kNP; ++k) red[k][threadIdx.x] = v[k];
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (threadIdx.x < s) {
#pragma unroll
      for (int k = 0; k <= kNP; ++k) red[k][threadIdx.x] += red[k][threadIdx.x + s];
    }
    __syncthreads();
  }
  if (threadIdx.x != 0) return;
  const double n = red[0][0];
  const double inv = n > 0 ? 1.0 / n : 0.0;
  a.stats[0] = float(red[1][0] * inv);               // loss
  a.stats[1] = float(red[2][0] * inv);               // logdiff
  a.stats[2] = float(red[3][0] * inv);               // clip fraction, low side
  a.stats[3] = float(red[4][0] * inv);               // clip fraction, high side
  a.stats[4] = float(red[5][0] * inv);               // mean k3
  a.stats[5] = float(red[kRatioPart][0] * inv);      // mean ratio
  a.stats[6] = float(n);                             // loss tokens
  a.stats[7] = a.n_traj > 0 ? float(red[kNP][0] / a.n_traj) : 0.f;  // mean |advantage|
}

__global__ __launch_bounds__(256) void grpo_scale_kernel(GrpoArgs a) {
  const int t = blockIdx.x * 256 + threadIdx.x;
  if (t >= a.T) return;
  const float n = a.stats[6];
  a.dlogp[t] = n > 0.f ? a.dlogp[t] / n : 0.f;
}

size_t grpo_ws_bytes(int T, int n_traj) {
  const size_t n_blocks = (size_t(T) + kTok - 1) / kTok;
  return al256(n_blocks * kNP * sizeof(float)) + al256(size_t(n_traj) * sizeof(float)) + 256;
}

hipError_t launch_grpo(int T, int n_traj, int G, float eps_lo, float eps_hi, float beta,
                       float adv_eps, const int32_t* traj_ptr, const float* reward,
                       const float* logp, const float* logp_old, const float* logp_ref,
                       const uint8_t* mask, float* adv_out, float* dlogp, float* stats, void* ws,
                       hipStream_t stream) {
  GrpoArgs a{};
  char* base = reinterpret_cast<char*>((reinterpret_cast<uintptr_t>(ws) + 255) & ~uintptr_t(255));
  const int n_blocks = (T + kTok - 1) / kTok;
  a.part = reinterpret_cast<float*>(base);
  a.adv = adv_out != nullptr
              ? adv_out
              : reinterpret_cast<float*>(base + al256(size_t(n_blocks) * kNP * sizeof(float)));
  a.traj_ptr = traj_ptr;
  a.reward = reward;
  a.logp = logp;
  a.logp_old = logp_old;
  a.logp_ref = logp_ref;
  a.mask = mask;
  a.dlogp = dlogp;
  a.stats = stats;
  a.T = T;
  a.n_traj = n_traj;
  a.G = G;
  a.eps_lo = eps_lo;
  a.eps_hi = eps_hi;
  a.beta = logp_ref != nullptr ? beta : 0.f;
  a.adv_eps = adv_eps;
  ProfScope prof("grpo", stream);
  const int n_groups = n_traj / G;
  hipLaunchKernelGGL(grpo_adv_kernel, dim3((n_groups + 255) / 256), dim3(256), 0, stream, a);
  if (T > 0)
    hipLaunchKernelGGL(grpo_token_kernel, dim3(n_blocks), dim3(kTok), 0, stream, a);
  hipLaunchKernelGGL(grpo_finish_kernel, dim3(1), dim3(256), 0, stream, a, n_blocks);
  if (T > 0)
    hipLaunchKernelGGL(grpo_scale_kernel, dim3((T + 255) / 256), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace mv
