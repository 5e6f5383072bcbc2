// GRPO token loss, its gradient into the per-token log-probs, and the drift
// diagnostics, on the outputs of the fused LM head (the same loss also runs
// inside the LM head's combine pass: mv_token_logprob_grpo; both use the
// per-token arithmetic of mv_grpo_dev.h).
//
// Four small launches (all HBM-trivial next to the LM-head GEMMs):
//   1. group-normalised advantage per trajectory;
//   2. per token: the trajectory by binary search of the packed offsets, the
//      ratio, the clipped surrogate and its gradient, the k3 reference KL and
//      the drift |logp - logp_old|; unnormalised gradient out, per-block
//      partial sums to the workspace (fixed-order tree in LDS);
//   3. one block sums the partials in block order (fp64) into the statistics;
//   4. the gradient is scaled by 1 / (number of loss tokens).
// Every reduction has a fixed order, so results are bitwise reproducible.
#include "mv_grpo_dev.h"

namespace mv {

namespace {
constexpr int kTok = 256;          // threads (= tokens) per block of the token pass
constexpr int kRatioPart = 6;
constexpr int kNP = kGrpoParts;
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
  float* part;               // [kNP][n_blocks] (counter-major)
  float* stats;              // 8 floats
  int T, n_traj, G;
  float eps_lo, eps_hi, beta, adv_eps;
};

__global__ __launch_bounds__(256) void grpo_adv_kernel(GrpoArgs a) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= a.n_traj) return;
  a.adv[i] = grpo_advantage(a.reward, a.G, i, a.adv_eps);
}

__global__ __launch_bounds__(kTok) void grpo_token_kernel(GrpoArgs a) {
  __shared__ float red[kNP][kTok];
  const int t = blockIdx.x * kTok + threadIdx.x;
  float v[kNP] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (t < a.T) {
    const int tr = grpo_traj_of(a.traj_ptr, a.n_traj, t);
    const bool on = a.mask == nullptr || a.mask[t] != 0;
    float g = 0.f;
    if (on)
      g = grpo_token_terms(a.logp[t], a.logp_old[t],
                           a.logp_ref != nullptr ? a.logp_ref + t : nullptr, a.adv[tr], a.eps_lo,
                           a.eps_hi, a.beta, v);
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
  if (threadIdx.x < kNP) a.part[size_t(threadIdx.x) * gridDim.x + blockIdx.x] = red[threadIdx.x][0];
}

// One block: the per-block partials (counter-major: counter k of block b at
// part[k * stride + b]) summed in fp64, thread-strided (16-byte loads where
// the rows allow them) then a fixed tree, into the statistics.
constexpr int kFinish = 512;
__global__ __launch_bounds__(kFinish) void grpo_finish_kernel(GrpoArgs a, int n_blocks,
                                                              int stride) {
  __shared__ double red[kNP + 1][kFinish];
  double v[kNP + 1] = {0, 0, 0, 0, 0, 0, 0, 0};
  const bool vec = (stride & 3) == 0 && (reinterpret_cast<uintptr_t>(a.part) & 15) == 0;
  const int n4 = vec ? n_blocks / 4 : 0;
#pragma unroll
  for (int k = 0; k < kNP; ++k) {
    const float* row = a.part + size_t(k) * stride;
    for (int b = threadIdx.x; b < n4; b += kFinish) {
      const float4 x = reinterpret_cast<const float4*>(row)[b];
      v[k] += x.x;
      v[k] += x.y;
      v[k] += x.z;
      v[k] += x.w;
    }
    for (int b = 4 * n4 + threadIdx.x; b < n_blocks; b += kFinish) v[k] += row[b];
  }
  for (int i = threadIdx.x; i < a.n_traj; i += kFinish) v[kNP] += fabs(double(a.adv[i]));
#pragma unroll
  for (int k = 0; k <= kNP; ++k) red[k][threadIdx.x] = v[k];
  __syncthreads();
  for (int s = kFinish / 2; s > 0; s >>= 1) {
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
  hipLaunchKernelGGL(grpo_adv_kernel, dim3((n_traj + 255) / 256), dim3(256), 0, stream, a);
  if (T > 0)
    hipLaunchKernelGGL(grpo_token_kernel, dim3(n_blocks), dim3(kTok), 0, stream, a);
  hipLaunchKernelGGL(grpo_finish_kernel, dim3(1), dim3(kFinish), 0, stream, a, n_blocks,
                     n_blocks);
  if (T > 0)
    hipLaunchKernelGGL(grpo_scale_kernel, dim3((T + 255) / 256), dim3(256), 0, stream, a);
  return hipGetLastError();
}

// Statistics of the GRPO loss that the LM head's combine pass evaluated per
// token (part: its per-block partials, counter k of block b at part[k *
// stride + b]; adv: the advantages its preparation pass wrote).
hipError_t launch_grpo_fused_finish(const float* part, int n_blocks, int stride, int n_traj,
                                    const float* adv, float* stats, hipStream_t stream) {
  GrpoArgs a{};
  a.part = const_cast<float*>(part);
  a.adv = const_cast<float*>(adv);
  a.stats = stats;
  a.n_traj = n_traj;
  hipLaunchKernelGGL(grpo_finish_kernel, dim3(1), dim3(kFinish), 0, stream, a, n_blocks, stride);
  return hipGetLastError();
}

}  // namespace mv
