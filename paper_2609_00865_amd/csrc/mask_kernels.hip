// Device materialisation of the visibility bits the attention kernels act on,
// and the clipped-surrogate gradient helper.
#include "mv_device.h"
#include "mv_predicate.h"

namespace mv {

// One thread per 32-bit word: word w of row i covers keys [32w, 32w + 32).
// The word's 64-key tile is looked up in the row's tile list exactly as the
// forward pass walks it; keys of unlisted tiles are 0, keys of full tiles 1,
// keys of partial tiles take the shared predicate.
__global__ void materialize_kernel(mv_mask_dev mk, int T, int row_begin, int row_end, int words,
                                   uint32_t* bits) {
  const int64_t gid = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t total = int64_t(row_end - row_begin) * words;
  if (gid >= total) return;
  const int i = row_begin + int(gid / words);
  const int w = int(gid % words);
  const int kt = (w * 32) / kFwdTileK;
  const int qt = i / kFwdTileQ;
  int lo = mk.q_ptr[qt], hi = mk.q_ptr[qt + 1];
  int ent = -1;
  while (lo < hi) {  // entries are sorted by key tile
    const int mid = (lo + hi) >> 1;
    const int kk = mk.k_list[mid] >> 1;
    if (kk == kt) {
      ent = mk.k_list[mid];
      break;
    }
    if (kk < kt) lo = mid + 1; else hi = mid;
  }
  uint32_t out = 0;
  if (ent >= 0) {
    const bool full = ent & 1;
    for (int b = 0; b < 32; ++b) {
      const int j = w * 32 + b;
      if (j >= T) break;
      if (full || mv_visible_iv(i, j, mk.omega[j], mk.iv_ptr, mk.iv)) out |= 1u << b;
    }
  }
  bits[gid] = out;
}

hipError_t launch_materialize(const mv_view_mask& m, int row_begin, int row_end, uint32_t* bits,
                              hipStream_t stream) {
  const int words = (m.T + 31) / 32;
  const int64_t total = int64_t(row_end - row_begin) * words;
  if (total == 0) return hipSuccess;
  const int64_t blocks = (total + 255) / 256;
  ProfScope p("materialize", stream);
  hipLaunchKernelGGL(materialize_kernel, dim3(unsigned(blocks)), dim3(256), 0, stream, m.d, m.T,
                     row_begin, row_end, words, bits);
  return hipGetLastError();
}

// d/dlogp of -scale * min(r A, clamp(r, 1-eps_lo, 1+eps_hi) A) with dr/dlogp = r.
__global__ void ppo_clip_kernel(int n, const float* ratio, const float* adv, float eps_lo,
                                float eps_hi, float scale, float* out) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= n) return;
  const float r = ratio[t], A = adv[t];
  const float rc = fminf(fmaxf(r, 1.f - eps_lo), 1.f + eps_hi);
  out[t] = (r * A <= rc * A) ? -scale * r * A : 0.f;
}

hipError_t launch_ppo_clip(int n, const float* ratio, const float* adv, float eps_lo,
                           float eps_hi, float scale, float* out, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  ProfScope p("ppo_clip", stream);
  hipLaunchKernelGGL(ppo_clip_kernel, dim3((n + 255) / 256), dim3(256), 0, stream, n, ratio, adv,
                     eps_lo, eps_hi, scale, out);
  return hipGetLastError();
}

}  // namespace mv
