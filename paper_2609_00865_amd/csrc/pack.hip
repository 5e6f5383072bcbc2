// Device side of the branch-replicated packing: the gather that builds the
// packed stream, its adjoint (deterministic sum over each token's copies),
// and the rotary embedding by per-segment position ids.  All three are
// bandwidth-bound streams of 16-byte (or head-row) accesses.
#include "mv_device.h"

namespace mv {

// One thread per 16-byte chunk of an output row.
__global__ __launch_bounds__(256) void pack_rows_kernel(const int32_t* __restrict__ src,
                                                        const u16* __restrict__ in, int W,
                                                        u16* __restrict__ out, int64_t n_chunks) {
  const int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= n_chunks) return;
  const int cpr = W / 8;
  const int64_t slot = idx / cpr;
  const int c = int(idx % cpr);
  st16(out + slot * W + c * 8, ld16(in + int64_t(src[slot]) * W + c * 8));
}

// One thread per 8 elements of a physical row: the copies' values summed in
// slot order in fp32.
__global__ __launch_bounds__(256) void unpack_sum_kernel(const int32_t* __restrict__ copy_ptr,
                                                         const int32_t* __restrict__ copy_slot,
                                                         const u16* __restrict__ in, int W,
                                                         int out_fp32, void* __restrict__ out,
                                                         int64_t n_chunks) {
  const int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= n_chunks) return;
  const int cpr = W / 8;
  const int64_t t = idx / cpr;
  const int c = int(idx % cpr);
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int k = copy_ptr[t]; k < copy_ptr[t + 1]; ++k) {
    const uint4 v = ld16(in + int64_t(copy_slot[k]) * W + c * 8);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc[2 * e] += bf16_to_f32(uint16_t(w[e] & 0xffff));
      acc[2 * e + 1] += bf16_to_f32(uint16_t(w[e] >> 16));
    }
  }
  if (out_fp32) {
    float* o = static_cast<float*>(out) + t * W + c * 8;
    *reinterpret_cast<float4*>(o) = make_float4(acc[0], acc[1], acc[2], acc[3]);
    *reinterpret_cast<float4*>(o + 4) = make_float4(acc[4], acc[5], acc[6], acc[7]);
  } else {
    uint4 v;
    v.x = pack2(acc[0], acc[1]);
    v.y = pack2(acc[2], acc[3]);
    v.z = pack2(acc[4], acc[5]);
    v.w = pack2(acc[6], acc[7]);
    st16(static_cast<u16*>(out) + t * W + c * 8, v);
  }
}

// One thread per (slot, frequency i): the angle pos * theta^(-2i/d) and its
// sine and cosine in double precision (positions reach 1e5 radians), then the
// pair (i, i + d/2) of every head rotated in fp32.
__global__ __launch_bounds__(256) void rope_kernel(const int32_t* __restrict__ pos,
                                                   const u16* x, int H, int d, double log_theta,
                                                   int direction, u16* out, int64_t n_items) {
  const int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= n_items) return;
  const int half = d / 2;
  const int64_t slot = idx / half;
  const int i = int(idx % half);
  const double a = double(pos[slot]) * exp(-(2.0 * i / d) * log_theta);
  double sd, cd;
  sincos(a, &sd, &cd);
  const float c = float(cd), s = direction > 0 ? float(sd) : -float(sd);
  for (int h = 0; h < H; ++h) {
    const int64_t base = (slot * H + h) * d;
    const float x0 = bf16_to_f32(x[base + i]), x1 = bf16_to_f32(x[base + i + half]);
    const float y0 = x0 * c - x1 * s, y1 = x1 * c + x0 * s;
    out[base + i] = uint16_t(bf16_bits(y0));
    out[base + i + half] = uint16_t(bf16_bits(y1));
  }
}

hipError_t launch_pack_rows(const mv_branch_pack& p, const void* in, int W, void* out,
                            hipStream_t stream) {
  const int64_t n = int64_t(p.N) * (W / 8);
  if (n == 0) return hipSuccess;
  ProfScope prof("pack", stream);
  hipLaunchKernelGGL(pack_rows_kernel, dim3(unsigned((n + 255) / 256)), dim3(256), 0, stream,
                     p.d_src, static_cast<const u16*>(in), W, static_cast<u16*>(out), n);
  return hipGetLastError();
}

hipError_t launch_unpack_sum(const mv_branch_pack& p, const void* in, int W, bool out_fp32,
                             void* out, hipStream_t stream) {
  const int64_t n = int64_t(p.T) * (W / 8);
  if (n == 0) return hipSuccess;
  ProfScope prof("unpack", stream);
  hipLaunchKernelGGL(unpack_sum_kernel, dim3(unsigned((n + 255) / 256)), dim3(256), 0, stream,
                     p.d_copy_ptr, p.d_copy_slot, static_cast<const u16*>(in), W,
                     out_fp32 ? 1 : 0, out, n);
  return hipGetLastError();
}

hipError_t launch_rope(const mv_branch_pack& p, const void* x, int H, int d, float theta,
                       int direction, void* out, hipStream_t stream) {
  const int64_t n = int64_t(p.N) * (d / 2);
  if (n == 0) return hipSuccess;
  ProfScope prof("rope", stream);
  hipLaunchKernelGGL(rope_kernel, dim3(unsigned((n + 255) / 256)), dim3(256), 0, stream, p.d_pos,
                     static_cast<const u16*>(x), H, d, std::log(double(theta)), direction,
                     static_cast<u16*>(out), n);
  return hipGetLastError();
}

}  // namespace mv
