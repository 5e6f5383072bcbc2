// Device side of the branch packings: the gather that builds the packed
// stream, its adjoint (deterministic sum over each token's copies), the
// rotary embedding by per-segment position ids, and the gather and the
// adjoint with the rotation fused into them (Q and K enter the packed layer
// rotated by their branch positions; dQ and dK leave it rotated back and
// summed over their copies in one pass).  All are bandwidth-bound streams
// of 16-byte (or head-row) accesses.
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

// Angles of the fused passes: theta^(-2i/d) per block in LDS (fp64), the
// angle pos * theta^(-2i/d) in fp64 (positions reach 1e5 radians), reduced
// to [-pi, pi] in fp64, then its cosine and sine in fp32.
__device__ __forceinline__ void rope_cs(int pos, double inv_freq, float& c, float& s) {
  const double a = double(pos) * inv_freq;
  const double k = rint(a * 0.15915494309189535);   // 1 / (2 pi)
  sincosf(float(fma(-k, 6.283185307179586, a)), &s, &c);
}

__device__ __forceinline__ void load_bf16x8(const u16* p, float (&x)[8]) {
  const uint4 v = ld16(p);
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    x[2 * e] = bf16_to_f32(uint16_t(w[e] & 0xffff));
    x[2 * e + 1] = bf16_to_f32(uint16_t(w[e] >> 16));
  }
}

__device__ __forceinline__ void store_bf16x8(u16* p, const float (&x)[8]) {
  uint4 v;
  v.x = pack2(x[0], x[1]);
  v.y = pack2(x[2], x[3]);
  v.z = pack2(x[4], x[5]);
  v.w = pack2(x[6], x[7]);
  st16(p, v);
}

__device__ __forceinline__ void fill_inv_freq(double* invf, int d, double log_theta) {
  for (int i = threadIdx.x; i < d / 2; i += blockDim.x) invf[i] = exp(-(2.0 * i / d) * log_theta);
  __syncthreads();
}

// out[slot] = R(pos[slot]) in[src[slot]]: one thread per (slot, 8-wide chunk
// of the first half of a head row); the chunk's eight angles once, then the
// pairs (i, i + d/2) of every head rotated in fp32 and rounded once to bf16.
__global__ __launch_bounds__(256) void pack_rope_kernel(const int32_t* __restrict__ src,
                                                        const int32_t* __restrict__ pos,
                                                        const u16* __restrict__ in, int H, int d,
                                                        double log_theta, u16* __restrict__ out,
                                                        int64_t n_items) {
  __shared__ double invf[128];
  fill_inv_freq(invf, d, log_theta);
  const int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= n_items) return;
  const int CH = d / 16, half = d / 2;
  const int64_t slot = idx / CH;
  const int c0 = int(idx % CH) * 8;
  float cs[8], sn[8];
  const int ps = pos[slot];
#pragma unroll
  for (int e = 0; e < 8; ++e) rope_cs(ps, invf[c0 + e], cs[e], sn[e]);
  const int64_t srow = src[slot];
  for (int h = 0; h < H; ++h) {
    const u16* x = in + (srow * H + h) * d + c0;
    float x0[8], x1[8], y0[8], y1[8];
    load_bf16x8(x, x0);
    load_bf16x8(x + half, x1);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      y0[e] = x0[e] * cs[e] - x1[e] * sn[e];
      y1[e] = x1[e] * cs[e] + x0[e] * sn[e];
    }
    u16* y = out + (slot * H + h) * d + c0;
    store_bf16x8(y, y0);
    store_bf16x8(y + half, y1);
  }
}

// out[t] = sum over the copies of token t, in slot order, of
// R(pos[slot])^T in[slot], in fp32, rounded once: one thread per (token,
// block of 4 heads, 8-wide chunk).
constexpr int kRopeHeads = 4;
__global__ __launch_bounds__(256) void unpack_rope_kernel(const int32_t* __restrict__ copy_ptr,
                                                          const int32_t* __restrict__ copy_slot,
                                                          const int32_t* __restrict__ pos,
                                                          const u16* __restrict__ in, int H,
                                                          int d, double log_theta, int out_fp32,
                                                          void* __restrict__ out,
                                                          int64_t n_items) {
  __shared__ double invf[128];
  fill_inv_freq(invf, d, log_theta);
  const int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= n_items) return;
  const int CH = d / 16, half = d / 2;
  const int NHB = (H + kRopeHeads - 1) / kRopeHeads;
  const int64_t t = idx / (CH * NHB);
  const int rem = int(idx % (CH * NHB));
  const int h0 = (rem / CH) * kRopeHeads;
  const int c0 = (rem % CH) * 8;
  float a0[kRopeHeads][8], a1[kRopeHeads][8];
#pragma unroll
  for (int j = 0; j < kRopeHeads; ++j)
#pragma unroll
    for (int e = 0; e < 8; ++e) a0[j][e] = a1[j][e] = 0.f;
  for (int k = copy_ptr[t]; k < copy_ptr[t + 1]; ++k) {
    const int64_t slot = copy_slot[k];
    float cs[8], sn[8];
    const int ps = pos[slot];
#pragma unroll
    for (int e = 0; e < 8; ++e) rope_cs(ps, invf[c0 + e], cs[e], sn[e]);
#pragma unroll
    for (int j = 0; j < kRopeHeads; ++j) {
      if (h0 + j >= H) break;
      const u16* x = in + (slot * H + h0 + j) * d + c0;
      float x0[8], x1[8];
      load_bf16x8(x, x0);
      load_bf16x8(x + half, x1);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        a0[j][e] += x0[e] * cs[e] + x1[e] * sn[e];
        a1[j][e] += x1[e] * cs[e] - x0[e] * sn[e];
      }
    }
  }
#pragma unroll
  for (int j = 0; j < kRopeHeads; ++j) {
    if (h0 + j >= H) break;
    const int64_t o = (t * H + h0 + j) * d + c0;
    if (out_fp32) {
      float* y = static_cast<float*>(out) + o;
      *reinterpret_cast<float4*>(y) = make_float4(a0[j][0], a0[j][1], a0[j][2], a0[j][3]);
      *reinterpret_cast<float4*>(y + 4) = make_float4(a0[j][4], a0[j][5], a0[j][6], a0[j][7]);
      *reinterpret_cast<float4*>(y + half) = make_float4(a1[j][0], a1[j][1], a1[j][2], a1[j][3]);
      *reinterpret_cast<float4*>(y + half + 4) =
          make_float4(a1[j][4], a1[j][5], a1[j][6], a1[j][7]);
    } else {
      u16* y = static_cast<u16*>(out) + o;
      store_bf16x8(y, a0[j]);
      store_bf16x8(y + half, a1[j]);
    }
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

hipError_t launch_pack_rope(const mv_branch_pack& p, const void* in, int H, int d, float theta,
                            void* out, hipStream_t stream) {
  const int64_t n = int64_t(p.N) * (d / 16);
  if (n == 0) return hipSuccess;
  ProfScope prof("pack_rope", stream);
  hipLaunchKernelGGL(pack_rope_kernel, dim3(unsigned((n + 255) / 256)), dim3(256), 0, stream,
                     p.d_src, p.d_pos, static_cast<const u16*>(in), H, d,
                     std::log(double(theta)), static_cast<u16*>(out), n);
  return hipGetLastError();
}

hipError_t launch_unpack_rope(const mv_branch_pack& p, const void* in, int H, int d, float theta,
                              bool out_fp32, void* out, hipStream_t stream) {
  const int64_t n = int64_t(p.T) * (d / 16) * ((H + kRopeHeads - 1) / kRopeHeads);
  if (n == 0) return hipSuccess;
  ProfScope prof("unpack_rope", stream);
  hipLaunchKernelGGL(unpack_rope_kernel, dim3(unsigned((n + 255) / 256)), dim3(256), 0, stream,
                     p.d_copy_ptr, p.d_copy_slot, p.d_pos, static_cast<const u16*>(in), H, d,
                     std::log(double(theta)), out_fp32 ? 1 : 0, out, n);
  return hipGetLastError();
}

}  // namespace mv
