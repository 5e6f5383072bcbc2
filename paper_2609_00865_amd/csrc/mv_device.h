// Device helpers for gfx950 (CDNA4): MFMA operand types, bf16 packing, and
// the block -> work mapping that keeps related blocks on one XCD.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "mv_internal.h"

namespace mv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16;

// D = A * B + C on a 32x32 tile with K = 16 (bf16 in, fp32 accumulate).
// Lane l supplies row (l % 32) of A and column (l % 32) of B, each as 8
// consecutive k values of group (l / 32); any permutation of k applied to both
// operands leaves D unchanged.  D element r of lane l is row
// (r / 4) * 8 + (l / 32) * 4 + r % 4, column l % 32.
__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// D = A * B + C on a 16x16 tile with K = 32.  Lane l supplies row (l % 16) of
// A and column (l % 16) of B, each as the 8 consecutive k values of group
// (l / 16); D element r of lane l is row (l / 16) * 4 + r, column l % 16.
__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

// M0, which these loads take as the LDS base, is a register the compiler
// may also use (and does not let inline asm clobber), so each helper saves it
// in a scratch SGPR and restores it right after the issue: from the
// compiler's view M0 is unchanged.  (The hardware reads M0 when the load is
// issued.)  The compiler's own LDS-DMA builtins are not used because it
// cannot tell which LDS buffer they write and would wait for every load in
// flight before any LDS read.
// 16 bytes per lane from global memory straight into LDS: lane l's data lands
// at LDS byte address lds + 16 l (lds is the wave's base, uniform across the
// wave).  The load is counted by vmcnt only; the compiler does not track it,
// so the caller waits with wait_vmcnt before a barrier that publishes it.
__device__ __forceinline__ void lds_load16(const void* src, uint32_t lds) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %1, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(src), "s"(__builtin_amdgcn_readfirstlane(lds))
      : "memory");
}

// A wave-uniform pointer taken through readfirstlane, so that it is held in
// scalar registers (the inline asm below takes scalar operands; the compiler
// may otherwise keep a uniform value in vector registers).
template <typename X>
__device__ __forceinline__ X* uniform_ptr(X* p) {
  const uint64_t a = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane(uint32_t(a));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(uint32_t(a >> 32));
  return reinterpret_cast<X*>((uint64_t(hi) << 32) | lo);
}

// A block-uniform 32-bit word read through the scalar data cache (a scalar
// load, tracked by lgkmcnt): it does not wait behind vector loads in flight,
// as a vector load of the same word would.  p must be uniform; the data must
// not change during the kernel.
__device__ __forceinline__ int sload_i32(const int* p) {
  int v;
  asm volatile("s_load_dword %0, %1, 0x0\n\ts_waitcnt lgkmcnt(0)"
               : "=s"(v)
               : "s"(uniform_ptr(p)));
  return v;
}

// s_waitcnt vmcnt(N) (the other counters left alone).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x70 | 0xF00);
}

__device__ __forceinline__ uint4 ld16(const void* p) { return *reinterpret_cast<const uint4*>(p); }

// A raw buffer over [base, base + bytes) (bytes < 2^32): loads take a 32-bit
// byte offset in a VGPR, and the hardware's range check returns zeros for an
// access at or past `bytes`, so the ragged end of a tile needs neither a
// clamped address nor a branch.  (The range check covers the VGPR offset; no
// SGPR offset is used.)  Word 3 is the gfx9 descriptor format (32-bit data).
typedef __amdgpu_buffer_rsrc_t rsrc_t;
__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(uniform_ptr(base)), 0,
                                           __builtin_amdgcn_readfirstlane(bytes), 0x00020000);
}
// 16 bytes per lane from a raw buffer straight into LDS: lane l's data
// lands at LDS byte address lds + 16 l (lds uniform across the wave).  As
// with lds_load16 the load is counted by vmcnt only; the caller waits with
// wait_vmcnt before the barrier that publishes it.  Offsets must stay in
// range (an out-of-range lane's LDS bytes are not relied upon).
__device__ __forceinline__ void buf_lds16(rsrc_t r, uint32_t off, uint32_t lds) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %3\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(off), "s"(r), "s"(__builtin_amdgcn_readfirstlane(lds))
      : "memory");
}
// 4 bytes per lane from a raw buffer straight into LDS (lane l at lds + 4 l).
__device__ __forceinline__ void buf_lds4(rsrc_t r, uint32_t off, uint32_t lds) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %3\n\tbuffer_load_dword %1, %2, 0 offen lds\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(off), "s"(r), "s"(__builtin_amdgcn_readfirstlane(lds))
      : "memory");
}
__device__ __forceinline__ uint4 buf_ld16(rsrc_t r, uint32_t off) {
  const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
  return make_uint4(v[0], v[1], v[2], v[3]);
}
__device__ __forceinline__ uint32_t buf_ld4(rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
}

__device__ __forceinline__ void st16(void* p, uint4 v) { *reinterpret_cast<uint4*>(p) = v; }

__device__ __forceinline__ uint32_t bf16_bits(float f) {
  return static_cast<uint32_t>(__builtin_bit_cast(uint16_t, static_cast<__bf16>(f)));
}

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __builtin_bit_cast(float, static_cast<uint32_t>(b) << 16);
}

// Two floats rounded to bf16 (nearest even) in one 32-bit word, lo in the low
// half: a single v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  const f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// Eight consecutive fp32 accumulator values as one bf16 MFMA operand.
__device__ __forceinline__ bf16x8 to_operand(const f32x16& acc, int base) {
  uint4 u;
  u.x = pack2(acc[base + 0], acc[base + 1]);
  u.y = pack2(acc[base + 2], acc[base + 3]);
  u.z = pack2(acc[base + 4], acc[base + 5]);
  u.w = pack2(acc[base + 6], acc[base + 7]);
  return as_bf16x8(u);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// max of x over lanes l and l ^ 32 (gfx950's permlane32_swap: a VALU op, no
// LDS round trip)
__device__ __forceinline__ float max_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, x),
                                                  __builtin_bit_cast(uint32_t, x), false, false);
  return fmaxf(__builtin_bit_cast(float, uint32_t(r[0])), __builtin_bit_cast(float, uint32_t(r[1])));
}

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

// Key tiles in LDS without padding (attention forward and dQ).  A tile of
// BK rows of D bf16 holds row r's D/8 16-byte chunks permuted: chunk c sits
// at position c ^ kv_swz<D>(r).  The permutation spreads both the row reads
// of an MFMA operand (16 rows, one chunk each) and the transposing reads (4
// rows x 4 chunks) over distinct banks; it depends on r % 16 only.
template <int D>
__device__ __forceinline__ int kv_swz(int r) {
  return D == 128 ? ((r & 3) << 2) | ((r >> 2) & 3) : (((r >> 1) & 1) << 2) | ((r >> 2) & 3);
}

// Row-read operand: 16 bytes (8 consecutive k) of chunk ch of row r.
template <int D>
__device__ __forceinline__ bf16x8 ld_row_swz(const char* tile, int r, int ch) {
  return as_bf16x8(ld16(tile + r * (D * 2) + ((ch ^ kv_swz<D>(r)) << 4)));
}

// MFMA operand read *across* the rows of a swizzled tile, with gfx950's
// transposing LDS read: within each group of 16 lanes, lane i receives
// element i % 4 of the 8-byte pieces addressed by lanes 4k + i / 4 (k = 0..3).
// Lane l = lane % 16 addresses rows rbase + g*4 + l/4 and + 8, columns
// col0 + 16((lane/16) % 2) + 4(l % 4) .. +4 (chunk col0/8 + 2((lane/16) % 2) +
// (l % 4)/2, half l % 2), so lane (c = lane % 32, g = lane / 32) receives
// column col0 + c of rows rbase + g*4 + {0,1,2,3} and rbase + 8 + g*4 +
// {0,1,2,3}: the k order of an MFMA accumulator's rows (see mfma32), so the
// result pairs with an operand taken straight from an accumulator.  rbase a
// multiple of 16, col0 of 32.
template <int D>
__device__ __forceinline__ bf16x8 ld_tr_swz(const char* tile, int rbase, int col0) {
  const int lane = threadIdx.x & 63, l = lane & 15;
  const int r = (lane >> 5) * 4 + (l >> 2);
  const int ch = (col0 >> 3) + ((lane >> 4) & 1) * 2 + ((l & 3) >> 1);
  const char* p0 = tile + (rbase + r) * (D * 2) + ((ch ^ kv_swz<D>(r)) << 4) + (l & 1) * 8;
  const char* p1 = tile + (rbase + r + 8) * (D * 2) + ((ch ^ kv_swz<D>(r + 8)) << 4) + (l & 1) * 8;
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p0));
  const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p1));
  typedef short i16x8 __attribute__((ext_vector_type(8)));
  const i16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return __builtin_bit_cast(bf16x8, v);
}

// Loads K and V tiles of BK key rows (one KV head; rows kv_row bytes apart
// in memory) straight into swizzled LDS tiles with 256 threads.  Load r of
// wave w fills chunk positions P = (r * 4 + w) * 64 + lane: row P / (D/8),
// position P % (D/8), i.e. chunk (P % (D/8)) ^ kv_swz<D>(row).  Rows past
// the last key read the last key (the caller masks them).
template <int D, int BK>
struct KvTileLoader {
  static constexpr int KLD = BK * D / 8 / 256;   // loads per thread and tensor
  static_assert(KLD >= 1, "tile too small for 256 threads");
  int row[KLD];
  uint32_t col[KLD];   // byte offset of the loaded chunk within its row
  uint32_t wv;         // LDS byte offset of this thread's wave within a tile
  // tid: the thread's index among the 256 that load (0..255)
  __device__ __forceinline__ explicit KvTileLoader(int tid) : wv(uint32_t(tid >> 6) * 1024) {
#pragma unroll
    for (int r = 0; r < KLD; ++r) {
      const int P = (r * 4 + (tid >> 6)) * 64 + (tid & 63);
      row[r] = P / (D / 8);
      col[r] = uint32_t((P % (D / 8)) ^ kv_swz<D>(P / (D / 8))) * 16;
    }
  }
  // one tensor's key tile kt into the tile at LDS byte address lds (KLD
  // loads per thread)
  __device__ __forceinline__ void issue_one(rsrc_t rs, int kt, int T, uint32_t kv_row,
                                            uint32_t lds) const {
#pragma unroll
    for (int r = 0; r < KLD; ++r) {
      const uint32_t off = uint32_t(min(kt * BK + row[r], T - 1)) * kv_row + col[r];
      buf_lds16(rs, off, lds + wv + r * 4096);
    }
  }
  // K and V of key tile kt into the tiles at LDS byte addresses ldsK, ldsV
  __device__ __forceinline__ void issue(rsrc_t krs, rsrc_t vrs, int kt, int T, uint32_t kv_row,
                                        uint32_t ldsK, uint32_t ldsV) const {
#pragma unroll
    for (int r = 0; r < KLD; ++r) {
      const uint32_t off = uint32_t(min(kt * BK + row[r], T - 1)) * kv_row + col[r];
      buf_lds16(krs, off, ldsK + wv + r * 4096);
      buf_lds16(vrs, off, ldsV + wv + r * 4096);
    }
  }
};

// LDS byte address of a __shared__ object
template <typename X>
__device__ __forceinline__ uint32_t lds_addr(X* p) {
  typedef __attribute__((address_space(3))) X lds_x;
  return (uint32_t)(uintptr_t)(lds_x*)p;
}

// The dispatcher deals consecutive block ids to the 8 XCDs round-robin.
// Returns (xcd, index of the block among those of its XCD).
__device__ __forceinline__ void xcd_split(int& xcd, int& local) {
  xcd = blockIdx.x % kNumXcd;
  local = blockIdx.x / kNumXcd;
}

}  // namespace mv
