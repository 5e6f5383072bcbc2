// Visibility predicate shared by every kernel that applies the view mask and
// by the host and device mask materialisers, so that the bits the tests see
// are the bits the attention computes with.
//
// Row i sees key j iff tau(j) <= i < omega(j), with tau(j) = j (a key is born
// at its own row; the diagonal is included) -- Eq. "4d-mask-def", Section 4.2.
#pragma once

#if defined(__HIPCC__)
#define MV_HD __host__ __device__ __forceinline__
#else
#define MV_HD inline
#endif

// (bitwise &: both comparisons are evaluated, so a vector unit selects
// instead of branching per element)
MV_HD bool mv_visible(int i, int j, int omega_j) { return (j <= i) & (i < omega_j); }

// The same test with the key given by its offset from a base key b: jo = j -
// b and di = i - b (j <= i iff jo <= di).  Kernels take b per lane and tile,
// so that jo is a compile-time constant per score element and the diagonal
// test compares against an immediate.
MV_HD bool mv_visible_rel(int di, int jo, int i, int omega_j) {
  return (jo <= di) & (i < omega_j);
}

// A key that a later edit restores has further live intervals.  Such a key is
// stored with the sign bit of omega set (the low 31 bits keep the end of its
// first interval) and its other intervals [b, e) in a per-key list: iv[2k],
// iv[2k + 1] for k in [iv_ptr[j], iv_ptr[j + 1]).  For every other key this is
// the single-interval test above.
MV_HD int mv_first_end(int omega_j) { return omega_j & 0x7fffffff; }

MV_HD bool mv_visible_iv(int i, int j, int omega_j, const int* iv_ptr, const int* iv) {
  if (omega_j >= 0) return j <= i && i < omega_j;
  if (j <= i && i < mv_first_end(omega_j)) return true;
  for (int k = iv_ptr[j]; k < iv_ptr[j + 1]; ++k)
    if (iv[2 * k] <= i && i < iv[2 * k + 1]) return true;
  return false;
}

// The predicate of a kernel specialised on whether the mask has interval
// lists at all: without them (IV = false) every omega is a key's only end.
template <bool IV>
MV_HD bool mv_visible_k(int i, int j, int omega_j, const int* iv_ptr, const int* iv) {
  return IV ? mv_visible_iv(i, j, omega_j, iv_ptr, iv) : mv_visible(i, j, omega_j);
}

#if defined(__HIPCC__)
// The visibility bits of one lane's 32 score elements of a 64-key tile whose
// keys may have several live intervals, in the attention kernels' layout:
// element e (bit e) is key j0 + (e / 16) * 32 + ((e % 16) / 4) * 8 + g * 4 +
// e % 4 for query row i; omega of the tile's key k at om[k].  Out of line: the
// interval walk stays off the register budget of the kernels' pipelined
// loops, which call it only for tiles that hold such a key.
[[maybe_unused]] static __device__ __noinline__ uint32_t
mv_visible_iv_bits(int i, int j0, int g, const int* om, const int* iv_ptr, const int* iv) {
  uint32_t bits = 0;
  for (int e = 0; e < 32; ++e) {
    const int k = (e >> 4) * 32 + ((e & 15) >> 2) * 8 + g * 4 + (e & 3);
    if (mv_visible_iv(i, j0 + k, om[k], iv_ptr, iv)) bits |= 1u << e;
  }
  return bits;
}
#endif
