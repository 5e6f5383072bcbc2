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

MV_HD bool mv_visible(int i, int j, int omega_j) { return j <= i && i < omega_j; }
