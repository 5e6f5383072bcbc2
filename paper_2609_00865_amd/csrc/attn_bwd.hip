// View-masked attention backward on gfx950: one backward for the packed
// trajectory instead of one per branch (Section 4.3, "Cost and deployment
// splits").  Three passes, all recomputing P from the forward's LSE:
//
//  1. D_i = <dO_i, O_i> per row and head, and the row's LSE in base-2 units
//     (HBM-bound, tiny).
//  2. dQ: per 128-row query tile and head, over the forward's tile list:
//     S^T = K Q^T, dP^T = V dO^T, dS^T = P^T o (dP^T - D), dQ^T += K^T dS^T.
//  3. dK/dV: per 128-key tile and KV head, over the contiguous row range that
//     sees some key of the tile, for every query head of the GQA group:
//     S = Q K^T, dV^T += dO^T P, dP = dO V^T, dK^T += Q^T dS.
//     Long ranges are cut into items that write fp32 partial tiles; a reduce
//     pass sums them in a fixed order (deterministic, no atomics).
// All stores write whole 16-byte or 8-byte runs of a row.
#include <mutex>
#include <type_traits>
#include <unordered_map>

#include "mv_device.h"
#include "mv_predicate.h"

namespace mv {

namespace {
constexpr float kLog2e = 1.4426950408889634f;
size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
}  // namespace

struct BwdArgs {
  const u16* q;
  const u16* k;
  const u16* v;
  const u16* o;
  const u16* dout;
  const float* lse;
  u16* dq;
  u16* dk;
  u16* dv;
  float* Dd;       // [Hq, T]
  float* L2;       // [Hq, T] LSE in base-2 units (LSE * log2 e), written by pass 1
  float* partial;  // [n_slots, Hkv, 2, 128, D]
  mv_mask_dev mask;
  int T, Hq, Hkv, n_qt, n_items;
  float scale, scale_log2;
};

// ---------------------------------------------------------------------------
// 1. D = rowsum(dO * O)
// ---------------------------------------------------------------------------
// D/8 consecutive lanes share one (row, head) vector, 16 bytes each, so a
// wave reads whole contiguous rows; the partial dot products are summed
// across those lanes.
template <int D>
__global__ __launch_bounds__(256) void bwd_pre_kernel(BwdArgs a) {
  constexpr int LPV = D / 8;   // lanes per vector
  const int64_t gid = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t vec = gid / LPV;   // row * Hq + head
  const bool ok = vec < int64_t(a.T) * a.Hq;
  float acc = 0.f;
  if (ok) {
    const size_t off = size_t(gid) * 8;   // = vec * D + (gid % LPV) * 8
    const uint4 x = ld16(a.o + off), y = ld16(a.dout + off);
    const uint32_t xs[4] = {x.x, x.y, x.z, x.w}, ys[4] = {y.x, y.y, y.z, y.w};
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      acc = fmaf(bf16_to_f32(xs[w] & 0xffff), bf16_to_f32(ys[w] & 0xffff), acc);
      acc = fmaf(bf16_to_f32(xs[w] >> 16), bf16_to_f32(ys[w] >> 16), acc);
    }
  }
#pragma unroll
  for (int m = LPV / 2; m > 0; m >>= 1) acc += __shfl_xor(acc, m);
  if (ok && gid % LPV == 0) {
    const int i = int(vec / a.Hq), h = int(vec % a.Hq);
    a.Dd[size_t(h) * a.T + i] = acc;
    a.L2[size_t(h) * a.T + i] = a.lse[size_t(h) * a.T + i] * kLog2e;
  }
}

// ---------------------------------------------------------------------------
// 2. dQ
// ---------------------------------------------------------------------------
template <int D, bool IV>
__global__ __launch_bounds__(256, 2) void bwd_dq_kernel(BwdArgs a) {
  constexpr int BQ = kFwdTileQ, BK = kFwdTileK;
  constexpr int KS = D / 16, DB = D / 32;

  // Two buffers: key tile e+1 lands while tile e is read.  K and V rows are
  // unpadded and swizzled (kv_swz): K is read along its rows and with the
  // transposing read, V along its rows.
  __shared__ __align__(1024) u16 sKbuf[2 * BK * D];
  __shared__ __align__(1024) u16 sVbuf[2 * BK * D];
  __shared__ __align__(16) int sOmbuf[2 * BK];

  int xcd, local;
  xcd_split(xcd, local);
  const int qrank = (local / a.Hq) * kNumXcd + xcd;
  const int h = local % a.Hq;
  if (qrank >= a.n_qt) return;
  const int qt = a.mask.qt_order[qrank];
  const int hk = h / (a.Hq / a.Hkv);
  const int T = a.T;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int c = lane & 31, g = lane >> 5;
  const int qrow = qt * BQ + wave * 32 + c;
  const bool qok = qrow < T;

  bf16x8 qf[KS], df[KS];
  {
    const size_t off = (size_t(qok ? qrow : 0) * a.Hq + h) * D + g * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      qf[ks] = as_bf16x8(qok ? ld16(a.q + off + ks * 16) : make_uint4(0, 0, 0, 0));
      df[ks] = as_bf16x8(qok ? ld16(a.dout + off + ks * 16) : make_uint4(0, 0, 0, 0));
    }
  }
  const float lse2 = qok ? a.lse[size_t(h) * T + qrow] * kLog2e : 0.f;
  const float Di = qok ? a.Dd[size_t(h) * T + qrow] : 0.f;

  f32x16 acc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[db][r] = 0.f;

  // K and V of KV head hk go from raw buffers straight into LDS.  Keys past
  // T read row T - 1 (their omega reads as 0, so no row sees them).
  const uint32_t kv_row = uint32_t(a.Hkv) * D * 2;   // bytes per key row
  const uint32_t kv_bytes = uint32_t(T) * kv_row - uint32_t(hk) * D * 2;
  const rsrc_t krs = make_rsrc(a.k + size_t(hk) * D, kv_bytes);
  const rsrc_t vrs = make_rsrc(a.v + size_t(hk) * D, kv_bytes);
  const rsrc_t omrs = make_rsrc(a.mask.omega, uint32_t(T) * 4);
  const KvTileLoader<D, BK> ldr(tid);
  int omreg = 0;
  auto issue_tile = [&](int kt, int buf) {
    const uint32_t st = uint32_t(buf) * BK * D * 2;
    ldr.issue(krs, vrs, kt, T, kv_row, lds_addr(sKbuf) + st, lds_addr(sVbuf) + st);
    omreg = int(buf_ld4(omrs, uint32_t(kt * BK + tid % BK) * 4));  // every thread: key tid % BK
  };

  // Tile e+1 is in flight while tile e is read; after the barrier that ends
  // tile e its buffer takes tile e+2.  The omega values go through registers
  // (written once their load has landed).  One barrier per tile.  Every row
  // tile lists at least its diagonal key tile; the list is read with scalar
  // loads, which do not wait behind the tile loads in flight.
  const int e0 = __builtin_amdgcn_readfirstlane(a.mask.q_ptr[qt]);
  const int e1 = __builtin_amdgcn_readfirstlane(a.mask.q_ptr[qt + 1]);
  issue_tile(sload_i32(a.mask.k_list + e0) >> 1, 0);
  wait_vmcnt<0>();
  sOmbuf[tid % BK] = omreg;   // identical copies
  if (e0 + 1 < e1) issue_tile(sload_i32(a.mask.k_list + e0 + 1) >> 1, 1);
  __syncthreads();
  for (int e = e0; e < e1; ++e) {
    const int ent = sload_i32(a.mask.k_list + e);
    const int kt = ent >> 1;
    const bool full = ent & 1;
    const int buf = (e - e0) & 1;
    const char* sK = reinterpret_cast<const char*>(sKbuf + buf * BK * D);
    const char* sV = reinterpret_cast<const char*>(sVbuf + buf * BK * D);
    const int* sOm = sOmbuf + buf * BK;
    const int j0 = kt * BK;
    // only a partial tile holding a key with several live intervals (masks
    // with restoring edits) walks the interval lists
    const bool tile_iv = IV && !full && __any(sOm[lane] < 0);

    // the tile's two 32-key halves one after the other: S^T and dP^T of a
    // half, its dS^T, then its share of dQ^T (half the live accumulators)
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      f32x16 s, dp;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        s[r] = 0.f;
        dp[r] = 0.f;
      }
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        s = mfma32(ld_row_swz<D>(sK, kb * 32 + c, ks * 2 + g), qf[ks], s);
        dp = mfma32(ld_row_swz<D>(sV, kb * 32 + c, ks * 2 + g), df[ks], dp);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) s[r] = fast_exp2(fmaf(s[r], a.scale_log2, -lse2));
      if (tile_iv) {
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const int4 om = *reinterpret_cast<const int4*>(&sOm[kb * 32 + q4 * 8 + g * 4]);
          const int omv[4] = {om.x, om.y, om.z, om.w};
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int r = q4 * 4 + u;
            const int key = j0 + kb * 32 + q4 * 8 + g * 4 + u;
            s[r] = mv_visible_iv(qrow, key, omv[u], a.mask.iv_ptr, a.mask.iv) ? s[r] : 0.f;
          }
        }
      } else if (!full) {  // block-uniform; per element a select, not a branch
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const int4 om = *reinterpret_cast<const int4*>(&sOm[kb * 32 + q4 * 8 + g * 4]);
          const int omv[4] = {om.x, om.y, om.z, om.w};
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int r = q4 * 4 + u;
            const int key = j0 + kb * 32 + q4 * 8 + g * 4 + u;
            s[r] = mv_visible(qrow, key, omv[u]) ? s[r] : 0.f;
          }
        }
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) s[r] = s[r] * (dp[r] - Di);
      const bf16x8 dsf[2] = {to_operand(s, 0), to_operand(s, 8)};
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
          // K^T operand: column block db of keys (2 kb + kk)*16.. in accumulator order
          acc[db] = mfma32(ld_tr_swz<D>(sK, (2 * kb + kk) * 16, db * 32), dsf[kk], acc[db]);
        }
    }
    // tile e+1 has landed (and its omega values are written) before the
    // barrier that publishes it; then tile e's buffer takes tile e+2
    wait_vmcnt<0>();
    if (e + 1 < e1) sOmbuf[(buf ^ 1) * BK + tid % BK] = omreg;
    __syncthreads();
    if (e + 2 < e1) issue_tile(sload_i32(a.mask.k_list + e + 2) >> 1, buf);
  }

  if (!qok) return;
  u16* out = a.dq + (size_t(qrow) * a.Hq + h) * D;
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      const int d0 = db * 32 + q4 * 8 + g * 4;
      uint2 w;
      w.x = pack2(acc[db][q4 * 4 + 0] * a.scale, acc[db][q4 * 4 + 1] * a.scale);
      w.y = pack2(acc[db][q4 * 4 + 2] * a.scale, acc[db][q4 * 4 + 3] * a.scale);
      *reinterpret_cast<uint2*>(out + d0) = w;
    }
}

// ---------------------------------------------------------------------------
// 3. dK / dV
// ---------------------------------------------------------------------------
template <int D, bool IV>
__global__ __launch_bounds__(256, 1) void bwd_dkdv_kernel(BwdArgs a) {
  constexpr int BK = kBwdTileK, BQ = kBwdBlockQ;
  constexpr int KS = D / 16, DB = D / 32;
  // Q and dO blocks, with the rows' LSE and D, go from raw buffers straight
  // into LDS; Q and dO rows are unpadded and swizzled (kv_swz), read along
  // their rows and with the transposing read.  Four buffers: while step st
  // accumulates dV, dK from its block, step st+1 computes S and dP from the
  // next one, and blocks st+2 and st+3 are in flight (each has two steps to
  // land).
  constexpr int NBUF = 4;
  __shared__ __align__(1024) u16 sQbuf[NBUF * BQ * D];
  __shared__ __align__(1024) u16 sdObuf[NBUF * BQ * D];
  __shared__ __align__(16) float sLbuf[NBUF * BQ];   // LSE * log2 e
  __shared__ __align__(16) float sDbuf[NBUF * BQ];
  // block of step st in buffer st % NBUF (buf below)
  auto qtile = [&](int buf) { return reinterpret_cast<const char*>(sQbuf + buf * BQ * D); };
  auto dotile = [&](int buf) { return reinterpret_cast<const char*>(sdObuf + buf * BQ * D); };

  int xcd, local;
  xcd_split(xcd, local);
  const int w = (local / a.Hkv) * kNumXcd + xcd;
  const int hk = local % a.Hkv;
  if (w >= a.n_items) return;
  const int kt = a.mask.bwd_items[4 * w + 0];
  const int qb0 = a.mask.bwd_items[4 * w + 1];
  const int qb1 = a.mask.bwd_items[4 * w + 2];
  const int slot = a.mask.bwd_items[4 * w + 3];
  const int om_min = a.mask.bwd_tiles[4 * kt + 0];
  const int T = a.T, G = a.Hq / a.Hkv;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int c = lane & 31, g = lane >> 5;
  const int j0 = kt * BK, j1 = min(T, j0 + BK);
  const int key = j0 + wave * 32 + c;
  const bool kok = key < T;
  const int om = kok ? a.mask.omega[key] : 0;

  bf16x8 kf[KS], vf[KS];
  {
    const size_t off = (size_t(kok ? key : 0) * a.Hkv + hk) * D + g * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      kf[ks] = as_bf16x8(kok ? ld16(a.k + off + ks * 16) : make_uint4(0, 0, 0, 0));
      vf[ks] = as_bf16x8(kok ? ld16(a.v + off + ks * 16) : make_uint4(0, 0, 0, 0));
    }
  }
  f32x16 dk[DB], dv[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      dk[db][r] = 0.f;
      dv[db][r] = 0.f;
    }

  const int nqb = qb1 - qb0;
  const int steps = nqb * G;
  const int h0 = hk * G;
  // Step st covers query block qb0 + st % nqb of head h0 + st / nqb.  Rows
  // past T read row T - 1 (finite values; no key is visible to them).  Every
  // wave issues the same number of loads per step (LPS): its share of Q and
  // dO, and the block's LSE (even waves) or D (odd waves; the second pair of
  // waves writes the same words again).
  const uint32_t q_row = uint32_t(a.Hq) * D * 2;     // bytes per query row
  const KvTileLoader<D, BQ> ldr(tid);
  constexpr int LPS = 2 * KvTileLoader<D, BQ>::KLD + 1;
  static_assert(BQ == 64, "one LSE / D word per lane");
  auto issue_step = [&](int st, int buf) {   // a step past the last reloads the last block
    const int sc_ = min(st, steps - 1);
    const int hh = h0 + sc_ / nqb, qb = qb0 + sc_ % nqb;
    const uint32_t bytes = uint32_t(T) * q_row - uint32_t(hh) * D * 2;
    ldr.issue(make_rsrc(a.q + size_t(hh) * D, bytes), make_rsrc(a.dout + size_t(hh) * D, bytes), qb,
              T, q_row, lds_addr(sQbuf) + buf * BQ * D * 2, lds_addr(sdObuf) + buf * BQ * D * 2);
    const bool odd = __builtin_amdgcn_readfirstlane(wave) & 1;   // wave-uniform
    const float* vec = (odd ? a.Dd : a.L2) + size_t(hh) * T;
    buf_lds4(make_rsrc(vec, uint32_t(T) * 4), uint32_t(min(qb * BQ + lane, T - 1)) * 4,
             (odd ? lds_addr(sDbuf) : lds_addr(sLbuf)) + buf * BQ * 4);
  };
  // before the barrier that ends step st: block st+2 landed (st+3 may fly)
  auto wait_step = [&](int st, int n_steps) {
    if (st + 3 < n_steps)
      wait_vmcnt<LPS>();
    else
      wait_vmcnt<0>();
  };

  // The work of a step runs in two halves (unit 2 st + mb: the block's
  // query rows mb*32 ..): S = Q K^T and dP = dO V^T of the half (rows: its
  // queries, lanes: this wave's keys), then P and dS as bf16 operands, then
  // its share of dV^T += dO^T P and dK^T += Q^T dS.
  f32x16 s, dp;
  auto scores_mfma = [&](int st, int mb) {
    const char* sQ = qtile(st % NBUF);
    const char* sdO = dotile(st % NBUF);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      s[r] = 0.f;
      dp[r] = 0.f;
    }
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      s = mfma32(ld_row_swz<D>(sQ, mb * 32 + c, ks * 2 + g), kf[ks], s);
      dp = mfma32(ld_row_swz<D>(sdO, mb * 32 + c, ks * 2 + g), vf[ks], dp);
    }
  };
  // rows of s/dp are queries mb*32 + q4*8 + g*4 + u of the block
  auto scores_valu = [&](int st, int mb, bf16x8 (&pf)[2], bf16x8 (&dsf)[2]) {
    const int buf = st % NBUF;
    const float* sL = sLbuf + buf * BQ;
    const float* sD = sDbuf + buf * BQ;
    const int i0 = (qb0 + st % nqb) * BQ;
    const bool full = (i0 >= j1 - 1) && (i0 + BQ <= om_min);
    // single-interval keys: row i sees this lane's key iff 0 <= i - key < om - key,
    // every row of a full step does (a select, not a branch, keeps the step
    // one scheduling region)
    const uint32_t range = full ? 0x7fffffffu : uint32_t(om - key);
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      const int qo = mb * 32 + q4 * 8 + g * 4;
      const float4 l4 = *reinterpret_cast<const float4*>(&sL[qo]);
      const float4 d4 = *reinterpret_cast<const float4*>(&sD[qo]);
      const float lv[4] = {l4.x, l4.y, l4.z, l4.w};
      const float dd[4] = {d4.x, d4.y, d4.z, d4.w};
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int r = q4 * 4 + u;
        float p = fast_exp2(fmaf(s[r], a.scale_log2, -lv[u]));
        if (IV) {
          if (!full && !mv_visible_iv(i0 + qo + u, key, om, a.mask.iv_ptr, a.mask.iv)) p = 0.f;
        } else {
          p = uint32_t(i0 + qo + u - key) < range ? p : 0.f;
        }
        s[r] = p;
        dp[r] = p * (dp[r] - dd[u]);
      }
    }
    pf[0] = to_operand(s, 0);
    pf[1] = to_operand(s, 8);
    dsf[0] = to_operand(dp, 0);
    dsf[1] = to_operand(dp, 8);
  };
  auto accumulate = [&](int st, int mb, const bf16x8 (&pf)[2], const bf16x8 (&dsf)[2]) {
    const char* sQ = qtile(st % NBUF);
    const char* sdO = dotile(st % NBUF);
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        // dO^T and Q^T operands: columns db*32.. of rows (2 mb + kk)*16.. in accumulator order
        dv[db] = mfma32(ld_tr_swz<D>(sdO, (2 * mb + kk) * 16, db * 32), pf[kk], dv[db]);
        dk[db] = mfma32(ld_tr_swz<D>(sQ, (2 * mb + kk) * 16, db * 32), dsf[kk], dk[db]);
      }
  };

  // Single-interval masks (IV = false): the same units, with every MFMA
  // interleaved with softmax work in a fixed issue order (a scheduling fence
  // after each group).  Unit n's S/dP (run in phase X of unit n-1) feed its
  // softmax elements 0..7 in phase Y of unit n-1 and 8..15 in its own phase
  // X; phase X issues unit n+1's S/dP MFMAs, phase Y unit n's dV/dK MFMAs;
  // operands are read two MFMAs ahead.  Score registers alternate by unit
  // parity; the row LSE, D and mask range of the unit in flight are kept.
  f32x16 sc[2], dc[2];
  float lv[16], dd[16];
  int ui0 = 0, umb = 0;
  uint32_t urange = 0;
  auto load_ctx = [&](int st, int mb, int buf) {
    const float* sL = sLbuf + buf * BQ;
    const float* sD = sDbuf + buf * BQ;
    ui0 = (qb0 + st % nqb) * BQ;
    umb = mb;
    const bool full = (ui0 >= j1 - 1) && (ui0 + BQ <= om_min);
    // a padding step past the last (st >= steps) sees nothing
    urange = st >= steps ? 0u : full ? 0x7fffffffu : uint32_t(om - key);
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      const int qo = mb * 32 + q4 * 8 + g * 4;
      const float4 l4 = *reinterpret_cast<const float4*>(&sL[qo]);
      const float4 d4 = *reinterpret_cast<const float4*>(&sD[qo]);
      lv[q4 * 4 + 0] = l4.x;
      lv[q4 * 4 + 1] = l4.y;
      lv[q4 * 4 + 2] = l4.z;
      lv[q4 * 4 + 3] = l4.w;
      dd[q4 * 4 + 0] = d4.x; dd[q4 * 4 + 1] = d4.y; dd[q4 * 4 + 2] = d4.z; dd[q4 * 4 + 3] = d4.w;
    }
  };
  // softmax element r (row umb*32 + (r/4)*8 + g*4 + r%4) of the unit in flight
  auto elem = [&](int par, int r) {
    float p = fast_exp2(fmaf(sc[par][r], a.scale_log2, -lv[r]));
    p = uint32_t(ui0 + umb * 32 + (r >> 2) * 8 + g * 4 + (r & 3) - key) < urange ? p : 0.f;
    sc[par][r] = p;
    dc[par][r] = p * (dc[par][r] - dd[r]);
  };
  // phase X of the unit in set par: the next unit's (st, mb) S/dP MFMAs into
  // set par ^ 1 (if NEXT) with elements 8..15 of this unit, then its operands
  auto phaseX = [&](auto next_tag, int par, int st, int mb, bf16x8 (&pfo)[2], bf16x8 (&dso)[2],
                    int buf) {
    constexpr bool NEXT = decltype(next_tag)::value;
    const char* sQ = qtile(buf);
    const char* sdO = dotile(buf);
    const int np = par ^ 1;
    auto opnd = [&](int j) {   // MFMA j: ks = j / 2, S (even) or dP (odd)
      return ld_row_swz<D>((j & 1) ? sdO : sQ, mb * 32 + c, (j >> 1) * 2 + g);
    };
    bf16x8 op[3];
    if constexpr (NEXT) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        sc[np][r] = 0.f;
        dc[np][r] = 0.f;
      }
      op[0] = opnd(0);
      op[1] = opnd(1);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < 2 * KS; ++j) {
      if constexpr (NEXT) {
        if (j + 2 < 2 * KS) op[(j + 2) % 3] = opnd(j + 2);
        if (j & 1)
          dc[np] = mfma32(op[j % 3], vf[j >> 1], dc[np]);
        else
          sc[np] = mfma32(op[j % 3], kf[j >> 1], sc[np]);
      }
      if ((j & 1) && 8 + (j >> 1) < 16) elem(par, 8 + (j >> 1));
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int r = 8 + KS; r < 16; ++r) elem(par, r);   // D = 64: the rest
    pfo[0] = to_operand(sc[par], 0);
    pfo[1] = to_operand(sc[par], 8);
    dso[0] = to_operand(dc[par], 0);
    dso[1] = to_operand(dc[par], 8);
  };
  // phase Y of unit (st, mb): its dV/dK MFMAs with elements 0..7 of the next
  // unit (st2, mb2) in set np, whose context is loaded first (if NEXT)
  auto phaseY = [&](auto next_tag, int st, int mb, const bf16x8 (&pfc)[2], const bf16x8 (&dsc)[2],
                    int np, int st2, int mb2, int buf, int buf2) {
    constexpr bool NEXT = decltype(next_tag)::value;
    if constexpr (NEXT) load_ctx(st2, mb2, buf2);
    const char* sQ = qtile(buf);
    const char* sdO = dotile(buf);
    // MFMA q: db = q / 4, kk = (q / 2) % 2, dV (even q) or dK (odd q)
    auto opnd = [&](int q) {
      return ld_tr_swz<D>((q & 1) ? sQ : sdO, (2 * mb + ((q >> 1) & 1)) * 16, (q >> 2) * 32);
    };
    constexpr int NQ = 4 * DB;
    bf16x8 op[3];
    op[0] = opnd(0);
    op[1] = opnd(1);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      if (q + 2 < NQ) op[(q + 2) % 3] = opnd(q + 2);
      const int db = q >> 2, kk = (q >> 1) & 1;
      if (q & 1)
        dk[db] = mfma32(op[q % 3], dsc[kk], dk[db]);
      else
        dv[db] = mfma32(op[q % 3], pfc[kk], dv[db]);
      if constexpr (NEXT) {
        if ((q & 1) && (q >> 1) < 8) elem(np, q >> 1);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (NEXT) {
#pragma unroll
      for (int r = NQ / 2; r < 8; ++r) elem(np, r);   // D = 64: the rest
    }
  };

  // Software pipeline over half-step units, one barrier per step: the next
  // unit's S and dP MFMAs are issued before this unit's dV and dK MFMAs, and
  // the next unit's exponentials follow them.  Block st+3 is requested into
  // the buffer step st-1 used (every wave finished with it before the last
  // barrier).
  bf16x8 pf[2], dsf[2];
  // Masks with restoring edits: only a key tile that holds a key with several
  // live intervals takes the plain loop with the interval walk; every other
  // tile runs the pipelined loop of single-interval masks.
  bool iv_tile = false;
  if constexpr (IV) iv_tile = __syncthreads_or(kok && om < 0) != 0;
  if (iv_tile) {
    issue_step(0, 0);
    if (steps > 1) issue_step(1, 1);
    if (steps > 2) issue_step(2, 2);
    wait_step(-1, steps);   // blocks 0 and 1 landed
    __syncthreads();
    scores_mfma(0, 0);
    scores_valu(0, 0, pf, dsf);
    for (int st = 0; st + 1 < steps; ++st) {
      if (st + 3 < steps) issue_step(st + 3, (st + 3) % NBUF);
      scores_mfma(st, 1);
      accumulate(st, 0, pf, dsf);
      scores_valu(st, 1, pf, dsf);
      scores_mfma(st + 1, 0);
      accumulate(st, 1, pf, dsf);
      scores_valu(st + 1, 0, pf, dsf);
      wait_step(st, steps);
      __syncthreads();
    }
    scores_mfma(steps - 1, 1);
    accumulate(steps - 1, 0, pf, dsf);
    scores_valu(steps - 1, 1, pf, dsf);
    accumulate(steps - 1, 1, pf, dsf);
  } else {
    // The step count is padded to a multiple of NBUF with steps that see
    // nothing (they reload the last block, so every operand is finite), and
    // the loop is unrolled NBUF times: every LDS buffer index is then a
    // compile-time constant and the fragment reads use immediate offsets.
    // The last step starts a unit past the end whose results are dropped.
    using yes = std::true_type;
    const int steps_pad = (steps + NBUF - 1) / NBUF * NBUF;
    static_assert(NBUF == 4, "unrolled four times");
    issue_step(0, 0);
    issue_step(1, 1);
    issue_step(2, 2);
    wait_step(-1, steps_pad);   // blocks 0 and 1 landed
    __syncthreads();
    // unit (0, 0): S/dP into set 0, its context, elements 0..7
    load_ctx(0, 0, 0);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      sc[0][r] = 0.f;
      dc[0][r] = 0.f;
    }
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      sc[0] = mfma32(ld_row_swz<D>(qtile(0), c, ks * 2 + g), kf[ks], sc[0]);
      dc[0] = mfma32(ld_row_swz<D>(dotile(0), c, ks * 2 + g), vf[ks], dc[0]);
    }
#pragma unroll
    for (int r = 0; r < 8; ++r) elem(0, r);
    auto iter = [&](int st, int u) {   // u = st % NBUF, a constant at each call
      if (st + 3 < steps_pad) issue_step(st + 3, (u + 3) & 3);
      phaseX(yes{}, 0, st, 1, pf, dsf, u);                           // S/dP of (st, 1); finish (st, 0)
      phaseY(yes{}, st, 0, pf, dsf, 1, st, 1, u, u);                 // dV/dK of (st, 0); start (st, 1)
      phaseX(yes{}, 1, st + 1, 0, pf, dsf, (u + 1) & 3);             // S/dP of (st+1, 0); finish (st, 1)
      phaseY(yes{}, st, 1, pf, dsf, 0, st + 1, 0, u, (u + 1) & 3);   // dV/dK of (st, 1); start (st+1, 0)
      wait_step(st, steps_pad);
      __syncthreads();
    };
    for (int st = 0; st < steps_pad; st += NBUF) {
      iter(st, 0);
      iter(st + 1, 1);
      iter(st + 2, 2);
      iter(st + 3, 3);
    }
  }

  if (!kok) return;
  if (slot < 0) {
    u16* pk = a.dk + (size_t(key) * a.Hkv + hk) * D;
    u16* pv = a.dv + (size_t(key) * a.Hkv + hk) * D;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int d0 = db * 32 + q4 * 8 + g * 4;
        uint2 wk, wv;
        wk.x = pack2(dk[db][q4 * 4 + 0] * a.scale, dk[db][q4 * 4 + 1] * a.scale);
        wk.y = pack2(dk[db][q4 * 4 + 2] * a.scale, dk[db][q4 * 4 + 3] * a.scale);
        wv.x = pack2(dv[db][q4 * 4 + 0], dv[db][q4 * 4 + 1]);
        wv.y = pack2(dv[db][q4 * 4 + 2], dv[db][q4 * 4 + 3]);
        *reinterpret_cast<uint2*>(pk + d0) = wk;
        *reinterpret_cast<uint2*>(pv + d0) = wv;
      }
  } else {
    float* base = a.partial + (size_t(slot) * a.Hkv + hk) * 2 * BK * D;
    float* pk = base + size_t(wave * 32 + c) * D;
    float* pv = base + size_t(BK) * D + size_t(wave * 32 + c) * D;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int d0 = db * 32 + q4 * 8 + g * 4;
        *reinterpret_cast<float4*>(pk + d0) =
            make_float4(dk[db][q4 * 4 + 0] * a.scale, dk[db][q4 * 4 + 1] * a.scale,
                        dk[db][q4 * 4 + 2] * a.scale, dk[db][q4 * 4 + 3] * a.scale);
        *reinterpret_cast<float4*>(pv + d0) =
            make_float4(dv[db][q4 * 4 + 0], dv[db][q4 * 4 + 1], dv[db][q4 * 4 + 2],
                        dv[db][q4 * 4 + 3]);
      }
  }
}

// Sum the fp32 partial tiles of every split key tile in slot order.
template <int D>
__global__ __launch_bounds__(256) void bwd_reduce_kernel(BwdArgs a, int n_red) {
  constexpr int BK = kBwdTileK;
  const int r = blockIdx.x / a.Hkv, hk = blockIdx.x % a.Hkv;
  if (r >= n_red) return;
  const int kt = a.mask.bwd_red[r];
  const int first = a.mask.bwd_tiles[4 * kt + 2], n = a.mask.bwd_tiles[4 * kt + 3];
  for (int e = threadIdx.x; e < 2 * BK * D / 4; e += blockDim.x) {
    const int which = e / (BK * D / 4);
    const int rem = e % (BK * D / 4);
    const int kk = rem / (D / 4), d0 = (rem % (D / 4)) * 4;
    const int key = kt * BK + kk;
    if (key >= a.T) continue;
    // partials summed in slot order (the result does not depend on
    // scheduling); four loads in flight
    const size_t stride = size_t(a.Hkv) * 2 * BK * D;   // floats from one slot to the next
    const float* p = a.partial + ((size_t(first) * a.Hkv + hk) * 2 + which) * BK * D +
                     size_t(kk) * D + d0;
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    int i = 0;
    for (; i + 4 <= n; i += 4) {
      float4 x[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) x[u] = *reinterpret_cast<const float4*>(p + (i + u) * stride);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        s.x += x[u].x;
        s.y += x[u].y;
        s.z += x[u].z;
        s.w += x[u].w;
      }
    }
    for (; i < n; ++i) {
      const float4 x = *reinterpret_cast<const float4*>(p + i * stride);
      s.x += x.x;
      s.y += x.y;
      s.z += x.z;
      s.w += x.w;
    }
    u16* out = (which == 0 ? a.dk : a.dv) + (size_t(key) * a.Hkv + hk) * D + d0;
    uint2 wv;
    wv.x = pack2(s.x, s.y);
    wv.y = pack2(s.z, s.w);
    *reinterpret_cast<uint2*>(out) = wv;
  }
}

// Scratch of mv_attn_bwd_noalloc: the backward's workspace (row statistics
// D and the fp32 partials of split key tiles) in a file-scope device array,
// one copy on every GPU the library runs on, held until the process ends.
// Every kernel that reads a byte of it writes that byte earlier in the same
// call, so nothing needs clearing; calls that overlap on one GPU race.
static __device__ __align__(256) unsigned char scratch[MV_ATTN_BWD_NOALLOC_SCRATCH_BYTES];

// The device address of `scratch` on the current device.  In host code the
// array's name is only a stand-in for the symbol, never a device address: the
// address comes from the runtime once per device and is kept.
hipError_t attn_bwd_scratch(void** ptr) {
  static std::mutex mu;
  static std::unordered_map<int, void*> addr;
  int dev = -1;
  if (hipError_t e = hipGetDevice(&dev); e != hipSuccess) return e;
  std::lock_guard<std::mutex> lk(mu);
  auto it = addr.find(dev);
  if (it == addr.end()) {
    void* p = nullptr;
    if (hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)); e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    it = addr.emplace(dev, p).first;
  }
  *ptr = it->second;
  return hipSuccess;
}

// D [Hq, T] | LSE * log2 e [Hq, T] | fp32 partials [n_slots, Hkv, 2, 128, D]
size_t attn_bwd_ws_bytes(const mv_view_mask& m, int Hq, int Hkv, int D) {
  return 2 * align256(size_t(Hq) * m.T * sizeof(float)) +
         align256(size_t(m.n_slots) * Hkv * 2 * kBwdTileK * D * sizeof(float)) + 256;
}

hipError_t launch_attn_bwd(const mv_view_mask& m, int Hq, int Hkv, int D, float scale,
                           const void* q, const void* k, const void* v, const void* o,
                           const void* dout, const float* lse, void* dq, void* dk, void* dv,
                           void* ws, hipStream_t stream, bool profile) {
  BwdArgs a;
  a.q = static_cast<const u16*>(q);
  a.k = static_cast<const u16*>(k);
  a.v = static_cast<const u16*>(v);
  a.o = static_cast<const u16*>(o);
  a.dout = static_cast<const u16*>(dout);
  a.lse = lse;
  a.dq = static_cast<u16*>(dq);
  a.dk = static_cast<u16*>(dk);
  a.dv = static_cast<u16*>(dv);
  char* base = static_cast<char*>(ws);
  base = reinterpret_cast<char*>((reinterpret_cast<uintptr_t>(base) + 255) & ~uintptr_t(255));
  const size_t row_stat = align256(size_t(Hq) * m.T * sizeof(float));
  a.Dd = reinterpret_cast<float*>(base);
  a.L2 = reinterpret_cast<float*>(base + row_stat);
  a.partial = reinterpret_cast<float*>(base + 2 * row_stat);
  a.mask = m.d;
  a.T = m.T;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.n_qt = m.n_qt;
  a.n_items = m.stats.bwd_items;
  a.scale = scale;
  a.scale_log2 = scale * kLog2e;

  const int64_t rows = int64_t(m.T) * Hq;
  const dim3 b256(256);
  const dim3 g_pre(unsigned((rows * (D / 8) + 255) / 256));
  const int per_xcd_q = (m.n_qt + kNumXcd - 1) / kNumXcd;
  const dim3 g_dq(per_xcd_q * Hq * kNumXcd);
  const int per_xcd_kv = (a.n_items + kNumXcd - 1) / kNumXcd;
  const dim3 g_kv(per_xcd_kv * Hkv * kNumXcd);
  const int n_red = int(m.bwd_red.size());
  const dim3 g_red(unsigned(std::max(1, n_red * Hkv)));
  // the general predicate only when some key has further live intervals
  const bool iv = !m.iv.empty();
  auto run = [&](auto pre, auto dkdv, auto red, auto dq) {
    { ProfScope p("attn_bwd_pre", stream, profile);
      hipLaunchKernelGGL(pre, g_pre, b256, 0, stream, a); }
    { ProfScope p("attn_bwd_dkdv", stream, profile);
      hipLaunchKernelGGL(dkdv, g_kv, b256, 0, stream, a); }
    if (n_red) {
      ProfScope p("attn_bwd_reduce", stream, profile);
      hipLaunchKernelGGL(red, g_red, b256, 0, stream, a, n_red);
    }
    { ProfScope p("attn_bwd_dq", stream, profile);
      hipLaunchKernelGGL(dq, g_dq, b256, 0, stream, a); }
  };
  if (D == 128 && iv)
    run(bwd_pre_kernel<128>, bwd_dkdv_kernel<128, true>, bwd_reduce_kernel<128>, bwd_dq_kernel<128, true>);
  else if (D == 128)
    run(bwd_pre_kernel<128>, bwd_dkdv_kernel<128, false>, bwd_reduce_kernel<128>, bwd_dq_kernel<128, false>);
  else if (iv)
    run(bwd_pre_kernel<64>, bwd_dkdv_kernel<64, true>, bwd_reduce_kernel<64>, bwd_dq_kernel<64, true>);
  else
    run(bwd_pre_kernel<64>, bwd_dkdv_kernel<64, false>, bwd_reduce_kernel<64>, bwd_dq_kernel<64, false>);
  return hipGetLastError();
}

}  // namespace mv
