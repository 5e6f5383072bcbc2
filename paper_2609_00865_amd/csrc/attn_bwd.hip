// View-masked attention backward on gfx950: one backward for the packed
// trajectory instead of one per branch (Section 4.3, "Cost and deployment
// splits").  Two passes (and a reduce), all recomputing P from the
// forward's LSE:
//
//  1. dQ: per 128-row query tile and head, over the forward's tile list:
//     S^T = K Q^T, dP^T = V dO^T, dS^T = P^T o (dP^T - D), dQ^T += K^T dS^T.
//     Each row's D = <dO_i, O_i> is taken in the prologue (every row and
//     head belongs to exactly one block) and stored negated, beside the
//     row's LSE in base-2 units, for the next pass.
//  2. dK/dV: per 128-key tile and KV head, over the contiguous row range that
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
  float* Dd;       // [Hq, T] -D = -rowsum(dO o O), written by the dQ pass
  float* L2;       // [Hq, T] LSE in base-2 units (LSE * log2 e), written by the dQ pass
  float* partial;  // [n_slots, Hkv, 2, 128, D]
  mv_mask_dev mask;
  int T, Hq, Hkv, n_qt, n_items;
  float scale, scale_log2;
};

// ---------------------------------------------------------------------------
// 1. dQ (and the rows' -D and LSE * log2 e)
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

  // Q and dO of the lane's row (d = ks*16 + g*8 .. +8), and D = <dO, O> of
  // the row: this lane's half of the products, then the partner lane's
  bf16x8 qf[KS], df[KS];
  float dsum = 0.f;
  {
    const size_t off = (size_t(qok ? qrow : 0) * a.Hq + h) * D + g * 8;
    const uint4 z = make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      qf[ks] = as_bf16x8(qok ? ld16(a.q + off + ks * 16) : z);
      const uint4 y = qok ? ld16(a.dout + off + ks * 16) : z;
      const uint4 x = qok ? ld16(a.o + off + ks * 16) : z;
      df[ks] = as_bf16x8(y);
      const uint32_t xs[4] = {x.x, x.y, x.z, x.w}, ys[4] = {y.x, y.y, y.z, y.w};
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        dsum = fmaf(bf16_to_f32(xs[w] & 0xffff), bf16_to_f32(ys[w] & 0xffff), dsum);
        dsum = fmaf(bf16_to_f32(xs[w] >> 16), bf16_to_f32(ys[w] >> 16), dsum);
      }
    }
  }
  dsum += __shfl_xor(dsum, 32);
  const float lse2 = qok ? a.lse[size_t(h) * T + qrow] * kLog2e : 0.f;
  const float nDi = -dsum;
  if (qok && g == 0) {   // for the dK/dV pass
    a.Dd[size_t(h) * T + qrow] = nDi;
    a.L2[size_t(h) * T + qrow] = lse2;
  }
  // -D_i in every element: the dP^T chain starts from it, so its MFMAs
  // deliver dP - D (lane = query row) and dS = P o (dP - D) is one multiply
  f32x16 negD;
#pragma unroll
  for (int r = 0; r < 16; ++r) negD[r] = nDi;

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
  // tile e in buffer BUF = (e - e0) & 1, a compile-time constant in each
  // half of the loop below (LDS addresses fold into immediate offsets)
  auto tile = [&](auto buf_tag, int e) {
    constexpr int buf = decltype(buf_tag)::value;
    const int ent = sload_i32(a.mask.k_list + e);
    const int kt = ent >> 1;
    const bool full = ent & 1;
    const char* sK = reinterpret_cast<const char*>(sKbuf + buf * BK * D);
    const char* sV = reinterpret_cast<const char*>(sVbuf + buf * BK * D);
    const int* sOm = sOmbuf + buf * BK;
    const int j0 = kt * BK;
    // only a partial tile holding a key with several live intervals (masks
    // with restoring edits) walks the interval lists
    const bool tile_iv = IV && !full && __any(sOm[lane] < 0);

    // The tile's MFMAs in one fixed sequence: S^T and dP^T of key half 0,
    // of half 1, then dQ^T += K^T dS^T of both halves.  The vector work of
    // a half runs beside the MFMAs that follow it: the exponentials of S
    // beside its dP MFMAs, half 0's dS beside half 1's S MFMAs, half 1's dS
    // beside half 0's dQ MFMAs; only the mask of a partial tile runs alone.
    constexpr int NS = 2 * KS;            // S and dP MFMAs of one half
    constexpr int NM = 2 * NS + 4 * DB;   // MFMAs of the tile
    f32x16 s[2], dp[2];
    bf16x8 dsf[2][2];
    auto opnd = [&](int m) {   // A operand of MFMA m
      if (m < 2 * NS) {
        const int kb = m / NS, j = m % NS;
        return ld_row_swz<D>(j < KS ? sK : sV, kb * 32 + c, (j % KS) * 2 + g);
      }
      const int q = m - 2 * NS, kb = q / (2 * DB), kk = (q % (2 * DB)) / DB, db = q % DB;
      return ld_tr_swz<D>(sK, (2 * kb + kk) * 16, db * 32);   // K^T, keys (2 kb + kk) * 16..
    };
    auto expo = [&](int kb, int i) { s[kb][i] = fast_exp2(fmaf(s[kb][i], a.scale_log2, -lse2)); };
    auto dso = [&](int kb, int i) {   // dp already holds dP - D
      dp[kb][i] = s[kb][i] * dp[kb][i];
      if ((i & 7) == 7) {
        dsf[kb][i >> 3] = to_operand(dp[kb], i & 8);
        asm volatile("" : "+v"(dsf[kb][i >> 3]));   // keeps it in its slot
      }
    };
    auto mask = [&](int kb) {   // partial tiles only (block-uniform)
      if (tile_iv) {
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const int4 om = *reinterpret_cast<const int4*>(&sOm[kb * 32 + q4 * 8 + g * 4]);
          const int omv[4] = {om.x, om.y, om.z, om.w};
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int r = q4 * 4 + u;
            const int key = j0 + kb * 32 + q4 * 8 + g * 4 + u;
            s[kb][r] = mv_visible_iv(qrow, key, omv[u], a.mask.iv_ptr, a.mask.iv) ? s[kb][r] : 0.f;
          }
        }
      } else {   // per element a select, not a branch
        const int di = qrow - (j0 + g * 4);   // keys relative to the lane's first
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const int4 om = *reinterpret_cast<const int4*>(&sOm[kb * 32 + q4 * 8 + g * 4]);
          const int omv[4] = {om.x, om.y, om.z, om.w};
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int r = q4 * 4 + u;
            const int jo = kb * 32 + q4 * 8 + u;   // key j0 + g * 4 + jo
            s[kb][r] = mv_visible_rel(di, jo, qrow, omv[u]) ? s[kb][r] : 0.f;
          }
        }
      }
    };
    // vector work of slot m: elements [16 (m - b) / n, 16 (m - b + 1) / n)
    // of a stretch of n slots starting at b
    auto spread = [&](int m, int b, int n, auto&& f) {
      if (m >= b && m < b + n) {
        const int i0 = 16 * (m - b) / n, i1 = 16 * (m - b + 1) / n;
#pragma unroll
        for (int i = i0; i < i1; ++i) f(i);
      }
    };
    bf16x8 op[3];
    op[0] = opnd(0);
    op[1] = opnd(1);
    __builtin_amdgcn_sched_barrier(0);
    auto slot = [&](int m) {
      if (m + 2 < NM) op[(m + 2) % 3] = opnd(m + 2);
      if (m < 2 * NS) {
        const int kb = m / NS, j = m % NS;
        if (j < KS)
          s[kb] = mfma32(op[m % 3], qf[j], j == 0 ? f32x16{} : s[kb]);
        else
          dp[kb] = mfma32(op[m % 3], df[j - KS], j == KS ? negD : dp[kb]);
      } else {
        const int q = m - 2 * NS, kb = q / (2 * DB), kk = (q % (2 * DB)) / DB, db = q % DB;
        acc[db] = mfma32(op[m % 3], dsf[kb][kk], acc[db]);
      }
      spread(m, KS + 1, KS - 1, [&](int i) { expo(0, i); });
      spread(m, NS + 1, KS - 1, [&](int i) { dso(0, i); });
      spread(m, NS + KS + 1, KS - 1, [&](int i) { expo(1, i); });
      spread(m, 2 * NS + 1, 2 * DB - 1, [&](int i) { dso(1, i); });
      __builtin_amdgcn_sched_barrier(0);
    };
#pragma unroll
    for (int m = 0; m < NS; ++m) slot(m);
    if (!full) mask(0);
#pragma unroll
    for (int m = NS; m < 2 * NS; ++m) slot(m);
    if (!full) mask(1);
#pragma unroll
    for (int m = 2 * NS; m < NM; ++m) slot(m);
    // tile e+1 has landed (and its omega values are written) before the
    // barrier that publishes it; then tile e's buffer takes tile e+2
    wait_vmcnt<0>();
    if (e + 1 < e1) sOmbuf[(buf ^ 1) * BK + tid % BK] = omreg;
    __syncthreads();
    if (e + 2 < e1) issue_tile(sload_i32(a.mask.k_list + e + 2) >> 1, buf);
  };
  for (int e = e0; e < e1; e += 2) {
    tile(std::integral_constant<int, 0>{}, e);
    if (e + 1 < e1) tile(std::integral_constant<int, 1>{}, e + 1);
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
// 2. dK / dV
// ---------------------------------------------------------------------------
// One workgroup per (128-key tile, KV head) work item, 8 waves: on each SIMD a
// score wave (waves 0-3) and an accumulating wave (waves 4-7) share 32 keys.
// For each 32-row unit of each 64-row query block (all query heads of the
// group), the score wave computes S = Q K^T and dP = dO V^T from its keys' K
// and V fragments (kept in registers), then P and dS = P (dP - D), and hands
// both to the accumulating wave as bf16 MFMA operands through LDS (16 bytes
// per lane and operand, in the lane order both waves use); the accumulating
// wave runs dV += dO^T P and dK += Q^T dS with the transposing LDS read.
// The score wave works one unit ahead, so one wave's softmax arithmetic runs
// beside the other's MFMAs, and each wave holds only half of the state (K/V
// fragments, or the dK/dV accumulators): that is what lets two waves share a
// SIMD.  One barrier per unit.  The accumulating waves also stream the query
// blocks (Q, dO, their rows' LSE and D) from raw buffers straight into LDS,
// three buffers: the block being accumulated, the block being scored, and
// one landing.
template <int D, bool IV>
__global__ __launch_bounds__(512, 1) void bwd_dkdv_kernel(BwdArgs a) {
  constexpr int BK = kBwdTileK, BQ = kBwdBlockQ;
  constexpr int KS = D / 16, DB = D / 32;
  constexpr int NBUF = 3;
  __shared__ __align__(1024) u16 sQbuf[NBUF * BQ * D];
  __shared__ __align__(1024) u16 sdObuf[NBUF * BQ * D];
  __shared__ __align__(16) float sLbuf[NBUF * BQ];   // LSE * log2 e
  __shared__ __align__(16) float sDbuf[NBUF * BQ];
  // P and dS operands of unit u in half u & 1: [half][pair][operand][lane]
  __shared__ __align__(16) bf16x8 sXbuf[2][4][4][64];
  // block of step st in buffer st % NBUF
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
  const int pair = wave & 3;
  const bool scorer = __builtin_amdgcn_readfirstlane(wave) < 4;   // wave-uniform
  const int c = lane & 31, g = lane >> 5;
  const int j0 = kt * BK, j1 = min(T, j0 + BK);
  const int key = j0 + pair * 32 + c;
  const bool kok = key < T;
  const int om = kok ? a.mask.omega[key] : 0;
  // masks with restoring edits: only a key tile holding a key with several
  // live intervals walks the interval lists
  bool iv_tile = false;
  if constexpr (IV) iv_tile = __syncthreads_or(kok && om < 0) != 0;

  const int nqb = qb1 - qb0;
  const int steps = nqb * G;
  const int h0 = hk * G;
  const int n_units = 2 * steps;   // unit u: step u / 2, rows (u % 2) * 32 .. of its block
  // Step st covers query block qb0 + st % nqb of head h0 + st / nqb.  Rows
  // past T read row T - 1 (finite values; no key is visible to them).  Every
  // accumulating wave issues the same number of loads per step (LPS): its
  // share of Q and dO, and the block's LSE (even waves) or D (odd waves; the
  // second pair of waves writes the same words again).
  const uint32_t q_row = uint32_t(a.Hq) * D * 2;     // bytes per query row
  constexpr int LPS = 2 * KvTileLoader<D, BQ>::KLD + 1;
  static_assert(BQ == 64, "one LSE / D word per lane");

  if (!scorer) {   // ---- accumulating waves: loads of steps 0 and 1
    const KvTileLoader<D, BQ> ldr(tid - 256);
    auto issue_step = [&](int st) {
      const int buf = st % NBUF;
      const int hh = h0 + st / nqb, qb = qb0 + st % nqb;
      const uint32_t bytes = uint32_t(T) * q_row - uint32_t(hh) * D * 2;
      ldr.issue(make_rsrc(a.q + size_t(hh) * D, bytes), make_rsrc(a.dout + size_t(hh) * D, bytes),
                qb, T, q_row, lds_addr(sQbuf) + buf * BQ * D * 2,
                lds_addr(sdObuf) + buf * BQ * D * 2);
      const bool odd = pair & 1;
      const float* vec = (odd ? a.Dd : a.L2) + size_t(hh) * T;
      buf_lds4(make_rsrc(vec, uint32_t(T) * 4), uint32_t(min(qb * BQ + lane, T - 1)) * 4,
               (odd ? lds_addr(sDbuf) : lds_addr(sLbuf)) + buf * BQ * 4);
    };
    issue_step(0);
    if (steps > 1) {
      issue_step(1);
      wait_vmcnt<LPS>();
    } else {
      wait_vmcnt<0>();
    }
    __syncthreads();   // block 0 landed

    f32x16 dk[DB], dv[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        dk[db][r] = 0.f;
        dv[db][r] = 0.f;
      }
    // interval u (between the barriers that end units u - 1 and u): unit u's
    // dV/dK here, unit u + 1 in the score wave.  Before the barrier that
    // ends it, the block the score waves read next (unit u + 2) has landed:
    // only the block issued after it may still be in flight.
    auto wait_for = [&](int u) {
      const int r = (u + 2) >> 1;
      const int last = min(steps - 1, u >= 0 ? (u >> 1) + 2 : 1);   // last block issued
      if (r < steps) {
        if (last > r)
          wait_vmcnt<LPS>();
        else
          wait_vmcnt<0>();
      }
    };
    wait_for(-1);
    __syncthreads();
    // unit u = 6 i + UM: its block's buffer (u / 2) % 3 = UM / 2, its rows
    // and operand half are compile-time constants, so every LDS address is a
    // per-lane base plus an immediate offset
    auto unit = [&](auto um_tag, int u) {
      constexpr int UM = decltype(um_tag)::value;
      constexpr int mb = UM & 1, buf = UM / 2;
      const int st = u >> 1;
      // block st+2 into the buffer block st-1 used (every wave is done with it)
      if (mb == 0 && st + 2 < steps) issue_step(st + 2);
      const bf16x8* x = &sXbuf[UM & 1][pair][0][lane];
      const bf16x8 pf[2] = {x[0], x[64]}, dsf[2] = {x[128], x[192]};
      const char* sQ = qtile(buf);
      const char* sdO = dotile(buf);
      // MFMA q: dV (even q) or dK (odd q) of db = (q / 2) % DB, operand kk =
      // q / (2 DB) (db before kk, so that no two neighbouring MFMAs of one
      // kind share an accumulator); operands read two MFMAs ahead
      auto opnd = [&](int q) {
        return ld_tr_swz<D>((q & 1) ? sQ : sdO, (2 * mb + q / (2 * DB)) * 16, ((q >> 1) % DB) * 32);
      };
      constexpr int NQ = 4 * DB;
      bf16x8 op[3];
      op[0] = opnd(0);
      op[1] = opnd(1);
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        if (q + 2 < NQ) op[(q + 2) % 3] = opnd(q + 2);
        const int db = (q >> 1) % DB, kk = q / (2 * DB);
        if (q & 1)
          dk[db] = mfma32(op[q % 3], dsf[kk], dk[db]);
        else
          dv[db] = mfma32(op[q % 3], pf[kk], dv[db]);
      }
      wait_for(u);
      __syncthreads();
    };
    using std::integral_constant;
    for (int u0 = 0; u0 < n_units; u0 += 6) {
      unit(integral_constant<int, 0>{}, u0);
      unit(integral_constant<int, 1>{}, u0 + 1);   // n_units is even
      if (u0 + 2 < n_units) {
        unit(integral_constant<int, 2>{}, u0 + 2);
        unit(integral_constant<int, 3>{}, u0 + 3);
      }
      if (u0 + 4 < n_units) {
        unit(integral_constant<int, 4>{}, u0 + 4);
        unit(integral_constant<int, 5>{}, u0 + 5);
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
      float* pk = base + size_t(pair * 32 + c) * D;
      float* pv = base + size_t(BK) * D + size_t(pair * 32 + c) * D;
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
    return;
  }

  // ---- score waves
  bf16x8 kf[KS], vf[KS];
  {
    const size_t off = (size_t(kok ? key : 0) * a.Hkv + hk) * D + g * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      kf[ks] = as_bf16x8(kok ? ld16(a.k + off + ks * 16) : make_uint4(0, 0, 0, 0));
      vf[ks] = as_bf16x8(kok ? ld16(a.v + off + ks * 16) : make_uint4(0, 0, 0, 0));
    }
  }
  __syncthreads();   // block 0 landed
  // unit v = 6 i + VM (computed in the interval before the accumulating
  // wave takes it): buffer VM / 2, rows and operand half constant
  auto unit = [&](auto vm_tag, int v) {
    constexpr int VM = decltype(vm_tag)::value;
    constexpr int mb = VM & 1, buf = VM / 2;
    const int st = v >> 1;
    const char* sQ = qtile(buf);
    const char* sdO = dotile(buf);
    // S^T and dP^T of the unit: rows are this wave's keys, lanes' columns
    // the unit's queries mb*32 + q4*8 + g*4 + e; operands two MFMAs ahead
    f32x16 s, dp;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      s[r] = 0.f;
      dp[r] = 0.f;
    }
    auto opnd = [&](int j) {   // MFMA j: ks = j / 2, S (even) or dP (odd)
      return ld_row_swz<D>((j & 1) ? sdO : sQ, mb * 32 + c, (j >> 1) * 2 + g);
    };
    bf16x8 op[3];
    op[0] = opnd(0);
    op[1] = opnd(1);
#pragma unroll
    for (int j = 0; j < 2 * KS; ++j) {
      if (j + 2 < 2 * KS) op[(j + 2) % 3] = opnd(j + 2);
      if (j & 1)
        dp = mfma32(op[j % 3], vf[j >> 1], dp);
      else
        s = mfma32(op[j % 3], kf[j >> 1], s);
    }
    const float* sL = sLbuf + buf * BQ;
    const float* sD = sDbuf + buf * BQ;   // -D
    const int i0 = (qb0 + st % nqb) * BQ;
    const bool full = (i0 >= j1 - 1) && (i0 + BQ <= om_min);   // block-uniform
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      const int qo = mb * 32 + q4 * 8 + g * 4;
      const float4 l4 = *reinterpret_cast<const float4*>(&sL[qo]);
      const float4 d4 = *reinterpret_cast<const float4*>(&sD[qo]);
      const float lv[4] = {l4.x, l4.y, l4.z, l4.w};
      const float nd[4] = {d4.x, d4.y, d4.z, d4.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) s[q4 * 4 + e] = fast_exp2(fmaf(s[q4 * 4 + e], a.scale_log2, -lv[e]));
      if (!full) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int i = i0 + qo + e;
          // single-interval keys: row i sees this lane's key iff 0 <= i -
          // key < om - key
          const bool vis = (IV && iv_tile) ? mv_visible_iv(i, key, om, a.mask.iv_ptr, a.mask.iv)
                                           : uint32_t(i - key) < uint32_t(om - key);
          s[q4 * 4 + e] = vis ? s[q4 * 4 + e] : 0.f;
        }
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) dp[q4 * 4 + e] = s[q4 * 4 + e] * (dp[q4 * 4 + e] + nd[e]);
    }
    bf16x8* x = &sXbuf[VM & 1][pair][0][lane];
    x[0] = to_operand(s, 0);
    x[64] = to_operand(s, 8);
    x[128] = to_operand(dp, 0);
    x[192] = to_operand(dp, 8);
    __syncthreads();
  };
  using std::integral_constant;
  for (int v0 = 0; v0 < n_units; v0 += 6) {
    unit(integral_constant<int, 0>{}, v0);
    unit(integral_constant<int, 1>{}, v0 + 1);
    if (v0 + 2 < n_units) {
      unit(integral_constant<int, 2>{}, v0 + 2);
      unit(integral_constant<int, 3>{}, v0 + 3);
    }
    if (v0 + 4 < n_units) {
      unit(integral_constant<int, 4>{}, v0 + 4);
      unit(integral_constant<int, 5>{}, v0 + 5);
    }
  }
  __syncthreads();   // the interval of the last unit's dV/dK
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

  const dim3 b256(256);
  const int per_xcd_q = (m.n_qt + kNumXcd - 1) / kNumXcd;
  const dim3 g_dq(per_xcd_q * Hq * kNumXcd);
  const int per_xcd_kv = (a.n_items + kNumXcd - 1) / kNumXcd;
  const dim3 g_kv(per_xcd_kv * Hkv * kNumXcd);
  const int n_red = int(m.bwd_red.size());
  const dim3 g_red(unsigned(std::max(1, n_red * Hkv)));
  // the general predicate only when some key has further live intervals
  const bool iv = !m.iv.empty();
  // dQ first: it writes the rows' -D and LSE * log2 e that dK/dV reads
  auto run = [&](auto dkdv, auto red, auto dq) {
    { ProfScope p("attn_bwd_dq", stream, profile);
      hipLaunchKernelGGL(dq, g_dq, b256, 0, stream, a); }
    { ProfScope p("attn_bwd_dkdv", stream, profile);
      hipLaunchKernelGGL(dkdv, g_kv, dim3(512), 0, stream, a); }
    if (n_red) {
      ProfScope p("attn_bwd_reduce", stream, profile);
      hipLaunchKernelGGL(red, g_red, b256, 0, stream, a, n_red);
    }
  };
  if (D == 128 && iv)
    run(bwd_dkdv_kernel<128, true>, bwd_reduce_kernel<128>, bwd_dq_kernel<128, true>);
  else if (D == 128)
    run(bwd_dkdv_kernel<128, false>, bwd_reduce_kernel<128>, bwd_dq_kernel<128, false>);
  else if (iv)
    run(bwd_dkdv_kernel<64, true>, bwd_reduce_kernel<64>, bwd_dq_kernel<64, true>);
  else
    run(bwd_dkdv_kernel<64, false>, bwd_reduce_kernel<64>, bwd_dq_kernel<64, false>);
  return hipGetLastError();
}

}  // namespace mv
