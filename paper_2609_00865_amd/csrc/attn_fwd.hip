// View-masked attention forward on gfx950.
//
// One workgroup = one 128-row query tile x one query head, 4 waves of 32 rows.
// For each 64-key tile the schedule lists (Section 4.2's mask, block-sparse as
// Appendix B.3 asks for), the block computes S^T = K Q^T with bf16 MFMA (keys
// on the accumulator rows, one query per lane, so the softmax statistics of a
// row stay inside a lane pair), applies the shared visibility predicate on
// partial tiles only, updates the online softmax in base 2, and accumulates
// O^T += V^T P^T with a second MFMA.  K and V go from buffer loads straight
// into LDS as unpadded rows with permuted 16-byte chunks (kv_swz); the V^T
// operand is read with the transposing LDS read.
//
// Each wave runs a two-stage software pipeline over the tile list: while the
// score MFMAs of tile t+1 run, the vector ALU turns the second half of tile
// t's scores into probabilities; while the PV MFMAs of tile t run, it turns
// the first half of tile t+1's.  Tiles take no row maxima: probabilities are
// taken against a score the row has already seen, and only a tile whose
// probabilities would grow past 2^16 takes its exact maximum and rescales
// (a slow path).  K and V have double buffers and one barrier per
// step: after it, tile t+2's K and tile t+1's V go into the buffers the
// previous step finished with, so each load has one step to land.  Query tiles are visited heaviest first and the heads of one query
// tile are kept on one XCD so that GQA heads share K/V in that XCD's L2.
#include <type_traits>

#include "mv_device.h"
#include "mv_predicate.h"

namespace mv {

struct FwdArgs {
  const u16* q;
  const u16* k;
  const u16* v;
  u16* o;
  float* lse;
  mv_mask_dev mask;
  int T, Hq, Hkv, n_qt;
  float scale_log2;
};

template <int D, bool IV>
__global__ __launch_bounds__(256, 2) void attn_fwd_kernel(FwdArgs a) {
  constexpr int BQ = kFwdTileQ, BK = kFwdTileK;
  constexpr int KS = D / 16;          // MFMA k-steps over the head dimension
  constexpr int DB = D / 32;          // 32-row blocks of O^T
  constexpr int NL = KvTileLoader<D, BK>::KLD;   // 16-byte loads per thread per K or V tile
  constexpr int NLK = NL + 1;                    // a K tile also brings its keys' omega
  static_assert(BK == 64, "one omega word per lane");
  static_assert(2 * KS == 16 || 2 * KS == 8, "score MFMAs per tile");
  // K and V each in two buffers (tile t in buffer t & 1); omega in four
  // (tile t in t & 3).  Rows are unpadded and swizzled (kv_swz).
  __shared__ __align__(1024) u16 sKbuf[2 * BK * D];
  __shared__ __align__(1024) u16 sVbuf[2 * BK * D];
  __shared__ __align__(16) int sOmbuf[4 * BK];

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

  // Q^T as the B operand: lane holds query qrow, d = ks*16 + g*8 .. +8
  bf16x8 qf[KS];
  {
    const u16* qp = a.q + (size_t(qok ? qrow : 0) * a.Hq + h) * D + g * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qf[ks] = as_bf16x8(qok ? ld16(qp + ks * 16) : make_uint4(0, 0, 0, 0));
  }

  f32x16 oacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[db][r] = 0.f;
  // running max (base-2 units of the scaled scores), the max the current
  // tile's probabilities use, and this lane's share of the row sum
  float m_run = -INFINITY, l_run = 0.f;

  // K and V of KV head hk go from raw buffers straight into LDS.  Keys past
  // T read row T - 1 (their omega reads as 0 through the range-checked
  // buffer, so no row sees them).
  const uint32_t kv_row = uint32_t(a.Hkv) * D * 2;   // bytes per key row
  const uint32_t kv_bytes = uint32_t(T) * kv_row - uint32_t(hk) * D * 2;
  const rsrc_t krs = make_rsrc(a.k + size_t(hk) * D, kv_bytes);
  const rsrc_t vrs = make_rsrc(a.v + size_t(hk) * D, kv_bytes);
  const rsrc_t omrs = make_rsrc(a.mask.omega, uint32_t(T) * 4);
  const KvTileLoader<D, BK> ldr(tid);
  // (block-uniform: the tile list is read with scalar loads, where no LDS
  // read is outstanding: such a load waits on lgkmcnt, which counts both)
  const int e0 = __builtin_amdgcn_readfirstlane(a.mask.q_ptr[qt]);
  const int n = __builtin_amdgcn_readfirstlane(a.mask.q_ptr[qt + 1]) - e0;   // >= 1
  const int* klist = a.mask.k_list + e0;
  // The list entry of tile t (key tile << 1 | full) is read once, with a
  // scalar load right after a barrier (no LDS read outstanding then), and
  // passed to the loads and the mask of that tile.
  auto issue_k = [&](int t, int ent) {   // K tile t and its omega values (NLK loads)
    const int kt = ent >> 1;
    ldr.issue_one(krs, kt, T, kv_row, lds_addr(sKbuf) + uint32_t(t & 1) * BK * D * 2);
    buf_lds4(omrs, uint32_t(kt * BK + lane) * 4, lds_addr(sOmbuf) + uint32_t(t & 3) * BK * 4);
  };
  auto issue_v = [&](int t, int ent) {   // V tile t (NL loads)
    const int kt = ent >> 1;
    ldr.issue_one(vrs, kt, T, kv_row, lds_addr(sVbuf) + uint32_t(t & 1) * BK * D * 2);
  };
  auto ktile = [&](int t) { return reinterpret_cast<const char*>(sKbuf + (t & 1) * BK * D); };
  auto vtile = [&](int t) { return reinterpret_cast<const char*>(sVbuf + (t & 1) * BK * D); };

  // Score sets: tile t's in sc[t & 1] (keys kb*32 + accumulator row).
  f32x16 sc[2][2];

  // S^T of tile t into set P, as MFMA j of 2 KS (block j % 2, k step j / 2)
  // with the K fragments read four MFMAs ahead.
  auto kfrag = [&](const char* sK, int j) {
    return ld_row_swz<D>(sK, (j & 1) * 32 + c, (j >> 1) * 2 + g);
  };
  // Mask of tile t's scores in set s (partial tiles only): invisible scores
  // become -inf.
  auto mask_tile = [&](f32x16 (&s)[2], int t, int ent) {
    if (!(ent & 1)) {   // block-uniform; per element a select, not a branch
      const int j0 = (ent >> 1) * BK;
      const int* sOm = sOmbuf + (t & 3) * BK;
      // a tile holding a key with several live intervals (only masks with
      // restoring edits have them) takes the out-of-line interval walk
      if (IV && __any(sOm[lane] < 0)) {
        const uint32_t vis = mv_visible_iv_bits(qrow, j0, g, sOm, a.mask.iv_ptr, a.mask.iv);
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) s[kb][r] = (vis >> (kb * 16 + r)) & 1u ? s[kb][r] : -INFINITY;
      } else {
        const int di = qrow - (j0 + g * 4);   // keys relative to the lane's first
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int q4 = 0; q4 < 4; ++q4) {
            const int4 om = *reinterpret_cast<const int4*>(&sOm[kb * 32 + q4 * 8 + g * 4]);
            const int omv[4] = {om.x, om.y, om.z, om.w};
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const int r = q4 * 4 + u;
              const int jo = kb * 32 + q4 * 8 + u;   // key j0 + g * 4 + jo
              s[kb][r] = mv_visible_rel(di, jo, qrow, omv[u]) ? s[kb][r] : -INFINITY;
            }
          }
      }
    }
  };
  // element i (0..31) of a tile: block i / 16, accumulator row i % 16
  auto tile_max = [&](const f32x16 (&s)[2]) {
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][r]);
    return max_halves(mx) * a.scale_log2;
  };
  // Probabilities are p = exp2(s * scale_log2 - m_run), where m_run is the
  // exact maximum of a tile this row has already scored (-inf until the row
  // has seen a key: then the offset is 0).  Tiles do not take their row
  // maxima: a tile whose probabilities reach 2^16 in some lane (its lane sum
  // of p exceeds that), or that a row meets with no key seen yet, takes the
  // slow path below.  So every p stays <= 2^16, far inside fp32 and the bf16
  // operand range, and the offset cancels in O = sum p v / sum p.
  auto m_off = [&]() { return m_run == -INFINITY ? 0.f : m_run; };
  auto pexp = [&](const f32x16 (&s)[2], int i, float mu) {
    return fast_exp2(fmaf(s[i >> 4][i & 15], a.scale_log2, -mu));
  };
  // eight probabilities as one bf16 MFMA operand
  auto pack8 = [](const float* p) {
    uint4 w;
    w.x = pack2(p[0], p[1]);
    w.y = pack2(p[2], p[3]);
    w.z = pack2(p[4], p[5]);
    w.w = pack2(p[6], p[7]);
    return as_bf16x8(w);
  };
  // Slow path for the tile with scores s: its exact maximum; if that is above
  // the row's offset, O and l are rescaled to it; then the tile's 32
  // probabilities are recomputed from the scores (kept unchanged until the
  // tile's PV products are issued) into the four operands and the lane sum.
  auto slow_tile = [&](const f32x16 (&s)[2], bf16x8 (&pf)[4], float& psum) {
    const float m_tile = tile_max(s);
    if (m_tile > m_run) {
      const float alpha = fast_exp2(m_run - m_tile);   // 0 when m_run is -inf
      m_run = m_tile;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[db][r] *= alpha;
    }
    const float mu = m_off();
    psum = 0.f;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      float p[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        p[u] = pexp(s, 8 * k + u, mu);
        psum += p[u];
      }
      pf[k] = pack8(p);
    }
  };

  // ---- prologue: K0, K1, V0 (the issue order the first wait assumes)
  const int ent0 = sload_i32(klist);
  int ent1 = n > 1 ? sload_i32(klist + 1) : 0;   // entry of the next tile
  issue_k(0, ent0);
  if (n > 1) issue_k(1, ent1);
  issue_v(0, ent0);
  if (n > 1)
    wait_vmcnt<NLK + NL>();
  else
    wait_vmcnt<NL>();
  __syncthreads();
  {
    const char* sK = ktile(0);
#pragma unroll
    for (int j = 0; j < 2 * KS; ++j)
      sc[0][j & 1] = mfma32(kfrag(sK, j), qf[j >> 1], j < 2 ? f32x16{} : sc[0][j & 1]);
  }
  mask_tile(sc[0], 0, ent0);
  m_run = tile_max(sc[0]);
  // operands of a tile, elements 8k .. 8k+7 in pf[k]; elements 0..15 of the
  // next tile are computed during the current tile's PV products, with their
  // lane sum in psum_a
  bf16x8 pf[4];
  float psum_a = 0.f;
  {
    const float mu = m_off();
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      float p[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        p[u] = pexp(sc[0], 8 * k + u, mu);
        psum_a += p[u];
      }
      pf[k] = pack8(p);
    }
  }

  // ---- one pipeline step: tile t (scores in set P, operands 0 and 1 of its
  // probabilities already in pf) and tile t+1 (scores into set P ^ 1).  On
  // the last tile (no t+1) the score MFMAs still run, on stale LDS, and their
  // results and probabilities are dropped: the interleaved phases stay free
  // of branches.
  auto step = [&](auto par_tag, int t) {
    constexpr int P = decltype(par_tag)::value;
    f32x16 (&cur)[2] = sc[P];
    f32x16 (&nxt)[2] = sc[P ^ 1];
    const bool next = t + 1 < n;   // block-uniform

    // one barrier per step: K[t+1] and V[t] landed, every wave done with
    // K[t] and V[t-1]; then K[t+2] and V[t+1] go into their buffers
    wait_vmcnt<0>();
    __syncthreads();
    const int ent2 = t + 2 < n ? sload_i32(klist + t + 2) : 0;
    if (t + 2 < n) issue_k(t + 2, ent2);
    if (next) issue_v(t + 1, ent1);

    // phase 1: S^T of tile t+1 (2 KS MFMAs) with tile t's elements 16..31
    // (spread evenly over the MFMA slots) and their bf16 operands
    const float mu = m_off();
    float psum = psum_a;
    {
      const char* sK = ktile(t + 1);
      bf16x8 kr[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) kr[j] = kfrag(sK, j);
      float p[16];
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int j = 0; j < 2 * KS; ++j) {
        nxt[j & 1] = mfma32(kr[j & 3], qf[j >> 1], j < 2 ? f32x16{} : nxt[j & 1]);
        if (j + 4 < 2 * KS) kr[j & 3] = kfrag(sK, j + 4);
        constexpr int NS = 2 * KS;
        const int i0 = 16 * j / NS, i1 = 16 * (j + 1) / NS;
#pragma unroll
        for (int i = i0; i < i1; ++i) {
          p[i] = pexp(cur, 16 + i, mu);
          psum += p[i];
        }
        if (i1 / 8 != i0 / 8) {   // operand 2 + k (elements 16 + 8k ..) complete
          const int k = i1 / 8 - 1;
          pf[2 + k] = pack8(p + 8 * k);
          // an empty asm that consumes the operand keeps its computation in
          // this phase (the compiler would otherwise sink it past the
          // barrier, next to the MFMAs that read it)
          asm volatile("" : "+v"(pf[2 + k]));
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    // rows past T never see a key and never ask for the slow path
    if (__any(!(psum <= 65536.f) || (qok && m_run == -INFINITY))) slow_tile(cur, pf, psum);
    l_run += psum;

    if (next) mask_tile(nxt, t + 1, ent1);
    ent1 = ent2;

    // phase 2: O^T += V^T P^T of tile t (4 DB MFMAs, V^T read four ahead)
    // with tile t+1's elements 0..15; operand k of tile t+1 replaces tile
    // t's operand k once the MFMAs that read the latter are issued
    {
      const float mu1 = m_off();
      const char* sV = vtile(t);
      auto vfrag = [&](int st) { return ld_tr_swz<D>(sV, (st / DB) * 16, (st % DB) * 32); };
      bf16x8 vr[4];
#pragma unroll
      for (int st = 0; st < 4; ++st) vr[st] = vfrag(st);
      float p[16];
      psum_a = 0.f;
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int st = 0; st < 4 * DB; ++st) {
        oacc[st % DB] = mfma32(vr[st & 3], pf[st / DB], oacc[st % DB]);
        if (st + 4 < 4 * DB) vr[st & 3] = vfrag(st + 4);
        constexpr int NS = 4 * DB;
        const int i0 = 16 * st / NS, i1 = 16 * (st + 1) / NS;
#pragma unroll
        for (int i = i0; i < i1; ++i) {
          p[i] = pexp(nxt, i, mu1);
          psum_a += p[i];
        }
        // operand k of tile t+1 (elements 8k ..) once complete and once the
        // MFMAs reading tile t's operand k (slots DB k .. DB k + DB - 1) are out
        if (i1 / 8 != i0 / 8) {
          const int k = i1 / 8 - 1;
          pf[k] = pack8(p + 8 * k);
          asm volatile("" : "+v"(pf[k]));
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      asm volatile("" : "+v"(psum_a));
    }
  };

  using p0 = std::integral_constant<int, 0>;
  using p1 = std::integral_constant<int, 1>;
  for (int t = 0; t < n; t += 2) {
    step(p0{}, t);
    if (t + 1 < n) step(p1{}, t + 1);
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (!qok) return;
  const float inv = 1.f / l_tot;
  u16* op = a.o + (size_t(qrow) * a.Hq + h) * D;
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      const int d0 = db * 32 + q4 * 8 + g * 4;
      uint2 w;
      w.x = pack2(oacc[db][q4 * 4 + 0] * inv, oacc[db][q4 * 4 + 1] * inv);
      w.y = pack2(oacc[db][q4 * 4 + 2] * inv, oacc[db][q4 * 4 + 3] * inv);
      *reinterpret_cast<uint2*>(op + d0) = w;
    }
  if (g == 0) a.lse[size_t(h) * T + qrow] = (m_run + __log2f(l_tot)) * 0.69314718055994531f;
}

hipError_t launch_attn_fwd(const mv_view_mask& m, int Hq, int Hkv, int D, float scale,
                           const void* q, const void* k, const void* v, void* o, float* lse,
                           hipStream_t stream) {
  FwdArgs a;
  a.q = static_cast<const u16*>(q);
  a.k = static_cast<const u16*>(k);
  a.v = static_cast<const u16*>(v);
  a.o = static_cast<u16*>(o);
  a.lse = lse;
  a.mask = m.d;
  a.T = m.T;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.n_qt = m.n_qt;
  a.scale_log2 = scale * 1.4426950408889634f;
  const int per_xcd = (m.n_qt + kNumXcd - 1) / kNumXcd;
  const dim3 grid(per_xcd * Hq * kNumXcd), block(256);
  ProfScope prof("attn_fwd", stream);
  // the general predicate only when some key has further live intervals
  const bool iv = !m.iv.empty();
  if (D == 128 && iv)
    hipLaunchKernelGGL((attn_fwd_kernel<128, true>), grid, block, 0, stream, a);
  else if (D == 128)
    hipLaunchKernelGGL((attn_fwd_kernel<128, false>), grid, block, 0, stream, a);
  else if (iv)
    hipLaunchKernelGGL((attn_fwd_kernel<64, true>), grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL((attn_fwd_kernel<64, false>), grid, block, 0, stream, a);
  return hipGetLastError();
}

}  // namespace mv
