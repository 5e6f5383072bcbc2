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
// operand is read with the transposing LDS read.  The next tile's loads are
// in flight during the current tile's math.  Query tiles are visited
// heaviest first and the heads of one query tile are kept on one XCD so that
// GQA heads share K/V in that XCD's L2.
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
  // Two buffers: key tile e+1 lands while tile e is read.  K and V rows are
  // unpadded and swizzled (kv_swz).
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
  float m_run = -INFINITY, l_run = 0.f;

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
  // tile lists at least its diagonal key tile.
  // (block-uniform: the tile list is read with scalar loads, which do not
  // wait behind the tile loads in flight)
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

    // S^T for keys [kb*32, kb*32+32) of the tile.  The two blocks' MFMAs
    // alternate, and the K fragments are read four MFMAs ahead (a fixed
    // order: each MFMA waits only for a read issued long before it).
    f32x16 s[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[kb][r] = 0.f;
    {
      auto kfrag = [&](int st) {   // step st: block st % 2, k step st / 2
        return ld_row_swz<D>(sK, (st & 1) * 32 + c, (st >> 1) * 2 + g);
      };
      bf16x8 kr[4];
#pragma unroll
      for (int st = 0; st < 4; ++st) kr[st] = kfrag(st);
#pragma unroll
      for (int st = 0; st < 2 * KS; ++st) {
        s[st & 1] = mfma32(kr[st & 3], qf[st >> 1], s[st & 1]);
        if (st + 4 < 2 * KS) kr[st & 3] = kfrag(st + 4);
        __builtin_amdgcn_sched_barrier(0);
      }
    }

    // scores stay raw (masked ones -inf); the running max m_run is in base-2
    // units of the scaled scores
    if (!full) {  // block-uniform; per element a select, not a branch
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const int4 om = *reinterpret_cast<const int4*>(&sOm[kb * 32 + q4 * 8 + g * 4]);
          const int omv[4] = {om.x, om.y, om.z, om.w};
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int r = q4 * 4 + u;
            const int key = j0 + kb * 32 + q4 * 8 + g * 4 + u;
            const bool vis = mv_visible_k<IV>(qrow, key, omv[u], a.mask.iv_ptr, a.mask.iv);
            s[kb][r] = vis ? s[kb][r] : -INFINITY;
          }
        }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    // Lazy rescaling: the running max moves only when a tile's max exceeds it
    // by more than 8 (base 2); until then p = exp2(x - m_run) <= 2^8, well
    // inside fp32 and the bf16 operand range, and O and l keep their scale.
    const float m_tile = mx * a.scale_log2;     // -inf for a fully masked row
    const bool grow = m_tile > m_run + 8.f;
    if (__any(grow)) {
      const float alpha = grow ? fast_exp2(m_run - m_tile) : 1.f;
      if (grow) m_run = m_tile;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[db][r] *= alpha;
    }
    const float m_use = (m_run == -INFINITY) ? 0.f : m_run;
    float psum = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = fast_exp2(fmaf(s[kb][r], a.scale_log2, -m_use));
        s[kb][r] = p;
        psum += p;
      }
    l_run += psum;

    bf16x8 pf[4];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) pf[ks] = to_operand(s[ks >> 1], (ks & 1) * 8);
    {
      // V^T operand of step st: column block st % DB, keys (st / DB)*16 ..
      // in accumulator order; read four MFMAs ahead as above
      auto vfrag = [&](int st) { return ld_tr_swz<D>(sV, (st / DB) * 16, (st % DB) * 32); };
      bf16x8 vr[4];
#pragma unroll
      for (int st = 0; st < 4; ++st) vr[st] = vfrag(st);
#pragma unroll
      for (int st = 0; st < 4 * DB; ++st) {
        oacc[st % DB] = mfma32(vr[st & 3], pf[st / DB], oacc[st % DB]);
        if (st + 4 < 4 * DB) vr[st & 3] = vfrag(st + 4);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    // tile e+1 has landed (and its omega values are written) before the
    // barrier that publishes it; then tile e's buffer takes tile e+2
    wait_vmcnt<0>();
    if (e + 1 < e1) sOmbuf[(buf ^ 1) * BK + tid % BK] = omreg;
    __syncthreads();
    if (e + 2 < e1) issue_tile(sload_i32(a.mask.k_list + e + 2) >> 1, buf);
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
