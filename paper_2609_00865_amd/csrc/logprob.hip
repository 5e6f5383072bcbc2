// Fused LM-head token log-prob, ratio and clip on gfx950.
//
// Forward: z = W h is produced 256 vocab rows x 256 tokens at a time by a bf16
// MFMA tile engine and reduced in registers to a per-token (max, sum of exp)
// over each wave's 128 vocab rows; the full logits are never stored.  A
// combine pass (one wave per token) takes the target logit z_{t,y_t} as an
// fp32 dot product, merges the partials into logsumexp and writes logp,
// ratio and the clipped ratio (the GRPO ratio of Appendix C, "Pitfall A, RL
// view"); its fused variant also evaluates the GRPO loss of each token and
// its gradient, and reduces the drift statistics (Eq. "logdiff") in the same
// pass.
//
// Backward: the logits tile is recomputed and turned into
// G_tv = g_t (onehot(y_t)_v - softmax(z_t)_v), stored once in bf16 (the tile
// writes -g_t softmax(z_t)_v everywhere, the per-token pass then rewrites the
// target entry), and a second pass of the same engine computes dH = G W from
// a transposed copy of W, so that both operands run along the vocabulary.
// dW = G^T H contracts over tokens, along which neither operand is
// contiguous: it has an engine of its own that stages both operands k-major
// and reads them with the transposing LDS read.
//
// Tile engine (logits, G, the KL passes, dH): 512 threads = 8 waves (two per
// SIMD) in a 2 x 4 grid over a 256 A-row x 256 token tile; each wave owns 128
// A rows x 64 tokens and runs MFMA 16x16x32.  64-wide k slices go from HBM
// straight into LDS (global_load_lds: no register staging and no LDS store
// instructions), two slices in flight, one barrier per slice; the next k
// step's operand fragments are read while the current step's MFMAs run.  An
// operand slice sits in LDS as [256 rows][64] bf16 without padding, with
// 16-byte chunk c of row r at chunk position c ^ (r & 7): the fragment reads
// (16 lanes = 16 consecutive rows at one chunk) hit distinct banks.  Tiles are
// ordered so that the blocks resident on one XCD at a time form a compact 2-D
// patch (a few token tiles x several A tiles) and share operand slices in that
// XCD's L2.
#include <algorithm>

#include "mv_grpo_dev.h"

namespace mv {

namespace {
constexpr int BA = 256, BT = 256, BKK = 64;
constexpr int NWAVES = 8;                  // waves per tile (2 x 4 grid)
// token tiles per raster group: 8 x 4 A tiles run side by side on an XCD
// for the products over the hidden dimension (measured ~1% faster than
// 4 x 8), 4 x 8 for dH and dW
constexpr int GROUP_T_H = 8, GROUP_T_V = 4;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.69314718055994531f;
// tile engine
constexpr int SLICE_B = 256 * BKK * 2;             // bytes of one operand's k slice
constexpr int NLD = SLICE_B / 1024 / NWAVES;       // direct loads per operand, thread and slice

// Panel layout of a bf16 matrix [R][K] (R padded to a multiple of 256, K a
// multiple of 64), used for G and W^T, the operands of the dH product whose
// k runs along the vocabulary: the 64-wide k slice of a 256-row block is one
// contiguous 32 KiB panel of 128-byte rows, so each slice load of a tile is
// one linear read instead of 256 rows a vocabulary row (~300 KB) apart.
constexpr int PANEL = 256 * 64;
__host__ __device__ inline size_t panel_index(int r, int k, int K) {
  return (size_t(r >> 8) * (K >> 6) + (k >> 6)) * PANEL + (r & 255) * 64 + (k & 63);
}
constexpr int FA = 8, FB = 4;                      // 16-row MFMA blocks per wave: A rows, tokens
static_assert(NLD * NWAVES * 1024 == SLICE_B, "slice split over the waves");
size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
int vocab_pad(int V) { return (V + BA - 1) / BA * BA; }
}  // namespace

enum { kModeLogits = 0, kModeGrad = 1, kModeDh = 2, kModeKL = 3, kModeKLGrad = 4 };

hipError_t launch_grpo_fused_finish(const float* part, int n_blocks, int stride, int n_traj,
                                    const float* adv, float* stats, hipStream_t stream);

struct LmArgs {
  const u16* h;       // [T, H]
  const u16* w;       // [V, H]
  const u16* wT;      // [H, Vp] (dH mode: W transposed, zero past V)
  const int32_t* tgt; // [T]
  const float* lse;   // [T] (grad mode)
  const float* g;     // [T] upstream dlogp (grad mode)
  const u16* G;       // [T, Vp] (dH and dW modes)
  u16* Gout;          // [T, Vp] (grad modes)
  u16* dh;            // [T, H] (dH mode)
  float2* part;       // [T, n_chunks] (logits mode)
  // KL modes: token row 2i is leaf i's teacher row, 2i + 1 its student row
  const u16* zero_row; // [H] zeros: the row read for an out-of-range leaf row index
  const u16* hT;      // teacher hidden states [*, H]
  const u16* hS;      // student hidden states [*, H]
  const int32_t* rowsT;
  const int32_t* rowsS;
  float4* partT;      // [n, n_chunks] (max, sum, cross, -) of the teacher
  float2* partS;      // [n, n_chunks] (max, sum) of the student
  const float* lseT;  // [n] (KL grad mode)
  const float* lseS;
  const float* dkl;   // [n] upstream gradient of each leaf's KL
  int n_leaves, n_rows_T, n_rows_S;
  int T, H, V, Vp, n_chunks;
  int Tg;              // rows of G: T rounded up to a multiple of 256 (zero past T)
  int nA, nT;         // tiles along the A side and along tokens
  // dH mode split over the vocabulary (K) when there are too few output
  // tiles to fill the chip: split s covers k slices [s*nk_split, ...) and
  // writes fp32 partials dh_part[s][t][H], summed in order by dh_reduce_kernel
  int k_split, nk_split;
  float* dh_part;
  float* dw;          // [V, H] fp32 (dW)
  int* bad_targets;   // count of target ids outside [-1, V) met by this call
};

// Output tile (a0, t0) and k split of this block.  Blocks are dealt to XCDs
// round-robin; each XCD gets a contiguous range of the rasterised tile order
// (groups of GT token tiles x all A tiles).  False: no tile (grid tail).
template <int GT>
__device__ __forceinline__ bool tile_of(const LmArgs& a, int n_splits, int& a0, int& t0,
                                        int& split) {
  const int n_out = a.nA * a.nT;
  const int n_tiles = n_out * n_splits;
  const int per_xcd = (n_tiles + kNumXcd - 1) / kNumXcd;
  int xcd, local;
  xcd_split(xcd, local);
  const int Lx = xcd * per_xcd + local;
  if (local >= per_xcd || Lx >= n_tiles) return false;
  split = Lx / n_out;
  const int L = Lx % n_out;
  const int grp = L / (GT * a.nA);
  const int rem = L % (GT * a.nA);
  const int t_in = min(GT, a.nT - grp * GT);
  a0 = (rem / t_in) * BA;
  t0 = (grp * GT + rem % t_in) * BT;
  return true;
}

template <int MODE>
__global__ __launch_bounds__(NWAVES * 64, 1) void lm_tile_kernel(LmArgs a) {
  __shared__ __align__(1024) u16 smem[2 * 2 * SLICE_B / 2];   // 2 slices x 2 operands

  int a0, t0, split;
  constexpr int GT = MODE == kModeDh ? GROUP_T_V : GROUP_T_H;
  if (!tile_of<GT>(a, MODE == kModeDh ? a.k_split : 1, a0, t0, split)) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wa = wave >> 2, wt = wave & 3;

  // A [a_rows][K] and B [T][K], both contiguous along k
  const int K = (MODE == kModeDh) ? a.Vp : a.H;
  const int a_rows = (MODE == kModeDh) ? a.H : a.V;
  const u16* A = (MODE == kModeDh) ? a.wT : a.w;
  const int kbeg = (MODE == kModeDh) ? split * a.nk_split : 0;
  const int nk = (MODE == kModeDh) ? min(K / BKK - kbeg, a.nk_split) : K / BKK;

  // Load i of this wave fills 16-byte slots (i * NWAVES + wave) * 64 + lane of
  // each operand's slice: row s / 8, k chunk (s % 8) ^ (row & 7).  Rows past
  // the operands are read from clamped (valid) rows; their products land in
  // output rows or columns that the epilogues skip.  The dH product reads
  // both operands (W^T and G) in the panel layout, the others row-major.
  constexpr bool PANELS = MODE == kModeDh;
  constexpr int SSTEP = PANELS ? PANEL : BKK;   // elements from one k slice of a row to the next
  const u16* srcA[NLD];
  const u16* srcB[NLD];
#pragma unroll
  for (int i = 0; i < NLD; ++i) {
    const int s = (i * NWAVES + wave) * 64 + lane;
    const int row = s >> 3, kc = (s & 7) ^ (row & 7);
    const int ar = min(a0 + row, a_rows - 1);
    const int t = min(t0 + row, a.T - 1);
    if (PANELS) {
      srcA[i] = A + panel_index(ar, kbeg * BKK, K) + kc * 8;
      srcB[i] = a.G + panel_index(t, kbeg * BKK, K) + kc * 8;
      continue;
    }
    const size_t koff = size_t(kbeg) * BKK + kc * 8;
    srcA[i] = A + size_t(ar) * K + koff;
    const u16* brow;
    if (MODE == kModeKL || MODE == kModeKLGrad) {
      // a row index outside its matrix reads as a zero hidden state
      const int r = (t & 1) ? a.rowsS[t >> 1] : a.rowsT[t >> 1];
      const int n_rows = (t & 1) ? a.n_rows_S : a.n_rows_T;
      brow = (r >= 0 && r < n_rows) ? ((t & 1) ? a.hS : a.hT) + size_t(r) * a.H : a.zero_row;
    } else {
      brow = a.h + size_t(t) * a.H;
    }
    srcB[i] = brow + koff;
  }
  typedef __attribute__((address_space(3))) u16 lds_u16;
  const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_u16*)smem;   // LDS byte address
  auto issue = [&](int kk) {
    const uint32_t st = lds0 + (kk & 1) * (2 * SLICE_B) + wave * 1024;
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      lds_load16(srcA[i] + size_t(kk) * SSTEP, st + i * NWAVES * 1024);
      lds_load16(srcB[i] + size_t(kk) * SSTEP, st + SLICE_B + i * NWAVES * 1024);
    }
  };

  const char* lds = reinterpret_cast<const char*>(smem);
  const int frow = lane & 15, fk = lane >> 4;
  bf16x8 fa[2][FA], fb[2][FB];
  // operand fragments of k step ks (0 or 1) of slice kk into register set buf
  auto read_frags = [&](int buf, int kk, int ks) {
    const char* sA = lds + (kk & 1) * (2 * SLICE_B);
    const char* sB = sA + SLICE_B;
    const int kc = ks * 4 + fk;
#pragma unroll
    for (int i = 0; i < FA; ++i) {
      const int row = wa * 128 + i * 16 + frow;
      fa[buf][i] = as_bf16x8(ld16(sA + (row * 8 + (kc ^ (row & 7))) * 16));
    }
#pragma unroll
    for (int j = 0; j < FB; ++j) {
      const int row = wt * 64 + j * 16 + frow;
      fb[buf][j] = as_bf16x8(ld16(sB + (row * 8 + (kc ^ (row & 7))) * 16));
    }
  };

  f32x4 acc[FA][FB];
#pragma unroll
  for (int i = 0; i < FA; ++i)
#pragma unroll
    for (int j = 0; j < FB; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto mma = [&](int buf) {
#pragma unroll
    for (int i = 0; i < FA; ++i)
#pragma unroll
      for (int j = 0; j < FB; ++j) acc[i][j] = mfma16(fa[buf][i], fb[buf][j], acc[i][j]);
  };

  issue(0);
  if (nk > 1) {
    issue(1);
    wait_vmcnt<2 * NLD>();   // slice 0 landed, slice 1 may still be in flight
  } else {
    wait_vmcnt<0>();
  }
  __syncthreads();
  read_frags(0, 0, 0);
  // (the last slice is peeled: a loop body without a path around the barrier
  // lets the second MFMA group start without waiting for the reads behind it)
  for (int kk = 0; kk + 1 < nk; ++kk) {
    read_frags(1, kk, 1);
    mma(0);
    // slice kk + 1 is the only one in flight; after the barrier it is visible
    // to every wave and every wave has read all of slice kk, whose buffer
    // then takes slice kk + 2
    wait_vmcnt<0>();
    __syncthreads();
    if (kk + 2 < nk) issue(kk + 2);
    read_frags(0, kk + 1, 0);
    mma(1);
  }
  read_frags(1, nk - 1, 1);
  mma(0);
  mma(1);

  // acc[i][j][r]: A row rb + i*16 + r, token tb + j*16
  const int rb = a0 + wa * 128 + (lane >> 4) * 4;
  const int tb = t0 + wt * 64 + (lane & 15);
  const bool full_v = a0 + BA <= a.V;  // block-uniform: no vocabulary padding in this tile
  const int chunk = (a0 + wa * 128) / 128;
  if (MODE == kModeLogits) {
#pragma unroll
    for (int j = 0; j < FB; ++j) {
      const int t = tb + j * 16;
      float mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < FA; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          if (!full_v && rb + i * 16 + r >= a.V) acc[i][j][r] = -INFINITY;
          mx = fmaxf(mx, acc[i][j][r]);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m2 = mx * kLog2e;                // -inf for a chunk of padding only
      const float mu = mx == -INFINITY ? 0.f : m2;
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < FA; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) s += fast_exp2(fmaf(acc[i][j][r], kLog2e, -mu));
      s += __shfl_xor(s, 16);
      s += __shfl_xor(s, 32);
      if (lane < 16 && t < a.T) a.part[size_t(t) * a.n_chunks + chunk] = make_float2(m2, s);
    }
  } else if (MODE == kModeGrad) {
    // -g_t softmax(z_t)_v everywhere (zero in the vocabulary padding; rows
    // T .. Tg - 1, which pad the dW product's k, are zeros too); the target
    // entry gets its one-hot term from lm_target_kernel afterwards.  The
    // tile's block of G is one contiguous 128 KiB run of four panels: it is
    // assembled in LDS in that order (the 16-byte chunks of each 128-byte
    // row permuted by the row's low bits, against bank conflicts) and written
    // with 16-byte stores that cover whole lines.
    char* sg = reinterpret_cast<char*>(smem);
    __syncthreads();   // every wave has read its last operand fragments
#pragma unroll
    for (int j = 0; j < FB; ++j) {
      const int t = tb + j * 16;
      const int tl = t - t0;                       // row within the tile's panels
      const int tc = min(t, a.T - 1);
      const int y = a.tgt[tc];
      // an id outside [0, V) carries no loss (-1 by convention; any other is
      // counted by lm_target_kernel)
      const float ng = (uint32_t(y) < uint32_t(a.V) && t < a.T) ? -a.g[tc] : 0.f;
      const float l2 = a.lse[tc] * kLog2e;
#pragma unroll
      for (int i = 0; i < FA; ++i) {
        const int vl = rb + i * 16 - a0;             // 4 consecutive entries vl ..
        float vals[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          vals[r] = ng * fast_exp2(fmaf(acc[i][j][r], kLog2e, -l2));
          if (!full_v && rb + i * 16 + r >= a.V) vals[r] = 0.f;
        }
        uint2 wv;
        wv.x = pack2(vals[0], vals[1]);
        wv.y = pack2(vals[2], vals[3]);
        const int c = vl & 63;
        *reinterpret_cast<uint2*>(sg + (vl >> 6) * 32768 + tl * 128 +
                                  ((((c >> 3) ^ (tl & 7)) << 4) | ((c & 7) * 2))) = wv;
      }
    }
    __syncthreads();
    uint4* gt = reinterpret_cast<uint4*>(a.Gout + panel_index(t0, a0, a.Vp));
#pragma unroll 4
    for (int k = tid; k < 128 * 1024 / 16; k += NWAVES * 64) {
      const int q = k >> 11, r = (k >> 3) & 255, c16 = k & 7;
      gt[k] = *reinterpret_cast<const uint4*>(sg + (q << 15) + (r << 7) + ((c16 ^ (r & 7)) << 4));
    }
  } else if (MODE == kModeKL) {
    // lanes c (even, teacher) and c ^ 1 (student) hold the same vocabulary
    // rows of one leaf; each lane keeps its own (max, sum of exp) and the
    // teacher also accumulates sum exp(zT - mT) * (zT - zS)
#pragma unroll
    for (int j = 0; j < FB; ++j) {
      const int t = tb + j * 16;
      const int leaf = t >> 1;
      float mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < FA; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (full_v || rb + i * 16 + r < a.V) mx = fmaxf(mx, acc[i][j][r]);
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m2 = mx * kLog2e;
      const float mu = mx == -INFINITY ? 0.f : m2;
      float sm = 0.f, cross = 0.f;
#pragma unroll
      for (int i = 0; i < FA; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float z = acc[i][j][r];
          const float zo = __shfl_xor(z, 1);  // the partner row's logit
          const bool ok = full_v || rb + i * 16 + r < a.V;
          const float e = ok ? fast_exp2(fmaf(z, kLog2e, -mu)) : 0.f;
          sm += e;
          cross += e * (z - zo);
        }
      sm += __shfl_xor(sm, 16);
      sm += __shfl_xor(sm, 32);
      cross += __shfl_xor(cross, 16);
      cross += __shfl_xor(cross, 32);
      if (lane < 16 && leaf < a.n_leaves) {
        const size_t o = size_t(leaf) * a.n_chunks + chunk;
        if (t & 1)
          a.partS[o] = make_float2(m2, sm);
        else
          a.partT[o] = make_float4(m2, sm, cross, 0.f);
      }
    }
  } else if (MODE == kModeKLGrad) {
    // student lanes write G = dkl * (q - p) for their leaf
#pragma unroll
    for (int j = 0; j < FB; ++j) {
      const int t = tb + j * 16;
      const int leaf = t >> 1;
      const bool student = (t & 1) && leaf < a.n_leaves;
      const int lc = leaf < a.n_leaves ? leaf : 0;
      const float gl = a.dkl[lc];
      const float lS = a.lseS[lc] * kLog2e, lT = a.lseT[lc] * kLog2e;
#pragma unroll
      for (int i = 0; i < FA; ++i) {
        u16* out = a.Gout + panel_index(lc, rb + i * 16, a.Vp);
        float vals[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float zS = acc[i][j][r];
          const float zT = __shfl_xor(zS, 1);
          const float q = fast_exp2(fmaf(zS, kLog2e, -lS));
          const float pt = fast_exp2(fmaf(zT, kLog2e, -lT));
          vals[r] = (full_v || rb + i * 16 + r < a.V) ? gl * (q - pt) : 0.f;
        }
        if (student) {
          uint2 wv;
          wv.x = pack2(vals[0], vals[1]);
          wv.y = pack2(vals[2], vals[3]);
          *reinterpret_cast<uint2*>(out) = wv;
        }
      }
    }
  } else {  // kModeDh: A rows are hidden columns
#pragma unroll
    for (int j = 0; j < FB; ++j) {
      const int t = tb + j * 16;
      if (t >= a.T) continue;
      if (a.k_split > 1) {
        float* out = a.dh_part + (size_t(split) * a.T + t) * a.H;
#pragma unroll
        for (int i = 0; i < FA; ++i) {
          const int hcol = rb + i * 16;
          if (hcol < a.H)
            *reinterpret_cast<float4*>(out + hcol) =
                make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
        }
      } else {
        u16* out = a.dh + size_t(t) * a.H;
#pragma unroll
        for (int i = 0; i < FA; ++i) {
          const int hcol = rb + i * 16;
          if (hcol < a.H) {
            uint2 wv;
            wv.x = pack2(acc[i][j][0], acc[i][j][1]);
            wv.y = pack2(acc[i][j][2], acc[i][j][3]);
            *reinterpret_cast<uint2*>(out + hcol) = wv;
          }
        }
      }
    }
  }
}

// dW[v][c] = sum_t G[t][v] H[t][c] (fp32 out).  Same tile shape as the tile
// engine (256 vocabulary rows x 256 hidden columns, 8 waves of 128 x 64) with
// MFMA 32x32x16; k = tokens, along which neither operand is contiguous.  Both
// k slices ([64 tokens][256]) go from HBM straight into LDS, two in flight,
// as unpadded 512-byte rows with 16-byte chunk c of token row r at position
// c ^ ((r & 3) << 2): the transposing operand reads (four token rows x 64
// bytes per 32 lanes) then hit distinct banks.  G's rows are padded with zeros
// to a multiple of 64 tokens (the grad pass writes them), so the last slice
// needs no masking: H rows past T are read clamped and meet zero G rows.
__global__ __launch_bounds__(NWAVES * 64, 1) void lm_dw_kernel(LmArgs a) {
  constexpr int WC = BT / (NWAVES / 2);    // hidden columns per wave (64)
  constexpr int NJ = WC / 32;
  __shared__ __align__(1024) u16 smem[2 * 2 * SLICE_B / 2];   // 2 slices x (G, H)

  int a0, t0, split;
  if (!tile_of<GROUP_T_V>(a, 1, a0, t0, split)) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c = lane & 31, g = lane >> 5;
  const int wa = wave / (NWAVES / 2), wt = wave % (NWAVES / 2);
  const int nk = a.Tg / BKK;

  // load i of this wave fills 16-byte slots (i * NWAVES + wave) * 64 + lane:
  // token row s / 32, chunk (s % 32) ^ ((row & 3) << 2)
  int gcol[NLD], hrow[NLD], hcol[NLD];
#pragma unroll
  for (int i = 0; i < NLD; ++i) {
    const int s = (i * NWAVES + wave) * 64 + lane;
    const int row = s >> 5, ch = (s & 31) ^ ((row & 3) << 2);
    gcol[i] = a0 + ch * 8;
    hrow[i] = row;
    hcol[i] = min(t0 + ch * 8, a.H - 8);   // hidden columns past H: outputs skipped
  }
  typedef __attribute__((address_space(3))) u16 lds_u16;
  const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_u16*)smem;
  auto issue = [&](int kk) {
    const uint32_t st = lds0 + (kk & 1) * (2 * SLICE_B) + wave * 1024;
    const int k0 = kk * BKK;
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      lds_load16(a.G + panel_index(k0 + hrow[i], gcol[i], a.Vp), st + i * NWAVES * 1024);
      const int t = min(k0 + hrow[i], a.T - 1);
      lds_load16(a.h + size_t(t) * a.H + hcol[i], st + SLICE_B + i * NWAVES * 1024);
    }
  };

  // transposing operand read in natural k order (rows g*8 + 0..7): lane l of a
  // 16-lane group reads token rows rb + (lane/32)*8 + l/4 and + 4, columns
  // col0 + ((lane/16) % 2)*16 + 4 (l % 4); with rb a multiple of 16 and col0 a
  // multiple of 32 the swizzle term of a lane is fixed
  const int l = lane & 15;
  const int rl = (lane >> 5) * 8 + (l >> 2);
  const int fl = (l >> 2) & 3;
  const int cl = ((((lane >> 4) & 1) * 2 + ((l & 3) >> 1)) << 3) + ((4 * (l & 3)) & 7);
  const char* lds = reinterpret_cast<const char*>(smem);
  auto tr = [&](const u16* tile, int rb, int cg) {   // cg = col0 / 32
    const u16* p0 = tile + (rb + rl) * 256 + (((cg ^ fl) << 5) + cl);
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p0));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p0 + 4 * 256));
    typedef short i16x8 __attribute__((ext_vector_type(8)));
    const i16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return __builtin_bit_cast(bf16x8, v);
  };
  bf16x8 af[2][4], bfr[2][NJ];
  auto read_frags = [&](int buf, int kk, int ks) {
    const u16* sG = reinterpret_cast<const u16*>(lds + (kk & 1) * (2 * SLICE_B));
    const u16* sH = reinterpret_cast<const u16*>(lds + (kk & 1) * (2 * SLICE_B) + SLICE_B);
#pragma unroll
    for (int i = 0; i < 4; ++i) af[buf][i] = tr(sG, ks * 16, wa * 4 + i);
#pragma unroll
    for (int j = 0; j < NJ; ++j) bfr[buf][j] = tr(sH, ks * 16, wt * NJ + j);
  };

  f32x16 acc[4][NJ];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  auto mma = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j) acc[i][j] = mfma32(af[buf][i], bfr[buf][j], acc[i][j]);
  };

  // four 16-token k steps per slice; one barrier per slice (as in the tile engine)
  issue(0);
  if (nk > 1) {
    issue(1);
    wait_vmcnt<2 * NLD>();
  } else {
    wait_vmcnt<0>();
  }
  __syncthreads();
  read_frags(0, 0, 0);
  for (int kk = 0; kk + 1 < nk; ++kk) {
    read_frags(1, kk, 1);
    mma(0);
    read_frags(0, kk, 2);
    mma(1);
    read_frags(1, kk, 3);
    mma(0);
    wait_vmcnt<0>();
    __syncthreads();
    if (kk + 2 < nk) issue(kk + 2);
    read_frags(0, kk + 1, 0);
    mma(1);
  }
  read_frags(1, nk - 1, 1);
  mma(0);
  read_frags(0, nk - 1, 2);
  mma(1);
  read_frags(1, nk - 1, 3);
  mma(0);
  mma(1);

  // acc[i][j][r]: vocabulary row a0 + wa*128 + i*32 + (r/4)*8 + g*4 + r%4,
  //               hidden column t0 + wt*WC + j*32 + c
  const int arow0 = a0 + wa * 128;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int hc = t0 + wt * WC + j * 32 + c;
    if (hc >= a.H) continue;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int v = arow0 + i * 32 + (r >> 2) * 8 + g * 4 + (r & 3);
        if (v < a.V) a.dw[size_t(v) * a.H + hc] = acc[i][j][r];
      }
  }
}

// Target logit z_{t,y_t} = h_t . W[y_t] in fp32 by one wave (lane k takes
// 16-byte chunks k, k + 64, ...; a fixed shuffle tree sums the lanes), so
// that the forward's combine and the backward's fix-up see the same value.
__device__ __forceinline__ float target_dot(const LmArgs& a, int t, int y, int lane) {
  const u16* hp = a.h + size_t(t) * a.H;
  const u16* wp = a.w + size_t(y) * a.H;
  float s = 0.f;
  for (int k = lane * 8; k < a.H; k += 512) {
    const uint4 hv = ld16(hp + k), wv = ld16(wp + k);
    const uint32_t hw[4] = {hv.x, hv.y, hv.z, hv.w}, ww[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      s = fmaf(bf16_to_f32(u16(hw[u])), bf16_to_f32(u16(ww[u])), s);
      s = fmaf(bf16_to_f32(u16(hw[u] >> 16)), bf16_to_f32(u16(ww[u] >> 16)), s);
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
  return s;
}

// Backward fix-up, one wave per token: rewrites G[t][y_t], which the grad
// tile left at -g_t p, to g_t (1 - p) with p = softmax(z_t)_{y_t} from the
// forward's lse.  An id outside [-1, V) is never used as an index: the token
// is treated as one without loss and counted in *bad_targets (this kernel
// sees every token exactly once per call).
__global__ __launch_bounds__(256) void lm_target_kernel(LmArgs a) {
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (t >= a.T) return;
  const int y = a.tgt[t];
  if (uint32_t(y) >= uint32_t(a.V)) {
    if (lane == 0 && y != -1) atomicAdd(a.bad_targets, 1);
    return;
  }
  const float s = target_dot(a, t, y, lane);
  if (lane != 0) return;
  const float p = fast_exp2(fmaf(s, kLog2e, -a.lse[t] * kLog2e));
  a.Gout[panel_index(t, y, a.Vp)] = u16(bf16_bits(a.g[t] * (1.f - p)));
}

// wT[h][v] = w[v][h] for v < V and 0 for V <= v < Vp, in the panel layout;
// 64 x 64 tiles through LDS.
__global__ __launch_bounds__(256) void transpose_w_kernel(const u16* w, u16* wT, int V, int H,
                                                          int Vp) {
  __shared__ u16 tile[64][72];
  const int v0 = blockIdx.x * 64, h0 = blockIdx.y * 64;
  const int tid = threadIdx.x;
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int idx = tid + q * 256;
    const int r = idx >> 3, c = (idx & 7) * 8;
    const uint4 val = v0 + r < V ? ld16(w + size_t(v0 + r) * H + h0 + c) : make_uint4(0, 0, 0, 0);
    st16(&tile[r][c], val);
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int idx = tid + q * 256;
    const int r = idx >> 3, c = (idx & 7) * 8;   // wT row h0 + r, columns v0 + c .. + 8
    uint32_t e[4];
#pragma unroll
    for (int u = 0; u < 4; ++u)
      e[u] = uint32_t(tile[c + 2 * u][r]) | (uint32_t(tile[c + 2 * u + 1][r]) << 16);
    st16(wT + panel_index(h0 + r, v0 + c, Vp), make_uint4(e[0], e[1], e[2], e[3]));
  }
}

// Outputs of the forward's combine pass; the GRPO fields are used only by the
// fused variant (mv_token_logprob_grpo).
struct CombineOut {
  const float* logp_old;
  float* logp;
  float* ratio;
  float* clipped;
  float* lse;
  float eps_lo, eps_hi;
  // GRPO loss fused into the pass
  const int32_t* traj_ptr;
  const float* reward;
  const float* logp_ref;     // null: no reference KL
  const uint8_t* mask;       // null: every token carries loss
  const float* adv;          // [n_traj] advantages from the preparation pass
  const int* n_loss_count;   // loss tokens counted by the preparation pass (mask given)
  int n_loss_fixed;          // the count when there is no mask (-1 otherwise)
  float* dlogp;
  float* part;               // [kGrpoParts][part_stride] (one column per block)
  int part_stride;
  int n_traj, G;
  float g_eps_lo, g_eps_hi, beta, adv_eps;
};

// One wave per token: the target logit, the merge of the per-chunk (max,
// sum) pairs into logsumexp, and the epilogue (logp, ratio, clip).  An id
// outside [-1, V) is never used as an index: the token is treated as one
// without loss and counted in *bad_targets.  GRPO: the wave finds the
// token's trajectory, lane 0 evaluates the token's loss terms and its
// gradient (already divided by the number of loss tokens), and the block's
// four tokens are summed in wave order into one column of per-block
// partials.
template <bool GRPO>
__global__ __launch_bounds__(256) void lm_combine_kernel(LmArgs a, CombineOut o) {
  __shared__ float red[4][kGrpoParts];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int t = __builtin_amdgcn_readfirstlane(blockIdx.x * 4 + wave);   // wave-uniform
  float v[kGrpoParts] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (t < a.T) {
    // GRPO: the token's inputs and trajectory first, so that their loads
    // land while the merge below runs
    bool on = false;
    float old_t = 0.f, ref_t = 0.f, adv_t = 0.f;
    if (GRPO) {
      on = o.mask == nullptr || o.mask[t] != 0;
      old_t = o.logp_old[t];
      if (o.logp_ref != nullptr) ref_t = o.logp_ref[t];
      adv_t = o.adv[grpo_traj_of_wave(o.traj_ptr, o.n_traj, t, lane)];
    }
    const int y = a.tgt[t];
    const bool scored = uint32_t(y) < uint32_t(a.V);
    float tl = 0.f;
    if (scored)
      tl = target_dot(a, t, y, lane);
    else if (lane == 0 && y != -1)
      atomicAdd(a.bad_targets, 1);
    const float2* p = a.part + size_t(t) * a.n_chunks;
    float m = -INFINITY;
    for (int i = lane; i < a.n_chunks; i += 64) m = fmaxf(m, p[i].x);
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
    float s = 0.f;
    for (int i = lane; i < a.n_chunks; i += 64) s += p[i].y * fast_exp2(p[i].x - m);
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
    if (lane == 0) {
      const float l = (m + __log2f(s)) * kLn2;
      o.lse[t] = l;
      const float lp = scored ? tl - l : 0.f;
      o.logp[t] = lp;
      if (o.logp_old != nullptr) {
        const float r = scored ? expf(lp - o.logp_old[t]) : 1.f;
        o.ratio[t] = r;
        o.clipped[t] = fminf(fmaxf(r, 1.f - o.eps_lo), 1.f + o.eps_hi);
      }
      if (GRPO) {
        float g = 0.f;
        if (on) {
          g = grpo_token_terms(lp, old_t, o.logp_ref != nullptr ? &ref_t : nullptr, adv_t,
                               o.g_eps_lo, o.g_eps_hi, o.beta, v);
          const float n = o.n_loss_fixed >= 0 ? float(o.n_loss_fixed) : float(*o.n_loss_count);
          g = g / n;   // n >= 1: this token is a loss token
        }
        o.dlogp[t] = g;
      }
    }
  }
  if (GRPO) {
    if (lane == 0)
#pragma unroll
      for (int k = 0; k < kGrpoParts; ++k) red[wave][k] = v[k];
    __syncthreads();
    if (threadIdx.x < kGrpoParts) {   // partials stored counter-major: [k][block]
      const int k = threadIdx.x;
      o.part[size_t(k) * o.part_stride + blockIdx.x] =
          ((red[0][k] + red[1][k]) + red[2][k]) + red[3][k];
    }
  }
}

// Merge one leaf's per-chunk teacher and student partials into both LSEs and
// KL(p || q) = sum_v p_v (zT_v - zS_v) - lseT + lseS.
__global__ __launch_bounds__(256) void kl_combine_kernel(LmArgs a, float* kl, float* lseT,
                                                         float* lseS) {
  const int leaf = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (leaf >= a.n_leaves) return;
  const float4* pt = a.partT + size_t(leaf) * a.n_chunks;
  const float2* ps = a.partS + size_t(leaf) * a.n_chunks;
  float mt = -INFINITY, ms = -INFINITY;
  for (int i = lane; i < a.n_chunks; i += 64) {
    mt = fmaxf(mt, pt[i].x);
    ms = fmaxf(ms, ps[i].x);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    mt = fmaxf(mt, __shfl_xor(mt, off));
    ms = fmaxf(ms, __shfl_xor(ms, off));
  }
  float st = 0.f, cr = 0.f, ss = 0.f;
  for (int i = lane; i < a.n_chunks; i += 64) {
    const float wt = fast_exp2(pt[i].x - mt);
    st += pt[i].y * wt;
    cr += pt[i].z * wt;
    ss += ps[i].y * fast_exp2(ps[i].x - ms);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    st += __shfl_xor(st, off);
    cr += __shfl_xor(cr, off);
    ss += __shfl_xor(ss, off);
  }
  if (lane != 0) return;
  const float l2t = __log2f(st), l2s = __log2f(ss);
  lseT[leaf] = (mt + l2t) * kLn2;
  lseS[leaf] = (ms + l2s) * kLn2;
  // lseS - lseT from the differences of its parts: no cancellation between
  // two terms of size log V, and exactly zero when both sides agree
  kl[leaf] = cr / st + ((ms - mt) + (l2s - l2t)) * kLn2;
}

// Vocabulary splits for a dH product: none when the output tiles already
// cover the CUs several times, otherwise the count (<= 8) with the least time
// per split slice, rounds of 256 resident blocks / splits (a larger count must
// gain 5% to be taken: each split adds an fp32 partial to write and reduce).
static int dh_splits(int n_tokens, int H) {
  const int tiles = ((H + BA - 1) / BA) * ((n_tokens + BT - 1) / BT);
  if (tiles >= 4 * 256) return 1;
  int best = 1;
  double best_t = (tiles + 255) / 256;
  for (int s = 2; s <= 8; ++s) {
    const double t = double((tiles * s + 255) / 256) / s;
    if (t < 0.95 * best_t) {
      best_t = t;
      best = s;
    }
  }
  return best;
}

static size_t dh_part_bytes(int T, int H) {
  const int splits = dh_splits(T, H);
  return splits > 1 ? align256(size_t(splits) * T * H * sizeof(float)) : 0;
}

// rows of a panel-layout matrix
static int panel_rows(int R) { return (R + 255) / 256 * 256; }

static size_t wT_bytes(int H, int V) {
  return align256(size_t(panel_rows(H)) * vocab_pad(V) * sizeof(u16));
}

size_t kl_fwd_ws_bytes(int n, int H, int V) {
  const int n_chunks = vocab_pad(V) / 128;
  return align256(size_t(n) * n_chunks * sizeof(float4)) +
         align256(size_t(n) * n_chunks * sizeof(float2)) + align256(size_t(H) * sizeof(u16)) +
         256;
}

// G [n, Vp] | dH partials | zero row [H] | W^T [H, Vp] (G and W^T in panels)
size_t kl_bwd_ws_bytes(int n, int H, int V) {
  return align256(size_t(panel_rows(n)) * vocab_pad(V) * sizeof(u16)) + dh_part_bytes(n, H) +
         align256(size_t(H) * sizeof(u16)) + wT_bytes(H, V) + 256;
}

__global__ __launch_bounds__(256) void zero_u16_kernel(u16* p, int n) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = 0;
}

static hipError_t zero_row(u16* p, int H, hipStream_t stream) {
  hipLaunchKernelGGL(zero_u16_kernel, dim3((H + 255) / 256), dim3(256), 0, stream, p, H);
  return hipGetLastError();
}

// Both log-prob workspaces start (at their first 256-byte aligned address)
// with a 256-byte status block: word 0 counts the target ids outside
// [-1, V) the last call met, word 1 the loss tokens of a fused GRPO forward.
// The call's own buffers follow it.
constexpr size_t kStatusBytes = 256;

// status | per-(token, chunk) (max, sum)
size_t logprob_fwd_ws_bytes(int T, int H, int V) {
  (void)H;
  const int n_chunks = vocab_pad(V) / 128;
  return kStatusBytes + align256(size_t(T) * n_chunks * sizeof(float2)) + 256;
}

// the forward's workspace | GRPO per-block partials (4 tokens a block) |
// advantages
static int combine_blocks(int T) { return (T + 3) / 4; }
// row stride of the counter-major partials (16-byte rows for the finish)
static int part_stride(int T) { return (combine_blocks(T) + 3) / 4 * 4; }
size_t logprob_grpo_ws_bytes(int T, int H, int V, int n_traj) {
  return logprob_fwd_ws_bytes(T, H, V) +
         align256(size_t(part_stride(T)) * kGrpoParts * sizeof(float)) +
         align256(size_t(n_traj) * sizeof(float));
}

static int g_rows(int T) { return panel_rows(T); }

// status | G [Tg, Vp] | dH partials | W^T [H, Vp] (G and W^T in panels)
size_t logprob_bwd_ws_bytes(int T, int H, int V) {
  return kStatusBytes + align256(size_t(g_rows(T)) * vocab_pad(V) * sizeof(u16)) +
         dh_part_bytes(T, H) + wT_bytes(H, V) + 256;
}

static char* align_ptr(void* p) {
  return reinterpret_cast<char*>((reinterpret_cast<uintptr_t>(p) + 255) & ~uintptr_t(255));
}

__global__ __launch_bounds__(64) void clear_status_kernel(int* status) {
  status[threadIdx.x] = 0;   // the whole 256-byte block
}

// The status block of a log-prob workspace, cleared on the stream (a kernel,
// not a memset, so that the call can be captured in a graph).
static int* clear_status(void* ws, hipStream_t stream) {
  int* st = reinterpret_cast<int*>(align_ptr(ws));
  hipLaunchKernelGGL(clear_status_kernel, dim3(1), dim3(64), 0, stream, st);
  return st;
}

int* logprob_status_word(const void* ws) {
  return reinterpret_cast<int*>(align_ptr(const_cast<void*>(ws)));
}

static dim3 gemm_grid(const LmArgs& a) {
  const int splits = a.k_split > 1 ? a.k_split : 1;
  const int per_xcd = (a.nA * a.nT * splits + kNumXcd - 1) / kNumXcd;
  return dim3(per_xcd * kNumXcd);
}

static hipError_t transpose_w(const u16* w, u16* wT, int V, int H, const char* name,
                              hipStream_t stream) {
  ProfScope p(name, stream);
  hipLaunchKernelGGL(transpose_w_kernel, dim3(vocab_pad(V) / 64, H / 64), dim3(256), 0, stream, w,
                     wT, V, H, vocab_pad(V));
  return hipGetLastError();
}

// dH[t][h] = sum over splits of the fp32 partials, in split order (the
// result does not depend on scheduling), rounded once to bf16.
__global__ __launch_bounds__(256) void dh_reduce_kernel(const float* part, u16* dh, int splits,
                                                        size_t n4) {
  const size_t i = size_t(blockIdx.x) * 256 + threadIdx.x;
  if (i >= n4) return;
  const float4* p = reinterpret_cast<const float4*>(part) + i;
  float4 acc = p[0];
  for (int s = 1; s < splits; ++s) {
    const float4 v = p[size_t(s) * n4];
    acc.x += v.x;
    acc.y += v.y;
    acc.z += v.z;
    acc.w += v.w;
  }
  uint2 w;
  w.x = pack2(acc.x, acc.y);
  w.y = pack2(acc.z, acc.w);
  reinterpret_cast<uint2*>(dh)[i] = w;
}

// dh[T, H] = G[T, Vp] W[Vp, H] (bf16 out) with b.wT = W^T [H, Vp], split over
// the vocabulary when the output alone would leave CUs idle; `part` is the
// fp32 partial area of the workspace (dh_part_bytes).
static hipError_t launch_dh(LmArgs b, float* part, const char* name, hipStream_t stream) {
  const int nk_total = b.Vp / BKK;
  int splits = std::min(dh_splits(b.T, b.H), nk_total);
  b.nk_split = (nk_total + splits - 1) / splits;
  splits = (nk_total + b.nk_split - 1) / b.nk_split;  // no empty split
  b.k_split = splits;
  b.dh_part = part;
  b.nA = (b.H + BA - 1) / BA;
  b.nT = (b.T + BT - 1) / BT;
  {
    ProfScope p(name, stream);
    hipLaunchKernelGGL(lm_tile_kernel<kModeDh>, gemm_grid(b), dim3(NWAVES * 64), 0, stream, b);
    if (splits > 1) {
      const size_t n4 = size_t(b.T) * b.H / 4;
      hipLaunchKernelGGL(dh_reduce_kernel, dim3(unsigned((n4 + 255) / 256)), dim3(256), 0, stream,
                         part, b.dh, splits, n4);
    }
  }
  return hipGetLastError();
}

// Preparation pass of the fused GRPO forward: the advantage of every
// trajectory (thread i < n_traj) and the loss tokens (the mask's nonzero
// entries, 1024 per block, added with one integer atomic per block: exact in
// any order).
__global__ __launch_bounds__(256) void grpo_prep_kernel(const uint8_t* mask, int T, int* count,
                                                        const float* reward, int n_traj, int G,
                                                        float adv_eps, float* adv) {
  __shared__ int wsum[4];
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n_traj) adv[i] = grpo_advantage(reward, G, i, adv_eps);
  if (mask == nullptr) return;   // block-uniform
  const int i0 = i * 4;
  int c = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) c += (i0 + k < T && mask[i0 + k] != 0) ? 1 : 0;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) c += __shfl_xor(c, off);
  if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = c;
  __syncthreads();
  if (threadIdx.x == 0) {
    const int tot = wsum[0] + wsum[1] + wsum[2] + wsum[3];
    if (tot) atomicAdd(count, tot);
  }
}

static hipError_t logprob_fwd_common(LmArgs& a, void* ws, const CombineOut& o, bool grpo,
                                     const uint8_t* grpo_mask, hipStream_t stream) {
  a.bad_targets = clear_status(ws, stream);
  a.part = reinterpret_cast<float2*>(align_ptr(ws) + kStatusBytes);
  a.nA = a.Vp / BA;
  a.nT = (a.T + BT - 1) / BT;
  if (grpo) {
    const int blocks = std::max((a.T + 1023) / 1024, (o.n_traj + 255) / 256);
    ProfScope p("grpo_prep", stream);
    hipLaunchKernelGGL(grpo_prep_kernel, dim3(unsigned(blocks)), dim3(256), 0, stream, grpo_mask,
                       a.T, a.bad_targets + 1, o.reward, o.n_traj, o.G, o.adv_eps,
                       const_cast<float*>(o.adv));
  }
  if (a.T == 0) return hipGetLastError();
  {
    ProfScope p("lm_logits", stream);
    hipLaunchKernelGGL(lm_tile_kernel<kModeLogits>, gemm_grid(a), dim3(NWAVES * 64), 0, stream, a);
  }
  {
    ProfScope p("lm_combine", stream);
    if (grpo)
      hipLaunchKernelGGL(lm_combine_kernel<true>, dim3(combine_blocks(a.T)), dim3(256), 0, stream,
                         a, o);
    else
      hipLaunchKernelGGL(lm_combine_kernel<false>, dim3(combine_blocks(a.T)), dim3(256), 0,
                         stream, a, o);
  }
  return hipGetLastError();
}

static LmArgs fwd_args(int T, int H, int V, const void* hidden, const void* weight,
                       const int32_t* target) {
  LmArgs a{};
  a.h = static_cast<const u16*>(hidden);
  a.w = static_cast<const u16*>(weight);
  a.tgt = target;
  a.T = T;
  a.H = H;
  a.V = V;
  a.Vp = vocab_pad(V);
  a.n_chunks = a.Vp / 128;
  return a;
}

hipError_t launch_logprob_fwd(int T, int H, int V, float eps_lo, float eps_hi, const void* hidden,
                              const void* weight, const int32_t* target, const float* logp_old,
                              float* logp, float* ratio, float* clipped, float* lse, void* ws,
                              hipStream_t stream) {
  LmArgs a = fwd_args(T, H, V, hidden, weight, target);
  CombineOut o{};
  o.logp_old = logp_old;
  o.logp = logp;
  o.ratio = ratio;
  o.clipped = clipped;
  o.lse = lse;
  o.eps_lo = eps_lo;
  o.eps_hi = eps_hi;
  return logprob_fwd_common(a, ws, o, false, nullptr, stream);
}

// The forward with the GRPO loss fused into its combine pass: count the loss
// tokens (mask given), the logits GEMM, the combine with the per-token loss
// terms and gradient, one block for the statistics and advantages.
hipError_t launch_logprob_grpo(int T, int H, int V, float eps_lo, float eps_hi,
                               const void* hidden, const void* weight, const int32_t* target,
                               const float* logp_old, int n_traj, int G, float g_eps_lo,
                               float g_eps_hi, float beta, float adv_eps, const int32_t* traj_ptr,
                               const float* reward, const float* logp_ref, const uint8_t* mask,
                               float* logp, float* ratio, float* clipped, float* lse,
                               float* adv_out, float* dlogp, float* stats, void* ws,
                               hipStream_t stream) {
  LmArgs a = fwd_args(T, H, V, hidden, weight, target);
  CombineOut o{};
  o.logp_old = logp_old;
  o.logp = logp;
  o.ratio = ratio;
  o.clipped = clipped;
  o.lse = lse;
  o.eps_lo = eps_lo;
  o.eps_hi = eps_hi;
  o.traj_ptr = traj_ptr;
  o.reward = reward;
  o.logp_ref = logp_ref;
  o.mask = mask;
  o.n_loss_count = reinterpret_cast<const int*>(align_ptr(ws)) + 1;
  o.n_loss_fixed = mask == nullptr ? T : -1;
  o.dlogp = dlogp;
  o.part = reinterpret_cast<float*>(align_ptr(ws) + kStatusBytes +
                                    align256(size_t(T) * a.n_chunks * sizeof(float2)));
  o.part_stride = part_stride(T);
  o.adv = adv_out != nullptr
              ? adv_out
              : reinterpret_cast<float*>(reinterpret_cast<char*>(o.part) +
                                         align256(size_t(part_stride(T)) * kGrpoParts *
                                                  sizeof(float)));
  o.n_traj = n_traj;
  o.G = G;
  o.g_eps_lo = g_eps_lo;
  o.g_eps_hi = g_eps_hi;
  o.beta = logp_ref != nullptr ? beta : 0.f;
  o.adv_eps = adv_eps;
  if (hipError_t e = logprob_fwd_common(a, ws, o, true, mask, stream); e != hipSuccess) return e;
  ProfScope p("grpo_finish", stream);
  return launch_grpo_fused_finish(o.part, combine_blocks(T), o.part_stride, n_traj, o.adv, stats,
                                  stream);
}

hipError_t launch_logprob_bwd(int T, int H, int V, const void* hidden, const void* weight,
                              const int32_t* target, const float* lse, const float* dlogp,
                              void* dhidden, void* ws, hipStream_t stream) {
  LmArgs a{};
  a.h = static_cast<const u16*>(hidden);
  a.w = static_cast<const u16*>(weight);
  a.tgt = target;
  a.lse = lse;
  a.g = dlogp;
  a.T = T;
  a.H = H;
  a.V = V;
  a.Vp = vocab_pad(V);
  a.Tg = g_rows(T);
  a.bad_targets = clear_status(ws, stream);
  char* base = align_ptr(ws) + kStatusBytes;
  u16* G = reinterpret_cast<u16*>(base);
  float* part = reinterpret_cast<float*>(base + align256(size_t(a.Tg) * a.Vp * sizeof(u16)));
  u16* wT = reinterpret_cast<u16*>(reinterpret_cast<char*>(part) + dh_part_bytes(T, H));
  a.Gout = G;
  a.G = G;
  a.wT = wT;
  a.dh = static_cast<u16*>(dhidden);
  a.nA = a.Vp / BA;
  a.nT = (T + BT - 1) / BT;
  if (hipError_t e = transpose_w(a.w, wT, V, H, "lm_wt", stream); e != hipSuccess) return e;
  {
    ProfScope p("lm_grad", stream);
    hipLaunchKernelGGL(lm_tile_kernel<kModeGrad>, gemm_grid(a), dim3(NWAVES * 64), 0, stream, a);
  }
  {
    ProfScope p("lm_target", stream);
    hipLaunchKernelGGL(lm_target_kernel, dim3((T + 3) / 4), dim3(256), 0, stream, a);
  }
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  return launch_dh(a, part, "lm_dh", stream);
}

// dW = G^T H from the G that launch_logprob_bwd left in its workspace.
hipError_t launch_logprob_dweight(int T, int H, int V, const void* hidden, const void* ws,
                                  float* dw, hipStream_t stream) {
  LmArgs a{};
  a.h = static_cast<const u16*>(hidden);
  a.G = reinterpret_cast<const u16*>(align_ptr(const_cast<void*>(ws)) + kStatusBytes);
  a.dw = dw;
  a.T = T;
  a.Tg = g_rows(T);
  a.H = H;
  a.V = V;
  a.Vp = vocab_pad(V);
  a.nA = a.Vp / BA;
  a.nT = (H + BT - 1) / BT;
  ProfScope p("lm_dw", stream);
  hipLaunchKernelGGL(lm_dw_kernel, gemm_grid(a), dim3(NWAVES * 64), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_kl_fwd(int n, int H, int V, const void* hT, int nT, const int32_t* rowsT,
                         const void* hS, int nS, const int32_t* rowsS, const void* weight,
                         float* kl, float* lseT, float* lseS, void* ws, hipStream_t stream) {
  LmArgs a{};
  a.n_rows_T = nT;
  a.n_rows_S = nS;
  a.w = static_cast<const u16*>(weight);
  a.hT = static_cast<const u16*>(hT);
  a.hS = static_cast<const u16*>(hS);
  a.rowsT = rowsT;
  a.rowsS = rowsS;
  a.n_leaves = n;
  a.T = 2 * n;
  a.H = H;
  a.V = V;
  a.Vp = vocab_pad(V);
  a.n_chunks = a.Vp / 128;
  char* base = align_ptr(ws);
  a.partT = reinterpret_cast<float4*>(base);
  a.partS = reinterpret_cast<float2*>(base + align256(size_t(n) * a.n_chunks * sizeof(float4)));
  u16* zrow = reinterpret_cast<u16*>(base + align256(size_t(n) * a.n_chunks * sizeof(float4)) +
                                     align256(size_t(n) * a.n_chunks * sizeof(float2)));
  a.zero_row = zrow;
  if (hipError_t e = zero_row(zrow, H, stream); e != hipSuccess) return e;
  a.nA = a.Vp / BA;
  a.nT = (a.T + BT - 1) / BT;
  {
    ProfScope p("kl_logits", stream);
    hipLaunchKernelGGL(lm_tile_kernel<kModeKL>, gemm_grid(a), dim3(NWAVES * 64), 0, stream, a);
  }
  {
    ProfScope p("kl_combine", stream);
    hipLaunchKernelGGL(kl_combine_kernel, dim3((n + 3) / 4), dim3(256), 0, stream, a, kl, lseT,
                       lseS);
  }
  return hipGetLastError();
}

hipError_t launch_kl_bwd(int n, int H, int V, const void* hT, int nT, const int32_t* rowsT,
                         const void* hS, int nS, const int32_t* rowsS, const void* weight,
                         const float* lseT, const float* lseS, const float* dkl, void* dh,
                         void* ws, hipStream_t stream) {
  LmArgs a{};
  a.n_rows_T = nT;
  a.n_rows_S = nS;
  a.w = static_cast<const u16*>(weight);
  a.hT = static_cast<const u16*>(hT);
  a.hS = static_cast<const u16*>(hS);
  a.rowsT = rowsT;
  a.rowsS = rowsS;
  a.lseT = lseT;
  a.lseS = lseS;
  a.dkl = dkl;
  a.n_leaves = n;
  a.T = 2 * n;
  a.H = H;
  a.V = V;
  a.Vp = vocab_pad(V);
  char* base = align_ptr(ws);
  u16* G = reinterpret_cast<u16*>(base);
  float* part = reinterpret_cast<float*>(base + align256(size_t(panel_rows(n)) * a.Vp * sizeof(u16)));
  u16* zrow = reinterpret_cast<u16*>(reinterpret_cast<char*>(part) + dh_part_bytes(n, H));
  u16* wT = reinterpret_cast<u16*>(reinterpret_cast<char*>(zrow) + align256(size_t(H) * sizeof(u16)));
  a.Gout = G;
  a.nA = a.Vp / BA;
  a.nT = (a.T + BT - 1) / BT;
  a.zero_row = zrow;
  if (hipError_t e = zero_row(zrow, H, stream); e != hipSuccess) return e;
  if (hipError_t e = transpose_w(a.w, wT, V, H, "kl_wt", stream); e != hipSuccess) return e;
  {
    ProfScope p("kl_grad", stream);
    hipLaunchKernelGGL(lm_tile_kernel<kModeKLGrad>, gemm_grid(a), dim3(NWAVES * 64), 0, stream, a);
  }
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  // dh = G W over the leaves
  LmArgs b{};
  b.w = a.w;
  b.wT = wT;
  b.G = G;
  b.dh = static_cast<u16*>(dh);
  b.T = n;
  b.H = H;
  b.V = V;
  b.Vp = a.Vp;
  return launch_dh(b, part, "kl_dh", stream);
}

}  // namespace mv
