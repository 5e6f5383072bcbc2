// Fused LM-head token log-prob, ratio and clip on gfx950.
//
// Forward: z = W h is produced 256 vocab rows x 256 tokens at a time by a bf16
// MFMA tile engine and reduced in registers to a per-token (max, sum of
// exp) over each wave's 128 vocab rows; the target logit is captured by the
// one lane that owns it.  The full logits are never stored.  A combine pass
// merges the partials into logsumexp and writes logp, ratio and the clipped
// ratio (the GRPO ratio of Appendix C, "Pitfall A, RL view").
//
// Backward: the logits tile is recomputed and turned into
// G_tv = g_t (onehot(y_t)_v - softmax(z_t)_v), stored once in bf16, and a
// second pass of the same engine computes dH = G W (contraction over the
// vocabulary).
//
// Tile engine: 512 threads = 8 waves (two per SIMD) in a 2 x 4 grid over a
// 256 A-row x 256 token tile; each wave owns 128 A-rows x 64 tokens (tokens on
// lanes), MFMA 32x32x16 (the dH pass reads its W^T operand from a row-major W
// slice with the transposing LDS read).  The 64-wide k slices are double-buffered in LDS with
// one barrier per slice: while a slice is multiplied, the next one is written
// from registers into the other buffer and the one after is loaded from HBM.
// Tiles are ordered so that the blocks resident on one XCD at a time form a
// compact 2-D patch (a few token tiles x several A tiles) and share operand
// slices in that XCD's L2.
#include <algorithm>

#include "mv_device.h"

namespace mv {

namespace {
constexpr int BA = 256, BT = 256, BKK = 64;
constexpr int PAD = BKK + 8;               // LDS row stride (bf16), conflict-free operand reads
// row stride of the row-major W slice of the dH pass: 576 bytes, so the four
// rows one transposing read touches start 16 banks apart
constexpr int WPAD = BA + 32;
constexpr int STAGE = (BA + BT) * PAD;     // one k slice of both operands
static_assert(BKK * WPAD <= BA * PAD, "dH pass W slice must fit the A region");
static_assert(BKK * WPAD <= BT * PAD, "dW pass hidden slice must fit the token region");
constexpr int NWAVES = 8;                 // waves per tile (2 x NWAVES/2 grid)
constexpr int GROUP_T = 4;                 // token tiles per raster group
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.69314718055994531f;
size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
int vocab_pad(int V) { return (V + BA - 1) / BA * BA; }
}  // namespace

enum { kModeLogits = 0, kModeGrad = 1, kModeDh = 2, kModeKL = 3, kModeKLGrad = 4, kModeDw = 5 };

struct LmArgs {
  const u16* h;       // [T, H]
  const u16* w;       // [V, H]
  const int32_t* tgt; // [T]
  const float* lse;   // [T] (grad mode)
  const float* g;     // [T] upstream dlogp (grad mode)
  const u16* G;       // [T, Vp] (dH mode)
  u16* Gout;          // [T, Vp] (grad mode)
  u16* dh;            // [T, H] (dH mode)
  float2* part;       // [T, n_chunks] (logits mode)
  float* tlogit;      // [T] (logits mode)
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
  int nA, nT;         // tiles along the A side and along tokens
  // dH mode split over the vocabulary (K) when there are too few output
  // tiles to fill the chip: split s covers k slices [s*nk_split, ...) and
  // writes fp32 partials dh_part[s][t][H], summed in order by dh_reduce_kernel
  int k_split, nk_split;
  float* dh_part;
  float* dw;          // [V, H] fp32 (dW mode)
};

template <int MODE, int NW>
__global__ __launch_bounds__(NW * 64, 1) void lm_gemm_kernel(LmArgs a) {
  constexpr int NT = NW * 64;              // threads
  constexpr int WTOK = BT / (NW / 2);      // tokens per wave (2 waves along the A side)
  constexpr int NJ = WTOK / 32;            // 32-token MFMA blocks per wave
  constexpr int LDA = (BA * BKK / 8) / NT; // 16-byte loads per thread, A slice
  constexpr int LDB = (BT * BKK / 8) / NT; // 16-byte loads per thread, token slice
  __shared__ __align__(16) u16 smem[2 * STAGE];

  // Blocks are dealt to XCDs round-robin; give each XCD a contiguous range of
  // the rasterised tile order (groups of GROUP_T token tiles x all A tiles).
  const int n_out = a.nA * a.nT;
  const int n_tiles = n_out * (MODE == kModeDh ? a.k_split : 1);
  const int per_xcd = (n_tiles + kNumXcd - 1) / kNumXcd;
  int xcd, local;
  xcd_split(xcd, local);
  const int Lx = xcd * per_xcd + local;
  if (local >= per_xcd || Lx >= n_tiles) return;
  const int split = Lx / n_out;            // 0 unless the dH product is split
  const int L = Lx % n_out;
  const int grp = L / (GROUP_T * a.nA);
  const int rem = L % (GROUP_T * a.nA);
  const int t_in = min(GROUP_T, a.nT - grp * GROUP_T);
  const int tt = grp * GROUP_T + rem % t_in;
  const int at = rem / t_in;
  const int a0 = at * BA, t0 = tt * BT;

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int c = lane & 31, g = lane >> 5;
  const int wa = wave / (NW / 2), wt = wave % (NW / 2);

  // dW mode: A rows = vocabulary, B "tokens" = hidden columns, k = tokens
  constexpr bool kT = (MODE == kModeDh || MODE == kModeDw);  // both stages k-major
  const int K = (MODE == kModeDh) ? a.Vp : (MODE == kModeDw ? a.T : a.H);
  const int a_rows = (MODE == kModeDh) ? a.H : a.V;
  const int b_rows = (MODE == kModeDw) ? a.H : a.T;
  const int kbeg = (MODE == kModeDh) ? split * a.nk_split : 0;
  const int nk = (MODE == kModeDh) ? min(K / BKK - kbeg, a.nk_split) : (K + BKK - 1) / BKK;
  // Out-of-range operand rows and columns are read from clamped (valid)
  // addresses instead of being masked, so loads never wait on a select: the
  // products they feed land in output rows, columns or vocabulary padding that
  // the epilogues skip or zero (and padding columns of G are stored as zero).
  // Tiles wholly inside the operands skip even the clamping.
  const bool interior = (t0 + BT <= b_rows) && (MODE == kModeDh ? (a0 + BA <= a.H) : (a0 + BA <= a_rows));

  f32x16 acc[4][NJ];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // each thread's token rows are fixed across k slices: resolve them once
  const u16* brow[LDB];
#pragma unroll
  for (int r = 0; r < LDB; ++r) {
    const int t = t0 + (tid + r * NT) / (BKK / 8);
    const int tc = (interior || t < a.T) ? t : 0;
    if (MODE == kModeDw) {
      brow[r] = nullptr;  // the dW stages are addressed per k slice
    } else if (MODE == kModeDh) {
      brow[r] = a.G + size_t(tc) * a.Vp;
    } else if (MODE == kModeKL || MODE == kModeKLGrad) {
      // a row index outside its matrix reads as a zero hidden state
      const int row = (tc & 1) ? a.rowsS[tc >> 1] : a.rowsT[tc >> 1];
      const int n_rows = (tc & 1) ? a.n_rows_S : a.n_rows_T;
      const bool row_ok = row >= 0 && row < n_rows;
      brow[r] = row_ok ? ((tc & 1) ? a.hS : a.hT) + size_t(row) * a.H : a.zero_row;
    } else {
      brow[r] = a.h + size_t(tc) * a.H;
    }
  }

  uint4 ra[LDA], rb[LDB];
  auto load = [&](int k0) {
    if (MODE == kModeDw) {
      // G slice [64 tokens][256 vocabulary] and H slice [64 tokens][256
      // hidden], both staged k-major and read with the transposing LDS read.
      // Token rows past T must add nothing (k is summed): the tail slice
      // zeroes them (a block-uniform branch, taken once per tile).
      auto stage = [&](bool tail) {
#pragma unroll
        for (int r = 0; r < LDA; ++r) {
          const int idx = tid + r * NT;
          const int row = idx / (BA / 8), cc = (idx % (BA / 8)) * 8;
          const int t = k0 + row;
          ra[r] = ld16(a.G + size_t(min(t, a.T - 1)) * a.Vp + a0 + cc);
          if (tail && t >= a.T) ra[r] = make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int r = 0; r < LDB; ++r) {
          const int idx = tid + r * NT;
          const int row = idx / (BT / 8), cc = (idx % (BT / 8)) * 8;
          const int t = k0 + row;
          rb[r] = ld16(a.h + size_t(min(t, a.T - 1)) * a.H + min(t0 + cc, a.H - 8));
          if (tail && t >= a.T) rb[r] = make_uint4(0, 0, 0, 0);
        }
      };
      if (k0 + BKK > a.T)
        stage(true);
      else
        stage(false);
      return;
    }
#pragma unroll
    for (int r = 0; r < LDA; ++r) {
      const int idx = tid + r * NT;
      if (MODE == kModeDh) {
        // W slice [64 vocab rows][256 hidden], staged row-major; the A = W^T
        // operand is read across its rows with the transposing LDS read
        const int row = idx / (BA / 8), cc = (idx % (BA / 8)) * 8;
        const int v = k0 + row;
        const u16* p = a.w + size_t(min(v, a.V - 1)) * a.H + min(a0 + cc, a.H - 8);
        ra[r] = ld16(p);
      } else {
        const int row = idx / (BKK / 8), cc = (idx % (BKK / 8)) * 8;
        const int v = a0 + row;
        const u16* p = a.w + size_t(min(v, a_rows - 1)) * a.H + k0 + cc;
        ra[r] = ld16(p);
      }
    }
#pragma unroll
    for (int r = 0; r < LDB; ++r) {
      const int cc = ((tid + r * NT) % (BKK / 8)) * 8;
      rb[r] = ld16(brow[r] + k0 + cc);
    }
  };
  auto store = [&](u16* sA) {
    u16* sB = sA + BA * PAD;
#pragma unroll
    for (int r = 0; r < LDA; ++r) {
      const int idx = tid + r * NT;
      if (kT) {
        const int row = idx / (BA / 8), cc = (idx % (BA / 8)) * 8;
        st16(&sA[row * WPAD + cc], ra[r]);
      } else {
        const int row = idx / (BKK / 8), cc = (idx % (BKK / 8)) * 8;
        st16(&sA[row * PAD + cc], ra[r]);
      }
    }
#pragma unroll
    for (int r = 0; r < LDB; ++r) {
      const int idx = tid + r * NT;
      if (MODE == kModeDw) {
        const int row = idx / (BT / 8), cc = (idx % (BT / 8)) * 8;
        st16(&sB[row * WPAD + cc], rb[r]);
      } else {
        const int row = idx / (BKK / 8), cc = (idx % (BKK / 8)) * 8;
        st16(&sB[row * PAD + cc], rb[r]);
      }
    }
  };

  if (nk > 0) {  // block-uniform
    load(kbeg * BKK);
    store(smem);
    if (nk > 1) load((kbeg + 1) * BKK);
    __syncthreads();
  }
  for (int kk = 0; kk < nk; ++kk) {
    const u16* sA = smem + (kk & 1) * STAGE;
    const u16* sB = sA + BA * PAD;
    // The next slice goes to the other buffer first (every wave finished
    // reading it before the last barrier), then the slice after it is
    // requested from HBM, so both overlap this slice's MFMAs.
    if (kk + 1 < nk) {
      store(smem + ((kk + 1) & 1) * STAGE);
      if (kk + 2 < nk) load((kbeg + kk + 2) * BKK);
    }
#pragma unroll
    for (int ks = 0; ks < BKK / 16; ++ks) {
      bf16x8 af[4], bf[NJ];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        af[i] = kT ? ld_operand_tr<WPAD, true>(sA, ks * 16, wa * 128 + i * 32)
                   : as_bf16x8(ld16(&sA[(wa * 128 + i * 32 + c) * PAD + ks * 16 + g * 8]));
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        bf[j] = (MODE == kModeDw)
                    ? ld_operand_tr<WPAD, true>(sB, ks * 16, wt * WTOK + j * 32)
                    : as_bf16x8(ld16(&sB[(wt * WTOK + j * 32 + c) * PAD + ks * 16 + g * 8]));
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j) acc[i][j] = mfma32(af[i], bf[j], acc[i][j]);
    }
    __syncthreads();
  }

  // acc[i][j][r]: A-row a0 + wa*128 + i*32 + (r/4)*8 + g*4 + r%4,
  //               token t0 + wt*WTOK + j*32 + c
  const int arow0 = a0 + wa * 128;
  if (MODE == kModeLogits) {
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int t = t0 + wt * WTOK + j * 32 + c;
      const int y = t < a.T ? a.tgt[t] : -1;
      float mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int v = arow0 + i * 32 + (r >> 2) * 8 + g * 4 + (r & 3);
          float z = acc[i][j][r];
          if (v == y) a.tlogit[t] = z;
          z = v < a.V ? z * kLog2e : -INFINITY;
          acc[i][j][r] = z;
          mx = fmaxf(mx, z);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float mu = mx == -INFINITY ? 0.f : mx;  // a chunk of vocabulary padding only
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) s += fast_exp2(acc[i][j][r] - mu);
      s += __shfl_xor(s, 32);
      if (g == 0 && t < a.T) a.part[size_t(t) * a.n_chunks + arow0 / 128] = make_float2(mx, s);
    }
  } else if (MODE == kModeGrad) {
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int t = t0 + wt * WTOK + j * 32 + c;
      if (t >= a.T) continue;
      const int y = a.tgt[t];
      const float gt = y >= 0 ? a.g[t] : 0.f;
      const float l2 = a.lse[t] * kLog2e;
      u16* out = a.Gout + size_t(t) * a.Vp;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          float vals[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int v = arow0 + i * 32 + q4 * 8 + g * 4 + u;
            const float p = fast_exp2(acc[i][j][q4 * 4 + u] * kLog2e - l2);
            vals[u] = v < a.V ? gt * ((v == y ? 1.f : 0.f) - p) : 0.f;
          }
          uint2 wv;
          wv.x = pack2(vals[0], vals[1]);
          wv.y = pack2(vals[2], vals[3]);
          *reinterpret_cast<uint2*>(out + arow0 + i * 32 + q4 * 8 + g * 4) = wv;
        }
    }
  } else if (MODE == kModeKL) {
    // lanes c (even, teacher) and c + 1 (student) hold the same vocabulary
    // rows of one leaf; each lane keeps its own (max, sum of exp) and the
    // teacher also accumulates sum exp(zT - mT) * (zT - zS)
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int t = t0 + wt * WTOK + j * 32 + c;
      const int leaf = t >> 1;
      float mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int v = arow0 + i * 32 + (r >> 2) * 8 + g * 4 + (r & 3);
          if (v < a.V) mx = fmaxf(mx, acc[i][j][r] * kLog2e);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float mu = mx == -INFINITY ? 0.f : mx;
      float sm = 0.f, cross = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int v = arow0 + i * 32 + (r >> 2) * 8 + g * 4 + (r & 3);
          const float z = acc[i][j][r];
          const float zo = __shfl_xor(z, 1);  // the partner row's logit
          const float e = v < a.V ? fast_exp2(z * kLog2e - mu) : 0.f;
          sm += e;
          cross += e * (z - zo);
        }
      sm += __shfl_xor(sm, 32);
      cross += __shfl_xor(cross, 32);
      if (g == 0 && leaf < a.n_leaves) {
        const size_t o = size_t(leaf) * a.n_chunks + arow0 / 128;
        if (t & 1)
          a.partS[o] = make_float2(mx, sm);
        else
          a.partT[o] = make_float4(mx, sm, cross, 0.f);
      }
    }
  } else if (MODE == kModeKLGrad) {
    // student lanes write G = dkl * (q - p) for their leaf
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int t = t0 + wt * WTOK + j * 32 + c;
      const int leaf = t >> 1;
      const bool student = (t & 1) && leaf < a.n_leaves;
      const int lc = leaf < a.n_leaves ? leaf : 0;
      const float gl = a.dkl[lc];
      const float lS = a.lseS[lc] * kLog2e, lT = a.lseT[lc] * kLog2e;
      u16* out = a.Gout + size_t(lc) * a.Vp;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          float vals[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int v = arow0 + i * 32 + q4 * 8 + g * 4 + u;
            const float zS = acc[i][j][q4 * 4 + u];
            const float zT = __shfl_xor(zS, 1);
            const float q = fast_exp2(zS * kLog2e - lS), pt = fast_exp2(zT * kLog2e - lT);
            vals[u] = v < a.V ? gl * (q - pt) : 0.f;
          }
          if (student) {
            uint2 wv;
            wv.x = pack2(vals[0], vals[1]);
            wv.y = pack2(vals[2], vals[3]);
            *reinterpret_cast<uint2*>(out + arow0 + i * 32 + q4 * 8 + g * 4) = wv;
          }
        }
    }
  } else if (MODE == kModeDw) {
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int hcol = t0 + wt * WTOK + j * 32 + c;
      if (hcol >= a.H) continue;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int v = arow0 + i * 32 + (r >> 2) * 8 + g * 4 + (r & 3);
          if (v < a.V) a.dw[size_t(v) * a.H + hcol] = acc[i][j][r];
        }
    }
  } else if (a.k_split > 1) {
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int t = t0 + wt * WTOK + j * 32 + c;
      if (t >= a.T) continue;
      float* out = a.dh_part + (size_t(split) * a.T + t) * a.H;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const int hcol = arow0 + i * 32 + q4 * 8 + g * 4;
          if (hcol >= a.H) continue;
          *reinterpret_cast<float4*>(out + hcol) =
              make_float4(acc[i][j][q4 * 4 + 0], acc[i][j][q4 * 4 + 1], acc[i][j][q4 * 4 + 2],
                          acc[i][j][q4 * 4 + 3]);
        }
    }
  } else {
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int t = t0 + wt * WTOK + j * 32 + c;
      if (t >= a.T) continue;
      u16* out = a.dh + size_t(t) * a.H;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const int hcol = arow0 + i * 32 + q4 * 8 + g * 4;
          if (hcol >= a.H) continue;
          uint2 wv;
          wv.x = pack2(acc[i][j][q4 * 4 + 0], acc[i][j][q4 * 4 + 1]);
          wv.y = pack2(acc[i][j][q4 * 4 + 2], acc[i][j][q4 * 4 + 3]);
          *reinterpret_cast<uint2*>(out + hcol) = wv;
        }
    }
  }
}

// Merge the per-chunk (max, sum) pairs of one token and finish the epilogue.
__global__ __launch_bounds__(256) void lm_combine_kernel(LmArgs a, const float* logp_old,
                                                         float* logp, float* ratio,
                                                         float* clipped, float* lse, float eps_lo,
                                                         float eps_hi) {
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (t >= a.T) return;
  const float2* p = a.part + size_t(t) * a.n_chunks;
  float m = -INFINITY;
  for (int i = lane; i < a.n_chunks; i += 64) m = fmaxf(m, p[i].x);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
  float s = 0.f;
  for (int i = lane; i < a.n_chunks; i += 64) s += p[i].y * fast_exp2(p[i].x - m);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
  if (lane != 0) return;
  const float l = (m + __log2f(s)) * kLn2;
  lse[t] = l;
  const int y = a.tgt[t];
  const float lp = y >= 0 ? a.tlogit[t] - l : 0.f;
  logp[t] = lp;
  if (logp_old != nullptr) {
    const float r = y >= 0 ? expf(lp - logp_old[t]) : 1.f;
    ratio[t] = r;
    clipped[t] = fminf(fmaxf(r, 1.f - eps_lo), 1.f + eps_hi);
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

size_t kl_fwd_ws_bytes(int n, int H, int V) {
  const int n_chunks = vocab_pad(V) / 128;
  return align256(size_t(n) * n_chunks * sizeof(float4)) +
         align256(size_t(n) * n_chunks * sizeof(float2)) + align256(size_t(H) * sizeof(u16)) +
         256;
}

size_t kl_bwd_ws_bytes(int n, int H, int V) {
  return align256(size_t(n) * vocab_pad(V) * sizeof(u16)) + dh_part_bytes(n, H) +
         align256(size_t(H) * sizeof(u16)) + 256;
}

__global__ __launch_bounds__(256) void zero_u16_kernel(u16* p, int n) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = 0;
}

static hipError_t zero_row(u16* p, int H, hipStream_t stream) {
  hipLaunchKernelGGL(zero_u16_kernel, dim3((H + 255) / 256), dim3(256), 0, stream, p, H);
  return hipGetLastError();
}

size_t logprob_fwd_ws_bytes(int T, int H, int V) {
  (void)H;
  const int n_chunks = vocab_pad(V) / 128;
  return align256(size_t(T) * n_chunks * sizeof(float2)) + align256(size_t(T) * sizeof(float)) +
         256;
}

size_t logprob_bwd_ws_bytes(int T, int H, int V) {
  return align256(size_t(T) * vocab_pad(V) * sizeof(u16)) + dh_part_bytes(T, H) + 256;
}

static char* align_ptr(void* p) {
  return reinterpret_cast<char*>((reinterpret_cast<uintptr_t>(p) + 255) & ~uintptr_t(255));
}


static dim3 gemm_grid(const LmArgs& a) {
  const int splits = a.k_split > 1 ? a.k_split : 1;
  const int per_xcd = (a.nA * a.nT * splits + kNumXcd - 1) / kNumXcd;
  return dim3(per_xcd * kNumXcd);
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



// dh[T, H] = G[T, Vp] W[Vp, H] (bf16 out), split over the vocabulary when the
// output alone would leave CUs idle; `part` is the fp32 partial area of the
// workspace (dh_part_bytes).
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
    hipLaunchKernelGGL((lm_gemm_kernel<kModeDh, NWAVES>), gemm_grid(b), dim3(NWAVES * 64), 0,
                       stream, b);
    if (splits > 1) {
      const size_t n4 = size_t(b.T) * b.H / 4;
      hipLaunchKernelGGL(dh_reduce_kernel, dim3(unsigned((n4 + 255) / 256)), dim3(256), 0, stream,
                         part, b.dh, splits, n4);
    }
  }
  return hipGetLastError();
}

hipError_t launch_logprob_fwd(int T, int H, int V, float eps_lo, float eps_hi, const void* hidden,
                              const void* weight, const int32_t* target, const float* logp_old,
                              float* logp, float* ratio, float* clipped, float* lse, void* ws,
                              hipStream_t stream) {
  LmArgs a{};
  a.h = static_cast<const u16*>(hidden);
  a.w = static_cast<const u16*>(weight);
  a.tgt = target;
  a.T = T;
  a.H = H;
  a.V = V;
  a.Vp = vocab_pad(V);
  a.n_chunks = a.Vp / 128;
  char* base = align_ptr(ws);
  a.part = reinterpret_cast<float2*>(base);
  a.tlogit = reinterpret_cast<float*>(base + align256(size_t(T) * a.n_chunks * sizeof(float2)));
  a.nA = a.Vp / BA;
  a.nT = (T + BT - 1) / BT;
  {
    ProfScope p("lm_logits", stream);
    hipLaunchKernelGGL((lm_gemm_kernel<kModeLogits, NWAVES>), gemm_grid(a), dim3(NWAVES * 64), 0,
                       stream, a);
  }
  {
    ProfScope p("lm_combine", stream);
    hipLaunchKernelGGL(lm_combine_kernel, dim3((T + 3) / 4), dim3(256), 0, stream, a, logp_old,
                       logp, ratio, clipped, lse, eps_lo, eps_hi);
  }
  return hipGetLastError();
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
  u16* G = reinterpret_cast<u16*>(align_ptr(ws));
  a.Gout = G;
  a.G = G;
  a.dh = static_cast<u16*>(dhidden);
  a.nA = a.Vp / BA;
  a.nT = (T + BT - 1) / BT;
  {
    ProfScope p("lm_grad", stream);
    hipLaunchKernelGGL((lm_gemm_kernel<kModeGrad, NWAVES>), gemm_grid(a), dim3(NWAVES * 64), 0,
                       stream, a);
  }
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  float* part = reinterpret_cast<float*>(reinterpret_cast<char*>(G) +
                                         align256(size_t(T) * a.Vp * sizeof(u16)));
  return launch_dh(a, part, "lm_dh", stream);
}

// dW = G^T H from the G that launch_logprob_bwd left in its workspace.
hipError_t launch_logprob_dweight(int T, int H, int V, const void* hidden, const void* ws,
                                  float* dw, hipStream_t stream) {
  LmArgs a{};
  a.h = static_cast<const u16*>(hidden);
  a.G = reinterpret_cast<const u16*>(align_ptr(const_cast<void*>(ws)));
  a.dw = dw;
  a.T = T;
  a.H = H;
  a.V = V;
  a.Vp = vocab_pad(V);
  a.nA = a.Vp / BA;
  a.nT = (H + BT - 1) / BT;
  ProfScope p("lm_dw", stream);
  hipLaunchKernelGGL((lm_gemm_kernel<kModeDw, NWAVES>), gemm_grid(a), dim3(NWAVES * 64), 0,
                     stream, a);
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
    hipLaunchKernelGGL((lm_gemm_kernel<kModeKL, NWAVES>), gemm_grid(a), dim3(NWAVES * 64), 0,
                       stream, a);
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
  u16* G = reinterpret_cast<u16*>(align_ptr(ws));
  a.Gout = G;
  a.nA = a.Vp / BA;
  a.nT = (a.T + BT - 1) / BT;
  u16* zrow = reinterpret_cast<u16*>(reinterpret_cast<char*>(G) +
                                     align256(size_t(n) * a.Vp * sizeof(u16)) +
                                     dh_part_bytes(n, H));
  a.zero_row = zrow;
  if (hipError_t e = zero_row(zrow, H, stream); e != hipSuccess) return e;
  {
    ProfScope p("kl_grad", stream);
    hipLaunchKernelGGL((lm_gemm_kernel<kModeKLGrad, NWAVES>), gemm_grid(a), dim3(NWAVES * 64), 0,
                       stream, a);
  }
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  // dh = G W over the leaves
  LmArgs b{};
  b.w = a.w;
  b.G = G;
  b.dh = static_cast<u16*>(dh);
  b.T = n;
  b.H = H;
  b.V = V;
  b.Vp = a.Vp;
  float* part = reinterpret_cast<float*>(reinterpret_cast<char*>(G) +
                                         align256(size_t(n) * a.Vp * sizeof(u16)));
  return launch_dh(b, part, "kl_dh", stream);
}

}  // namespace mv
