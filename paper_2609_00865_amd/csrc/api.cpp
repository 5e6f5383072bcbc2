// C ABI of libmv: argument validation, workspace sizing and kernel dispatch.
// Validation is complete before anything is enqueued, so a failing call
// launches nothing.
#include <atomic>
#include <cmath>
#include <cstring>
#include <mutex>
#include <sstream>

#include "mv_internal.h"

namespace mv {

thread_local std::string g_last_error;

void set_error(const std::string& msg) { g_last_error = msg; }

namespace {
struct ProfRecord {
  std::string name;
  hipEvent_t start, stop;
};
std::atomic<bool> g_prof_on{false};
std::mutex g_prof_mu;
std::vector<ProfRecord> g_prof;

void prof_clear_locked() {
  for (auto& r : g_prof) {
    (void)hipEventDestroy(r.start);
    (void)hipEventDestroy(r.stop);
  }
  g_prof.clear();
}
}  // namespace

ProfScope::ProfScope(const char* name, hipStream_t stream, bool allowed)
    : name_(name), stream_(stream) {
  if (!allowed || !g_prof_on.load(std::memory_order_relaxed)) return;
  if (hipEventCreate(&start_) != hipSuccess) {
    start_ = nullptr;
    return;
  }
  (void)hipEventRecord(start_, stream_);
}

ProfScope::~ProfScope() {
  if (start_ == nullptr) return;
  hipEvent_t stop = nullptr;
  if (hipEventCreate(&stop) != hipSuccess) {
    (void)hipEventDestroy(start_);
    return;
  }
  (void)hipEventRecord(stop, stream_);
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof.push_back({name_, start_, stop});
}

hipError_t launch_attn_fwd(const mv_view_mask& m, int Hq, int Hkv, int D, float scale,
                           const void* q, const void* k, const void* v, void* o, float* lse,
                           hipStream_t stream);
hipError_t launch_attn_bwd(const mv_view_mask& m, int Hq, int Hkv, int D, float scale,
                           const void* q, const void* k, const void* v, const void* o,
                           const void* dout, const float* lse, void* dq, void* dk, void* dv,
                           void* ws, hipStream_t stream, bool profile = true);
size_t attn_bwd_ws_bytes(const mv_view_mask& m, int Hq, int Hkv, int D);
hipError_t attn_bwd_scratch(void** ptr);
hipError_t launch_materialize(const mv_view_mask& m, int row_begin, int row_end, uint32_t* bits,
                              hipStream_t stream);
hipError_t launch_ppo_clip(int n, const float* ratio, const float* adv, float eps_lo,
                           float eps_hi, float scale, float* out, hipStream_t stream);
size_t logprob_fwd_ws_bytes(int T, int H, int V);
size_t logprob_bwd_ws_bytes(int T, int H, int V);
hipError_t launch_logprob_fwd(int T, int H, int V, float eps_lo, float eps_hi, const void* hidden,
                              const void* weight, const int32_t* target, const float* logp_old,
                              float* logp, float* ratio, float* clipped, float* lse, void* ws,
                              hipStream_t stream);
hipError_t launch_logprob_bwd(int T, int H, int V, const void* hidden, const void* weight,
                              const int32_t* target, const float* lse, const float* dlogp,
                              void* dhidden, void* ws, hipStream_t stream);
hipError_t launch_logprob_dweight(int T, int H, int V, const void* hidden, const void* ws,
                                  float* dw, hipStream_t stream);
int* logprob_status_word(const void* ws);
size_t logprob_grpo_ws_bytes(int T, int H, int V, int n_traj);
hipError_t launch_logprob_grpo(int T, int H, int V, float eps_lo, float eps_hi,
                               const void* hidden, const void* weight, const int32_t* target,
                               const float* logp_old, int n_traj, int G, float g_eps_lo,
                               float g_eps_hi, float beta, float adv_eps, const int32_t* traj_ptr,
                               const float* reward, const float* logp_ref, const uint8_t* mask,
                               float* logp, float* ratio, float* clipped, float* lse,
                               float* adv_out, float* dlogp, float* stats, void* ws,
                               hipStream_t stream);
size_t grpo_ws_bytes(int T, int n_traj);
hipError_t launch_grpo(int T, int n_traj, int G, float eps_lo, float eps_hi, float beta,
                       float adv_eps, const int32_t* traj_ptr, const float* reward,
                       const float* logp, const float* logp_old, const float* logp_ref,
                       const uint8_t* mask, float* adv_out, float* dlogp, float* stats, void* ws,
                       hipStream_t stream);
size_t kl_fwd_ws_bytes(int n, int H, int V);
size_t kl_bwd_ws_bytes(int n, int H, int V);
hipError_t launch_kl_fwd(int n, int H, int V, const void* hT, int nT, const int32_t* rowsT,
                         const void* hS, int nS, const int32_t* rowsS, const void* weight,
                         float* kl, float* lseT, float* lseS, void* ws, hipStream_t stream);
hipError_t launch_kl_bwd(int n, int H, int V, const void* hT, int nT, const int32_t* rowsT,
                         const void* hS, int nS, const int32_t* rowsS, const void* weight,
                         const float* lseT, const float* lseS, const float* dkl, void* dh,
                         void* ws, hipStream_t stream);

}  // namespace mv

namespace {

mv_status fail(mv_status s, const std::string& msg) {
  mv::set_error(msg);
  return s;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

mv_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return MV_OK;
  return fail(MV_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

mv_status check_attn(const mv_view_mask* m, const mv_attn_shape* s) {
  if (m == nullptr || s == nullptr) return fail(MV_ERR_INVALID_ARG, "null mask or shape");
  if (s->total_tokens != m->T) {
    std::ostringstream os;
    os << "shape.total_tokens " << s->total_tokens << " != mask total_tokens " << m->T;
    return fail(MV_ERR_SHAPE, os.str());
  }
  if (s->n_heads_q <= 0 || s->n_heads_kv <= 0 || s->n_heads_q % s->n_heads_kv != 0)
    return fail(MV_ERR_SHAPE, "n_heads_q must be a positive multiple of n_heads_kv");
  if (s->head_dim != 64 && s->head_dim != 128)
    return fail(MV_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  if (!std::isfinite(s->softmax_scale)) return fail(MV_ERR_INVALID_ARG, "softmax_scale not finite");
  // the kernels address each tensor with 32-bit byte offsets
  if (int64_t(s->total_tokens) * s->n_heads_q * s->head_dim * 2 >= (int64_t(1) << 32))
    return fail(MV_ERR_UNSUPPORTED, "each of Q, K, V, O must be under 4 GiB");
  return MV_OK;
}

mv_status check_uploaded(const mv_view_mask* m) {
  if (m->dev == nullptr) return fail(MV_ERR_STATE, "mask has not been uploaded");
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return fail(MV_ERR_HIP, "hipGetDevice failed");
  if (dev != m->device) return fail(MV_ERR_STATE, "mask was uploaded to another device");
  return MV_OK;
}

float attn_scale(const mv_attn_shape* s) {
  return s->softmax_scale > 0.f ? s->softmax_scale : 1.f / std::sqrt(float(s->head_dim));
}

mv_status check_ptrs(std::initializer_list<const void*> ps) {
  for (const void* p : ps) {
    if (p == nullptr) return fail(MV_ERR_INVALID_ARG, "null device pointer");
    if (!aligned16(p)) return fail(MV_ERR_INVALID_ARG, "device pointer not 16-byte aligned");
  }
  return MV_OK;
}

mv_status check_logprob(const mv_logprob_shape* s) {
  if (s == nullptr) return fail(MV_ERR_INVALID_ARG, "null shape");
  if (s->n_tokens < 0 || s->hidden <= 0 || s->vocab <= 0)
    return fail(MV_ERR_SHAPE, "n_tokens >= 0, hidden > 0, vocab > 0 required");
  if (s->hidden % 64 != 0) return fail(MV_ERR_UNSUPPORTED, "hidden must be a multiple of 64");
  if (int64_t(s->n_tokens) * s->hidden >= (int64_t(1) << 31) ||
      int64_t(s->vocab) * s->hidden >= (int64_t(1) << 31))
    return fail(MV_ERR_UNSUPPORTED, "hidden/weight larger than 2^31 elements");
  if (!(s->eps_low >= 0.f && s->eps_low < 1.f && s->eps_high >= 0.f && std::isfinite(s->eps_high)))
    return fail(MV_ERR_INVALID_ARG, "clip range must satisfy 0 <= eps_low < 1, 0 <= eps_high");
  return MV_OK;
}

mv_status check_grpo(const mv_grpo_shape* s) {
  if (s == nullptr) return fail(MV_ERR_INVALID_ARG, "null shape");
  if (s->n_tokens < 0 || s->n_traj <= 0 || s->group_size <= 0)
    return fail(MV_ERR_SHAPE, "n_tokens >= 0, n_traj > 0, group_size > 0 required");
  if (s->n_traj % s->group_size != 0)
    return fail(MV_ERR_SHAPE, "n_traj must be a multiple of group_size");
  if (!(s->eps_low >= 0.f && s->eps_low < 1.f && s->eps_high >= 0.f && s->eps_high < 1.f))
    return fail(MV_ERR_INVALID_ARG, "clip eps must lie in [0, 1)");
  if (!(s->beta >= 0.f) || !(s->adv_eps >= 0.f))
    return fail(MV_ERR_INVALID_ARG, "beta and adv_eps must be >= 0");
  return MV_OK;
}

mv_status check_kl(const mv_kl_shape* s) {
  if (s == nullptr) return fail(MV_ERR_INVALID_ARG, "null shape");
  if (s->n_leaves < 0 || s->hidden <= 0 || s->vocab <= 0 || s->n_rows_teacher < 0 ||
      s->n_rows_student < 0)
    return fail(MV_ERR_SHAPE, "n_leaves >= 0, hidden > 0, vocab > 0, row counts >= 0 required");
  if (s->hidden % 64 != 0) return fail(MV_ERR_UNSUPPORTED, "hidden must be a multiple of 64");
  if (int64_t(s->vocab) * s->hidden >= (int64_t(1) << 31) || s->n_leaves > (1 << 29))
    return fail(MV_ERR_UNSUPPORTED, "operands larger than 2^31 elements");
  return MV_OK;
}

}  // namespace

extern "C" {

const char* mv_status_string(mv_status s) {
  switch (s) {
    case MV_OK: return "MV_OK";
    case MV_ERR_INVALID_ARG: return "MV_ERR_INVALID_ARG";
    case MV_ERR_BAD_RECORD: return "MV_ERR_BAD_RECORD";
    case MV_ERR_SHAPE: return "MV_ERR_SHAPE";
    case MV_ERR_UNSUPPORTED: return "MV_ERR_UNSUPPORTED";
    case MV_ERR_WORKSPACE: return "MV_ERR_WORKSPACE";
    case MV_ERR_HIP: return "MV_ERR_HIP";
    case MV_ERR_STATE: return "MV_ERR_STATE";
  }
  return "MV_ERR_UNKNOWN";
}

const char* mv_last_error(void) { return mv::g_last_error.c_str(); }

int32_t mv_version(void) { return (1 << 16) | 0; }

mv_status mv_view_mask_materialize(const mv_view_mask* m, int32_t row_begin, int32_t row_end,
                                   uint32_t* dev_bits, hipStream_t stream) {
  if (m == nullptr || dev_bits == nullptr) return fail(MV_ERR_INVALID_ARG, "null argument");
  if (row_begin < 0 || row_end > m->T || row_begin > row_end)
    return fail(MV_ERR_INVALID_ARG, "row range outside [0, total_tokens]");
  if (mv_status s = check_uploaded(m); s != MV_OK) return s;
  return hip_status(mv::launch_materialize(*m, row_begin, row_end, dev_bits, stream),
                    "materialize launch");
}

mv_status mv_attn_fwd(const mv_view_mask* m, const mv_attn_shape* s, const void* q, const void* k,
                      const void* v, void* o, float* lse, hipStream_t stream) {
  if (mv_status st = check_attn(m, s); st != MV_OK) return st;
  if (mv_status st = check_ptrs({q, k, v, o, lse}); st != MV_OK) return st;
  if (mv_status st = check_uploaded(m); st != MV_OK) return st;
  return hip_status(mv::launch_attn_fwd(*m, s->n_heads_q, s->n_heads_kv, s->head_dim,
                                        attn_scale(s), q, k, v, o, lse, stream),
                    "attention forward launch");
}

size_t mv_attn_bwd_workspace_bytes(const mv_view_mask* m, const mv_attn_shape* s) {
  if (m == nullptr || s == nullptr || check_attn(m, s) != MV_OK) return 0;
  return mv::attn_bwd_ws_bytes(*m, s->n_heads_q, s->n_heads_kv, s->head_dim);
}

mv_status mv_attn_bwd(const mv_view_mask* m, const mv_attn_shape* s, const void* q, const void* k,
                      const void* v, const void* o, const void* dout, const float* lse, void* dq,
                      void* dk, void* dv, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (mv_status st = check_attn(m, s); st != MV_OK) return st;
  if (mv_status st = check_ptrs({q, k, v, o, dout, lse, dq, dk, dv, ws}); st != MV_OK) return st;
  const size_t need = mv::attn_bwd_ws_bytes(*m, s->n_heads_q, s->n_heads_kv, s->head_dim);
  if (ws_bytes < need) {
    std::ostringstream os;
    os << "attention backward workspace has " << ws_bytes << " bytes, needs " << need;
    return fail(MV_ERR_WORKSPACE, os.str());
  }
  if (mv_status st = check_uploaded(m); st != MV_OK) return st;
  return hip_status(mv::launch_attn_bwd(*m, s->n_heads_q, s->n_heads_kv, s->head_dim,
                                        attn_scale(s), q, k, v, o, dout, lse, dq, dk, dv, ws,
                                        stream),
                    "attention backward launch");
}

mv_status mv_attn_bwd_noalloc(const mv_view_mask* m, const mv_attn_shape* s, const void* q,
                              const void* k, const void* v, const void* o, const void* dout,
                              const float* lse, void* dq, void* dk, void* dv,
                              hipStream_t stream) {
  if (mv_status st = check_attn(m, s); st != MV_OK) return st;
  if (mv_status st = check_ptrs({q, k, v, o, dout, lse, dq, dk, dv}); st != MV_OK) return st;
  const size_t need = mv::attn_bwd_ws_bytes(*m, s->n_heads_q, s->n_heads_kv, s->head_dim);
  if (need > MV_ATTN_BWD_NOALLOC_SCRATCH_BYTES) {
    std::ostringstream os;
    os << "attention backward needs " << need << " bytes of scratch; the static scratch of "
       << "mv_attn_bwd_noalloc holds " << size_t(MV_ATTN_BWD_NOALLOC_SCRATCH_BYTES)
       << " (use mv_attn_bwd with a workspace)";
    return fail(MV_ERR_WORKSPACE, os.str());
  }
  if (mv_status st = check_uploaded(m); st != MV_OK) return st;
  void* scratch = nullptr;
  if (hipError_t e = mv::attn_bwd_scratch(&scratch); e != hipSuccess)
    return hip_status(e, "scratch address");
  return hip_status(mv::launch_attn_bwd(*m, s->n_heads_q, s->n_heads_kv, s->head_dim,
                                        attn_scale(s), q, k, v, o, dout, lse, dq, dk, dv, scratch,
                                        stream, /*profile=*/false),
                    "attention backward launch");
}

size_t mv_token_logprob_workspace_bytes(const mv_logprob_shape* s) {
  if (check_logprob(s) != MV_OK) return 0;
  return mv::logprob_fwd_ws_bytes(s->n_tokens, s->hidden, s->vocab);
}

mv_status mv_token_logprob(const mv_logprob_shape* s, const void* hidden, const void* weight,
                           const int32_t* target, const float* logp_old, float* logp, float* ratio,
                           float* clipped, float* lse, void* ws, size_t ws_bytes,
                           hipStream_t stream) {
  if (mv_status st = check_logprob(s); st != MV_OK) return st;
  if (s->n_tokens == 0) return MV_OK;
  if (mv_status st = check_ptrs({hidden, weight, ws}); st != MV_OK) return st;
  if (target == nullptr || logp == nullptr || lse == nullptr)
    return fail(MV_ERR_INVALID_ARG, "target, logp and lse are required");
  if ((logp_old == nullptr) != (ratio == nullptr) || (ratio == nullptr) != (clipped == nullptr))
    return fail(MV_ERR_INVALID_ARG, "logp_old, ratio and clipped must be all set or all null");
  const size_t need = mv::logprob_fwd_ws_bytes(s->n_tokens, s->hidden, s->vocab);
  if (ws_bytes < need) {
    std::ostringstream os;
    os << "log-prob workspace has " << ws_bytes << " bytes, needs " << need;
    return fail(MV_ERR_WORKSPACE, os.str());
  }
  return hip_status(mv::launch_logprob_fwd(s->n_tokens, s->hidden, s->vocab, s->eps_low,
                                           s->eps_high, hidden, weight, target, logp_old, logp,
                                           ratio, clipped, lse, ws, stream),
                    "log-prob forward launch");
}

size_t mv_token_logprob_grpo_workspace_bytes(const mv_logprob_shape* s,
                                             const mv_grpo_shape* g) {
  if (check_logprob(s) != MV_OK || check_grpo(g) != MV_OK) return 0;
  return mv::logprob_grpo_ws_bytes(s->n_tokens, s->hidden, s->vocab, g->n_traj);
}

mv_status mv_token_logprob_grpo(const mv_logprob_shape* s, const mv_grpo_shape* g,
                                const void* hidden, const void* weight, const int32_t* target,
                                const float* logp_old, const int32_t* traj_ptr,
                                const float* reward, const float* logp_ref,
                                const uint8_t* loss_mask, float* logp, float* ratio,
                                float* clipped, float* lse, float* advantage, float* dlogp,
                                mv_grpo_stats* stats, void* ws, size_t ws_bytes,
                                hipStream_t stream) {
  if (mv_status st = check_logprob(s); st != MV_OK) return st;
  if (mv_status st = check_grpo(g); st != MV_OK) return st;
  if (g->n_tokens != s->n_tokens)
    return fail(MV_ERR_SHAPE, "the GRPO shape's n_tokens must equal the log-prob shape's");
  if (traj_ptr == nullptr || reward == nullptr || stats == nullptr || ws == nullptr)
    return fail(MV_ERR_INVALID_ARG, "traj_ptr, reward, stats and workspace are required");
  if (s->n_tokens > 0) {
    if (mv_status st = check_ptrs({hidden, weight}); st != MV_OK) return st;
    if (target == nullptr || logp_old == nullptr || logp == nullptr || ratio == nullptr ||
        clipped == nullptr || lse == nullptr || dlogp == nullptr)
      return fail(MV_ERR_INVALID_ARG,
                  "target, logp_old, logp, ratio, clipped, lse and dlogp are required");
  }
  if (logp_ref == nullptr && g->beta != 0.f)
    return fail(MV_ERR_INVALID_ARG, "beta > 0 needs logp_ref");
  const size_t need = mv::logprob_grpo_ws_bytes(s->n_tokens, s->hidden, s->vocab, g->n_traj);
  if (ws_bytes < need) {
    std::ostringstream os;
    os << "log-prob GRPO workspace has " << ws_bytes << " bytes, needs " << need;
    return fail(MV_ERR_WORKSPACE, os.str());
  }
  return hip_status(
      mv::launch_logprob_grpo(s->n_tokens, s->hidden, s->vocab, s->eps_low, s->eps_high, hidden,
                              weight, target, logp_old, g->n_traj, g->group_size, g->eps_low,
                              g->eps_high, g->beta, g->adv_eps, traj_ptr, reward, logp_ref,
                              loss_mask, logp, ratio, clipped, lse, advantage, dlogp,
                              reinterpret_cast<float*>(stats), ws, stream),
      "log-prob GRPO forward launch");
}

size_t mv_token_logprob_bwd_workspace_bytes(const mv_logprob_shape* s) {
  if (check_logprob(s) != MV_OK) return 0;
  return mv::logprob_bwd_ws_bytes(s->n_tokens, s->hidden, s->vocab);
}

mv_status mv_token_logprob_bwd(const mv_logprob_shape* s, const void* hidden, const void* weight,
                               const int32_t* target, const float* lse, const float* dlogp,
                               void* dhidden, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (mv_status st = check_logprob(s); st != MV_OK) return st;
  if (s->n_tokens == 0) return MV_OK;
  if (mv_status st = check_ptrs({hidden, weight, dhidden, ws}); st != MV_OK) return st;
  if (target == nullptr || lse == nullptr || dlogp == nullptr)
    return fail(MV_ERR_INVALID_ARG, "target, lse and dlogp are required");
  const size_t need = mv::logprob_bwd_ws_bytes(s->n_tokens, s->hidden, s->vocab);
  if (ws_bytes < need) {
    std::ostringstream os;
    os << "log-prob backward workspace has " << ws_bytes << " bytes, needs " << need;
    return fail(MV_ERR_WORKSPACE, os.str());
  }
  return hip_status(mv::launch_logprob_bwd(s->n_tokens, s->hidden, s->vocab, hidden, weight,
                                           target, lse, dlogp, dhidden, ws, stream),
                    "log-prob backward launch");
}

size_t mv_sdcc_kl_workspace_bytes(const mv_kl_shape* s) {
  if (check_kl(s) != MV_OK) return 0;
  return mv::kl_fwd_ws_bytes(s->n_leaves, s->hidden, s->vocab);
}

size_t mv_sdcc_kl_bwd_workspace_bytes(const mv_kl_shape* s) {
  if (check_kl(s) != MV_OK) return 0;
  return mv::kl_bwd_ws_bytes(s->n_leaves, s->hidden, s->vocab);
}

mv_status mv_sdcc_kl(const mv_kl_shape* s, const void* hT, const int32_t* rowsT, const void* hS,
                     const int32_t* rowsS, const void* weight, float* kl, float* lseT, float* lseS,
                     void* ws, size_t ws_bytes, hipStream_t stream) {
  if (mv_status st = check_kl(s); st != MV_OK) return st;
  if (s->n_leaves == 0) return MV_OK;
  if (mv_status st = check_ptrs({hT, hS, weight, ws}); st != MV_OK) return st;
  if (rowsT == nullptr || rowsS == nullptr || kl == nullptr || lseT == nullptr || lseS == nullptr)
    return fail(MV_ERR_INVALID_ARG, "row indices and per-leaf outputs are required");
  const size_t need = mv::kl_fwd_ws_bytes(s->n_leaves, s->hidden, s->vocab);
  if (ws_bytes < need) {
    std::ostringstream os;
    os << "KL workspace has " << ws_bytes << " bytes, needs " << need;
    return fail(MV_ERR_WORKSPACE, os.str());
  }
  return hip_status(mv::launch_kl_fwd(s->n_leaves, s->hidden, s->vocab, hT, s->n_rows_teacher,
                                      rowsT, hS, s->n_rows_student, rowsS, weight, kl, lseT, lseS, ws, stream),
                    "KL forward launch");
}

mv_status mv_sdcc_kl_bwd(const mv_kl_shape* s, const void* hT, const int32_t* rowsT,
                         const void* hS, const int32_t* rowsS, const void* weight,
                         const float* lseT, const float* lseS, const float* dkl, void* dh,
                         void* ws, size_t ws_bytes, hipStream_t stream) {
  if (mv_status st = check_kl(s); st != MV_OK) return st;
  if (s->n_leaves == 0) return MV_OK;
  if (mv_status st = check_ptrs({hT, hS, weight, dh, ws}); st != MV_OK) return st;
  if (rowsT == nullptr || rowsS == nullptr || lseT == nullptr || lseS == nullptr || dkl == nullptr)
    return fail(MV_ERR_INVALID_ARG, "row indices, LSEs and dkl are required");
  const size_t need = mv::kl_bwd_ws_bytes(s->n_leaves, s->hidden, s->vocab);
  if (ws_bytes < need) {
    std::ostringstream os;
    os << "KL backward workspace has " << ws_bytes << " bytes, needs " << need;
    return fail(MV_ERR_WORKSPACE, os.str());
  }
  return hip_status(mv::launch_kl_bwd(s->n_leaves, s->hidden, s->vocab, hT, s->n_rows_teacher,
                                      rowsT, hS, s->n_rows_student, rowsS, weight, lseT, lseS, dkl, dh, ws, stream),
                    "KL backward launch");
}

float mv_sdcc_lambda(int32_t step, int32_t total_steps, float lambda_max, float warmup_frac) {
  const double warm = double(warmup_frac) * double(total_steps);
  if (warm <= 0.0 || step >= warm) return lambda_max;
  if (step <= 0) return 0.f;
  return float(double(lambda_max) * double(step) / warm);
}

mv_status mv_profile_enable(int32_t on) {
  std::lock_guard<std::mutex> lk(mv::g_prof_mu);
  mv::prof_clear_locked();
  mv::g_prof_on.store(on != 0);
  return MV_OK;
}

mv_status mv_profile_read(const char* kernel, double* total_ms, int32_t* count) {
  if (kernel == nullptr || total_ms == nullptr || count == nullptr)
    return fail(MV_ERR_INVALID_ARG, "null argument");
  std::lock_guard<std::mutex> lk(mv::g_prof_mu);
  double tot = 0.0;
  int32_t n = 0;
  for (auto& r : mv::g_prof) {
    if (r.name != kernel) continue;
    if (hipEventSynchronize(r.stop) != hipSuccess) return fail(MV_ERR_HIP, "event wait failed");
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess)
      return fail(MV_ERR_HIP, "event timing failed");
    tot += ms;
    ++n;
  }
  *total_ms = tot;
  *count = n;
  return MV_OK;
}

mv_status mv_token_logprob_dweight(const mv_logprob_shape* s, const void* hidden,
                                   const void* ws, size_t ws_bytes, float* dweight,
                                   hipStream_t stream) {
  if (mv_status st = check_logprob(s); st != MV_OK) return st;
  if (s->n_tokens == 0) return MV_OK;
  if (mv_status st = check_ptrs({hidden, ws, dweight}); st != MV_OK) return st;
  const size_t need = mv::logprob_bwd_ws_bytes(s->n_tokens, s->hidden, s->vocab);
  if (ws_bytes < need) {
    std::ostringstream os;
    os << "workspace has " << ws_bytes << " bytes, the backward's holds " << need;
    return fail(MV_ERR_WORKSPACE, os.str());
  }
  return hip_status(mv::launch_logprob_dweight(s->n_tokens, s->hidden, s->vocab, hidden, ws,
                                               dweight, stream),
                    "LM-head weight gradient launch");
}

mv_status mv_token_logprob_bad_targets(const void* ws, int32_t* host_count,
                                       hipStream_t stream) {
  if (ws == nullptr || host_count == nullptr) return fail(MV_ERR_INVALID_ARG, "null argument");
  int32_t v = 0;
  if (hipError_t e = hipMemcpyAsync(&v, mv::logprob_status_word(ws), sizeof(v),
                                    hipMemcpyDeviceToHost, stream);
      e != hipSuccess)
    return hip_status(e, "status copy");
  if (hipError_t e = hipStreamSynchronize(stream); e != hipSuccess)
    return hip_status(e, "status wait");
  *host_count = v;
  return MV_OK;
}

size_t mv_grpo_loss_workspace_bytes(const mv_grpo_shape* s) {
  if (check_grpo(s) != MV_OK) return 0;
  return mv::grpo_ws_bytes(s->n_tokens, s->n_traj);
}

mv_status mv_grpo_loss(const mv_grpo_shape* s, const int32_t* traj_ptr, const float* reward,
                       const float* logp, const float* logp_old, const float* logp_ref,
                       const uint8_t* loss_mask, float* advantage, float* dlogp,
                       mv_grpo_stats* stats, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (mv_status st = check_grpo(s); st != MV_OK) return st;
  if (traj_ptr == nullptr || reward == nullptr || stats == nullptr || ws == nullptr)
    return fail(MV_ERR_INVALID_ARG, "traj_ptr, reward, stats and workspace are required");
  if (s->n_tokens > 0 && (logp == nullptr || logp_old == nullptr || dlogp == nullptr))
    return fail(MV_ERR_INVALID_ARG, "logp, logp_old and dlogp are required");
  if (logp_ref == nullptr && s->beta != 0.f)
    return fail(MV_ERR_INVALID_ARG, "beta > 0 needs logp_ref");
  const size_t need = mv::grpo_ws_bytes(s->n_tokens, s->n_traj);
  if (ws_bytes < need) {
    std::ostringstream os;
    os << "GRPO workspace has " << ws_bytes << " bytes, needs " << need;
    return fail(MV_ERR_WORKSPACE, os.str());
  }
  return hip_status(mv::launch_grpo(s->n_tokens, s->n_traj, s->group_size, s->eps_low,
                                    s->eps_high, s->beta, s->adv_eps, traj_ptr, reward, logp,
                                    logp_old, logp_ref, loss_mask, advantage, dlogp,
                                    reinterpret_cast<float*>(stats), ws, stream),
                    "GRPO loss launch");
}

mv_status mv_ppo_clip_dlogp(int32_t n, const float* ratio, const float* adv, float eps_low,
                            float eps_high, float scale, float* dlogp, hipStream_t stream) {
  if (n < 0) return fail(MV_ERR_INVALID_ARG, "n must be >= 0");
  if (n > 0 && (ratio == nullptr || adv == nullptr || dlogp == nullptr))
    return fail(MV_ERR_INVALID_ARG, "null pointer");
  return hip_status(mv::launch_ppo_clip(n, ratio, adv, eps_low, eps_high, scale, dlogp, stream),
                    "ppo clip launch");
}

}  // extern "C"
