// Internal declarations of libmv: the view-mask object, tile constants and
// kernel launchers.  Not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <string>
#include <vector>

#include "../../include/mv.h"

namespace mv {

// Forward / dQ schedule: 128-row query tiles x 64-key key tiles.
constexpr int kFwdTileQ = 128;
constexpr int kFwdTileK = 64;
// dK/dV schedule: 128-key key tiles visited by 64-row query blocks; a key
// tile's row range is cut into work items of at most kBwdChunk query blocks.
constexpr int kBwdTileK = 128;
constexpr int kBwdBlockQ = 64;
constexpr int kBwdChunk = 32;
// Blocks are dealt to the 8 XCDs round-robin by the dispatcher.
constexpr int kNumXcd = 8;

void set_error(const std::string& msg);

// Brackets one kernel launch with HIP events when profiling is enabled (and
// `allowed`: a caller that must not create events passes false).
class ProfScope {
 public:
  ProfScope(const char* name, hipStream_t stream, bool allowed = true);
  ~ProfScope();
  ProfScope(const ProfScope&) = delete;
  ProfScope& operator=(const ProfScope&) = delete;

 private:
  const char* name_;
  hipStream_t stream_;
  hipEvent_t start_ = nullptr;
};

}  // namespace mv

// Device-side view of an uploaded mask (all int32 arrays).
struct mv_mask_dev {
  const int32_t* omega;      // [T] death row of each key
  const int32_t* kt_minmax;  // [n_kt64 * 2] min/max omega per 64-key tile
  const int32_t* q_ptr;      // [n_qt + 1] CSR row pointers per 128-row tile
  const int32_t* k_list;     // [nnz] (kt64 << 1) | full_flag, ascending kt
  const int32_t* qt_order;   // [n_qt] query tiles, heaviest first
  const int32_t* bwd_items;  // [n_items * 4] (kt128, qb_begin, qb_end, slot)
  const int32_t* bwd_tiles;  // [n_kt128 * 4] (min omega, max omega, first slot, n slots)
  const int32_t* bwd_red;    // [n_red] key tiles whose partials are reduced
  const int32_t* iv_ptr;     // [T + 1] per-key ranges of further live intervals
  const int32_t* iv;         // [2 * n_iv] (begin, end) of those intervals
};

struct mv_view_mask {
  int32_t T = 0;
  int32_t n_qt = 0, n_kt64 = 0, n_kt128 = 0;
  std::vector<int32_t> omega, kt_minmax, q_ptr, k_list, qt_order;
  std::vector<int32_t> bwd_items, bwd_tiles, bwd_red;
  std::vector<int32_t> iv_ptr, iv;  // further live intervals of restored keys
  int32_t n_slots = 0;
  int32_t kind = MV_VIEW_LIVE;
  std::vector<int32_t> leaf_token, leaf_teacher, leaf_student;  // diverging leaves
  mv_mask_stats stats{};
  // device copy
  size_t off[10] = {0};
  size_t bytes = 0;
  void* dev = nullptr;
  int device = -1;
  mv_mask_dev d{};
  int32_t first_end(int32_t j) const { return omega[j] & 0x7fffffff; }
  // end of the key's last live interval
  int32_t last_end(int32_t j) const {
    return iv_ptr[j + 1] > iv_ptr[j] ? iv[2 * (iv_ptr[j + 1] - 1) + 1] : first_end(j);
  }
  bool visible(int32_t i, int32_t j) const;
};

struct mv_branch_pack {
  int32_t T = 0, N = 0;
  std::vector<int32_t> src, pos, target, seg_begin;
  std::vector<uint8_t> owner;
  std::vector<int32_t> copy_ptr, copy_slot;  // per physical token, its slots in order
  mv_pack_stats stats{};
  mv_view_mask* mask = nullptr;              // block-diagonal causal mask, owned
  // device copy
  size_t off[4] = {0};
  size_t bytes = 0;
  void* dev = nullptr;
  int device = -1;
  const int32_t* d_src = nullptr;
  const int32_t* d_pos = nullptr;
  const int32_t* d_copy_ptr = nullptr;
  const int32_t* d_copy_slot = nullptr;
};

namespace mv {
hipError_t launch_pack_rows(const mv_branch_pack& p, const void* in, int W, void* out,
                            hipStream_t stream);
hipError_t launch_unpack_sum(const mv_branch_pack& p, const void* in, int W, bool out_fp32,
                             void* out, hipStream_t stream);
hipError_t launch_rope(const mv_branch_pack& p, const void* x, int H, int d, float theta,
                       int direction, void* out, hipStream_t stream);
hipError_t launch_pack_rope(const mv_branch_pack& p, const void* in, int H, int d, float theta,
                            void* out, hipStream_t stream);
hipError_t launch_unpack_rope(const mv_branch_pack& p, const void* in, int H, int d, float theta,
                              bool out_fp32, void* out, hipStream_t stream);
}  // namespace mv
