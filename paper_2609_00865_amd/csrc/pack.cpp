// Host construction of the branch-replicated packing (Appendix G): one
// segment per branch layer (Appendix B.1), holding the keys live just before
// the layer's first row and then the layer's rows, with position ids that
// restart per segment.  The live keys before row J are the keys j < J whose
// lifetime (Eq. "4d-mask-def"; several intervals for a key that an edit
// restores) holds row J; no edit fires inside a layer, so causal attention
// over the segment reproduces every row's view.
#include <algorithm>
#include <sstream>

#include "mv_internal.h"

namespace {

mv_status bad(mv_status s, const std::string& msg) {
  mv::set_error(msg);
  return s;
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

mv_status check_ready(const mv_branch_pack* p) {
  if (p == nullptr) return bad(MV_ERR_INVALID_ARG, "null pack");
  if (p->dev == nullptr) return bad(MV_ERR_STATE, "pack layout not uploaded");
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return bad(MV_ERR_HIP, "hipGetDevice failed");
  if (dev != p->device) return bad(MV_ERR_STATE, "pack uploaded to another device");
  return MV_OK;
}

mv_status hip_ok(hipError_t e, const char* what) {
  if (e == hipSuccess) return MV_OK;
  return bad(MV_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

}  // namespace

extern "C" {

mv_status mv_build_branch_pack(const mv_trajectory* trajs, int32_t n_traj, int32_t total_tokens,
                               mv_branch_pack** out) {
  if (out == nullptr) return bad(MV_ERR_INVALID_ARG, "out is null");
  *out = nullptr;
  // validates the record and gives the key lifetimes
  mv_view_mask* live = nullptr;
  if (mv_status st = mv_build_view_mask(trajs, n_traj, total_tokens, &live); st != MV_OK)
    return st;
  try {
    auto* p = new mv_branch_pack();
    p->T = total_tokens;
    p->seg_begin.push_back(0);
    int64_t pairs = 0;
    for (int32_t t = 0; t < n_traj; ++t) {
      const mv_trajectory& tr = trajs[t];
      std::vector<int32_t> bounds{tr.begin};
      for (int32_t k = 0; k < tr.n_edits; ++k) bounds.push_back(tr.edits[k].junction);
      bounds.push_back(tr.end);
      for (size_t k = 0; k + 1 < bounds.size(); ++k) {
        const int32_t first = bounds[k], end = bounds[k + 1];
        int32_t p_in_seg = 0;
        for (int32_t j = tr.begin; j < first; ++j) {
          if (!live->visible(first, j)) continue;  // not in row `first`'s view
          p->src.push_back(j);
          p->pos.push_back(p_in_seg++);
          p->owner.push_back(0);
          p->target.push_back(-1);
        }
        for (int32_t r = first; r < end; ++r) {
          p->src.push_back(r);
          p->pos.push_back(p_in_seg++);
          p->owner.push_back(1);
          p->target.push_back(r + 1 < tr.end ? r + 1 : -1);
        }
        pairs += int64_t(p_in_seg) * (p_in_seg + 1) / 2;
        p->seg_begin.push_back(int32_t(p->src.size()));
      }
    }
    mv_view_mask_free(live);
    if (p->src.size() > size_t(1) << 30) {
      delete p;
      return bad(MV_ERR_UNSUPPORTED, "packed stream longer than 2^30 slots");
    }
    p->N = int32_t(p->src.size());
    // copies of each physical token, in slot order
    p->copy_ptr.assign(p->T + 1, 0);
    for (int32_t s : p->src) ++p->copy_ptr[s + 1];
    int32_t max_copies = 0;
    for (int32_t t = 0; t < p->T; ++t) {
      max_copies = std::max(max_copies, p->copy_ptr[t + 1]);
      p->copy_ptr[t + 1] += p->copy_ptr[t];
    }
    p->copy_slot.resize(p->N);
    std::vector<int32_t> fill(p->copy_ptr.begin(), p->copy_ptr.end() - 1);
    for (int32_t i = 0; i < p->N; ++i) p->copy_slot[fill[p->src[i]]++] = i;
    // the block-diagonal causal mask: every segment a trajectory without edits
    const int32_t n_seg = int32_t(p->seg_begin.size()) - 1;
    std::vector<mv_trajectory> segs(n_seg);
    for (int32_t s = 0; s < n_seg; ++s)
      segs[s] = mv_trajectory{p->seg_begin[s], p->seg_begin[s + 1], 0, nullptr};
    if (mv_status st = mv_build_view_mask(segs.data(), n_seg, p->N, &p->mask); st != MV_OK) {
      delete p;
      return st;
    }
    p->stats = mv_pack_stats{p->T, p->N, n_seg, max_copies, pairs};
    size_t off = 0;
    const size_t sizes[4] = {size_t(p->N), size_t(p->N), size_t(p->T) + 1, size_t(p->N)};
    for (int i = 0; i < 4; ++i) {
      p->off[i] = off;
      off += align256(sizes[i] * sizeof(int32_t));
    }
    p->bytes = off;
    *out = p;
    return MV_OK;
  } catch (const std::exception& e) {
    mv_view_mask_free(live);
    return bad(MV_ERR_INVALID_ARG, std::string("host allocation failed: ") + e.what());
  }
}

mv_status mv_branch_pack_stats(const mv_branch_pack* p, mv_pack_stats* out) {
  if (p == nullptr || out == nullptr) return bad(MV_ERR_INVALID_ARG, "null argument");
  *out = p->stats;
  return MV_OK;
}

mv_status mv_branch_pack_layout(const mv_branch_pack* p, int32_t* src, int32_t* pos,
                                uint8_t* owner, int32_t* target, int32_t* seg_begin) {
  if (p == nullptr) return bad(MV_ERR_INVALID_ARG, "null pack");
  if (src) std::copy(p->src.begin(), p->src.end(), src);
  if (pos) std::copy(p->pos.begin(), p->pos.end(), pos);
  if (owner) std::copy(p->owner.begin(), p->owner.end(), owner);
  if (target) std::copy(p->target.begin(), p->target.end(), target);
  if (seg_begin) std::copy(p->seg_begin.begin(), p->seg_begin.end(), seg_begin);
  return MV_OK;
}

mv_view_mask* mv_branch_pack_mask(mv_branch_pack* p) { return p ? p->mask : nullptr; }

size_t mv_branch_pack_device_bytes(const mv_branch_pack* p) { return p ? p->bytes : 0; }

mv_status mv_branch_pack_upload(mv_branch_pack* p, void* dev_buf, size_t bytes,
                                hipStream_t stream) {
  if (p == nullptr || dev_buf == nullptr) return bad(MV_ERR_INVALID_ARG, "null pack or buffer");
  if ((reinterpret_cast<uintptr_t>(dev_buf) & 255) != 0)
    return bad(MV_ERR_INVALID_ARG, "pack buffer must be 256-byte aligned");
  if (bytes < p->bytes) {
    std::ostringstream os;
    os << "pack buffer has " << bytes << " bytes, needs " << p->bytes;
    return bad(MV_ERR_WORKSPACE, os.str());
  }
  const std::vector<int32_t>* arrs[4] = {&p->src, &p->pos, &p->copy_ptr, &p->copy_slot};
  char* base = static_cast<char*>(dev_buf);
  for (int i = 0; i < 4; ++i) {
    if (arrs[i]->empty()) continue;
    if (mv_status st = hip_ok(hipMemcpyAsync(base + p->off[i], arrs[i]->data(),
                                             arrs[i]->size() * sizeof(int32_t),
                                             hipMemcpyHostToDevice, stream),
                              "pack upload");
        st != MV_OK)
      return st;
  }
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return bad(MV_ERR_HIP, "hipGetDevice failed");
  p->dev = dev_buf;
  p->device = dev;
  auto at = [&](int i) { return reinterpret_cast<const int32_t*>(base + p->off[i]); };
  p->d_src = at(0);
  p->d_pos = at(1);
  p->d_copy_ptr = at(2);
  p->d_copy_slot = at(3);
  return MV_OK;
}

void mv_branch_pack_free(mv_branch_pack* p) {
  if (p == nullptr) return;
  mv_view_mask_free(p->mask);
  delete p;
}

mv_status mv_pack_rows(const mv_branch_pack* p, const void* in, int32_t width, void* out,
                       hipStream_t stream) {
  if (mv_status st = check_ready(p); st != MV_OK) return st;
  if (width <= 0 || width % 8 != 0) return bad(MV_ERR_UNSUPPORTED, "width must be a positive multiple of 8");
  if (in == nullptr || out == nullptr || !aligned16(in) || !aligned16(out))
    return bad(MV_ERR_INVALID_ARG, "null or misaligned tensor");
  return hip_ok(mv::launch_pack_rows(*p, in, width, out, stream), "pack launch");
}

mv_status mv_unpack_rows_sum(const mv_branch_pack* p, const void* in, int32_t width,
                             int32_t out_fp32, void* out, hipStream_t stream) {
  if (mv_status st = check_ready(p); st != MV_OK) return st;
  if (width <= 0 || width % 8 != 0) return bad(MV_ERR_UNSUPPORTED, "width must be a positive multiple of 8");
  if (in == nullptr || out == nullptr || !aligned16(in) || !aligned16(out))
    return bad(MV_ERR_INVALID_ARG, "null or misaligned tensor");
  return hip_ok(mv::launch_unpack_sum(*p, in, width, out_fp32 != 0, out, stream), "unpack launch");
}

mv_status mv_rope(const mv_branch_pack* p, const void* x, int32_t n_heads, int32_t head_dim,
                  float theta, int32_t direction, void* out, hipStream_t stream) {
  if (mv_status st = check_ready(p); st != MV_OK) return st;
  if (n_heads <= 0 || head_dim <= 0 || head_dim % 2 != 0 || head_dim > 256)
    return bad(MV_ERR_UNSUPPORTED, "n_heads > 0 and an even head_dim <= 256 required");
  if (!(theta > 1.f)) return bad(MV_ERR_INVALID_ARG, "theta must be > 1");
  if (direction != 1 && direction != -1) return bad(MV_ERR_INVALID_ARG, "direction must be +1 or -1");
  if (x == nullptr || out == nullptr) return bad(MV_ERR_INVALID_ARG, "null tensor");
  return hip_ok(mv::launch_rope(*p, x, n_heads, head_dim, theta, direction, out, stream),
                "rope launch");
}

}  // extern "C"
