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

namespace {

// Shared by both packings.  Replicated (shared = false): segment k holds the
// whole branch sequence S_k = (keys live just before J_k, in physical order)
// ++ (rows J_k .. J_{k+1}), under a block-diagonal causal mask.  Shared trunk
// (shared = true): S_k begins with the d_k tokens it shares with S_{k-1} (the
// tokens before the first one edit k removes, at the same positions, so
// their keys and values are the same at every layer); segment k holds only
// S_k[d_k:], and its rows read the shared prefix from the slots of earlier
// segments.  That visibility is again one lifetime per slot: it is the record
// over the packed stream whose edit at the start of segment k evicts the
// slots holding S_{k-1}[d_k:].
mv_status build_pack(const mv_trajectory* trajs, int32_t n_traj, int32_t total_tokens,
                     bool shared, mv_branch_pack** out) {
  if (out == nullptr) return bad(MV_ERR_INVALID_ARG, "out is null");
  *out = nullptr;
  // validates the record and gives the key lifetimes
  mv_view_mask* live = nullptr;
  if (mv_status st = mv_build_view_mask(trajs, n_traj, total_tokens, &live); st != MV_OK)
    return st;
  mv_branch_pack* p = nullptr;
  try {
    p = new mv_branch_pack();
    p->T = total_tokens;
    p->seg_begin.push_back(0);
    int64_t pairs = 0;
    // shared trunk: one record per trajectory over its packed slots
    std::vector<mv_trajectory> rec;
    std::vector<std::vector<mv_edit>> rec_edits;
    std::vector<std::vector<mv_span>> rec_spans;
    for (int32_t t = 0; t < n_traj; ++t) {
      const mv_trajectory& tr = trajs[t];
      std::vector<int32_t> bounds{tr.begin};
      for (int32_t k = 0; k < tr.n_edits; ++k) bounds.push_back(tr.edits[k].junction);
      bounds.push_back(tr.end);
      const int32_t traj_slot0 = int32_t(p->src.size());
      std::vector<int32_t> prev_seq, prev_slots;   // S_{k-1} and the slots holding it
      std::vector<std::pair<int32_t, std::vector<int32_t>>> evictions;   // (junction, slots)
      for (size_t k = 0; k + 1 < bounds.size(); ++k) {
        const int32_t first = bounds[k], end = bounds[k + 1];
        std::vector<int32_t> seq;
        for (int32_t j = tr.begin; j < first; ++j)
          if (live->visible(first, j)) seq.push_back(j);   // in row `first`'s view
        const size_t n_before = seq.size();
        for (int32_t r = first; r < end; ++r) seq.push_back(r);
        size_t d = 0;   // common prefix with the previous branch
        if (shared && k > 0)
          while (d < prev_seq.size() && d < seq.size() && prev_seq[d] == seq[d]) ++d;
        std::vector<int32_t> slots(prev_slots.begin(), prev_slots.begin() + d);
        const int32_t seg0 = int32_t(p->src.size());
        if (shared && k > 0 && d < prev_slots.size())
          evictions.push_back({seg0, std::vector<int32_t>(prev_slots.begin() + d, prev_slots.end())});
        for (size_t q = d; q < seq.size(); ++q) {
          const int32_t j = seq[q];
          slots.push_back(int32_t(p->src.size()));
          p->src.push_back(j);
          p->pos.push_back(int32_t(q));
          const bool own = q >= n_before;
          p->owner.push_back(own ? 1 : 0);
          p->target.push_back(own && j + 1 < tr.end ? j + 1 : -1);
        }
        if (!shared) pairs += int64_t(seq.size()) * (int64_t(seq.size()) + 1) / 2;
        p->seg_begin.push_back(int32_t(p->src.size()));
        prev_seq.swap(seq);
        prev_slots.swap(slots);
      }
      if (shared) {
        // the record of this trajectory's slots: each eviction as sorted spans
        std::vector<mv_edit> edits;
        for (auto& ev : evictions) {
          std::vector<int32_t>& sl = ev.second;
          std::sort(sl.begin(), sl.end());
          rec_spans.emplace_back();
          for (int32_t x : sl) {
            if (!rec_spans.back().empty() && rec_spans.back().back().end == x)
              rec_spans.back().back().end = x + 1;
            else
              rec_spans.back().push_back(mv_span{x, x + 1});
          }
          mv_edit e{};
          e.junction = ev.first;
          e.n_evict = int32_t(rec_spans.back().size());
          e.summary = mv_span{0, 0};
          edits.push_back(e);
        }
        rec_edits.push_back(std::move(edits));
        rec.push_back(mv_trajectory{traj_slot0, int32_t(p->src.size()), 0, nullptr});
      }
    }
    mv_view_mask_free(live);
    live = nullptr;
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
    const int32_t n_seg = int32_t(p->seg_begin.size()) - 1;
    mv_status st = MV_OK;
    if (shared) {
      // (edit spans are attached only now: the span vectors no longer move)
      size_t si = 0;
      for (size_t t = 0; t < rec.size(); ++t) {
        for (auto& e : rec_edits[t]) e.evict = rec_spans[si++].data();
        rec[t].n_edits = int32_t(rec_edits[t].size());
        rec[t].edits = rec_edits[t].data();
      }
      st = mv_build_view_mask(rec.data(), int32_t(rec.size()), p->N, &p->mask);
      if (st == MV_OK) pairs = p->mask->stats.visible_pairs;
    } else {
      // the block-diagonal causal mask: every segment a trajectory without edits
      std::vector<mv_trajectory> segs(n_seg);
      for (int32_t s = 0; s < n_seg; ++s)
        segs[s] = mv_trajectory{p->seg_begin[s], p->seg_begin[s + 1], 0, nullptr};
      st = mv_build_view_mask(segs.data(), n_seg, p->N, &p->mask);
    }
    if (st != MV_OK) {
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
    delete p;
    return bad(MV_ERR_INVALID_ARG, std::string("host allocation failed: ") + e.what());
  }
}

}  // namespace

extern "C" {

mv_status mv_build_branch_pack(const mv_trajectory* trajs, int32_t n_traj, int32_t total_tokens,
                               mv_branch_pack** out) {
  return build_pack(trajs, n_traj, total_tokens, false, out);
}

mv_status mv_build_shared_trunk_pack(const mv_trajectory* trajs, int32_t n_traj,
                                     int32_t total_tokens, mv_branch_pack** out) {
  return build_pack(trajs, n_traj, total_tokens, true, out);
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

mv_status mv_pack_rows_rope(const mv_branch_pack* p, const void* in, int32_t n_heads,
                            int32_t head_dim, float theta, void* out, hipStream_t stream) {
  if (mv_status st = check_ready(p); st != MV_OK) return st;
  if (n_heads <= 0 || head_dim <= 0 || head_dim % 16 != 0 || head_dim > 256)
    return bad(MV_ERR_UNSUPPORTED, "n_heads > 0 and head_dim a multiple of 16, <= 256 required");
  if (!(theta > 1.f)) return bad(MV_ERR_INVALID_ARG, "theta must be > 1");
  if (in == nullptr || out == nullptr || !aligned16(in) || !aligned16(out))
    return bad(MV_ERR_INVALID_ARG, "null or misaligned tensor");
  if (in == out) return bad(MV_ERR_INVALID_ARG, "out must not alias in");
  return hip_ok(mv::launch_pack_rope(*p, in, n_heads, head_dim, theta, out, stream),
                "pack+rope launch");
}

mv_status mv_unpack_rows_sum_rope(const mv_branch_pack* p, const void* in, int32_t n_heads,
                                  int32_t head_dim, float theta, int32_t out_fp32, void* out,
                                  hipStream_t stream) {
  if (mv_status st = check_ready(p); st != MV_OK) return st;
  if (n_heads <= 0 || head_dim <= 0 || head_dim % 16 != 0 || head_dim > 256)
    return bad(MV_ERR_UNSUPPORTED, "n_heads > 0 and head_dim a multiple of 16, <= 256 required");
  if (!(theta > 1.f)) return bad(MV_ERR_INVALID_ARG, "theta must be > 1");
  if (in == nullptr || out == nullptr || !aligned16(in) || !aligned16(out))
    return bad(MV_ERR_INVALID_ARG, "null or misaligned tensor");
  if (in == out) return bad(MV_ERR_INVALID_ARG, "out must not alias in");
  return hip_ok(mv::launch_unpack_rope(*p, in, n_heads, head_dim, theta, out_fp32 != 0, out,
                                       stream),
                "unpack+rope launch");
}

}  // extern "C"
