// Host construction of the view mask: eviction records -> key lifetimes
// omega(j) (Eq. "4d-mask-def", Section 4.2) -> block-sparse tile schedules.
//
// The paper notes that a dense per-query mask is costly (Section 4.3, "Cost
// and deployment splits") and that a real FLOP saving needs a block-sparse
// kernel (Appendix B.3).  Here the mask is never materialised: each key keeps
// one integer, and the passes visit only tiles holding a visible pair.
#include <algorithm>
#include <array>
#include <cstring>
#include <map>
#include <numeric>
#include <sstream>

#include "mv_internal.h"
#include "mv_predicate.h"

namespace {

mv_status bad(mv_status s, const std::string& msg) {
  mv::set_error(msg);
  return s;
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Lifetimes of every key from the record: a key is live from its own row
// until an edit evicts it (omega, the end of its first interval), and again
// from each edit that restores it until the next eviction or the trajectory
// end (the further intervals of keys that re-enter, kept in a per-key list).
mv_status validate_and_fill_lifetimes(const mv_trajectory* trajs, int32_t n_traj, int32_t T,
                                      std::vector<int32_t>& omega, std::vector<int32_t>& iv_ptr,
                                      std::vector<int32_t>& iv) {
  omega.assign(T, 0);
  std::vector<int32_t> open_at(T, -1);     // start of the key's current live interval
  std::vector<uint8_t> first_closed(T, 0);
  std::vector<std::array<int32_t, 3>> extra;  // (key, begin, end)
  int32_t pos = 0;
  auto check_spans = [&](int32_t t, int32_t k, const char* what, const mv_span* sp, int32_t n,
                         int32_t lo, int32_t hi) -> mv_status {
    if (n < 0 || (n > 0 && sp == nullptr))
      return bad(MV_ERR_INVALID_ARG, std::string("edit ") + what + ": null pointer or negative count");
    int32_t prev_end = lo;
    for (int32_t s = 0; s < n; ++s) {
      if (sp[s].begin < prev_end || sp[s].end <= sp[s].begin || sp[s].end > hi) {
        std::ostringstream os;
        os << "trajectory " << t << " edit " << k << " " << what << " span " << s << " ["
           << sp[s].begin << ", " << sp[s].end
           << ") must be non-empty, sorted, disjoint and inside [" << lo << ", " << hi << ")";
        return bad(MV_ERR_BAD_RECORD, os.str());
      }
      prev_end = sp[s].end;
    }
    return MV_OK;
  };
  for (int32_t t = 0; t < n_traj; ++t) {
    const mv_trajectory& tr = trajs[t];
    if (tr.begin != pos || tr.end <= tr.begin || tr.end > T) {
      std::ostringstream os;
      os << "trajectory " << t << " [" << tr.begin << ", " << tr.end
         << ") does not continue the packing at " << pos;
      return bad(MV_ERR_BAD_RECORD, os.str());
    }
    for (int32_t j = tr.begin; j < tr.end; ++j) open_at[j] = j;
    if (tr.n_edits < 0 || (tr.n_edits > 0 && tr.edits == nullptr))
      return bad(MV_ERR_INVALID_ARG, "trajectory edits: null pointer or negative count");
    int32_t last_j = tr.begin;
    for (int32_t k = 0; k < tr.n_edits; ++k) {
      const mv_edit& e = tr.edits[k];
      if (e.junction <= last_j || e.junction >= tr.end) {
        std::ostringstream os;
        os << "trajectory " << t << " edit " << k << ": junction " << e.junction
           << " must be in (" << last_j << ", " << tr.end << ") and increasing";
        return bad(MV_ERR_BAD_RECORD, os.str());
      }
      last_j = e.junction;
      if (mv_status st = check_spans(t, k, "evict", e.evict, e.n_evict, tr.begin, e.junction);
          st != MV_OK)
        return st;
      if (mv_status st =
              check_spans(t, k, "restore", e.restore, e.n_restore, tr.begin, e.junction);
          st != MV_OK)
        return st;
      for (int32_t s = 0; s < e.n_evict; ++s) {
        const mv_span sp = e.evict[s];
        for (int32_t j = sp.begin; j < sp.end; ++j) {
          if (open_at[j] < 0) {
            std::ostringstream os;
            os << "token " << j << " is evicted at row " << e.junction << " but is not live";
            return bad(MV_ERR_BAD_RECORD, os.str());
          }
          if (!first_closed[j]) {
            omega[j] = e.junction;
            first_closed[j] = 1;
          } else {
            extra.push_back({j, open_at[j], e.junction});
          }
          open_at[j] = -1;
        }
        if (e.summary.begin < e.summary.end &&
            std::max(sp.begin, e.summary.begin) < std::min(sp.end, e.summary.end))
          return bad(MV_ERR_BAD_RECORD, "summary block intersects its own eviction set");
      }
      for (int32_t s = 0; s < e.n_restore; ++s) {
        const mv_span sp = e.restore[s];
        for (int32_t j = sp.begin; j < sp.end; ++j) {
          if (open_at[j] >= 0 || open_at[j] == -2) {
            std::ostringstream os;
            os << "token " << j << " is restored at row " << e.junction
               << " but is live (or evicted by the same edit)";
            return bad(MV_ERR_BAD_RECORD, os.str());
          }
        }
      }
      // a token evicted by this edit cannot come back in the same edit
      for (int32_t s = 0; s < e.n_evict; ++s)
        for (int32_t j = e.evict[s].begin; j < e.evict[s].end; ++j) open_at[j] = -2;
      for (int32_t s = 0; s < e.n_restore; ++s)
        for (int32_t j = e.restore[s].begin; j < e.restore[s].end; ++j) {
          if (open_at[j] == -2) {
            std::ostringstream os;
            os << "token " << j << " is evicted and restored by the same edit at row "
               << e.junction;
            return bad(MV_ERR_BAD_RECORD, os.str());
          }
          open_at[j] = e.junction;
        }
      for (int32_t s = 0; s < e.n_evict; ++s)
        for (int32_t j = e.evict[s].begin; j < e.evict[s].end; ++j) open_at[j] = -1;
      if (e.summary.begin != e.summary.end &&
          (e.summary.begin > e.summary.end || e.summary.begin < tr.begin || e.summary.end > tr.end))
        return bad(MV_ERR_BAD_RECORD, "summary block outside its trajectory");
    }
    for (int32_t j = tr.begin; j < tr.end; ++j) {
      if (open_at[j] < 0) continue;
      if (!first_closed[j]) {
        omega[j] = tr.end;
        first_closed[j] = 1;
      } else {
        extra.push_back({j, open_at[j], tr.end});
      }
    }
    pos = tr.end;
  }
  if (pos != T) return bad(MV_ERR_BAD_RECORD, "trajectories do not cover [0, total_tokens)");
  // per-key lists of further intervals, in order
  std::stable_sort(extra.begin(), extra.end(),
                   [](const auto& a, const auto& b) { return a[0] < b[0]; });
  iv_ptr.assign(T + 1, 0);
  iv.clear();
  iv.reserve(2 * extra.size());
  for (const auto& x : extra) {
    ++iv_ptr[x[0] + 1];
    iv.push_back(x[1]);
    iv.push_back(x[2]);
  }
  for (int32_t j = 0; j < T; ++j) iv_ptr[j + 1] += iv_ptr[j];
  for (int32_t j = 0; j < T; ++j)
    if (iv_ptr[j + 1] > iv_ptr[j]) omega[j] |= int32_t(0x80000000u);
  return MV_OK;
}

// Diverging leaves (Definition "trajectory tree", Appendix B.1; Section 5.1):
// a token t of the final compressed walk is scored under the live view of
// row t-1 and, on the final walk, under the row of the last surviving token
// before t.  The two conditioning sets differ iff some key j < t is live at
// row t-1 but not in the final walk, or (a key that re-entered) in the final
// walk but not live at row t-1.  A difference array over t counts those keys
// for every t at once from the keys' intervals.
void build_leaves(mv_view_mask& m, const mv_trajectory* trajs, int32_t n_traj) {
  m.leaf_token.clear();
  m.leaf_teacher.clear();
  m.leaf_student.clear();
  for (int32_t k = 0; k < n_traj; ++k) {
    const int32_t b = trajs[k].begin, e = trajs[k].end;
    // diff over t in [b, e]: key j counts at t iff (t-1 live) != (j final)
    std::vector<int32_t> diff(e - b + 2, 0);
    auto add = [&](int32_t t0, int32_t t1, int32_t v) {  // t in [t0, t1)
      if (t0 >= t1) return;
      diff[t0 - b] += v;
      diff[t1 - b] -= v;
    };
    for (int32_t j = b; j < e; ++j) {
      const bool final = m.last_end(j) == e;
      // live at row t-1 for t-1 in an interval [lo, hi): t in [lo+1, hi+1),
      // restricted to t > j
      std::vector<std::pair<int32_t, int32_t>> ivs{{j, m.first_end(j)}};
      for (int32_t q = m.iv_ptr[j]; q < m.iv_ptr[j + 1]; ++q)
        ivs.push_back({m.iv[2 * q], m.iv[2 * q + 1]});
      if (final) {
        // counts where not live: t in (j, e] minus the live ranges
        add(j + 1, e + 1, 1);
        for (const auto& iv : ivs) add(iv.first + 1, iv.second + 1, -1);
      } else {
        for (const auto& iv : ivs) add(iv.first + 1, iv.second + 1, 1);
      }
    }
    int32_t run = 0, last_survivor = -1;
    for (int32_t t = b + 1; t < e; ++t) {
      run += diff[t - b];
      if (m.last_end(t - 1) == e) last_survivor = t - 1;
      if (m.last_end(t) == e && run > 0 && last_survivor >= 0) {
        m.leaf_token.push_back(t);
        m.leaf_teacher.push_back(t - 1);
        m.leaf_student.push_back(last_survivor);
      }
    }
  }
  m.stats.n_leaves = int32_t(m.leaf_token.size());
}

void build_stats(mv_view_mask& m) {
  const int32_t T = m.T;
  int64_t pairs = 0;
  std::vector<int32_t> diff(T + 1, 0);
  int32_t segs = 0;
  for (int32_t j = 0; j < T; ++j) {
    pairs += m.first_end(j) - j;
    diff[j] += 1;
    diff[m.first_end(j)] -= 1;
    for (int32_t q = m.iv_ptr[j]; q < m.iv_ptr[j + 1]; ++q) {
      pairs += m.iv[2 * q + 1] - m.iv[2 * q];
      diff[m.iv[2 * q]] += 1;
      diff[m.iv[2 * q + 1]] -= 1;
    }
    if (j == 0 || m.omega[j] != m.omega[j - 1]) ++segs;
  }
  int32_t run = 0, mx = 0;
  for (int32_t i = 0; i < T; ++i) {
    run += diff[i];
    mx = std::max(mx, run);
  }
  m.stats.visible_pairs = pairs;
  m.stats.total_tokens = T;
  m.stats.max_view = mx;
  m.stats.n_segments = segs;
}

void build_fwd_schedule(mv_view_mask& m) {
  const int32_t T = m.T, BQ = mv::kFwdTileQ, BK = mv::kFwdTileK;
  m.n_kt64 = (T + BK - 1) / BK;
  m.n_qt = (T + BQ - 1) / BQ;
  m.kt_minmax.resize(2 * size_t(m.n_kt64));
  for (int32_t kt = 0; kt < m.n_kt64; ++kt) {
    // lo: the first row some key of the tile is not live at (full tiles end
    // there); hi: the end of the last live interval of any key (no row from
    // there on sees the tile)
    int32_t lo = INT32_MAX, hi = 0;
    for (int32_t j = kt * BK; j < std::min(T, (kt + 1) * BK); ++j) {
      lo = std::min(lo, m.first_end(j));
      hi = std::max(hi, m.last_end(j));
    }
    m.kt_minmax[2 * kt] = lo;
    m.kt_minmax[2 * kt + 1] = hi;
  }
  m.q_ptr.assign(m.n_qt + 1, 0);
  m.k_list.clear();
  int64_t full = 0, partial = 0, skipped = 0;
  for (int32_t qt = 0; qt < m.n_qt; ++qt) {
    const int32_t i0 = qt * BQ, i1 = std::min(T, i0 + BQ);
    const int32_t kt_end = (i1 - 1) / BK + 1;
    for (int32_t kt = 0; kt < kt_end; ++kt) {
      const int32_t j0 = kt * BK, j1 = std::min(T, j0 + BK);
      const int32_t lo = m.kt_minmax[2 * kt], hi = m.kt_minmax[2 * kt + 1];
      if (j1 - 1 <= i0) {
        // every key precedes every row: visible pairs exist iff some key is
        // still alive at the tile's first row
        if (hi <= i0) {
          ++skipped;
          continue;
        }
        // full tiles skip the predicate, so they must hold no padding keys
        const bool is_full = lo >= i1 && j0 + BK <= T;
        m.k_list.push_back((kt << 1) | (is_full ? 1 : 0));
        (is_full ? full : partial) += 1;
      } else {
        // the tile meets the diagonal: row r = max(j0, i0) sees key r
        m.k_list.push_back(kt << 1);
        ++partial;
      }
    }
    m.q_ptr[qt + 1] = int32_t(m.k_list.size());
  }
  m.qt_order.resize(m.n_qt);
  std::iota(m.qt_order.begin(), m.qt_order.end(), 0);
  std::stable_sort(m.qt_order.begin(), m.qt_order.end(), [&](int32_t a, int32_t b) {
    return (m.q_ptr[a + 1] - m.q_ptr[a]) > (m.q_ptr[b + 1] - m.q_ptr[b]);
  });
  m.stats.tiles_full = int32_t(full);
  m.stats.tiles_partial = int32_t(partial);
  m.stats.fwd_tile_pairs = int64_t(full + partial) * BQ * BK;
  m.stats.tiles_skipped = int32_t(skipped);
}

void build_bwd_schedule(mv_view_mask& m) {
  const int32_t T = m.T, BK = mv::kBwdTileK, BQ = mv::kBwdBlockQ, CH = mv::kBwdChunk;
  m.n_kt128 = (T + BK - 1) / BK;
  m.bwd_tiles.assign(4 * size_t(m.n_kt128), 0);
  m.bwd_items.clear();
  m.bwd_red.clear();
  int32_t slot = 0;
  std::vector<std::array<int32_t, 4>> items;
  for (int32_t kt = 0; kt < m.n_kt128; ++kt) {
    const int32_t j0 = kt * BK, j1 = std::min(T, j0 + BK);
    int32_t lo = INT32_MAX, hi = 0;
    for (int32_t j = j0; j < j1; ++j) {
      lo = std::min(lo, m.first_end(j));
      hi = std::max(hi, m.last_end(j));
    }
    // rows seeing some key of the tile form the contiguous range [j0, hi)
    const int32_t qb0 = j0 / BQ, qb1 = (hi + BQ - 1) / BQ;
    const int32_t n = qb1 - qb0, chunks = (n + CH - 1) / CH;
    m.bwd_tiles[4 * kt + 0] = lo;
    m.bwd_tiles[4 * kt + 1] = hi;
    if (chunks == 1) {
      items.push_back({kt, qb0, qb1, -1});
      m.bwd_tiles[4 * kt + 2] = -1;
      m.bwd_tiles[4 * kt + 3] = 0;
    } else {
      m.bwd_tiles[4 * kt + 2] = slot;
      m.bwd_tiles[4 * kt + 3] = chunks;
      for (int32_t c = 0; c < chunks; ++c)
        items.push_back({kt, qb0 + c * CH, std::min(qb1, qb0 + (c + 1) * CH), slot + c});
      slot += chunks;
      m.bwd_red.push_back(kt);
    }
  }
  // Work order.  Items of eight neighbouring key tiles with the same chunk
  // index walk nearly the same query blocks (each start two blocks later), so
  // they form a group that should run side by side on one XCD, sharing the
  // Q / dO stream in its L2.  Groups go longest first (a greedy balance of
  // the tail); the dispatcher deals consecutive items to the 8 XCDs round
  // robin, so run r of 8 items in group order is placed at the positions
  // that XCD r % 8 takes next.
  std::vector<std::array<int32_t, 4>> order;
  {
    std::map<std::pair<int32_t, int32_t>, std::vector<std::array<int32_t, 4>>> groups;
    for (const auto& it : items) {
      const int32_t c = (it[1] - it[0] * BK / BQ) / CH;
      groups[{it[0] / 8, c}].push_back(it);
    }
    std::vector<std::vector<std::array<int32_t, 4>>*> gl;
    for (auto& kv : groups) gl.push_back(&kv.second);
    auto len = [](const std::vector<std::array<int32_t, 4>>* g) {
      int32_t n = 0;
      for (const auto& it : *g) n = std::max(n, it[2] - it[1]);
      return n;
    };
    std::stable_sort(gl.begin(), gl.end(), [&](auto* a, auto* b) { return len(a) > len(b); });
    for (auto* g : gl) order.insert(order.end(), g->begin(), g->end());
  }
  const size_t n_items = order.size(), full = n_items / 64 * 64;
  for (size_t p = 0; p < n_items; ++p) {
    size_t q = p;
    if (p < full) {
      const size_t local = p / 8, x = p % 8;
      q = ((local / 8) * 8 + x) * 8 + local % 8;
    }
    items[p] = order[q];
  }
  int64_t bwd_pairs = 0;
  for (const auto& it : items) bwd_pairs += int64_t(it[2] - it[1]) * BQ * BK;
  m.stats.bwd_tile_pairs = bwd_pairs;
  m.bwd_items.reserve(items.size() * 4);
  for (const auto& it : items) m.bwd_items.insert(m.bwd_items.end(), it.begin(), it.end());
  m.n_slots = slot;
  m.stats.bwd_items = int32_t(items.size());
  m.stats.bwd_partial_slots = slot;
}

void layout_device(mv_view_mask& m) {
  const std::vector<int32_t>* arrs[10] = {&m.omega,     &m.kt_minmax, &m.q_ptr,    &m.k_list,
                                          &m.qt_order,  &m.bwd_items, &m.bwd_tiles, &m.bwd_red,
                                          &m.iv_ptr,    &m.iv};
  size_t off = 0;
  for (int i = 0; i < 10; ++i) {
    m.off[i] = off;
    off = align256(off + std::max<size_t>(1, arrs[i]->size()) * sizeof(int32_t));
  }
  m.bytes = off;
}

}  // namespace

extern "C" {

mv_status mv_build_view_mask_kind(const mv_trajectory* trajs, int32_t n_traj,
                                  int32_t total_tokens, int32_t kind, mv_view_mask** out) {
  if (out == nullptr) return bad(MV_ERR_INVALID_ARG, "out is null");
  *out = nullptr;
  if (trajs == nullptr || n_traj <= 0) return bad(MV_ERR_INVALID_ARG, "no trajectories");
  if (total_tokens <= 0 || total_tokens > (1 << 30))
    return bad(MV_ERR_INVALID_ARG, "total_tokens must be in [1, 2^30]");
  if (kind != MV_VIEW_LIVE && kind != MV_VIEW_FINAL)
    return bad(MV_ERR_INVALID_ARG, "kind must be MV_VIEW_LIVE or MV_VIEW_FINAL");
  try {
    auto* m = new mv_view_mask();
    m->T = total_tokens;
    m->kind = kind;
    mv_status s =
        validate_and_fill_lifetimes(trajs, n_traj, total_tokens, m->omega, m->iv_ptr, m->iv);
    if (s != MV_OK) {
      delete m;
      return s;
    }
    build_leaves(*m, trajs, n_traj);
    if (kind == MV_VIEW_FINAL) {
      // the final compressed walk applies every edit: a key of the final walk
      // is seen by every later row, any other key by its own row only
      for (int32_t t = 0; t < n_traj; ++t)
        for (int32_t j = trajs[t].begin; j < trajs[t].end; ++j)
          m->omega[j] = m->last_end(j) == trajs[t].end ? trajs[t].end : j + 1;
      std::fill(m->iv_ptr.begin(), m->iv_ptr.end(), 0);
      m->iv.clear();
    }
    build_stats(*m);
    build_fwd_schedule(*m);
    build_bwd_schedule(*m);
    layout_device(*m);
    *out = m;
    return MV_OK;
  } catch (const std::exception& e) {
    return bad(MV_ERR_INVALID_ARG, std::string("host allocation failed: ") + e.what());
  }
}

mv_status mv_build_view_mask(const mv_trajectory* trajs, int32_t n_traj, int32_t total_tokens,
                             mv_view_mask** out) {
  return mv_build_view_mask_kind(trajs, n_traj, total_tokens, MV_VIEW_LIVE, out);
}

mv_status mv_build_view_mask_tiled(const mv_trajectory* trajs, int32_t n_traj,
                                   int32_t total_tokens, int32_t tile_q, int32_t tile_k,
                                   mv_view_mask** out) {
  static_assert(MV_TILE_Q == mv::kFwdTileQ && MV_TILE_K == mv::kFwdTileK,
                "the header's tile shape is the kernels'");
  if (tile_q != MV_TILE_Q || tile_k != MV_TILE_K) {
    std::ostringstream os;
    os << "tile shape " << tile_q << " x " << tile_k << " unsupported: the kernels are built for "
       << MV_TILE_Q << " x " << MV_TILE_K;
    return bad(MV_ERR_UNSUPPORTED, os.str());
  }
  return mv_build_view_mask(trajs, n_traj, total_tokens, out);
}

mv_status mv_view_mask_leaves(const mv_view_mask* m, int32_t* tokens, int32_t* teacher_rows,
                              int32_t* student_rows, int32_t capacity, int32_t* n_out) {
  if (m == nullptr || n_out == nullptr) return bad(MV_ERR_INVALID_ARG, "null argument");
  const int32_t n = int32_t(m->leaf_token.size());
  *n_out = n;
  if (capacity < n) {
    if (tokens == nullptr && teacher_rows == nullptr && student_rows == nullptr && capacity == 0)
      return MV_OK;  // size query
    return bad(MV_ERR_WORKSPACE, "leaf arrays smaller than the number of diverging leaves");
  }
  if (n > 0 && (tokens == nullptr || teacher_rows == nullptr || student_rows == nullptr))
    return bad(MV_ERR_INVALID_ARG, "null leaf array");
  for (int32_t i = 0; i < n; ++i) {
    tokens[i] = m->leaf_token[i];
    teacher_rows[i] = m->leaf_teacher[i];
    student_rows[i] = m->leaf_student[i];
  }
  return MV_OK;
}

size_t mv_view_mask_device_bytes(const mv_view_mask* m) { return m ? m->bytes : 0; }

mv_status mv_view_mask_upload(mv_view_mask* m, void* dev_buf, size_t bytes, hipStream_t stream) {
  if (m == nullptr || dev_buf == nullptr) return bad(MV_ERR_INVALID_ARG, "null mask or buffer");
  if ((reinterpret_cast<uintptr_t>(dev_buf) & 255) != 0)
    return bad(MV_ERR_INVALID_ARG, "mask buffer must be 256-byte aligned");
  if (bytes < m->bytes) {
    std::ostringstream os;
    os << "mask buffer has " << bytes << " bytes, needs " << m->bytes;
    return bad(MV_ERR_WORKSPACE, os.str());
  }
  const std::vector<int32_t>* arrs[10] = {&m->omega,     &m->kt_minmax, &m->q_ptr,
                                          &m->k_list,    &m->qt_order,  &m->bwd_items,
                                          &m->bwd_tiles, &m->bwd_red,   &m->iv_ptr,
                                          &m->iv};
  char* base = static_cast<char*>(dev_buf);
  for (int i = 0; i < 10; ++i) {
    if (arrs[i]->empty()) continue;
    hipError_t e = hipMemcpyAsync(base + m->off[i], arrs[i]->data(),
                                  arrs[i]->size() * sizeof(int32_t), hipMemcpyHostToDevice, stream);
    if (e != hipSuccess) return bad(MV_ERR_HIP, std::string("mask upload: ") + hipGetErrorString(e));
  }
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return bad(MV_ERR_HIP, "hipGetDevice failed");
  m->dev = dev_buf;
  m->device = dev;
  auto at = [&](int i) { return reinterpret_cast<const int32_t*>(base + m->off[i]); };
  m->d = mv_mask_dev{at(0), at(1), at(2), at(3), at(4), at(5), at(6), at(7), at(8), at(9)};
  return MV_OK;
}

mv_status mv_view_mask_stats(const mv_view_mask* m, mv_mask_stats* out) {
  if (m == nullptr || out == nullptr) return bad(MV_ERR_INVALID_ARG, "null argument");
  *out = m->stats;
  return MV_OK;
}

mv_status mv_view_mask_death(const mv_view_mask* m, int32_t* host_out) {
  if (m == nullptr || host_out == nullptr) return bad(MV_ERR_INVALID_ARG, "null argument");
  for (int32_t j = 0; j < m->T; ++j) host_out[j] = m->first_end(j);
  return MV_OK;
}

mv_status mv_view_mask_intervals(const mv_view_mask* m, int32_t* iv_ptr, int32_t* iv,
                                 int32_t capacity, int32_t* n_out) {
  if (m == nullptr || n_out == nullptr) return bad(MV_ERR_INVALID_ARG, "null argument");
  const int32_t n = int32_t(m->iv.size() / 2);
  *n_out = n;
  if (iv_ptr != nullptr) std::copy(m->iv_ptr.begin(), m->iv_ptr.end(), iv_ptr);
  if (iv == nullptr) return MV_OK;
  if (capacity < n) return bad(MV_ERR_WORKSPACE, "interval array smaller than the interval count");
  std::copy(m->iv.begin(), m->iv.end(), iv);
  return MV_OK;
}

mv_status mv_view_mask_materialize_host(const mv_view_mask* m, int32_t row_begin, int32_t row_end,
                                        uint32_t* host_bits) {
  if (m == nullptr || host_bits == nullptr) return bad(MV_ERR_INVALID_ARG, "null argument");
  if (row_begin < 0 || row_end > m->T || row_begin > row_end)
    return bad(MV_ERR_INVALID_ARG, "row range outside [0, total_tokens]");
  const int32_t T = m->T, words = (T + 31) / 32;
  std::memset(host_bits, 0, size_t(row_end - row_begin) * words * sizeof(uint32_t));
  for (int32_t i = row_begin; i < row_end; ++i) {
    uint32_t* row = host_bits + size_t(i - row_begin) * words;
    const int32_t qt = i / mv::kFwdTileQ;
    for (int32_t e = m->q_ptr[qt]; e < m->q_ptr[qt + 1]; ++e) {
      const int32_t kt = m->k_list[e] >> 1;
      const bool full = m->k_list[e] & 1;
      for (int32_t j = kt * mv::kFwdTileK; j < std::min(T, (kt + 1) * mv::kFwdTileK); ++j)
        if (full || m->visible(i, j)) row[j >> 5] |= 1u << (j & 31);
    }
  }
  return MV_OK;
}

void mv_view_mask_free(mv_view_mask* m) { delete m; }

}  // extern "C"

bool mv_view_mask::visible(int32_t i, int32_t j) const {
  return mv_visible_iv(i, j, omega[j], iv_ptr.data(), iv.data());
}
