// Decode session, host side: stream tree, block pool, block-table regions
// and the per-step schedule (App. E, the masked parallel decoding loop).
// No HIP calls: the launch lives with the other entry points that enqueue
// device work.
#include "session.hpp"

#include <algorithm>
#include <cstring>
#include <limits>
#include <memory>
#include <new>

using padoc::clear_error;
using padoc::set_error;

namespace {

constexpr int32_t kBlk = 16;     // tokens per paged block
constexpr int32_t kMinCls = 2;   // smallest block-table region: 4 entries (64 tokens)
constexpr int64_t kI32Max = std::numeric_limits<int32_t>::max();

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

int32_t class_for(int64_t entries) {
  int32_t c = kMinCls;
  while ((int64_t(1) << c) < entries) ++c;
  return c;
}

bool alloc_region(padoc_session* s, int32_t cls, int64_t& off) {
  if (cls >= (int32_t)s->free_regions.size()) s->free_regions.resize(cls + 1);
  auto& fl = s->free_regions[cls];
  if (!fl.empty()) {
    off = fl.back();
    fl.pop_back();
    return true;
  }
  const int64_t n = int64_t(1) << cls;
  if (s->bt_top + n > s->desc.block_table_capacity) return false;
  off = s->bt_top;
  s->bt_top += n;
  return true;
}

void free_region(padoc_session* s, int32_t cls, int64_t off) {
  s->free_regions[cls].push_back(off);
  std::fill(s->bt_host.begin() + off, s->bt_host.begin() + off + (int64_t(1) << cls), -1);
}

void erase_sorted(std::vector<int32_t>& v, int32_t id) {
  auto it = std::lower_bound(v.begin(), v.end(), id);
  if (it != v.end() && *it == id) v.erase(it);
}

// Release `id` and then its ancestors while they are closed and have no kept
// child: blocks back to the pool, region back to its free list.
void release_upwards(padoc_session* s, int32_t id) {
  while (id >= 0) {
    padoc_session::Stream& x = s->st[id];
    if (x.open || !x.kept || x.kept_children > 0) return;
    x.kept = false;
    for (auto it = x.blocks.rbegin(); it != x.blocks.rend(); ++it) s->free_blocks.push_back(*it);
    x.blocks.clear();
    x.blocks.shrink_to_fit();
    if (x.cls >= 0) free_region(s, x.cls, x.bt_off);
    x.cls = -1;
    erase_sorted(s->kept_ids, id);
    if (x.parent >= 0) --s->st[x.parent].kept_children;
    id = x.parent;
  }
}

padoc_status check_session(const padoc_session* s) {
  if (!s) return set_error(PADOC_ERR_ARG, "session is null");
  return PADOC_OK;
}

padoc_status check_unprepared(const padoc_session* s) {
  if (s->prepared)
    return set_error(PADOC_ERR_MODE, "a prepared step has not been launched or committed");
  return PADOC_OK;
}

// The step's tree: every kept stream in id order with its length after the
// step (lengths as they stand when n_new is null); a stream moving to a new
// block-table region (moving_to >= 0) is placed there.
void fill_tree(padoc_session* s, const int32_t* n_new, const int32_t* n_query, std::vector<padoc_segment>& seg,
               std::vector<int32_t>& seg_id) {
  seg.clear();
  seg_id.clear();
  int64_t q = 0;
  size_t row = 0;
  for (int32_t id : s->kept_ids) {
    padoc_session::Stream& x = s->st[id];
    padoc_segment g{};
    g.parent = x.parent >= 0 ? s->st[x.parent].index : -1;  // kept parents come first
    g.fork = x.fork;
    g.len = x.len;
    g.q_len = 0;
    g.kv_off = x.moving_to >= 0 ? x.moving_to : (x.cls >= 0 ? x.bt_off : 0);
    g.q_off = q;
    if (row < s->open_ids.size() && s->open_ids[row] == id) {
      if (n_new) {
        g.len += n_new[row];
        g.q_len = n_query[row];
        q += n_query[row];
      }
      ++row;
    }
    x.index = (int32_t)seg.size();
    seg.push_back(g);
    seg_id.push_back(id);
  }
}

}  // namespace

namespace padoc {
void session_free_host(padoc_session* s) { delete s; }
}  // namespace padoc

extern "C" padoc_status padoc_session_create(const padoc_session_desc* d, padoc_session** out) {
  clear_error();
  if (!out) return set_error(PADOC_ERR_ARG, "out is null");
  *out = nullptr;
  if (!d) return set_error(PADOC_ERR_ARG, "desc is null");
  if (d->dtype != PADOC_F32 && d->dtype != PADOC_BF16)
    return set_error(PADOC_ERR_DTYPE, "dtype %d is not PADOC_F32 or PADOC_BF16", (int)d->dtype);
  if (d->num_blocks < 0 || d->num_blocks > kI32Max)
    return set_error(PADOC_ERR_ARG, "num_blocks=%lld must be in [0, 2^31-1]", (long long)d->num_blocks);
  if (d->block_table_capacity < 0 || d->block_table_capacity > kI32Max)
    return set_error(PADOC_ERR_ARG, "block_table_capacity=%lld must be in [0, 2^31-1]",
                     (long long)d->block_table_capacity);
  // Head counts, head_dim, scale and schedule knobs are checked by a probe
  // plan of an empty tree (the same checks every step's plan passes).
  padoc_tree_desc probe{};
  probe.num_heads_q = d->num_heads_q;
  probe.num_heads_kv = d->num_heads_kv;
  probe.head_dim = d->head_dim;
  probe.softmax_scale = d->softmax_scale;
  probe.dtype = d->dtype;
  probe.block_size = kBlk;
  probe.num_kv_rows = d->num_blocks;
  probe.block_table_len = d->block_table_capacity;
  probe.max_chunk_keys = d->max_chunk_keys;
  probe.target_workgroups = d->target_workgroups;
  try {
    std::unique_ptr<padoc_session> s(new padoc_session());
    padoc_status st = padoc::build_plan(&probe, s->plan);
    if (st != PADOC_OK) return st;
    s->desc = *d;
    s->free_blocks.resize((size_t)d->num_blocks);
    for (int64_t i = 0; i < d->num_blocks; ++i) s->free_blocks[(size_t)i] = (int32_t)(d->num_blocks - 1 - i);
    s->bt_host.assign((size_t)d->block_table_capacity, -1);
    *out = s.release();
  } catch (const std::bad_alloc&) {
    return set_error(PADOC_ERR_ARG, "out of host memory creating the session");
  }
  return PADOC_OK;
}

extern "C" padoc_status padoc_session_open(padoc_session* s, int32_t parent, int32_t fork, int32_t* id) {
  clear_error();
  padoc_status st = check_session(s);
  if (st != PADOC_OK) return st;
  if ((st = check_unprepared(s)) != PADOC_OK) return st;
  if (!id) return set_error(PADOC_ERR_ARG, "id is null");
  if (parent < -1 || parent >= (int32_t)s->st.size())
    return set_error(PADOC_ERR_ARG, "parent %d is not a stream of this session", parent);
  if (parent >= 0 && !s->st[parent].kept)
    return set_error(PADOC_ERR_ARG, "parent %d has been released", parent);
  if (parent < 0 ? fork != 0 : (fork < 0 || fork > s->st[parent].len))
    return set_error(PADOC_ERR_TREE, "fork %d outside [0, %d] (parent %d)", fork,
                     parent < 0 ? 0 : s->st[parent].len, parent);
  if ((int64_t)s->st.size() >= kI32Max) return set_error(PADOC_ERR_ARG, "too many streams");
  try {
    padoc_session::Stream x;
    x.parent = parent;
    x.fork = fork;
    const int32_t nid = (int32_t)s->st.size();
    s->st.push_back(std::move(x));
    s->open_ids.push_back(nid);
    s->kept_ids.push_back(nid);
    if (parent >= 0) ++s->st[parent].kept_children;
    *id = nid;
  } catch (const std::bad_alloc&) {
    return set_error(PADOC_ERR_ARG, "out of host memory");
  }
  return PADOC_OK;
}

extern "C" padoc_status padoc_session_close(padoc_session* s, int32_t id) {
  clear_error();
  padoc_status st = check_session(s);
  if (st != PADOC_OK) return st;
  if ((st = check_unprepared(s)) != PADOC_OK) return st;
  if (id < 0 || id >= (int32_t)s->st.size() || !s->st[id].open)
    return set_error(PADOC_ERR_ARG, "stream %d is not open", id);
  s->st[id].open = false;
  erase_sorted(s->open_ids, id);
  release_upwards(s, id);
  return PADOC_OK;
}

extern "C" padoc_status padoc_session_select(const padoc_session* s, int32_t max_rows, const int64_t* priority,
                                             int32_t* n_new, int32_t* n_query) {
  clear_error();
  padoc_status st = check_session(s);
  if (st != PADOC_OK) return st;
  const size_t R = s->open_ids.size();
  if (R > 0 && (!n_new || !n_query)) return set_error(PADOC_ERR_ARG, "null pointer");
  if (max_rows < 0) return set_error(PADOC_ERR_ARG, "max_rows = %d is negative", max_rows);
  try {
    std::vector<int32_t> order(R);
    for (size_t i = 0; i < R; ++i) order[i] = (int32_t)i;
    const size_t take = max_rows == 0 ? R : std::min(R, (size_t)max_rows);
    // rows are in ascending stream id, so without priorities the first
    // `take` rows are the oldest streams; with them, the largest priority
    // first, equal priorities by ascending id
    if (priority && take < R)
      std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return priority[a] > priority[b]; });
    for (size_t i = 0; i < R; ++i) n_new[i] = n_query[i] = 0;
    for (size_t i = 0; i < take; ++i) n_new[order[i]] = n_query[order[i]] = 1;
  } catch (const std::bad_alloc&) {
    return set_error(PADOC_ERR_ARG, "out of host memory");
  }
  return PADOC_OK;
}

extern "C" padoc_status padoc_session_prepare(padoc_session* s, const int32_t* n_new_in, const int32_t* n_query_in,
                                              int32_t* n_kv_rows, int32_t* n_q_rows, size_t* workspace_bytes) {
  clear_error();
  padoc_status st = check_session(s);
  if (st != PADOC_OK) return st;
  if ((st = check_unprepared(s)) != PADOC_OK) return st;
  const size_t R = s->open_ids.size();
  try {
    std::vector<int32_t> ones;
    if (!n_new_in || !n_query_in) ones.assign(R, 1);
    const int32_t* n_new = n_new_in ? n_new_in : ones.data();
    const int32_t* n_query = n_query_in ? n_query_in : ones.data();
    int64_t total_new = 0, total_q = 0, need_blocks = 0;
    for (size_t i = 0; i < R; ++i) {
      const padoc_session::Stream& x = s->st[s->open_ids[i]];
      if (n_new[i] < 0 || n_query[i] < 0 || n_query[i] > n_new[i])
        return set_error(PADOC_ERR_ARG, "row %zu: need 0 <= n_query (%d) <= n_new (%d)", i, n_query[i], n_new[i]);
      if ((int64_t)x.len + n_new[i] > kI32Max) return set_error(PADOC_ERR_BOUNDS, "stream length exceeds 2^31-1");
      total_new += n_new[i];
      total_q += n_query[i];
      need_blocks += ceil_div((int64_t)x.len + n_new[i], kBlk) - (int64_t)x.blocks.size();
    }
    if (total_new > kI32Max || total_q > kI32Max) return set_error(PADOC_ERR_BOUNDS, "step exceeds 2^31-1 rows");
    if (need_blocks > (int64_t)s->free_blocks.size())
      return set_error(PADOC_ERR_BOUNDS, "the step needs %lld blocks, the pool has %zu free", (long long)need_blocks,
                       s->free_blocks.size());
    // Region moves (tentative until the plan is built).
    struct Move {
      int32_t id, cls;
      int64_t off;
    };
    std::vector<Move> moves;
    auto undo = [&] {
      for (const Move& m : moves) {
        s->free_regions[m.cls].push_back(m.off);
        s->st[m.id].moving_to = -1;
      }
    };
    for (size_t i = 0; i < R; ++i) {
      const int32_t id = s->open_ids[i];
      const padoc_session::Stream& x = s->st[id];
      const int64_t nb = ceil_div((int64_t)x.len + n_new[i], kBlk);
      if (nb == 0 || (x.cls >= 0 && (int64_t(1) << x.cls) >= nb)) continue;
      Move m{id, class_for(nb), 0};
      if (!alloc_region(s, m.cls, m.off)) {
        undo();
        return set_error(PADOC_ERR_BOUNDS, "the block table (%lld entries) cannot hold the step",
                         (long long)s->desc.block_table_capacity);
      }
      moves.push_back(m);
      s->st[id].moving_to = m.off;
    }
    // The step's schedule.
    fill_tree(s, n_new, n_query, s->seg, s->seg_id);
    padoc_tree_desc d{};
    d.n_seg = (int32_t)s->seg.size();
    d.seg = s->seg.data();
    d.num_heads_q = s->desc.num_heads_q;
    d.num_heads_kv = s->desc.num_heads_kv;
    d.head_dim = s->desc.head_dim;
    d.softmax_scale = s->desc.softmax_scale;
    d.dtype = s->desc.dtype;
    d.block_size = kBlk;
    d.num_kv_rows = s->desc.num_blocks;
    d.num_q_rows = total_q;
    d.block_table_len = s->desc.block_table_capacity;
    d.max_chunk_keys = s->desc.max_chunk_keys;
    d.target_workgroups = s->desc.target_workgroups;
    st = padoc::build_plan(&d, s->plan);
    if (st != PADOC_OK) {
      undo();
      return st;
    }
    // Commit: blocks, regions, patches, slots of the new rows.
    s->new_slot.resize((size_t)total_new * 2);
    s->patch.clear();
    s->row_id.assign(s->open_ids.begin(), s->open_ids.end());
    s->row_n_new.assign(n_new, n_new + R);
    s->new_off.resize(R + 1);
    s->q_off.resize(R + 1);
    s->new_off[0] = s->q_off[0] = 0;
    for (size_t i = 0; i < R; ++i) {
      s->new_off[i + 1] = s->new_off[i] + n_new[i];
      s->q_off[i + 1] = s->q_off[i] + n_query[i];
    }
    for (const Move& m : moves) {
      padoc_session::Stream& x = s->st[m.id];
      x.moving_to = -1;
      if (x.cls >= 0) free_region(s, x.cls, x.bt_off);
      x.cls = m.cls;
      x.bt_off = m.off;
      for (size_t j = 0; j < x.blocks.size(); ++j) {
        s->bt_host[(size_t)x.bt_off + j] = x.blocks[j];
        s->patch.push_back((int32_t)(x.bt_off + (int64_t)j));
        s->patch.push_back(x.blocks[j]);
      }
    }
    for (size_t i = 0; i < R; ++i) {
      padoc_session::Stream& x = s->st[s->open_ids[i]];
      const int64_t nb = ceil_div((int64_t)x.len + n_new[i], kBlk);
      while ((int64_t)x.blocks.size() < nb) {
        const int32_t b = s->free_blocks.back();
        s->free_blocks.pop_back();
        const int64_t e = x.bt_off + (int64_t)x.blocks.size();
        x.blocks.push_back(b);
        s->bt_host[(size_t)e] = b;
        s->patch.push_back((int32_t)e);
        s->patch.push_back(b);
      }
      int32_t* sl = s->new_slot.data() + 2 * (size_t)s->new_off[i];
      for (int32_t j = 0; j < n_new[i]; ++j) {
        const int32_t pos = x.len + j;
        sl[2 * j] = x.blocks[pos / kBlk];
        sl[2 * j + 1] = pos % kBlk;
      }
      x.len += n_new[i];
    }
    s->off_patch = align256((size_t)total_new * 8);
    s->rec_bytes = s->off_patch + s->patch.size() * 4;
    s->ws_records = align256(s->rec_bytes);
    s->ws_bytes = s->ws_records + s->plan.ws_bytes;
    s->prepared = true;
    if (n_kv_rows) *n_kv_rows = (int32_t)total_new;
    if (n_q_rows) *n_q_rows = (int32_t)total_q;
    if (workspace_bytes) *workspace_bytes = s->ws_bytes;
  } catch (const std::bad_alloc&) {
    return set_error(PADOC_ERR_ARG, "out of host memory preparing the step");
  }
  return PADOC_OK;
}

extern "C" padoc_status padoc_session_commit(padoc_session* s) {
  clear_error();
  padoc_status st = check_session(s);
  if (st != PADOC_OK) return st;
  if (!s->prepared) return set_error(PADOC_ERR_MODE, "no step is prepared");
  s->prepared = false;
  return PADOC_OK;
}

extern "C" padoc_status padoc_session_view_get(const padoc_session* cs, padoc_session_view* v) {
  clear_error();
  padoc_status st = check_session(cs);
  if (st != PADOC_OK) return st;
  if (!v) return set_error(PADOC_ERR_ARG, "view is null");
  padoc_session* s = const_cast<padoc_session*>(cs);
  std::memset(v, 0, sizeof(*v));
  if (!s->prepared) {
    try {
      fill_tree(s, nullptr, nullptr, s->seg, s->seg_id);
      s->row_id.assign(s->open_ids.begin(), s->open_ids.end());
    } catch (const std::bad_alloc&) {
      return set_error(PADOC_ERR_ARG, "out of host memory");
    }
  }
  v->n_seg = (int32_t)s->seg.size();
  v->seg = s->seg.data();
  v->seg_id = s->seg_id.data();
  v->n_rows = (int32_t)s->row_id.size();
  v->row_id = s->row_id.data();
  if (s->prepared) {
    v->new_off = s->new_off.data();
    v->q_off = s->q_off.data();
    v->new_slot = s->new_slot.data();
    v->n_patch = (int32_t)(s->patch.size() / 2);
    v->patch = s->patch.data();
    v->plan = &s->plan;
    v->workspace_bytes = s->ws_bytes;
  }
  v->block_table = s->bt_host.data();
  v->free_blocks = (int64_t)s->free_blocks.size();
  return PADOC_OK;
}
