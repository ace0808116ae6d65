// Host planner: tree validation, ancestor closure and the tile / split-KV
// schedules of the two entry points.  No HIP calls.
//
// Visibility (Sec. 3.2 ancestor sets; App. C tree-varlen relation): query
// token p of segment s sees keys [0, F(s,t)) of every proper ancestor t
// (F = fork offset of the child of t on the path to s) and keys [0, p] of s.
// Every key range a work item visits is therefore a prefix [0, lim) of one
// segment, with lim depending only on the query token; the schedule records,
// per range, the largest and smallest lim over the item's tokens and (when
// they differ) the per-token limits.  Key tiles below the smallest limit need
// no mask; keys at or past the largest are never visited, and segments no
// token of the item sees are never listed, so non-ancestor tiles are skipped
// by construction (the block-skipping idea of App. C, "Flex Attention").
#include "plan.hpp"

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <limits>
#include <map>
#include <memory>
#include <new>
#include <tuple>
#include <utility>

namespace padoc {

namespace {
thread_local std::string t_err;
}

padoc_status set_error(padoc_status st, const char* fmt, ...) {
  char buf[768];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  t_err = buf;
  return st;
}

void clear_error() { t_err.clear(); }
const char* last_error() { return t_err.c_str(); }

namespace {

constexpr int64_t kI32Max = std::numeric_limits<int32_t>::max();

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
int64_t round_up(int64_t a, int64_t b) { return ceil_div(a, b) * b; }
size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Proper ancestors of every segment as (ancestor, fork offset into it)
// pairs, root first, stored flat.
struct AncList {
  using Pair = std::pair<int32_t, int32_t>;
  struct Span {
    const Pair *b, *e;
    const Pair* begin() const { return b; }
    const Pair* end() const { return e; }
  };
  std::vector<int64_t> off;  // n + 1 entries
  std::vector<Pair> a;
  Span operator[](int32_t s) const { return {a.data() + off[s], a.data() + off[s + 1]}; }
};

// A set of query tokens processed together (one work item per KV head and
// key chunk): entries begin .. begin+count-1 of the builder's token list.
struct Task {
  int32_t begin, count;
};

// A visible segment of a task: each token's limit (keys [0, lim) visible)
// is at the builder's vlim[lim_off + i].
struct VisRange {
  int32_t t;
  int32_t n_keys;  // max lim
  int64_t lim_off;
};

// A key chunk [kb, kb+len) of the VisRange with index r.
struct Piece {
  int32_t r, kb, len;
};

// Sort work items by cost, highest first, keeping the order of equal costs.
void sort_by_cost(std::vector<padoc::WorkRec>& w, std::vector<padoc::WorkRec>& tmp) {
  int32_t mx = 0;
  for (const auto& x : w) mx = std::max(mx, x.cost);
  if (mx > (1 << 16)) {
    std::stable_sort(w.begin(), w.end(), [](const padoc::WorkRec& a, const padoc::WorkRec& b) { return a.cost > b.cost; });
    return;
  }
  std::vector<int32_t> start(mx + 2, 0);
  for (const auto& x : w) ++start[mx - x.cost + 1];
  for (int32_t c = 0; c <= mx; ++c) start[c + 1] += start[c];
  tmp.assign(w.begin(), w.end());
  for (const auto& x : tmp) w[start[mx - x.cost]++] = x;
}

// Working vectors of the planner, kept per thread so that repeated planning
// (a new schedule every decode step) reuses their memory.
struct Scratch {
  std::vector<int32_t> tseg, tpos, vlim, slot, touched, l;
  std::vector<char> sees;
  AncList anc;
  std::vector<int64_t> viewers;
  std::vector<int32_t> root, at, fill;
  std::vector<Task> tasks, stasks, ptasks;
  std::vector<VisRange> vis, svis, pvis;
  std::vector<size_t> svis_at, pvis_at;
  std::vector<Piece> pieces;
  std::vector<std::pair<size_t, int32_t>> parts;
  std::vector<padoc::WorkRec> sitems, pitems, tmp;
  std::vector<std::tuple<int32_t, int64_t, int32_t, uint32_t>> xkeys;
  std::vector<uint32_t> xgroup, xorder;
  std::vector<int64_t> xcost;
};
thread_local Scratch t_scratch;

// Tile items that read the same keys -- the column groups of one key chunk
// of one KV head -- are placed on one XCD: workgroup b runs on XCD b % 8,
// each XCD has an L2 cache of its own, and the tile items run at the same
// time, so the K/V tiles one of them reads are L2 hits for the others.
// Groups go to the XCDs largest first, each to the least loaded; within an
// XCD items keep their (cost) order; a position whose XCD has no item left
// takes one from the XCD with the most items left.
void xcd_group(std::vector<padoc::WorkRec>& w, const std::vector<padoc::RangeRec>& ranges, Scratch& S) {
  constexpr int kXcd = 8;
  const uint32_t n = (uint32_t)w.size();
  if (n <= 1) return;
  auto& keys = S.xkeys;
  keys.resize(n);
  for (uint32_t i = 0; i < n; ++i) {
    const padoc::RangeRec& r = ranges[w[i].rng_begin];
    keys[i] = {w[i].kvh, r.kv_start, r.key_begin, i};
  }
  std::sort(keys.begin(), keys.end());
  auto& grp = S.xgroup;  // group of item i
  auto& cost = S.xcost;  // cost of group g
  grp.assign(n, 0);
  cost.clear();
  for (uint32_t k = 0; k < n; ++k) {
    const bool same = k > 0 && std::get<0>(keys[k]) == std::get<0>(keys[k - 1]) &&
                      std::get<1>(keys[k]) == std::get<1>(keys[k - 1]) && std::get<2>(keys[k]) == std::get<2>(keys[k - 1]);
    if (!same) cost.push_back(0);
    const uint32_t i = std::get<3>(keys[k]);
    grp[i] = (uint32_t)cost.size() - 1;
    cost.back() += w[i].cost;
  }
  const uint32_t ng = (uint32_t)cost.size();
  auto& order = S.xorder;  // groups, costliest first
  order.resize(ng);
  for (uint32_t g = 0; g < ng; ++g) order[g] = g;
  std::stable_sort(order.begin(), order.end(), [&](uint32_t a, uint32_t b) { return cost[a] > cost[b]; });
  int64_t load[kXcd] = {};
  std::vector<int32_t> xcd_of(ng);
  for (uint32_t g : order) {
    const int x = (int)(std::min_element(load, load + kXcd) - load);
    xcd_of[g] = x;
    load[x] += cost[g];
  }
  std::vector<std::vector<uint32_t>> lists(kXcd);
  for (uint32_t i = 0; i < n; ++i) lists[xcd_of[grp[i]]].push_back(i);  // items keep their order
  size_t next[kXcd] = {};
  S.tmp.assign(w.begin(), w.end());
  for (uint32_t p = 0; p < n; ++p) {
    int x = (int)(p % kXcd);
    if (next[x] == lists[x].size()) {
      size_t most = 0;
      for (int y = 0; y < kXcd; ++y)
        if (lists[y].size() - next[y] > most) {
          most = lists[y].size() - next[y];
          x = y;
        }
    }
    w[p] = S.tmp[lists[x][next[x]++]];
  }
}

class Builder {
 public:
  Builder(padoc_plan& p, Scratch& s)
      : P(p), S(s), tseg(s.tseg), tpos(s.tpos), vlim(s.vlim), sees(s.sees), anc_(s.anc), slot_(s.slot),
        touched_(s.touched), l_(s.l) {
    tseg.clear();
    tpos.clear();
    vlim.clear();
    slot_.assign(p.seg.size(), -1);
  }

  padoc_plan& P;
  Scratch& S;
  // Token list of all tasks: segment and position of each query token.
  std::vector<int32_t>&tseg, &tpos;
  // Per-token limits of the visible ranges.
  std::vector<int32_t>& vlim;
  // Tokens of the last emit_ranges call that see at least one key.
  std::vector<char>& sees;

  // visible() for a task of one private segment's query tokens: the only
  // private segment they see is their own (an ancestor whose keys they see
  // is seen by another segment's queries, so it is shared), with the limit
  // position + 1 of each token.
  void visible_own(const Task& task, std::vector<VisRange>& out) {
    VisRange v{tseg[task.begin], 0, (int64_t)vlim.size()};
    for (int32_t i = task.begin; i < task.begin + task.count; ++i) {
      vlim.push_back(tpos[i] + 1);
      v.n_keys = std::max(v.n_keys, tpos[i] + 1);
    }
    out.push_back(v);
  }

  // Appends to `out` the segments visible to any token of `task` for which
  // include(t) holds, in ascending segment order.
  template <class Pred>
  void visible(const Task& task, Pred include, std::vector<VisRange>& out) {
    touched_.clear();
    const int32_t e = task.begin + task.count;
    for (int32_t i = task.begin; i < e; ++i) {
      const int32_t s = tseg[i];
      for (const auto& a : anc_[s])
        if (a.second > 0 && include(a.first)) touch(a.first);
      if (include(s)) touch(s);
    }
    std::sort(touched_.begin(), touched_.end());
    for (int32_t t : touched_) {
      slot_[t] = (int32_t)out.size();
      out.push_back({t, 0, (int64_t)vlim.size()});
      vlim.resize(vlim.size() + task.count, 0);
    }
    for (int32_t i = task.begin; i < e; ++i) {
      const int32_t s = tseg[i], k = i - task.begin;
      for (const auto& a : anc_[s])
        if (a.second > 0 && include(a.first)) set(out[slot_[a.first]], k, a.second);
      if (include(s)) set(out[slot_[s]], k, tpos[i] + 1);
    }
    for (int32_t t : touched_) slot_[t] = -1;
  }

  int32_t add_tokens(const Task& task) {
    const int32_t begin = (int32_t)P.toks.size();
    for (int32_t i = task.begin; i < task.begin + task.count; ++i) {
      const padoc_segment& s = P.seg[tseg[i]];
      P.toks.push_back((int32_t)(s.q_off + (tpos[i] - (s.len - s.q_len))));
    }
    return begin;
  }

  // Emit the range records of pieces[0 .. n_pieces) (ranges of `vis`);
  // returns {rng_begin, rng_count, cost} and marks in sees[] the tokens that
  // see at least one key.
  void emit_ranges(const std::vector<VisRange>& vis, const Piece* pieces, size_t n_pieces, int32_t ntok,
                   int32_t& rng_begin, int32_t& rng_count, int32_t& cost) {
    rng_begin = (int32_t)P.ranges.size();
    rng_count = 0;
    cost = 1;
    sees.assign(ntok, 0);
    l_.resize(ntok);
    for (size_t k = 0; k < n_pieces; ++k) {
      const Piece& pc = pieces[k];
      const VisRange& r = vis[pc.r];
      const int32_t* lim = vlim.data() + r.lim_off;
      int32_t mx = 0, mn = std::numeric_limits<int32_t>::max();
      for (int32_t i = 0; i < ntok; ++i) {
        int32_t v = lim[i] - pc.kb;
        v = v < 0 ? 0 : (v > pc.len ? pc.len : v);
        l_[i] = v;
        mx = std::max(mx, v);
        mn = std::min(mn, v);
        if (v > 0) sees[i] = 1;
      }
      if (mx == 0) continue;
      const padoc_segment& t = P.seg[r.t];
      padoc::RangeRec rr{};
      rr.kv_start = P.block_size ? t.kv_off + pc.kb / P.block_size : t.kv_off + pc.kb;
      rr.n_keys = mx;
      rr.min_lim = mn;
      rr.seg = r.t;
      rr.key_begin = pc.kb;
      if (mn == mx) {
        rr.lim_off = -1;
      } else {
        rr.lim_off = (int32_t)P.lims.size();
        P.lims.insert(P.lims.end(), l_.begin(), l_.end());
      }
      P.ranges.push_back(rr);
      ++rng_count;
      cost += (int32_t)ceil_div(mx, P.tile_keys);
    }
  }

 private:
  void touch(int32_t t) {
    if (slot_[t] == -1) {
      slot_[t] = -2;
      touched_.push_back(t);
    }
  }
  void set(VisRange& r, int32_t k, int32_t lim) {
    vlim[r.lim_off + k] = lim;
    r.n_keys = std::max(r.n_keys, lim);
  }

  const AncList& anc_;
  std::vector<int32_t>&slot_, &touched_, &l_;
};

padoc_status validate(const padoc_tree_desc* d) {
  if (d->n_seg < 0) return set_error(PADOC_ERR_ARG, "n_seg = %d is negative", d->n_seg);
  if (d->n_seg > 0 && !d->seg) return set_error(PADOC_ERR_ARG, "seg is null with n_seg = %d", d->n_seg);
  if (d->dtype != PADOC_F32 && d->dtype != PADOC_BF16)
    return set_error(PADOC_ERR_DTYPE, "dtype %d is not PADOC_F32 or PADOC_BF16", (int)d->dtype);
  if (d->num_heads_q <= 0 || d->num_heads_kv <= 0)
    return set_error(PADOC_ERR_SHAPE, "head counts must be positive (Hq=%d, Hkv=%d)", d->num_heads_q,
                     d->num_heads_kv);
  if (d->num_heads_q % d->num_heads_kv != 0)
    return set_error(PADOC_ERR_SHAPE, "Hq=%d is not a multiple of Hkv=%d", d->num_heads_q, d->num_heads_kv);
  if (d->num_heads_q / d->num_heads_kv > 64)
    return set_error(PADOC_ERR_SHAPE, "Hq/Hkv=%d exceeds 64", d->num_heads_q / d->num_heads_kv);
  if (d->head_dim != 64 && d->head_dim != 128)
    return set_error(PADOC_ERR_SHAPE, "head_dim=%d is not 64 or 128", d->head_dim);
  if (d->num_heads_kv > 4096)  // kernels address a 64-key K/V tile with 32-bit offsets
    return set_error(PADOC_ERR_SHAPE, "Hkv=%d exceeds 4096", d->num_heads_kv);
  if (!std::isfinite(d->softmax_scale) || !(d->softmax_scale > 0.f))
    return set_error(PADOC_ERR_ARG, "softmax_scale must be positive and finite");
  if (d->block_size != 0 && d->block_size != kBlock)
    return set_error(PADOC_ERR_ARG, "block_size=%d is not 0 (packed) or 16 (paged)", d->block_size);
  if (d->num_kv_rows < 0 || d->num_q_rows < 0 || d->block_table_len < 0)
    return set_error(PADOC_ERR_ARG, "negative buffer size");
  if (d->num_q_rows > kI32Max) return set_error(PADOC_ERR_BOUNDS, "num_q_rows exceeds 2^31-1");
  if (d->max_chunk_keys < 0 || d->max_chunk_keys % kTileKeys != 0 || d->max_chunk_keys > padoc::kMaxItemKeys)
    return set_error(PADOC_ERR_ARG, "max_chunk_keys=%d must be a multiple of %d in [0, %d]", d->max_chunk_keys,
                     kTileKeys, padoc::kMaxItemKeys);
  if (d->target_workgroups < 0) return set_error(PADOC_ERR_ARG, "target_workgroups is negative");
  const int32_t n = d->n_seg;
  for (int32_t i = 0; i < n; ++i) {
    const padoc_segment& s = d->seg[i];
    if (s.parent < -1 || s.parent >= i)
      return set_error(PADOC_ERR_TREE, "segment %d: parent %d is not -1 or an earlier segment", i, s.parent);
    if (s.len < 0) return set_error(PADOC_ERR_TREE, "segment %d: len %d is negative", i, s.len);
    if (s.q_len < 0 || s.q_len > s.len)
      return set_error(PADOC_ERR_TREE, "segment %d: q_len %d outside [0, len=%d]", i, s.q_len, s.len);
    if (s.parent < 0) {
      if (s.fork != 0) return set_error(PADOC_ERR_TREE, "segment %d: a root must have fork 0 (got %d)", i, s.fork);
    } else if (s.fork < 0 || s.fork > d->seg[s.parent].len) {
      return set_error(PADOC_ERR_TREE, "segment %d: fork %d outside [0, len(parent %d)=%d]", i, s.fork,
                       s.parent, d->seg[s.parent].len);
    }
    if (s.kv_off < 0) return set_error(PADOC_ERR_BOUNDS, "segment %d: kv_off %lld is negative", i, (long long)s.kv_off);
    if (d->block_size == 0) {
      if (s.kv_off + s.len > d->num_kv_rows)
        return set_error(PADOC_ERR_BOUNDS, "segment %d: K/V rows [%lld, %lld) exceed num_kv_rows=%lld", i,
                         (long long)s.kv_off, (long long)(s.kv_off + s.len), (long long)d->num_kv_rows);
    } else {
      const int64_t nb = ceil_div(s.len, d->block_size);
      if (s.kv_off + nb > d->block_table_len)
        return set_error(PADOC_ERR_BOUNDS, "segment %d: block-table entries [%lld, %lld) exceed block_table_len=%lld",
                         i, (long long)s.kv_off, (long long)(s.kv_off + nb), (long long)d->block_table_len);
      if (d->block_table_host) {
        for (int64_t b = s.kv_off; b < s.kv_off + nb; ++b) {
          const int32_t id = d->block_table_host[b];
          if (id < 0 || id >= d->num_kv_rows)
            return set_error(PADOC_ERR_BOUNDS, "segment %d: block_table[%lld]=%d outside the pool of %lld blocks",
                             i, (long long)b, id, (long long)d->num_kv_rows);
        }
      }
    }
    if (s.q_off < 0 || s.q_off + s.q_len > d->num_q_rows)
      return set_error(PADOC_ERR_BOUNDS, "segment %d: query rows [%lld, %lld) exceed num_q_rows=%lld", i,
                       (long long)s.q_off, (long long)(s.q_off + s.q_len), (long long)d->num_q_rows);
  }
  // Query rows of different segments must not overlap (outputs would race).
  std::vector<std::pair<int64_t, int32_t>> qr;
  for (int32_t i = 0; i < n; ++i)
    if (d->seg[i].q_len > 0) qr.push_back({d->seg[i].q_off, i});
  std::sort(qr.begin(), qr.end());
  for (size_t j = 1; j < qr.size(); ++j) {
    const padoc_segment& a = d->seg[qr[j - 1].second];
    if (a.q_off + a.q_len > qr[j].first)
      return set_error(PADOC_ERR_BOUNDS, "query rows of segments %d and %d overlap", qr[j - 1].second, qr[j].second);
  }
  return PADOC_OK;
}

void build_forward(padoc_plan& P, Builder& B) {
  // Tokens are packed into tasks of tile_tokens; consecutive siblings share
  // tasks (their ancestor ranges coincide), a root starts its own.
  const int32_t n = (int32_t)P.seg.size();
  auto& tasks = B.S.tasks;
  tasks.clear();
  Task cur{0, 0};
  int64_t group = std::numeric_limits<int64_t>::min();
  auto flush = [&] {
    if (cur.count > 0) tasks.push_back(cur);
    cur = {(int32_t)B.tseg.size(), 0};
  };
  for (int32_t s = 0; s < n; ++s) {
    const padoc_segment& sg = P.seg[s];
    if (sg.q_len == 0) continue;
    const int64_t g = sg.parent >= 0 ? (int64_t)sg.parent : -(int64_t)s - 1;
    if (g != group) {
      flush();
      group = g;
    }
    for (int32_t p = sg.len - sg.q_len; p < sg.len; ++p) {
      B.tseg.push_back(s);
      B.tpos.push_back(p);
      if (++cur.count == P.tile_tokens) flush();
    }
  }
  flush();
  auto& vis = B.S.vis;
  auto& pieces = B.S.pieces;
  for (const Task& task : tasks) {
    vis.clear();
    B.vlim.clear();
    B.visible(task, [](int32_t) { return true; }, vis);
    pieces.clear();
    for (size_t r = 0; r < vis.size(); ++r) pieces.push_back({(int32_t)r, 0, vis[r].n_keys});
    const int32_t tok_begin = B.add_tokens(task);
    int32_t rb, rc, cost;
    B.emit_ranges(vis, pieces.data(), pieces.size(), task.count, rb, rc, cost);
    for (int32_t g = 0; g < P.Hkv; ++g) {
      padoc::WorkRec w{};
      w.direct[0] = -1;
      w.tok_begin = tok_begin;
      w.ntok = task.count;
      w.rng_begin = rb;
      w.rng_count = rc;
      w.kvh = g;
      w.out_base = 0;
      w.cost = cost;
      w.col0 = 0;
      w.ncol = task.count * P.G;
      P.work.push_back(w);
    }
  }
}

// Backward (packed bf16): key-major items.  For each segment t and each run of
// up to kBwdKeys of its keys [kb, kb+nk), the query tokens that see any of
// them: t's own queries at positions p >= kb (they see keys <= p), and every
// query of every descendant s whose fork offset into t, F(s, t), exceeds kb
// (they see keys < F).  Each token's limit is stored relative to kb and
// clipped to nk.  A run's columns (token x head) form one item per KV head,
// except that runs longer than about one compute unit's share of all the
// 32-column blocks (total / (target_workgroups / 4), at least 64 blocks) are
// cut into equal block-aligned pieces, whose items add into the same dK/dV
// rows; whole runs store their rows.
void build_backward(padoc_plan& P, const AncList& anc, int32_t target_workgroups) {
  const int32_t n = (int32_t)P.seg.size();
  std::vector<std::vector<std::pair<int32_t, int32_t>>> desc(n);  // (s, F(s, t)) per t
  for (int32_t s = 0; s < n; ++s)
    for (const auto& a : anc[s]) desc[a.first].push_back({s, a.second});
  auto qrow = [&](int32_t s, int32_t p) {
    const padoc_segment& sg = P.seg[s];
    return (int32_t)(sg.q_off + (p - (sg.len - sg.q_len)));
  };
  struct Run {
    int64_t key_row0;
    int32_t nk, tok_begin, ntok, lim_begin;
  };
  std::vector<Run> runs;
  int64_t total_blocks = 0;
  for (int32_t t = 0; t < n; ++t) {
    const padoc_segment& tg = P.seg[t];
    for (int32_t kb = 0; kb < tg.len; kb += kBwdKeys) {
      const int32_t nk = std::min(kBwdKeys, tg.len - kb);
      const int32_t tok_begin = (int32_t)P.btoks.size(), lim_begin = (int32_t)P.blims.size();
      for (int32_t p = std::max(kb, tg.len - tg.q_len); p < tg.len; ++p) {
        P.btoks.push_back(qrow(t, p));
        P.blims.push_back(std::min(p + 1 - kb, nk));
      }
      for (const auto& d : desc[t]) {
        const padoc_segment& sg = P.seg[d.first];
        if (d.second <= kb || sg.q_len == 0) continue;
        for (int32_t p = sg.len - sg.q_len; p < sg.len; ++p) {
          P.btoks.push_back(qrow(d.first, p));
          P.blims.push_back(std::min(d.second - kb, nk));
        }
      }
      const int32_t ntok = (int32_t)P.btoks.size() - tok_begin;
      if (ntok == 0) continue;
      runs.push_back({tg.kv_off + kb, nk, tok_begin, ntok, lim_begin});
      total_blocks += ceil_div((int64_t)ntok * P.G, 32) * P.Hkv;
    }
  }
  const int64_t tw = target_workgroups > 0 ? target_workgroups : 1024;
  const int64_t cap = std::max<int64_t>(64, ceil_div(total_blocks * 4, tw));
  for (const Run& r : runs) {
    const int64_t cols = (int64_t)r.ntok * P.G;
    const int64_t blocks = ceil_div(cols, 32);
    const int64_t pieces = ceil_div(blocks, cap);
    const int64_t step = ceil_div(blocks, pieces) * 32;
    for (int64_t c0 = 0; c0 < cols; c0 += step) {
      for (int32_t g = 0; g < P.Hkv; ++g) {
        padoc::BwdRec b{};
        b.key_row0 = r.key_row0;
        b.n_keys = r.nk;
        b.tok_begin = r.tok_begin;
        b.ntok = r.ntok;
        b.lim_begin = r.lim_begin;
        b.col0 = (int32_t)c0;
        b.ncol = (int32_t)std::min<int64_t>(step, cols - c0);
        b.kvh = g;
        b.cost = (int32_t)ceil_div(b.ncol, 32);
        P.bwd.push_back(b);
      }
    }
  }
  std::stable_sort(P.bwd.begin(), P.bwd.end(),
                   [](const padoc::BwdRec& a, const padoc::BwdRec& b) { return a.cost > b.cost; });
}

// Decode.  A segment is shared when a query token of another segment sees
// any of it (page prefix, layout stream), private otherwise (a branch seen
// only by its own queries).  Shared keys are processed by matrix-core tile
// items: per page, the tokens that see shared segments are cut into items of
// at most 256 columns, so siblings share every K/V tile (loaded from HBM once
// per item and key chunk).  Private keys are streamed by wavefront items of
// 16 columns.  Both kinds run in one launch and write split partials; the
// combine map lists them per (query row, KV head) in creation order, and
// every row with partials is merged by the combine kernel.
void build_decode(padoc_plan& P, Builder& B, const AncList& anc, const padoc_tree_desc* d) {
  const int32_t n = (int32_t)P.seg.size();
  const int32_t G = P.G;
  const int32_t NTs = std::max(1, kTileCols / G);
  const int32_t NTp = std::max(1, kPrivateCols / G);
  Scratch& S = B.S;
  auto& viewers = S.viewers;
  viewers.assign(n, 0);
  for (int32_t s = 0; s < n; ++s)
    if (P.seg[s].q_len > 0)
      for (const auto& a : anc[s])
        if (a.second > 0) viewers[a.first] += P.seg[s].q_len;
  auto shared = [&](int32_t t) { return viewers[t] > 0; };
  auto priv = [&](int32_t t) { return viewers[t] == 0; };
  auto& root = S.root;
  root.resize(n);
  for (int32_t s = 0; s < n; ++s) root[s] = P.seg[s].parent < 0 ? s : root[P.seg[s].parent];

  // Shared tasks: per page (ascending root), the query tokens of every
  // segment that sees a shared key, in segment then position order, cut
  // into tasks of NTs tokens.  Private tasks: NTp consecutive query tokens
  // of one private segment.
  auto& stasks = S.stasks;
  auto& ptasks = S.ptasks;
  stasks.clear();
  ptasks.clear();
  {
    auto sees_shared = [&](int32_t s) {
      if (P.seg[s].q_len == 0) return false;
      if (shared(s)) return true;
      for (const auto& a : anc[s])
        if (a.second > 0) return true;
      return false;
    };
    auto& at = S.at;
    at.assign(n + 1, 0);
    for (int32_t s = 0; s < n; ++s)
      if (sees_shared(s)) at[root[s] + 1] += P.seg[s].q_len;
    for (int32_t r = 0; r < n; ++r) at[r + 1] += at[r];
    const int32_t total = at[n];
    B.tseg.resize(total);
    B.tpos.resize(total);
    auto& fill = S.fill;
    fill.assign(at.begin(), at.end() - 1);
    for (int32_t s = 0; s < n; ++s) {
      if (!sees_shared(s)) continue;
      const padoc_segment& sg = P.seg[s];
      for (int32_t p = sg.len - sg.q_len; p < sg.len; ++p) {
        const int32_t i = fill[root[s]]++;
        B.tseg[i] = s;
        B.tpos[i] = p;
      }
    }
    for (int32_t r = 0; r < n; ++r)
      for (int32_t b = at[r]; b < at[r + 1]; b += NTs) stasks.push_back({b, std::min(NTs, at[r + 1] - b)});
    for (int32_t s = 0; s < n; ++s) {
      const padoc_segment& sg = P.seg[s];
      if (sg.q_len == 0 || shared(s)) continue;
      for (int32_t b = sg.len - sg.q_len; b < sg.len; b += NTp) {
        Task t{(int32_t)B.tseg.size(), 0};
        for (int32_t p = b; p < std::min(sg.len, b + NTp); ++p) {
          B.tseg.push_back(s);
          B.tpos.push_back(p);
          ++t.count;
        }
        ptasks.push_back(t);
      }
    }
  }
  // Chunk sizes.  Shared keys: at most 3/16 x target_workgroups tile items
  // (see below).  Private keys: about target_workgroups x 2 wavefronts' worth
  // of equal pieces.
  auto& svis = S.svis;
  auto& pvis = S.pvis;
  auto& svis_at = S.svis_at;
  auto& pvis_at = S.pvis_at;
  svis.clear();
  pvis.clear();
  svis_at.assign(1, 0);
  pvis_at.assign(1, 0);
  int64_t total_p = 0;
  for (const Task& t : stasks) {
    B.visible(t, shared, svis);
    svis_at.push_back(svis.size());
  }
  for (const Task& t : ptasks) {
    B.visible_own(t, pvis);
    const int64_t splits = ceil_div((int64_t)t.count * G, kPrivateCols);
    for (size_t r = pvis_at.back(); r < pvis.size(); ++r) total_p += round_up(pvis[r].n_keys, 32) * P.Hkv * splits;
    pvis_at.push_back(pvis.size());
  }
  const int64_t tw = d->target_workgroups > 0 ? d->target_workgroups : 1024;
  auto chunk_keys = [&](int64_t total, int64_t pieces) {
    if (d->max_chunk_keys > 0) return (int64_t)d->max_chunk_keys;
    const int64_t ch = round_up(std::max<int64_t>(1, ceil_div(total, pieces)), 64);
    return std::min<int64_t>(std::max<int64_t>(ch, 512), padoc::kMaxItemKeys);
  };
  const int64_t CHp = chunk_keys(total_p, 2 * tw);
  // Shared keys: every tile item takes a whole compute unit (its registers)
  // for its duration, and the private items stream keys on the units the
  // tile items leave free.  The tile items are capped at three quarters of
  // the target_workgroups / 4 units (one round), so that from the start at
  // least a quarter of the units read private keys, while the shared keys
  // still get most of the matrix cores; a step over the cap would need a
  // second round of tile items.  Smallest chunk (a multiple of 64 from 128
  // up to 8192) whose items (over all tasks and KV heads) fit, else 8192: a
  // small step (one page) gets short chunks, so its few shared keys still
  // spread over many compute units instead of forming a few long serial
  // chains (below 128 keys an item's fixed latency stays while the combine
  // gets more partials per row).
  auto shared_items = [&](int64_t CH) {
    int64_t n = 0;
    for (size_t i = 0; i + 1 < svis_at.size(); ++i) {
      int64_t room = 0;
      for (size_t r = svis_at[i]; r < svis_at[i + 1]; ++r)
        for (int32_t kb = 0; kb < svis[r].n_keys;) {
          if (room <= 0) {
            ++n;
            room = CH;
          }
          const int32_t take = (int32_t)std::min<int64_t>(svis[r].n_keys - kb, room);
          kb += take;
          room -= round_up(take, 64);
        }
    }
    return n * P.Hkv;
  };
  int64_t CHs = d->max_chunk_keys;
  if (CHs <= 0) {
    const int64_t target = std::max<int64_t>(1, tw * 3 / 16);
    int64_t lo = 2, hi = 128;  // chunk = 64 * k keys
    if (shared_items(64 * hi) > target) {
      lo = hi;
    } else {
      while (lo < hi) {
        const int64_t mid = (lo + hi) / 2;
        if (shared_items(64 * mid) <= target)
          hi = mid;
        else
          lo = mid + 1;
      }
    }
    CHs = 64 * lo;
  }

  // (row * Hkv + kvh, slot) of every partial, in creation order.
  auto& parts = S.parts;
  auto& sitems = S.sitems;
  auto& pitems = S.pitems;
  parts.clear();
  sitems.clear();
  pitems.clear();
  auto emit = [&](const Task& task, int32_t tok_begin, const std::vector<VisRange>& vis, const Piece* pieces,
                  size_t n_pieces, int32_t width, std::vector<padoc::WorkRec>& out) {
    const int32_t ntok = task.count;
    int32_t rb, rc, cost;
    B.emit_ranges(vis, pieces, n_pieces, ntok, rb, rc, cost);
    if (rc == 0) return;
    for (int32_t kvh = 0; kvh < P.Hkv; ++kvh) {
      const int32_t base = (int32_t)P.n_slots;
      for (int32_t i = 0; i < ntok; ++i)
        if (B.sees[i]) parts.push_back({(size_t)P.toks[tok_begin + i] * P.Hkv + kvh, base + i * G});
      P.n_slots += (int64_t)ntok * G;
      for (int32_t c0 = 0; c0 < ntok * G; c0 += width) {
        padoc::WorkRec w{};
        w.direct[0] = -1;
        w.tok_begin = tok_begin;
        w.ntok = ntok;
        w.rng_begin = rb;
        w.rng_count = rc;
        w.kvh = kvh;
        w.out_base = base;
        w.cost = cost;
        w.col0 = c0;
        w.ncol = std::min(width, ntok * G - c0);
        out.push_back(w);
      }
    }
  };
  // Cut the visible ranges vis[r0 .. r1) into chunks of at most CH keys
  // (each piece counted rounded up to 64) and emit each chunk; returns the
  // number of chunks.
  auto& chunk = S.pieces;
  auto cut_emit = [&](const Task& task, int32_t tok_begin, const std::vector<VisRange>& vis, size_t r0, size_t r1,
                      int64_t CH, int32_t width, std::vector<padoc::WorkRec>& out) {
    int32_t n_chunks = 0;
    int64_t room = CH;
    chunk.clear();
    for (size_t r = r0; r < r1; ++r) {
      int32_t kb = 0;
      while (kb < vis[r].n_keys) {
        if (room <= 0) {
          emit(task, tok_begin, vis, chunk.data(), chunk.size(), width, out);
          ++n_chunks;
          chunk.clear();
          room = CH;
        }
        const int32_t take = (int32_t)std::min<int64_t>(vis[r].n_keys - kb, room);
        chunk.push_back({(int32_t)r, kb, take});
        kb += take;
        room -= round_up(take, 64);
      }
    }
    if (!chunk.empty()) {
      emit(task, tok_begin, vis, chunk.data(), chunk.size(), width, out);
      ++n_chunks;
    }
    return n_chunks;
  };
  for (size_t i = 0; i < stasks.size(); ++i) {
    const int32_t tb = B.add_tokens(stasks[i]);
    cut_emit(stasks[i], tb, svis, svis_at[i], svis_at[i + 1], CHs, kTileCols, sitems);
  }
  for (size_t i = 0; i < ptasks.size(); ++i) {
    const int32_t tb = B.add_tokens(ptasks[i]);
    if (ptasks[i].count != 1) {
      cut_emit(ptasks[i], tb, pvis, pvis_at[i], pvis_at[i + 1], CHp, kPrivateCols, pitems);
      continue;
    }
    // One query token (the usual decode step): what cut_emit makes of its
    // one range [0, n) -- chunks of CHp keys, each fully visible (no
    // limits), one partial per KV head -- written out directly.
    const VisRange& v = pvis[pvis_at[i]];
    const padoc_segment& sg = P.seg[v.t];
    for (int32_t kb = 0; kb < v.n_keys; kb += (int32_t)CHp) {
      const int32_t take = (int32_t)std::min<int64_t>(v.n_keys - kb, CHp);
      padoc::RangeRec rr{};
      rr.kv_start = sg.kv_off + kb / P.block_size;
      rr.n_keys = take;
      rr.min_lim = take;
      rr.lim_off = -1;
      rr.seg = v.t;
      rr.key_begin = kb;
      const int32_t rb = (int32_t)P.ranges.size();
      P.ranges.push_back(rr);
      const int32_t cost = 1 + (int32_t)ceil_div(take, P.tile_keys);
      for (int32_t kvh = 0; kvh < P.Hkv; ++kvh) {
        const int32_t base = (int32_t)P.n_slots;
        parts.push_back({(size_t)P.toks[tb] * P.Hkv + kvh, base});
        P.n_slots += G;
        for (int32_t c0 = 0; c0 < G; c0 += kPrivateCols) {
          padoc::WorkRec w{};
          // the range and the Q row, copied so the kernel's first K/V loads
          // wait for one record instead of three
          w.direct[0] = rr.kv_start <= INT32_MAX ? (int32_t)rr.kv_start : -1;
          w.direct[1] = take;
          w.direct[2] = P.toks[tb];
          w.tok_begin = tb;
          w.ntok = 1;
          w.rng_begin = rb;
          w.rng_count = 1;
          w.kvh = kvh;
          w.out_base = base;
          w.cost = cost;
          w.col0 = c0;
          w.ncol = std::min(kPrivateCols, G - c0);
          pitems.push_back(w);
        }
      }
    }
  }
  sort_by_cost(sitems, S.tmp);
  xcd_group(sitems, P.ranges, S);
  sort_by_cost(pitems, S.tmp);
  P.work.reserve(sitems.size() + pitems.size());
  P.work.assign(sitems.begin(), sitems.end());
  P.work.insert(P.work.end(), pitems.begin(), pitems.end());
  P.n_work_shared = (int32_t)sitems.size();
  // Private items are taken from kPrivateQueues queues (queue of workgroup b:
  // b % kPrivateQueues) by every wavefront of the launch: the tile
  // workgroups' after their item, and workgroups of their own on the compute
  // units the tile items leave free (target_workgroups / 4 units).  Every
  // queue gets at least one such workgroup, so that no queue waits for the
  // tile items to end.
  P.n_private_groups = 0;
  if (!pitems.empty()) {
    const int64_t groups = ceil_div((int64_t)pitems.size(), 8);
    const int64_t free_units = std::max<int64_t>(0, tw / 4 - (int64_t)sitems.size());
    P.n_private_groups = (int32_t)std::max<int64_t>(std::min(groups, free_units), padoc::kPrivateQueues);
  }

  // Combine map: slots per (row, KV head) in creation order (stable counting
  // sort of the partials by row).
  const size_t n_rows = (size_t)P.num_q_rows * P.Hkv;
  P.comb_ptr.assign(n_rows + 1, 0);
  for (const auto& pr : parts) ++P.comb_ptr[pr.first + 1];
  for (size_t r = 0; r < n_rows; ++r) P.comb_ptr[r + 1] += P.comb_ptr[r];
  P.comb_slot.resize(parts.size());
  {
    auto& fill = S.fill;
    fill.assign(P.comb_ptr.begin(), P.comb_ptr.end() - 1);
    for (const auto& pr : parts) P.comb_slot[fill[pr.first]++] = pr.second;
  }
  for (size_t r = 0; r < n_rows; ++r)
    if (P.comb_ptr[r + 1] > P.comb_ptr[r]) P.comb_rows.push_back((int32_t)r);
}

template <class T>
void put(std::vector<unsigned char>& blob, size_t off, const std::vector<T>& v) {
  if (!v.empty()) std::memcpy(blob.data() + off, v.data(), v.size() * sizeof(T));
}

// Backward workspace: the forward schedule (dQ items), the backward
// schedule, then sum(dO * O) per (row, head) and the fp32 dK / dV
// accumulators.
void serialise_backward(padoc_plan& P) {
  P.boff_bwd = 0;
  P.boff_btoks = align256(P.boff_bwd + P.bwd.size() * sizeof(padoc::BwdRec));
  P.boff_blims = align256(P.boff_btoks + P.btoks.size() * 4);
  const size_t bytes = P.boff_blims + P.blims.size() * 4;
  P.bwd_blob.assign(bytes, 0);
  put(P.bwd_blob, P.boff_bwd, P.bwd);
  put(P.bwd_blob, P.boff_btoks, P.btoks);
  put(P.bwd_blob, P.boff_blims, P.blims);
  P.bws_off_blob = align256(P.blob.size());
  P.bws_off_dd = align256(P.bws_off_blob + bytes);
  P.bws_off_dk = align256(P.bws_off_dd + (size_t)P.num_q_rows * P.Hq * 4);
  const size_t acc = (size_t)P.num_kv_rows * P.Hkv * P.D * 4;
  P.bws_off_dv = align256(P.bws_off_dk + acc);
  P.bws_bytes = std::max<size_t>(256, align256(P.bws_off_dv + acc));
}

void serialise(padoc_plan& P) {
  P.off_work = 0;
  P.off_ranges = align256(P.off_work + P.work.size() * sizeof(padoc::WorkRec));
  P.off_lims = align256(P.off_ranges + P.ranges.size() * sizeof(padoc::RangeRec));
  P.off_toks = align256(P.off_lims + P.lims.size() * 4);
  P.off_comb_slot = align256(P.off_toks + P.toks.size() * 4);
  P.off_comb_rows = align256(P.off_comb_slot + P.comb_slot.size() * 4);
  P.off_next = align256(P.off_comb_rows + P.comb_rows.size() * 16);
  const size_t blob_bytes = P.off_next + padoc::kPrivateQueues * 256;  // queue counters, 256 bytes apart
  P.off_part_o = align256(blob_bytes);
  P.off_part_ml = align256(P.off_part_o + (size_t)P.n_slots * P.D * 4);
  P.ws_bytes = std::max<size_t>(256, align256(P.off_part_ml + (size_t)P.n_slots * 8));
  // Every byte is written once: the sections, the zero padding after each
  // (up to the next 256-byte offset) and the zeroed queue counters (a plan
  // rebuilt every decode step does not clear the whole blob first).
  P.blob.resize(blob_bytes);
  unsigned char* b = P.blob.data();
  auto section = [&](size_t off, const void* src, size_t bytes, size_t end) {
    if (bytes) std::memcpy(b + off, src, bytes);
    std::memset(b + off + bytes, 0, end - off - bytes);
  };
  section(P.off_work, P.work.data(), P.work.size() * sizeof(padoc::WorkRec), P.off_ranges);
  section(P.off_ranges, P.ranges.data(), P.ranges.size() * sizeof(padoc::RangeRec), P.off_lims);
  section(P.off_lims, P.lims.data(), P.lims.size() * 4, P.off_toks);
  section(P.off_toks, P.toks.data(), P.toks.size() * 4, P.off_comb_slot);
  section(P.off_comb_slot, P.comb_slot.data(), P.comb_slot.size() * 4, P.off_comb_rows);
  // merged pairs as device records {row*Hkv + kvh, first, end, 0}: the
  // combine kernel finds a pair and its slot list with one load
  int32_t* rec = reinterpret_cast<int32_t*>(b + P.off_comb_rows);
  for (size_t i = 0; i < P.comb_rows.size(); ++i) {
    const int32_t rk = P.comb_rows[i];
    const int32_t r4[4] = {rk, P.comb_ptr[rk], P.comb_ptr[rk + 1], 0};
    std::memcpy(rec + 4 * i, r4, sizeof r4);
  }
  std::memset(b + P.off_comb_rows + P.comb_rows.size() * 16, 0, blob_bytes - P.off_comb_rows - P.comb_rows.size() * 16);
}

}  // namespace

padoc_status build_plan(const padoc_tree_desc* d, padoc_plan& P) {
  padoc_status st = validate(d);
  if (st != PADOC_OK) return st;
  try {
    ++P.build_id;
    P.kind = d->block_size == 0 ? 0 : 1;
    P.Hq = d->num_heads_q;
    P.Hkv = d->num_heads_kv;
    P.G = d->num_heads_q / d->num_heads_kv;
    P.D = d->head_dim;
    P.scale = d->softmax_scale;
    P.dtype = d->dtype;
    P.block_size = d->block_size;
    P.num_kv_rows = d->num_kv_rows;
    P.num_q_rows = d->num_q_rows;
    P.block_table_len = d->block_table_len;
    P.seg.assign(d->seg, d->seg + d->n_seg);
    P.tile_cols = kTileCols;
    P.tile_keys = P.kind == 1 ? 32 : kTileKeys;  // decode ranges are classified per 32-key step
    P.tile_tokens = std::max(1, P.tile_cols / P.G);
    P.work.clear();
    P.n_work_shared = 0;
    P.n_private_groups = 0;
    P.ranges.clear();
    P.lims.clear();
    P.toks.clear();
    {
      std::lock_guard<std::mutex> lk(P.tc_mu);
      P.tc_built = false;
      P.tile_class.clear();
      P.tile_class_off.clear();
    }
    P.comb_ptr.clear();
    P.comb_slot.clear();
    P.comb_rows.clear();
    P.n_slots = 0;
    P.bwd.clear();
    P.btoks.clear();
    P.blims.clear();
    P.bwd_blob.clear();
    P.blob.clear();
    Scratch& S = t_scratch;
    AncList& anc = S.anc;
    anc.off.assign((size_t)d->n_seg + 1, 0);
    for (int32_t s = 0; s < d->n_seg; ++s) {
      const int32_t par = P.seg[s].parent;
      anc.off[s + 1] = anc.off[s] + (par >= 0 ? anc.off[par + 1] - anc.off[par] + 1 : 0);
    }
    anc.a.resize((size_t)anc.off[d->n_seg]);
    for (int32_t s = 0; s < d->n_seg; ++s) {
      const int32_t par = P.seg[s].parent;
      if (par < 0) continue;
      std::copy(anc.a.begin() + anc.off[par], anc.a.begin() + anc.off[par + 1], anc.a.begin() + anc.off[s]);
      anc.a[anc.off[s + 1] - 1] = {par, P.seg[s].fork};
    }
    Builder B(P, S);
    if (P.kind == 0)
      build_forward(P, B);
    else
      build_decode(P, B, anc, d);
    if (P.n_slots > kI32Max) return set_error(PADOC_ERR_ARG, "schedule too large (%lld partial slots)", (long long)P.n_slots);
    if ((int64_t)P.lims.size() > kI32Max || (int64_t)P.ranges.size() > kI32Max)
      return set_error(PADOC_ERR_ARG, "schedule too large");
    // a paged tile item stages the block ids of all its tiles (one per thread)
    for (int32_t i = 0; P.kind == 1 && i < P.n_work_shared; ++i) {
      const padoc::WorkRec& w = P.work[i];
      int64_t nt = 0;
      for (int32_t r = 0; r < w.rng_count; ++r) nt += ceil_div(P.ranges[w.rng_begin + r].n_keys, kTileKeys);
      if (nt > padoc::kMaxItemTiles)
        return set_error(PADOC_ERR_ARG, "internal: shared item %d has %lld tiles (at most %d)", i, (long long)nt,
                         padoc::kMaxItemTiles);
    }
    // Costliest items first: the hardware dispatcher then assigns work
    // greedily to the first free compute unit (longest-processing-time
    // order).  Decode items are already ordered by workgroup.
    if (P.kind == 0) sort_by_cost(P.work, S.tmp);
    serialise(P);
    if (P.kind == 0 && P.dtype == PADOC_BF16) {
      build_backward(P, anc, d->target_workgroups);
      if ((int64_t)P.btoks.size() > kI32Max || (int64_t)P.bwd.size() > kI32Max)
        return set_error(PADOC_ERR_ARG, "backward schedule too large");
      serialise_backward(P);
    }
  } catch (const std::bad_alloc&) {
    return set_error(PADOC_ERR_ARG, "out of host memory while planning");
  }
  return PADOC_OK;
}

}  // namespace padoc

using namespace padoc;

extern "C" padoc_status padoc_tree_layout(padoc_segment* seg, int32_t n, int32_t block_size) {
  clear_error();
  if (n < 0 || (n > 0 && !seg)) return set_error(PADOC_ERR_ARG, "bad segment array (n=%d)", n);
  if (block_size < 0) return set_error(PADOC_ERR_ARG, "block_size %d is negative", block_size);
  int64_t kv = 0, q = 0;
  for (int32_t i = 0; i < n; ++i) {
    seg[i].kv_off = kv;
    seg[i].q_off = q;
    kv += block_size == 0 ? seg[i].len : ceil_div(seg[i].len, block_size);
    q += seg[i].q_len;
  }
  return PADOC_OK;
}

extern "C" padoc_status padoc_tree_from_pages(const padoc_page* pages, int32_t n_pages, int32_t block_size,
                                              padoc_segment* out, int32_t capacity, int32_t* n_out) {
  clear_error();
  if (!n_out) return set_error(PADOC_ERR_ARG, "n_out is null");
  *n_out = 0;
  if (n_pages < 0 || (n_pages > 0 && !pages)) return set_error(PADOC_ERR_ARG, "bad page array (n_pages=%d)", n_pages);
  if (block_size < 0) return set_error(PADOC_ERR_ARG, "block_size %d is negative", block_size);
  int64_t need = 0;
  for (int32_t i = 0; i < n_pages; ++i) {
    const padoc_page& p = pages[i];
    if (p.n_branches < 0) return set_error(PADOC_ERR_ARG, "page %d: n_branches %d is negative", i, p.n_branches);
    if (p.n_branches > 0 && (!p.branch_fork || !p.branch_len || !p.branch_q_len))
      return set_error(PADOC_ERR_ARG, "page %d: branch arrays are null", i);
    need += 2 + (int64_t)p.n_branches;
  }
  if (need > kI32Max) return set_error(PADOC_ERR_ARG, "too many segments (%lld)", (long long)need);
  *n_out = (int32_t)need;
  if (need > capacity || (need > 0 && !out))
    return set_error(PADOC_ERR_ARG, "capacity %d < %lld segments needed", capacity, (long long)need);
  int32_t k = 0;
  for (int32_t i = 0; i < n_pages; ++i) {
    const padoc_page& p = pages[i];
    const int32_t root = k;
    out[k++] = padoc_segment{-1, 0, p.prefix_len, p.prefix_q_len, 0, 0};
    const int32_t stream = k;
    out[k++] = padoc_segment{root, p.prefix_len, p.stream_len, p.stream_q_len, 0, 0};
    for (int32_t b = 0; b < p.n_branches; ++b)
      out[k++] = padoc_segment{stream, p.branch_fork[b], p.branch_len[b], p.branch_q_len[b], 0, 0};
  }
  return padoc_tree_layout(out, k, block_size);
}

extern "C" padoc_status padoc_tree_depths(const padoc_segment* seg, int32_t n, int64_t* d_seq, int64_t* d_crit) {
  clear_error();
  if (n < 0) return set_error(PADOC_ERR_ARG, "n = %d is negative", n);
  if (n > 0 && (!seg || !d_seq || !d_crit)) return set_error(PADOC_ERR_ARG, "null pointer");
  try {
    std::vector<int64_t> start(n, 0);
    std::vector<int32_t> root(n);
    for (int32_t s = 0; s < n; ++s) {
      const padoc_segment& g = seg[s];
      if (g.len < 0) return set_error(PADOC_ERR_TREE, "segment %d: negative length", s);
      if (g.parent < -1 || g.parent >= s)
        return set_error(PADOC_ERR_TREE, "segment %d: parent %d is not an earlier segment", s, g.parent);
      d_seq[s] = d_crit[s] = 0;
      if (g.parent < 0) {
        root[s] = s;
        continue;
      }
      if (g.fork < 0 || g.fork > seg[g.parent].len)
        return set_error(PADOC_ERR_TREE, "segment %d: fork %d outside [0, %d]", s, g.fork, seg[g.parent].len);
      root[s] = root[g.parent];
      // below a root the stream starts at step 0; deeper, after the parent's
      // first `fork` tokens
      start[s] = seg[g.parent].parent < 0 ? 0 : start[g.parent] + g.fork;
      d_seq[root[s]] += g.len;
      d_crit[root[s]] = std::max(d_crit[root[s]], start[s] + g.len);
    }
  } catch (const std::bad_alloc&) {
    return set_error(PADOC_ERR_ARG, "out of host memory");
  }
  return PADOC_OK;
}

extern "C" padoc_status padoc_tree_remaining(const padoc_segment* seg, int32_t n, const int32_t* progress,
                                             int64_t* remaining) {
  clear_error();
  if (n < 0) return set_error(PADOC_ERR_ARG, "n = %d is negative", n);
  if (n > 0 && (!seg || !remaining)) return set_error(PADOC_ERR_ARG, "null pointer");
  auto done = [&](int32_t s) -> int32_t { return progress ? progress[s] : 0; };
  try {
    // started: a child of a root starts with the page; deeper, once its
    // parent has started and produced the `fork` tokens it conditions on
    std::vector<int32_t> root(n);
    std::vector<char> started(n, 0);
    for (int32_t s = 0; s < n; ++s) {
      const padoc_segment& g = seg[s];
      if (g.len < 0) return set_error(PADOC_ERR_TREE, "segment %d: negative length", s);
      if (g.parent < -1 || g.parent >= s)
        return set_error(PADOC_ERR_TREE, "segment %d: parent %d is not an earlier segment", s, g.parent);
      if (g.parent < 0) {
        root[s] = s;
        continue;  // roots are prefilled: their progress is not read
      }
      const int32_t p = g.parent;
      if (g.fork < 0 || g.fork > seg[p].len)
        return set_error(PADOC_ERR_TREE, "segment %d: fork %d outside [0, %d]", s, g.fork, seg[p].len);
      root[s] = root[p];
      started[s] = seg[p].parent < 0 || (started[p] && done(p) >= g.fork);
      if (done(s) < 0 || done(s) > g.len)
        return set_error(PADOC_ERR_ARG, "segment %d: progress %d outside [0, %d]", s, done(s), g.len);
      if (done(s) > 0 && !started[s])
        return set_error(PADOC_ERR_ARG, "segment %d has progress %d before its parent reached its fork", s, done(s));
    }
    // Children have larger indices than their parents, so one pass from the
    // last segment down sees every child's remaining path before its parent.
    // A decoded segment's path: its own tokens still to come, or, through a
    // child not started yet, the steps until that child's fork point plus
    // the child's whole path.  Started segments run on their own: the page
    // ends with the longest of their paths.
    for (int32_t s = 0; s < n; ++s) remaining[s] = 0;
    for (int32_t s = n - 1; s >= 0; --s) {
      const padoc_segment& g = seg[s];
      if (g.parent < 0) continue;
      remaining[s] = std::max<int64_t>(remaining[s], (int64_t)g.len - done(s));
      if (started[s])
        remaining[root[s]] = std::max(remaining[root[s]], remaining[s]);
      else
        remaining[g.parent] = std::max(remaining[g.parent], (int64_t)(g.fork - done(g.parent)) + remaining[s]);
    }
  } catch (const std::bad_alloc&) {
    return set_error(PADOC_ERR_ARG, "out of host memory");
  }
  return PADOC_OK;
}

extern "C" padoc_status padoc_plan_create(const padoc_tree_desc* d, padoc_plan** out) {
  clear_error();
  if (!out) return set_error(PADOC_ERR_ARG, "out is null");
  *out = nullptr;
  if (!d) return set_error(PADOC_ERR_ARG, "desc is null");
  std::unique_ptr<padoc_plan> P(new (std::nothrow) padoc_plan());
  if (!P) return set_error(PADOC_ERR_ARG, "out of host memory while planning");
  const padoc_status st = padoc::build_plan(d, *P);
  if (st == PADOC_OK) *out = P.release();
  return st;
}

extern "C" padoc_status padoc_plan_workspace_bytes(const padoc_plan* plan, size_t* bytes) {
  clear_error();
  if (!plan || !bytes) return set_error(PADOC_ERR_ARG, "null argument");
  *bytes = plan->ws_bytes;
  return PADOC_OK;
}

extern "C" padoc_status padoc_plan_backward_workspace_bytes(const padoc_plan* plan, size_t* bytes) {
  clear_error();
  if (!plan || !bytes) return set_error(PADOC_ERR_ARG, "null argument");
  if (plan->kind != 0) return set_error(PADOC_ERR_MODE, "the backward needs a packed plan (block_size 0)");
  if (plan->dtype != PADOC_BF16) return set_error(PADOC_ERR_DTYPE, "the backward supports bf16 plans only");
  *bytes = plan->bws_bytes;
  return PADOC_OK;
}

extern "C" padoc_status padoc_plan_export(const padoc_plan* P, padoc_schedule_view* v) {
  clear_error();
  if (!P || !v) return set_error(PADOC_ERR_ARG, "null argument");
  std::memset(v, 0, sizeof(*v));
  v->kind = P->kind;
  v->tile_cols = P->tile_cols;
  v->tile_keys = P->tile_keys;
  v->n_work = (int32_t)P->work.size();
  v->work = P->work.data();
  v->n_work_shared = P->n_work_shared;
  v->n_range = (int32_t)P->ranges.size();
  v->ranges = P->ranges.data();
  v->n_lim = (int32_t)P->lims.size();
  v->lims = P->lims.data();
  v->n_tok = (int32_t)P->toks.size();
  v->toks = P->toks.data();
  // Tile classes are derived from the ranges on the first export (the
  // kernels classify tiles from n_keys and min_lim themselves).
  {
    std::lock_guard<std::mutex> lk(P->tc_mu);
    if (!P->tc_built) {
      P->tile_class_off.reserve(P->ranges.size());
      for (const auto& r : P->ranges) {
        P->tile_class_off.push_back((int64_t)P->tile_class.size());
        const int32_t nkt = (int32_t)ceil_div(r.n_keys, P->tile_keys);
        for (int32_t kt = 0; kt < nkt; ++kt)
          P->tile_class.push_back((int64_t)(kt + 1) * P->tile_keys <= r.min_lim ? 1 : 2);
      }
      P->tc_built = true;
    }
  }
  v->n_tile_class = (int64_t)P->tile_class.size();
  v->tile_class = P->tile_class.data();
  v->tile_class_off = P->tile_class_off.data();
  v->n_comb_ptr = (int64_t)P->comb_ptr.size();
  v->comb_ptr = P->comb_ptr.data();
  v->n_comb = (int64_t)P->comb_slot.size();
  v->comb_slot = P->comb_slot.data();
  v->n_comb_rows = (int64_t)P->comb_rows.size();
  v->comb_rows = P->comb_rows.data();
  v->n_bwd = (int32_t)P->bwd.size();
  v->bwd = P->bwd.data();
  v->n_btok = (int64_t)P->btoks.size();
  v->btoks = P->btoks.data();
  v->n_blim = (int64_t)P->blims.size();
  v->blims = P->blims.data();
  v->n_slots = P->n_slots;
  v->workspace_bytes = P->ws_bytes;
  return PADOC_OK;
}

extern "C" const char* padoc_last_error(void) { return padoc::last_error(); }
