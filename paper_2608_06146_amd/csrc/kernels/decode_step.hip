// One decode step of the live streams over the paged cache (App. E; Attn
// equation with the ancestor mask), bf16: the shared-key tile items and the
// private-key items in one launch.
//
// Workgroups 0 .. n_shared-1 each run one shared tile item on all 8
// wavefronts (fwd_item: every sibling column of a KV head against each K/V
// tile).  Then every wavefront of the launch -- of the tile workgroups and of
// the workgroups after them -- takes private items, one at a time, from
// queues (atomic counters that the schedule upload zeroes), in the plan's
// order (largest first).  A workgroup fills a compute unit's registers and
// workgroups are dispatched in index order, so the tile items hold n_shared
// compute units (the planner keeps them to part of the chip) while private
// items stream keys on the rest, and the tile items' units join in as they
// finish: the matrix-core-bound shared keys and the HBM-bound private keys
// overlap, and no wavefront idles while private items are left.  Every item
// writes split partials; the combine kernel merges them.
//
// Private item (a branch's own history, seen only by its own queries): up to
// 16 columns (query token x head) on one wavefront, streaming the item's
// paged keys from HBM straight into matrix-core operand registers, 32 keys
// per step.
//
// Per step, with v_mfma_f32_16x16x32_bf16 (lane l: row/column l%16, group
// g = l/16 holding eight consecutive K-dimension elements; K blocks are
// chunk-major, so every 16-byte K load of a lane group is part of a full
// 128-byte line):
//   S^T = K Q^T     two 16-key M blocks; row m of block mb holds key
//                   8*(m/4) + 4*mb + m%4, so each lane's eight scores are the
//                   keys 8g .. 8g+7 of the step
//   online softmax  one column per lane group (4 lanes x 8 scores)
//   O^T += V^T P^T  P^T is the lane's 8 scores; V^T comes from d-major V
//                   blocks ([d][16 tokens]) as one 16-byte load per lane.
// Two register sets hold the K and V of two future steps: a set is refilled
// right after its last use, so every load has two steps of compute to land.
// The item's records and the block ids are scalar loads (their own wait
// counter), and a step's block ids are requested one step before its K/V
// loads, so no wait for metadata also waits for K/V data in flight; the
// column maxima use lane-swap instructions rather than LDS shuffles.
// Keys past a range's end are never used: their scores are masked and V
// elements past the end are zeroed before they reach a product.  Outputs are
// split partials (unnormalised O, running max in log2 units, sum).
#include <type_traits>

#include "device_common.hpp"
#include "fwd_item.hpp"

namespace padoc {

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8_t as_bf16x8(const uint4& u) { return *reinterpret_cast<const bf16x8_t*>(&u); }

// Key (within a 32-key step) held by row m of 16-key M block mb.
__device__ __forceinline__ int step_key(int mb, int m) { return 8 * (m >> 2) + 4 * mb + (m & 3); }

// Register sets of a private item's K/V pipeline: steps in flight.
constexpr int kSets = 2;

// Private work item `item` on the wavefront whose lane index is `lane`.
template <int D>
__device__ __forceinline__ void private_item(const TileParams& p, int item, int lane) {
  constexpr int NDS = D / 32;  // K-slices (32 d each) of the score product
  constexpr int NDM = D / 16;  // 16-row blocks of O^T
  const WorkRec w = load_scalar(p.work + item);
  // A one-range, one-token item without limits carries its range and its Q
  // row in the work record: its first loads wait for one record, not three.
  const bool direct = w.direct[0] >= 0;
  const int n = lane & 15, g = lane >> 4;
  const int G = p.G;
  const int kvh = w.kvh;
  const int64_t Hkv = p.Hkv;
  const int col = w.col0 + n;
  const int t = col / G;
  const bool valid = n < w.ncol && t < w.ntok;
  const int32_t qrow = !valid ? 0 : direct ? w.direct[2] : p.toks[w.tok_begin + t];
  const int32_t hq = kvh * G + (col - t * G);
  const uint16_t* Kc = static_cast<const uint16_t*>(p.k);
  const uint16_t* Vc = static_cast<const uint16_t*>(p.v);
  const int32_t* bt = p.block_table;

  // Q fragments (B operand): column n, d = ds*32 + 8g .. +7.
  bf16x8_t bq[NDS];
  const uint16_t* qp = static_cast<const uint16_t*>(p.q) + ((int64_t)qrow * p.Hq + hq) * D + 8 * g;
#pragma unroll
  for (int ds = 0; ds < NDS; ++ds)
    bq[ds] = as_bf16x8(valid ? *reinterpret_cast<const uint4*>(qp + ds * 32) : make_uint4(0, 0, 0, 0));

  // Step cursors over the item's ranges: C = step being computed, L = next
  // step to load (two ahead of C once the pipeline is full).
  // No implicit padding: copies of a padded struct keep the padding in
  // memory (the compiler would place it in LDS).
  struct Cursor {
    int ri, st;
    RangeRec R;
    int ok, unused;
  };
  auto advance = [&](Cursor& c) __attribute__((always_inline)) {
    if (++c.st * 32 >= c.R.n_keys) {
      c.st = 0;
      if (++c.ri < w.rng_count)
        c.R = load_scalar(p.ranges + w.rng_begin + c.ri);
      else
        c.ok = 0;
    }
  };
  RangeRec R0;
  if (direct) {
    R0.kv_start = w.direct[0];
    R0.n_keys = w.direct[1];
    R0.min_lim = w.direct[1];
    R0.lim_off = -1;
    R0.seg = 0;
    R0.key_begin = 0;
    R0.reserved = 0;
  } else {
    R0 = load_scalar(p.ranges + w.rng_begin);
  }
  Cursor C{0, 0, R0, 1, 0};
  Cursor L = C;  // once exhausted (ok = 0) it still names a valid step of the last range

  uint4 kf[kSets][2][NDS];  // [set][M block][K-slice]
  uint4 vf[kSets][NDM];     // [set][16-row d block]
  int vkeep[kSets];
  int64_t blk[kSets][2];    // [set][block of the step's first/second 16 keys]
  int32_t nid[2];       // block ids of the load cursor's step, requested ahead

  auto fetch_ids = [&](const Cursor& c) __attribute__((always_inline)) {
    const int kb = c.st * 32;
    const int32_t* b = bt + c.R.kv_start + (kb >> 4);
    nid[0] = load_scalar(b);
    nid[1] = load_scalar(b + ((kb + 16 < c.R.n_keys) ? 1 : 0));
  };
  // Loads of set X for the load cursor's step.  Past the item's last step
  // (real = false) the same loads read this lane's Q row instead (cached,
  // in bounds, never used): every step issues the same loads, so the
  // compiler's waits for a set stay exact (a load under a branch would make
  // it wait for every load in flight).
  auto load_k = [&](int X, bool real) __attribute__((always_inline)) {
    blk[X][0] = nid[0];
    blk[X][1] = nid[1];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
      // dims ds*32 + 8g .. +7 = chunk 4ds + g; with the chunk-major block
      // layout the 16 lanes of a group read two full 128-byte lines
      const int key = step_key(mb, n);
      const uint16_t* kp = Kc + paged_k_offset<D>(blk[X][key >> 4], kvh, (int32_t)Hkv, key & 15, g);
#pragma unroll
      for (int ds = 0; ds < NDS; ++ds)
        kf[X][mb][ds] = load_stream16(real ? kp + ds * 4 * (kBlock * 8) : qp + ds * 32);
    }
  };
  auto load_v = [&](const Cursor& c, int X, bool real) __attribute__((always_inline)) {
    const int keep = c.R.n_keys - (c.st * 32 + 8 * g);  // keys 8g .. 8g+7 of the step
    const uint16_t* vp = Vc + ((blk[X][g >> 1] * Hkv + kvh) * D + n) * kBlock + 8 * (g & 1);
#pragma unroll
    for (int dm = 0; dm < NDM; ++dm)
      vf[X][dm] = load_stream16(real ? vp + dm * 16 * kBlock : qp + dm * 16);
    vkeep[X] = keep;
  };

  float m_run = -INFINITY, l_part = 0.f;
  f32x4_t acc[NDM];
#pragma unroll
  for (int dm = 0; dm < NDM; ++dm) acc[dm] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  // This column's limit in the compute cursor's range: the range's length
  // when it has no limits, else the entry of the column's token (scalar
  // loads of the item's tokens' entries, picked per lane).
  int lim = 0;
  const int t_lo = w.col0 / G, t_hi = min(w.ntok - 1, (w.col0 + kPrivateCols - 1) / G);
  auto load_lim = [&]() __attribute__((always_inline)) {
    if (C.R.lim_off < 0) {
      lim = C.R.n_keys;
      return;
    }
    int v = 0;
    for (int i = t_lo; i <= t_hi; ++i) {
      const int32_t li = load_scalar(p.lims + C.R.lim_off + i);
      v = t == i ? li : v;
    }
    lim = valid ? v : 0;
  };
  load_lim();
  const float sl2 = p.scale_log2;

  // Prologue: steps 0 .. kSets-1 into sets 0 .. kSets-1, the block ids of
  // step kSets.  Branch-free: an exhausted load cursor still names a valid
  // step.
  fetch_ids(L);
  load_k(0, true);
  load_v(L, 0, true);
  advance(L);
#pragma unroll
  for (int X = 1; X < kSets; ++X) {
    const bool real = L.ok;
    fetch_ids(L);
    load_k(X, real);
    load_v(L, X, real);
    advance(L);
  }
  fetch_ids(L);

  // Step of the compute cursor on register set X, then refill set X with the
  // load cursor's step (kSets ahead) and request the block ids of the step
  // after it; false once the item's last step is done.
  auto step = [&](auto xc) __attribute__((always_inline)) -> bool {
    constexpr int X = decltype(xc)::value;
    const int kb = C.st * 32;
    f32x4_t S[2];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
      S[mb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ds = 0; ds < NDS; ++ds)
        S[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kf[X][mb][ds]), bq[ds], S[mb], 0, 0, 0);
    }
    const bool more = L.ok;
    load_k(X, more);  // set X's K is consumed
    if (kb + 32 > C.R.min_lim) {
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (kb + 8 * g + 4 * mb + i >= lim) S[mb][i] = -INFINITY;
    }
    float mx = fmaxf(fmaxf(fmaxf(S[0][0], S[0][1]), fmaxf(S[0][2], S[0][3])),
                     fmaxf(fmaxf(S[1][0], S[1][1]), fmaxf(S[1][2], S[1][3])));
    mx = max_lane_halves(max_lane_rows(mx));
    const float m_new = fmaxf(m_run, mx * sl2);
    const float m_sub = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = fast_exp2(m_run - m_sub);
    m_run = m_new;
    float e[8];
    float ls = 0.f;
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        e[4 * mb + i] = fast_exp2(fmaf(S[mb][i], sl2, -m_sub));
        ls += e[4 * mb + i];
      }
    l_part = fmaf(l_part, alpha, ls);
    bf16x8_t pb;
#pragma unroll
    for (int s = 0; s < 8; ++s) pb[s] = (__bf16)e[s];
#pragma unroll
    for (int dm = 0; dm < NDM; ++dm) {
      acc[dm] *= alpha;
      acc[dm] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(keep_first(vf[X][dm], vkeep[X])), pb, acc[dm], 0, 0, 0);
    }
    load_v(L, X, more);  // set X's V is consumed
    advance(L);
    fetch_ids(L);  // used by the next step's K loads
    const int ri_before = C.ri;
    advance(C);
    if (!C.ok) return false;
    if (C.ri != ri_before) load_lim();
    return true;
  };
  for (bool go = true; go;)
    tile::static_for<kSets>([&](auto xc) __attribute__((always_inline)) {
      if (go) go = step(xc);
    });

  float lt = l_part + __shfl_xor(l_part, 16);
  lt += __shfl_xor(lt, 32);
  if (!valid) return;
  const int64_t slot = (int64_t)w.out_base + col;
  float* op = p.part_o + slot * D + 4 * g;
#pragma unroll
  for (int dm = 0; dm < NDM; ++dm)
    *reinterpret_cast<float4*>(op + dm * 16) = make_float4(acc[dm][0], acc[dm][1], acc[dm][2], acc[dm][3]);
  if (g == 0) {
    p.part_ml[2 * slot] = m_run;
    p.part_ml[2 * slot + 1] = lt;
  }
}

// Private items are dealt to kQueues queues (item j to queue j % kQueues),
// one per XCD: workgroup b runs on XCD b % 8, and a wavefront takes from
// the queue of its workgroup's index, so the atomics of a queue stay within
// one XCD's compute units and the 8 counters (256 bytes apart) are served in
// parallel.  The wavefronts of the workgroups after the tile items start with
// a fixed item each (no atomic on the launch's critical start); every later
// item comes from the queue's counter.
constexpr int kQueues = kPrivateQueues;

__device__ __forceinline__ int take_private(int* ctr, int lane) {
  int v = 0;
  if (lane == 0) v = atomicAdd(ctr, 1);
  return __builtin_amdgcn_readfirstlane(v);
}

template <int D>
__global__ __launch_bounds__(tile::kThreads) void decode_step_kernel(TileParams p, int n_shared, int n_private,
                                                                     int n_groups, int* next) {
  const int b = blockIdx.x;
  if (b < n_shared) tile::fwd_item<D, true>(p, b);
  if (n_private <= 0) return;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int q = b % kQueues;
  const int n_q = (n_private - q + kQueues - 1) / kQueues;  // items q, q + 8, ... below n_private
  // Private-only workgroups of queue q: b0, b0 + 8, ... below n_shared + n_groups.
  const int end = n_shared + n_groups;
  const int b0 = n_shared + (q - n_shared % kQueues + kQueues) % kQueues;
  const int n_first = b0 < end ? ((end - 1 - b0) / kQueues + 1) * tile::kWaves : 0;
  int* ctr = next + q * 64;
  // An index is taken only when the wavefront is free: one reserved ahead
  // would sit behind a long item while another wavefront idles.
  int k = b >= n_shared ? ((b - b0) / kQueues) * tile::kWaves + wave : n_first + take_private(ctr, lane);
  while (k < n_q) {
    private_item<D>(p, n_shared + q + kQueues * k, lane);
    k = n_first + take_private(ctr, lane);
  }
}

}  // namespace

// n_groups: workgroups after the tile items (they take private items only).
// `next`: kQueues counters 256 bytes apart, zero at launch.
hipError_t launch_decode_step_bf16(const TileParams& p, int n_shared, int n_private, int n_groups, int* next, int D,
                                   hipStream_t stream) {
  const int n_blocks = n_shared + n_groups;
  if (n_blocks <= 0) return hipSuccess;
  const dim3 grid(n_blocks), block(tile::kThreads);
  if (D == 64)
    hipLaunchKernelGGL((decode_step_kernel<64>), grid, block, 0, stream, p, n_shared, n_private, n_groups, next);
  else
    hipLaunchKernelGGL((decode_step_kernel<128>), grid, block, 0, stream, p, n_shared, n_private, n_groups, next);
  return hipGetLastError();
}

}  // namespace padoc
