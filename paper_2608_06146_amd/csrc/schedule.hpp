// Device-side schedule records and kernel parameter blocks.
//
// The planner (host/plan.cpp) serialises these records into the caller's
// workspace; the kernels read them.  The record layouts are the ones the C
// ABI exports for inspection (padoc_work_view / padoc_range_view).
#pragma once

#include <stdint.h>

#include "padoc_attn.h"  // include/ is on the include path

namespace padoc {

using WorkRec = padoc_work_view;    // 48 bytes
using RangeRec = padoc_range_view;  // 32 bytes
using BwdRec = padoc_bwd_view;      // 40 bytes
static_assert(sizeof(WorkRec) == 48, "work record is 48 bytes");
static_assert(sizeof(RangeRec) == 32, "range record is 32 bytes");
static_assert(sizeof(BwdRec) == 40, "backward record is 40 bytes");

// Key tile of every kernel (keys staged per step) and columns per work item.
constexpr int kTileKeys = 64;
constexpr int kTileCols = 256;
constexpr int kBlock = 16;  // paged KV block (tokens)
constexpr int kPrivateCols = 16;  // columns of a private decode item (one wavefront)
constexpr int kPrivateQueues = 8;  // decode: private item queues (one per XCD)
constexpr int kBwdKeys = 128;     // keys of a backward key-major item (4 x 32)
constexpr int kMaxItemKeys = 8192;  // decode: keys of a chunk (item) at most
constexpr int kMaxItemTiles = kMaxItemKeys / kTileKeys;  // tiles of a paged tile item at most

// Everything a tile kernel needs.  Pointers are device pointers.
struct TileParams {
  const void* q;          // [n_q, Hq, D]
  const void* k;          // packed [T, Hkv, D] or paged [blocks, Hkv, 16, D]
  const void* v;
  void* o;                // final mode: [n_q, Hq, D]
  float* lse;             // final mode: [n_q, Hq]
  const int32_t* block_table;  // paged mode
  const WorkRec* work;
  const RangeRec* ranges;
  const int32_t* lims;
  const int32_t* toks;
  float* part_o;          // partial mode: [slots, D] unnormalised accumulators
  float* part_ml;         // partial mode: [slots, 2] (running max in log2 units, sum)
  int32_t Hq, Hkv, G;
  float scale_log2;       // softmax_scale * log2(e)
};

// Backward of the packed forward (bf16).
struct BwdParams {
  const void* q;     // [n_q, Hq, D]
  const void* k;     // [T, Hkv, D]
  const void* v;
  const void* o;     // [n_q, Hq, D]
  const float* lse;  // [n_q, Hq]
  const void* dout;  // [n_q, Hq, D]
  void* dq;          // [n_q, Hq, D]
  void* dk;          // [T, Hkv, D]
  void* dv;
  float* dd;         // workspace [n_q, Hq]: sum_d dout * o
  float* dk_acc;     // workspace [T, Hkv, D] fp32
  float* dv_acc;
  const WorkRec* work;  // the forward's query-major items (dQ)
  const RangeRec* ranges;
  const int32_t* lims;
  const int32_t* toks;
  const BwdRec* bwd;    // key-major items (dK, dV)
  const int32_t* btoks;
  const int32_t* blims;
  int64_t n_q, T;
  int32_t Hq, Hkv, G;
  float scale, scale_log2;
};

struct CombineParams {
  const int32_t* comb_slot;  // partial slots, grouped by (row, KV head)
  const int4* comb_rows;     // per merged pair: {row*Hkv + kvh, first, end, 0} into comb_slot
  int64_t n_rows;
  const float* part_o;
  const float* part_ml;
  void* o;
  float* lse;
  int64_t n_q;
  int32_t Hq, Hkv, G;
  int32_t* next;  // decode: the step kernel's kPrivateQueues queue counters (256 bytes apart), zeroed for the next call
};

}  // namespace padoc
