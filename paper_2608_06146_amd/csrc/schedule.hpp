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
static_assert(sizeof(WorkRec) == 48, "work record is 48 bytes");
static_assert(sizeof(RangeRec) == 32, "range record is 32 bytes");

// Key tile of every kernel (keys staged per step) and columns per work item.
constexpr int kTileKeys = 64;
constexpr int kTileCols = 256;
constexpr int kBlock = 16;  // paged KV block (tokens)
constexpr int kPrivateCols = 16;  // columns of a private decode item (one wavefront)

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
  const int32_t* comb_ptr;   // decode: partial slots per (row, KV head) ...
  const int32_t* comb_slot;  // ... merged by items with fin = 1
  int32_t Hq, Hkv, G;
  float scale_log2;       // softmax_scale * log2(e)
};

struct CombineParams {
  const int32_t* comb_ptr;   // [n_q * Hkv + 1]
  const int32_t* comb_slot;
  const int32_t* comb_rows;  // (row*Hkv + kvh) pairs to merge
  int64_t n_rows;
  const float* part_o;
  const float* part_ml;
  void* o;
  float* lse;
  int64_t n_q;
  int32_t Hq, Hkv, G;
};

}  // namespace padoc
