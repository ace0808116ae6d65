// Host-side plan: validated tree + serialised schedule.  Pure C++17, no HIP
// calls, so it builds and runs on machines without a GPU.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <mutex>
#include <string>
#include <vector>

#include "../schedule.hpp"

struct padoc_plan {
  int32_t kind = 0;  // 0 forward (final O/LSE), 1 decode (partials + combine)
  int32_t Hq = 0, Hkv = 0, G = 0, D = 0;
  float scale = 0.f;
  padoc_dtype dtype = PADOC_BF16;
  int32_t block_size = 0;
  int64_t num_kv_rows = 0, num_q_rows = 0, block_table_len = 0;
  std::vector<padoc_segment> seg;

  int32_t tile_cols = padoc::kTileCols;
  int32_t tile_keys = padoc::kTileKeys;
  int32_t tile_tokens = 0;  // tokens per work item = tile_cols / G

  std::vector<padoc::WorkRec> work;
  int32_t n_work_shared = 0;  // decode: work[0 .. n_work_shared) are tile items
  int32_t n_private_groups = 0;  // decode: workgroups that only take private items
  std::vector<padoc::RangeRec> ranges;
  std::vector<int32_t> lims;
  std::vector<int32_t> toks;
  // Export only, filled on the first padoc_plan_export after a build.
  mutable std::vector<int8_t> tile_class;
  mutable std::vector<int64_t> tile_class_off;  // per range: first entry in tile_class
  mutable std::mutex tc_mu;
  mutable bool tc_built = false;
  std::vector<int32_t> comb_ptr;
  std::vector<int32_t> comb_slot;
  std::vector<int32_t> comb_rows;  // (row*Hkv + kvh) pairs the combine kernel merges
  int64_t n_slots = 0;

  // Backward (packed bf16 plans): key-major items and their token lists.
  std::vector<padoc::BwdRec> bwd;
  std::vector<int32_t> btoks, blims;
  std::vector<unsigned char> bwd_blob;  // bwd, btoks, blims (uploaded by padoc_tree_attn_bwd)
  size_t boff_bwd = 0, boff_btoks = 0, boff_blims = 0;
  size_t bws_off_blob = 0, bws_off_dd = 0, bws_off_dk = 0, bws_off_dv = 0, bws_bytes = 0;
  mutable std::once_flag bpin_once;
  mutable void* bpinned = nullptr;

  // Serialised schedule (uploaded into the workspace before every launch).
  std::vector<unsigned char> blob;
  size_t off_work = 0, off_ranges = 0, off_lims = 0, off_toks = 0;
  size_t off_comb_slot = 0, off_comb_rows = 0, off_part_o = 0, off_part_ml = 0;
  size_t off_next = 0;  // decode: private item queue counters (zeros in the blob)
  size_t ws_bytes = 0;

  // Incremented by every build of the plan (plans rebuilt in place).
  uint64_t build_id = 0;

  // Pinned host copy of `blob` (made on the first launch after a build, so
  // the schedule upload is a true asynchronous DMA; freed by
  // padoc_plan_destroy), the build it holds, and for rebuilt plans an event
  // (hipEvent_t) after the last upload that read it.
  mutable std::mutex pin_mu;
  mutable void* pinned = nullptr;
  mutable size_t pinned_cap = 0;
  mutable uint64_t pinned_build = 0;
  mutable void* pin_ev = nullptr;
  // The workspace the last schedule upload of this build went to (under
  // pin_mu): padoc_branch_decode_resident refuses any other.
  mutable const void* up_ws = nullptr;
  mutable uint64_t up_build = 0;
};

namespace padoc {

// Validate `desc` and build its schedule into `plan`, replacing what the plan
// held (its vectors keep their memory, so rebuilding one plan per decode
// step allocates little).  Host only.
padoc_status build_plan(const padoc_tree_desc* desc, padoc_plan& plan);

// Thread-local error state shared by every C entry point.
padoc_status set_error(padoc_status st, const char* fmt, ...);
void clear_error();
const char* last_error();

}  // namespace padoc
