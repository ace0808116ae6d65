// Decode session state: the streams of every page being decoded, the pool
// of paged-cache blocks and the block-table regions they occupy, and the
// prepared step.  Pure C++17 host code; the launch (HIP) side only reads it
// and owns the pinned staging buffers.
#pragma once

#include <stdint.h>

#include <vector>

#include "plan.hpp"

struct padoc_session {
  padoc_session_desc desc{};

  struct Stream {
    int32_t parent = -1, fork = 0, len = 0;
    bool open = true;
    bool kept = true;  // false once released (blocks and region returned)
    int32_t kept_children = 0;
    int64_t bt_off = 0;  // first entry of the block-table region
    int32_t cls = -1;    // region holds 1 << cls entries; -1 = no region yet
    std::vector<int32_t> blocks;
    // per step: index in the step's tree, and a region the stream moves to
    // (-1: none) while the step is being prepared
    int32_t index = -1;
    int64_t moving_to = -1;
  };
  std::vector<Stream> st;
  std::vector<int32_t> open_ids, kept_ids;  // ascending
  std::vector<int32_t> free_blocks;         // stack of pool block ids
  std::vector<std::vector<int64_t>> free_regions;  // per size class
  int64_t bt_top = 0;                       // table entries handed out so far
  std::vector<int32_t> bt_host;             // host copy of the device table

  // The prepared step.
  bool prepared = false;
  padoc_plan plan;
  std::vector<padoc_segment> seg;
  std::vector<int32_t> seg_id, row_id, new_off, q_off, new_slot, patch;
  std::vector<int32_t> row_n_new;
  size_t off_patch = 0, rec_bytes = 0;  // workspace: slots at 0, patches at off_patch
  size_t ws_records = 0, ws_bytes = 0;  // records area (aligned), total

  // Launch side: two pinned staging buffers and the events of their last
  // uploads (hipEvent_t), created on the first launch.
  void* stage[2] = {nullptr, nullptr};
  size_t stage_cap[2] = {0, 0};
  void* stage_ev[2] = {nullptr, nullptr};
  int stage_next = 0;
};

namespace padoc {

// Host side of padoc_session_destroy (frees no device or pinned memory).
void session_free_host(padoc_session* s);

}  // namespace padoc
