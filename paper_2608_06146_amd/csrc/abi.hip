// C entry points that launch work: argument checks, schedule upload into the
// caller's workspace, and the kernel launches on the caller's stream.
#include <hip/hip_runtime.h>

#include <cstring>

#include "host/plan.hpp"

namespace padoc {
hipError_t launch_tile_mfma_bf16(const TileParams& p, int n_work, int D, bool paged, hipStream_t s);
hipError_t launch_decode_private_bf16(const TileParams& p, int n_items, int D, hipStream_t s);
hipError_t launch_tile_valu_f32(const TileParams& p, int n_work, int D, bool paged, hipStream_t s);
hipError_t launch_lse_combine(const CombineParams& p, int D, bool bf16, hipStream_t s);
hipError_t launch_tree_attn_bwd(const BwdParams& p, int n_work, int n_bwd, int D, hipStream_t s);

namespace {
thread_local hipEvent_t t_ev_before = nullptr;
thread_local hipEvent_t t_ev_after = nullptr;

padoc_status hip_fail(const char* what, hipError_t e) {
  return set_error(PADOC_ERR_HIP, "%s failed: %s (%d)", what, hipGetErrorString(e), (int)e);
}

template <class T>
const T* at(void* ws, size_t off) {
  return reinterpret_cast<const T*>(static_cast<char*>(ws) + off);
}

padoc_status check_common(const padoc_plan* P, const void* q, const void* k, const void* v, const void* o,
                          const float* lse, void* ws, size_t ws_bytes) {
  if (!P) return set_error(PADOC_ERR_ARG, "plan is null");
  if (!P->work.empty()) {
    if (!q || !k || !v || !o || !lse) return set_error(PADOC_ERR_ARG, "a tensor pointer is null");
    if (((uintptr_t)q | (uintptr_t)k | (uintptr_t)v | (uintptr_t)o) & 15)
      return set_error(PADOC_ERR_ARG, "q, k, v and o must be 16-byte aligned");
    if (((uintptr_t)lse) & 3) return set_error(PADOC_ERR_ARG, "lse must be 4-byte aligned");
  }
  if (!ws) return set_error(PADOC_ERR_WORKSPACE, "workspace is null");
  if (((uintptr_t)ws) & 255) return set_error(PADOC_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (ws_bytes < P->ws_bytes)
    return set_error(PADOC_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu the plan needs", ws_bytes,
                     P->ws_bytes);
  return PADOC_OK;
}

// The plan's schedule in pinned host memory (made once per plan).
const void* pinned_blob(const padoc_plan* P) {
  std::call_once(P->pin_once, [P] {
    void* h = nullptr;
    hipError_t e = hipHostMalloc(&h, P->blob.size(), hipHostMallocDefault);
    if (e == hipSuccess) {
      std::memcpy(h, P->blob.data(), P->blob.size());
      P->pinned = h;
    }
    P->pin_status = (int)e;
  });
  return P->pinned ? P->pinned : P->blob.data();
}

// The plan's backward schedule in pinned host memory (made once per plan).
const void* pinned_bwd_blob(const padoc_plan* P) {
  std::call_once(P->bpin_once, [P] {
    void* h = nullptr;
    if (hipHostMalloc(&h, P->bwd_blob.size(), hipHostMallocDefault) == hipSuccess) {
      std::memcpy(h, P->bwd_blob.data(), P->bwd_blob.size());
      P->bpinned = h;
    }
  });
  return P->bpinned ? P->bpinned : P->bwd_blob.data();
}

padoc_status run(const padoc_plan* P, const void* q, const void* k, const void* v, const int32_t* bt, void* o,
                 float* lse, void* ws, hipStream_t stream) {
  if (P->work.empty()) return PADOC_OK;
  hipError_t e = hipMemcpyAsync(ws, pinned_blob(P), P->blob.size(), hipMemcpyHostToDevice, stream);
  if (e != hipSuccess) return hip_fail("hipMemcpyAsync(schedule)", e);
  TileParams tp{};
  tp.q = q;
  tp.k = k;
  tp.v = v;
  tp.o = o;
  tp.lse = lse;
  tp.block_table = bt;
  tp.work = at<WorkRec>(ws, P->off_work);
  tp.ranges = at<RangeRec>(ws, P->off_ranges);
  tp.lims = at<int32_t>(ws, P->off_lims);
  tp.toks = at<int32_t>(ws, P->off_toks);
  tp.part_o = reinterpret_cast<float*>(static_cast<char*>(ws) + P->off_part_o);
  tp.part_ml = reinterpret_cast<float*>(static_cast<char*>(ws) + P->off_part_ml);
  tp.comb_ptr = at<int32_t>(ws, P->off_comb_ptr);
  tp.comb_slot = at<int32_t>(ws, P->off_comb_slot);
  tp.Hq = P->Hq;
  tp.Hkv = P->Hkv;
  tp.G = P->G;
  tp.scale_log2 = P->scale * 1.4426950408889634f;
  const bool paged = P->block_size != 0;
  const bool partial = P->kind == 1;  // decode plans: wave items, split-KV partials
  const int n_work = (int)P->work.size();
  if (t_ev_before && t_ev_after) {
    e = hipEventRecord(t_ev_before, stream);
    if (e != hipSuccess) return hip_fail("hipEventRecord", e);
  }
  if (P->dtype == PADOC_BF16) {
    if (!paged) {
      e = launch_tile_mfma_bf16(tp, n_work, P->D, false, stream);
    } else {
      // Shared keys (all sibling columns per tile) on the tile kernel, then
      // private keys on the streaming kernel, whose epilogue also merges the
      // shared partials of its rows (they are complete: same stream, earlier).
      TileParams tq = tp;
      tq.work = tp.work + P->n_work_shared;
      e = launch_tile_mfma_bf16(tp, P->n_work_shared, P->D, true, stream);
      if (e == hipSuccess) e = launch_decode_private_bf16(tq, n_work - P->n_work_shared, P->D, stream);
    }
  } else {
    e = launch_tile_valu_f32(tp, n_work, P->D, paged, stream);
  }
  if (e != hipSuccess) return hip_fail("tile kernel launch", e);
  if (partial) {
    CombineParams cp{};
    cp.comb_ptr = at<int32_t>(ws, P->off_comb_ptr);
    cp.comb_slot = at<int32_t>(ws, P->off_comb_slot);
    cp.comb_rows = at<int32_t>(ws, P->off_comb_rows);
    cp.n_rows = (int64_t)P->comb_rows.size();
    cp.part_o = tp.part_o;
    cp.part_ml = tp.part_ml;
    cp.o = o;
    cp.lse = lse;
    cp.n_q = P->num_q_rows;
    cp.Hq = P->Hq;
    cp.Hkv = P->Hkv;
    cp.G = P->G;
    e = launch_lse_combine(cp, P->D, P->dtype == PADOC_BF16, stream);
    if (e != hipSuccess) return hip_fail("combine kernel launch", e);
  }
  if (t_ev_before && t_ev_after) {
    e = hipEventRecord(t_ev_after, stream);
    if (e != hipSuccess) return hip_fail("hipEventRecord", e);
  }
  return PADOC_OK;
}
}  // namespace
}  // namespace padoc

using namespace padoc;

extern "C" padoc_status padoc_tree_attn_fwd(const padoc_plan* plan, const void* q, const void* k, const void* v,
                                            void* o, float* lse, void* workspace, size_t workspace_bytes,
                                            hipStream_t stream) {
  clear_error();
  padoc_status st = check_common(plan, q, k, v, o, lse, workspace, workspace_bytes);
  if (st != PADOC_OK) return st;
  if (plan->kind != 0)
    return set_error(PADOC_ERR_MODE, "plan was built for paged K/V (block_size 16); use padoc_branch_decode");
  return run(plan, q, k, v, nullptr, o, lse, workspace, stream);
}

extern "C" padoc_status padoc_branch_decode(const padoc_plan* plan, const void* q, const void* k_cache,
                                            const void* v_cache, const int32_t* block_table, void* o, float* lse,
                                            void* workspace, size_t workspace_bytes, hipStream_t stream) {
  clear_error();
  padoc_status st = check_common(plan, q, k_cache, v_cache, o, lse, workspace, workspace_bytes);
  if (st != PADOC_OK) return st;
  if (plan->kind != 1)
    return set_error(PADOC_ERR_MODE, "plan was built for packed K/V (block_size 0); use padoc_tree_attn_fwd");
  if (!plan->work.empty() && !block_table) return set_error(PADOC_ERR_ARG, "block_table is null");
  return run(plan, q, k_cache, v_cache, block_table, o, lse, workspace, stream);
}

extern "C" padoc_status padoc_tree_attn_bwd(const padoc_plan* plan, const void* q, const void* k, const void* v,
                                            const void* o, const float* lse, const void* dout, void* dq, void* dk,
                                            void* dv, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  clear_error();
  if (!plan) return set_error(PADOC_ERR_ARG, "plan is null");
  if (plan->kind != 0)
    return set_error(PADOC_ERR_MODE, "the backward needs a packed plan (block_size 0)");
  if (plan->dtype != PADOC_BF16) return set_error(PADOC_ERR_DTYPE, "the backward supports bf16 plans only");
  if (!workspace) return set_error(PADOC_ERR_WORKSPACE, "workspace is null");
  if (((uintptr_t)workspace) & 255) return set_error(PADOC_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (workspace_bytes < plan->bws_bytes)
    return set_error(PADOC_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu the backward needs",
                     workspace_bytes, plan->bws_bytes);
  const bool any_q = plan->num_q_rows > 0, any_kv = plan->num_kv_rows > 0;
  if ((any_q && (!q || !o || !lse || !dout || !dq)) || (any_kv && (!k || !v || !dk || !dv)))
    return set_error(PADOC_ERR_ARG, "a tensor pointer is null");
  if (((uintptr_t)q | (uintptr_t)k | (uintptr_t)v | (uintptr_t)o | (uintptr_t)dout | (uintptr_t)dq |
       (uintptr_t)dk | (uintptr_t)dv) & 15)
    return set_error(PADOC_ERR_ARG, "q, k, v, o, dout, dq, dk and dv must be 16-byte aligned");
  if (((uintptr_t)lse) & 3) return set_error(PADOC_ERR_ARG, "lse must be 4-byte aligned");
  if (!any_q && !any_kv) return PADOC_OK;
  char* ws = static_cast<char*>(workspace);
  hipError_t e = hipSuccess;
  if (!plan->blob.empty()) e = hipMemcpyAsync(ws, pinned_blob(plan), plan->blob.size(), hipMemcpyHostToDevice, stream);
  if (e == hipSuccess && !plan->bwd_blob.empty())
    e = hipMemcpyAsync(ws + plan->bws_off_blob, pinned_bwd_blob(plan), plan->bwd_blob.size(), hipMemcpyHostToDevice,
                       stream);
  if (e != hipSuccess) return hip_fail("hipMemcpyAsync(schedule)", e);
  BwdParams bp{};
  bp.q = q;
  bp.k = k;
  bp.v = v;
  bp.o = o;
  bp.lse = lse;
  bp.dout = dout;
  bp.dq = dq;
  bp.dk = dk;
  bp.dv = dv;
  bp.dd = reinterpret_cast<float*>(ws + plan->bws_off_dd);
  bp.dk_acc = reinterpret_cast<float*>(ws + plan->bws_off_dk);
  bp.dv_acc = reinterpret_cast<float*>(ws + plan->bws_off_dv);
  bp.work = at<WorkRec>(ws, plan->off_work);
  bp.ranges = at<RangeRec>(ws, plan->off_ranges);
  bp.lims = at<int32_t>(ws, plan->off_lims);
  bp.toks = at<int32_t>(ws, plan->off_toks);
  bp.bwd = at<BwdRec>(ws, plan->bws_off_blob + plan->boff_bwd);
  bp.btoks = at<int32_t>(ws, plan->bws_off_blob + plan->boff_btoks);
  bp.blims = at<int32_t>(ws, plan->bws_off_blob + plan->boff_blims);
  bp.n_q = plan->num_q_rows;
  bp.T = plan->num_kv_rows;
  bp.Hq = plan->Hq;
  bp.Hkv = plan->Hkv;
  bp.G = plan->G;
  bp.scale = plan->scale;
  bp.scale_log2 = plan->scale * 1.4426950408889634f;
  if (t_ev_before && t_ev_after) {
    e = hipEventRecord(t_ev_before, stream);
    if (e != hipSuccess) return hip_fail("hipEventRecord", e);
  }
  e = launch_tree_attn_bwd(bp, (int)plan->work.size(), (int)plan->bwd.size(), plan->D, stream);
  if (e != hipSuccess) return hip_fail("backward kernel launch", e);
  if (t_ev_before && t_ev_after) {
    e = hipEventRecord(t_ev_after, stream);
    if (e != hipSuccess) return hip_fail("hipEventRecord", e);
  }
  return PADOC_OK;
}

extern "C" void padoc_plan_destroy(padoc_plan* plan) {
  if (!plan) return;
  if (plan->pinned) (void)hipHostFree(plan->pinned);
  if (plan->bpinned) (void)hipHostFree(plan->bpinned);
  delete plan;
}

extern "C" padoc_status padoc_set_kernel_events(hipEvent_t before, hipEvent_t after) {
  clear_error();
  if ((before == nullptr) != (after == nullptr))
    return set_error(PADOC_ERR_ARG, "pass both events or neither");
  t_ev_before = before;
  t_ev_after = after;
  return PADOC_OK;
}

extern "C" const char* padoc_version(void) { return "padoc_attn 0.1.0 (gfx950)"; }
