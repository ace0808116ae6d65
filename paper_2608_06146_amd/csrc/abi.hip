// C entry points that launch work: argument checks, schedule upload into the
// caller's workspace, and the kernel launches on the caller's stream.
#include <hip/hip_runtime.h>

#include <cstring>
#include <mutex>

#include "host/plan.hpp"
#include "host/session.hpp"

namespace padoc {
hipError_t launch_tile_mfma_bf16(const TileParams& p, int n_work, int D, hipStream_t s);
hipError_t launch_decode_step_bf16(const TileParams& p, int n_shared, int n_private, int n_groups, int* next, int D,
                                   hipStream_t s);
hipError_t launch_tile_valu_f32(const TileParams& p, int n_work, int D, bool paged, hipStream_t s);
hipError_t launch_lse_combine(const CombineParams& p, int D, bool bf16, hipStream_t s);
hipError_t launch_tree_attn_bwd(const BwdParams& p, int n_work, int n_bwd, int D, hipStream_t s);
hipError_t launch_relayout_kv(const void* k_rows, const void* v_rows, void* k_cache, void* v_cache, int64_t n_blocks,
                              int Hkv, int D, int elem_bytes, hipStream_t stream);
hipError_t launch_append_kv(const void* k_new, const void* v_new, void* k_cache, void* v_cache, const int32_t* slots,
                            int64_t n_rows, int Hkv, int D, bool bf16, const int32_t* patch, int64_t n_patch,
                            int32_t* block_table, hipStream_t s);

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

// The plan's schedule in pinned host memory, copied once per build of the
// plan.  A plan rebuilt in place (a session's per-step plan) overwrites the
// copy only after the upload that last read it has completed.
const void* pinned_blob(const padoc_plan* P) {
  std::lock_guard<std::mutex> lk(P->pin_mu);
  if (P->pinned_build != P->build_id) {
    if (P->pin_ev) (void)hipEventSynchronize(static_cast<hipEvent_t>(P->pin_ev));
    if (P->pinned && P->pinned_cap < P->blob.size()) {
      (void)hipHostFree(P->pinned);
      P->pinned = nullptr;
      P->pinned_cap = 0;
    }
    if (!P->pinned && !P->blob.empty()) {
      void* h = nullptr;
      if (hipHostMalloc(&h, P->blob.size(), hipHostMallocDefault) == hipSuccess) {
        P->pinned = h;
        P->pinned_cap = P->blob.size();
      }
    }
    if (P->pinned) std::memcpy(P->pinned, P->blob.data(), P->blob.size());
    P->pinned_build = P->build_id;
  }
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

// Copy plan P's schedule (with zeroed work-queue counters) into workspace
// ws on `stream`; `pinned`: from the plan's pinned host copy (made on first
// use), else straight from the plan's own host memory, allocating nothing.
padoc_status upload_schedule(const padoc_plan* P, void* ws, hipStream_t stream, bool pinned) {
  hipError_t e =
      hipMemcpyAsync(ws, pinned ? pinned_blob(P) : P->blob.data(), P->blob.size(), hipMemcpyHostToDevice, stream);
  if (e != hipSuccess) return hip_fail("hipMemcpyAsync(schedule)", e);
  std::lock_guard<std::mutex> lk(P->pin_mu);
  P->up_ws = ws;
  P->up_build = P->build_id;
  if (pinned && P->build_id > 1) {
    // a rebuilt plan: mark when its pinned copy may be overwritten
    if (!P->pin_ev) {
      hipEvent_t ev = nullptr;
      if (hipEventCreateWithFlags(&ev, hipEventDisableTiming) == hipSuccess) P->pin_ev = ev;
    }
    if (P->pin_ev) {
      e = hipEventRecord(static_cast<hipEvent_t>(P->pin_ev), stream);
      if (e != hipSuccess) return hip_fail("hipEventRecord", e);
    }
  }
  return PADOC_OK;
}

// Launch the attention of plan P.  `upload`: copy the schedule into the
// workspace first (else the caller already did); `events`: record the
// profiling events around the kernels.
// `pinned`: upload from the plan's pinned host copy (made on first use);
// else straight from the plan's own host memory, allocating nothing.
padoc_status run(const padoc_plan* P, const void* q, const void* k, const void* v, const int32_t* bt, void* o,
                 float* lse, void* ws, hipStream_t stream, bool upload = true, bool events = true,
                 bool pinned = true) {
  if (P->work.empty()) return PADOC_OK;
  hipError_t e = hipSuccess;
  if (upload) {
    padoc_status st = upload_schedule(P, ws, stream, pinned);
    if (st != PADOC_OK) return st;
  }
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
  tp.Hq = P->Hq;
  tp.Hkv = P->Hkv;
  tp.G = P->G;
  tp.scale_log2 = P->scale * 1.4426950408889634f;
  const bool paged = P->block_size != 0;
  const bool partial = P->kind == 1;  // decode plans: wave items, split-KV partials
  const int n_work = (int)P->work.size();
  if (events && t_ev_before && t_ev_after) {
    e = hipEventRecord(t_ev_before, stream);
    if (e != hipSuccess) return hip_fail("hipEventRecord", e);
  }
  if (P->dtype == PADOC_BF16) {
    if (!paged)
      e = launch_tile_mfma_bf16(tp, n_work, P->D, stream);
    else  // shared-key tile items and private-key items in one launch
      e = launch_decode_step_bf16(tp, P->n_work_shared, n_work - P->n_work_shared, P->n_private_groups,
                                  reinterpret_cast<int*>(static_cast<char*>(ws) + P->off_next), P->D, stream);
  } else {
    e = launch_tile_valu_f32(tp, n_work, P->D, paged, stream);
  }
  if (e != hipSuccess) return hip_fail("tile kernel launch", e);
  if (partial) {
    CombineParams cp{};
    cp.comb_slot = at<int32_t>(ws, P->off_comb_slot);
    cp.comb_rows = at<int4>(ws, P->off_comb_rows);
    cp.n_rows = (int64_t)P->comb_rows.size();
    cp.part_o = tp.part_o;
    cp.part_ml = tp.part_ml;
    cp.o = o;
    cp.lse = lse;
    cp.n_q = P->num_q_rows;
    cp.Hq = P->Hq;
    cp.Hkv = P->Hkv;
    cp.G = P->G;
    cp.next = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + P->off_next);
    e = launch_lse_combine(cp, P->D, P->dtype == PADOC_BF16, stream);
    if (e != hipSuccess) return hip_fail("combine kernel launch", e);
  }
  if (events && t_ev_before && t_ev_after) {
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

extern "C" padoc_status padoc_plan_upload(const padoc_plan* plan, void* workspace, size_t workspace_bytes,
                                          hipStream_t stream) {
  clear_error();
  if (!plan) return set_error(PADOC_ERR_ARG, "plan is null");
  if (plan->kind != 1) return set_error(PADOC_ERR_MODE, "padoc_plan_upload takes decode plans (block_size 16)");
  if (!workspace) return set_error(PADOC_ERR_WORKSPACE, "workspace is null");
  if (((uintptr_t)workspace) & 255) return set_error(PADOC_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (workspace_bytes < plan->ws_bytes)
    return set_error(PADOC_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu the plan needs",
                     workspace_bytes, plan->ws_bytes);
  if (plan->work.empty()) return PADOC_OK;
  return upload_schedule(plan, workspace, stream, /*pinned=*/true);
}

extern "C" padoc_status padoc_branch_decode_resident(const padoc_plan* plan, const void* q, const void* k_cache,
                                                     const void* v_cache, const int32_t* block_table, void* o,
                                                     float* lse, void* workspace, size_t workspace_bytes,
                                                     hipStream_t stream) {
  clear_error();
  padoc_status st = check_common(plan, q, k_cache, v_cache, o, lse, workspace, workspace_bytes);
  if (st != PADOC_OK) return st;
  if (plan->kind != 1)
    return set_error(PADOC_ERR_MODE, "plan was built for packed K/V (block_size 0); use padoc_tree_attn_fwd");
  if (!plan->work.empty() && !block_table) return set_error(PADOC_ERR_ARG, "block_table is null");
  if (plan->work.empty()) return PADOC_OK;
  {
    std::lock_guard<std::mutex> lk(plan->pin_mu);
    if (plan->up_ws != workspace || plan->up_build != plan->build_id)
      return set_error(PADOC_ERR_MODE,
                       "the workspace does not hold this plan's schedule (upload it with padoc_plan_upload after "
                       "every build of the plan)");
  }
  return run(plan, q, k_cache, v_cache, block_table, o, lse, workspace, stream, /*upload=*/false);
}

// Workspace of padoc_branch_decode_no_alloc: one array per GPU the library
// runs on, held until the process ends.  Host code never passes `scratch`
// itself to a kernel or a copy (on the host it names a stand-in, not device
// memory): it uses the device address hipGetSymbolAddress returns.
constexpr size_t kNoAllocScratchBytes = PADOC_NO_ALLOC_WORKSPACE_BYTES;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace padoc {
namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxDevices] = {};

// Device address of the current device's copy of `scratch`, looked up on
// the first call made with that device current.
padoc_status scratch_of_current_device(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail("hipGetDevice", e);
  if (dev < 0 || dev >= kMaxDevices) return set_error(PADOC_ERR_ARG, "device %d is out of range", dev);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail("hipGetSymbolAddress(scratch)", e);
    if (!p) return set_error(PADOC_ERR_HIP, "hipGetSymbolAddress(scratch) returned no address");
    g_scratch_addr[dev] = p;
  }
  *out = g_scratch_addr[dev];
  return PADOC_OK;
}
}  // namespace
}  // namespace padoc

extern "C" padoc_status padoc_branch_decode_no_alloc(const padoc_plan* plan, const void* q, const void* k_cache,
                                                     const void* v_cache, const int32_t* block_table, void* o,
                                                     float* lse, hipStream_t stream) {
  clear_error();
  if (!plan) return set_error(PADOC_ERR_ARG, "plan is null");
  if (plan->kind != 1)
    return set_error(PADOC_ERR_MODE, "plan was built for packed K/V (block_size 0); use padoc_tree_attn_fwd");
  if (plan->ws_bytes > kNoAllocScratchBytes)
    return set_error(PADOC_ERR_WORKSPACE,
                     "the plan needs %zu bytes of workspace; padoc_branch_decode_no_alloc holds at most %zu "
                     "(use padoc_branch_decode with a caller workspace)",
                     plan->ws_bytes, kNoAllocScratchBytes);
  void* ws = nullptr;
  padoc_status st = scratch_of_current_device(&ws);
  if (st != PADOC_OK) return st;
  st = check_common(plan, q, k_cache, v_cache, o, lse, ws, kNoAllocScratchBytes);
  if (st != PADOC_OK) return st;
  if (!plan->work.empty() && !block_table) return set_error(PADOC_ERR_ARG, "block_table is null");
  return run(plan, q, k_cache, v_cache, block_table, o, lse, ws, stream, /*upload=*/true, /*events=*/true,
             /*pinned=*/false);
}

extern "C" padoc_status padoc_cache_from_rows(const void* k_rows, const void* v_rows, void* k_cache, void* v_cache,
                                              int64_t num_blocks, int32_t num_heads_kv, int32_t head_dim,
                                              padoc_dtype dtype, hipStream_t stream) {
  clear_error();
  if (num_blocks < 0) return set_error(PADOC_ERR_ARG, "num_blocks = %lld is negative", (long long)num_blocks);
  if (num_heads_kv < 1) return set_error(PADOC_ERR_SHAPE, "num_heads_kv = %d must be >= 1", num_heads_kv);
  if (head_dim != 64 && head_dim != 128) return set_error(PADOC_ERR_SHAPE, "head_dim = %d is not 64 or 128", head_dim);
  if (dtype != PADOC_BF16 && dtype != PADOC_F32)
    return set_error(PADOC_ERR_DTYPE, "dtype %d is not PADOC_F32 or PADOC_BF16", (int)dtype);
  if (num_blocks == 0) return PADOC_OK;
  if (!k_rows || !v_rows || !k_cache || !v_cache) return set_error(PADOC_ERR_ARG, "null buffer pointer");
  if (k_rows == k_cache || v_rows == v_cache || k_rows == v_cache || v_rows == k_cache)
    return set_error(PADOC_ERR_ARG, "source and destination buffers must be distinct");
  if (num_blocks > INT64_MAX / ((int64_t)num_heads_kv * 16 * head_dim * 4))
    return set_error(PADOC_ERR_BOUNDS, "num_blocks = %lld overflows the cache size", (long long)num_blocks);
  const hipError_t e = launch_relayout_kv(k_rows, v_rows, k_cache, v_cache, num_blocks, num_heads_kv, head_dim,
                                          dtype == PADOC_BF16 ? 2 : 4, stream);
  if (e != hipSuccess) return hip_fail("relayout kernel launch", e);
  return PADOC_OK;
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
  if (plan->pin_ev) (void)hipEventDestroy(static_cast<hipEvent_t>(plan->pin_ev));
  if (plan->pinned) (void)hipHostFree(plan->pinned);
  if (plan->bpinned) (void)hipHostFree(plan->bpinned);
  delete plan;
}

// One step of a decode session: upload the step's slot list, block-table
// patches and schedule in one copy, append the new K/V rows (and patch the
// table), then the attention kernels.
extern "C" padoc_status padoc_session_launch(padoc_session* s, const void* q, const void* k_new, const void* v_new,
                                             void* o, float* lse, void* workspace, size_t workspace_bytes,
                                             hipStream_t stream) {
  clear_error();
  if (!s) return set_error(PADOC_ERR_ARG, "session is null");
  if (!s->prepared) return set_error(PADOC_ERR_MODE, "no step is prepared");
  const padoc_session_desc& d = s->desc;
  if (!d.k_cache || !d.v_cache || !d.block_table)
    return set_error(PADOC_ERR_ARG, "the session was created without device caches and block table");
  if (((uintptr_t)d.k_cache | (uintptr_t)d.v_cache) & 15)
    return set_error(PADOC_ERR_ARG, "the caches must be 16-byte aligned");
  const int64_t n_new = s->new_off.back(), n_q = s->q_off.back();
  const size_t esz = d.dtype == PADOC_BF16 ? 2 : 4;
  if (n_new > 0 && (!k_new || !v_new)) return set_error(PADOC_ERR_ARG, "k_new / v_new is null");
  if (((uintptr_t)k_new | (uintptr_t)v_new) & (esz - 1))
    return set_error(PADOC_ERR_ARG, "k_new / v_new are not aligned to their element size");
  const padoc_plan* P = &s->plan;
  if (n_q > 0) {
    if (!q || !o || !lse) return set_error(PADOC_ERR_ARG, "q, o or lse is null");
    if (((uintptr_t)q | (uintptr_t)o) & 15) return set_error(PADOC_ERR_ARG, "q and o must be 16-byte aligned");
    if (((uintptr_t)lse) & 3) return set_error(PADOC_ERR_ARG, "lse must be 4-byte aligned");
  }
  if (!workspace) return set_error(PADOC_ERR_WORKSPACE, "workspace is null");
  if (((uintptr_t)workspace) & 255) return set_error(PADOC_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (workspace_bytes < s->ws_bytes)
    return set_error(PADOC_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu the step needs",
                     workspace_bytes, s->ws_bytes);
  const int64_t n_patch = (int64_t)s->patch.size() / 2;
  const size_t up = s->ws_records + P->blob.size();
  char* ws = static_cast<char*>(workspace);
  hipError_t e = hipSuccess;
  if (up > 0) {
    const int k = s->stage_next;
    if (s->stage_ev[k]) {
      e = hipEventSynchronize(static_cast<hipEvent_t>(s->stage_ev[k]));
      if (e != hipSuccess) return hip_fail("hipEventSynchronize(staging)", e);
    } else {
      hipEvent_t ev = nullptr;
      e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
      if (e != hipSuccess) return hip_fail("hipEventCreateWithFlags", e);
      s->stage_ev[k] = ev;
    }
    if (s->stage_cap[k] < up) {
      if (s->stage[k]) (void)hipHostFree(s->stage[k]);
      s->stage[k] = nullptr;
      s->stage_cap[k] = 0;
      const size_t cap = up + up / 2;
      void* h = nullptr;
      e = hipHostMalloc(&h, cap, hipHostMallocDefault);
      if (e != hipSuccess) return hip_fail("hipHostMalloc(staging)", e);
      s->stage[k] = h;
      s->stage_cap[k] = cap;
    }
    char* h = static_cast<char*>(s->stage[k]);
    if (n_new > 0) std::memcpy(h, s->new_slot.data(), (size_t)n_new * 8);
    if (n_patch > 0) std::memcpy(h + s->off_patch, s->patch.data(), (size_t)n_patch * 8);
    if (!P->blob.empty()) std::memcpy(h + s->ws_records, P->blob.data(), P->blob.size());
    e = hipMemcpyAsync(ws, h, up, hipMemcpyHostToDevice, stream);
    if (e != hipSuccess) return hip_fail("hipMemcpyAsync(step)", e);
    e = hipEventRecord(static_cast<hipEvent_t>(s->stage_ev[k]), stream);
    if (e != hipSuccess) return hip_fail("hipEventRecord", e);
    s->stage_next = k ^ 1;
  }
  // From here on the step is enqueued: it is complete on the host side even
  // if a later launch fails (the device state is then undefined).
  s->prepared = false;
  if (t_ev_before && t_ev_after) {
    e = hipEventRecord(t_ev_before, stream);
    if (e != hipSuccess) return hip_fail("hipEventRecord", e);
  }
  if (n_new > 0 || n_patch > 0) {
    e = launch_append_kv(k_new, v_new, d.k_cache, d.v_cache, at<int32_t>(ws, 0), n_new, d.num_heads_kv, d.head_dim,
                         d.dtype == PADOC_BF16, at<int32_t>(ws, s->off_patch), n_patch, d.block_table, stream);
    if (e != hipSuccess) return hip_fail("append kernel launch", e);
  }
  padoc_status st = run(P, q, d.k_cache, d.v_cache, d.block_table, o, lse, ws + s->ws_records, stream,
                        /*upload=*/false, /*events=*/false);
  if (st != PADOC_OK) return st;
  if (t_ev_before && t_ev_after) {
    e = hipEventRecord(t_ev_after, stream);
    if (e != hipSuccess) return hip_fail("hipEventRecord", e);
  }
  return PADOC_OK;
}

extern "C" void padoc_session_destroy(padoc_session* s) {
  if (!s) return;
  for (int k = 0; k < 2; ++k) {
    if (s->stage_ev[k]) (void)hipEventDestroy(static_cast<hipEvent_t>(s->stage_ev[k]));
    if (s->stage[k]) (void)hipHostFree(s->stage[k]);
  }
  if (s->plan.pin_ev) (void)hipEventDestroy(static_cast<hipEvent_t>(s->plan.pin_ev));
  if (s->plan.pinned) (void)hipHostFree(s->plan.pinned);
  if (s->plan.bpinned) (void)hipHostFree(s->plan.bpinned);
  session_free_host(s);
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
