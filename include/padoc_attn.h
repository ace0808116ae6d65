/*
 * libpadoc_attn -- ancestor-masked attention over a packed token tree
 * (PaDoc, "Layout-Grounded Parallel Decoding for Document Parsing").
 *
 * The operation (Sec. 3.2 ancestor sets; App. C "Attention Backends"; App. E
 * masked parallel decoding and its Attn equation):
 *
 *   A page is a tree of segments.  The root is the page prefix X (image and
 *   prompt tokens); the layout stream is its child; content branches Y_k are
 *   children of the stream.  A query token at position p of segment s attends
 *   to every key at position j of segment t such that
 *       t == s and j <= p                      (causal inside its own node), or
 *       t is a proper ancestor of s and j < F   (F = fork offset of the child
 *                                                of t on the path to s),
 *   and computes O = softmax(scale * q K^T) V over exactly those keys and
 *   LSE = ln(sum over those keys of exp(scale * q.k)).  Pages never see each
 *   other.  The descriptor allows trees of any depth (parent index < own).
 *
 * Two entry points:
 *   padoc_tree_attn_fwd  -- packed variable-length forward: K/V of all tokens
 *                           in packed order (the training / branch-creation
 *                           form, App. C tree-varlen relation
 *                           Q_M -> K_M, Q_{Y_k} -> [K_{M<=f_k}; K_{Y_k}]).
 *   padoc_branch_decode  -- one step of masked parallel decoding (App. E,
 *                           algorithm steps "append" then "decode") over a
 *                           paged KV cache: every live stream's newest
 *                           q_len tokens query their ancestors + own history;
 *                           keys shared by sibling streams are read once.
 *   padoc_tree_attn_bwd  -- gradient of the packed forward (the paper trains
 *                           with the tree-varlen backend, App. C): dQ, dK, dV
 *                           of sum(dO * O); a key shared by several segments
 *                           (page prefix, layout stream) receives the sum over
 *                           every query that sees it.
 *
 * Layouts (row-major, head dimension innermost, everything contiguous):
 *   Q, O     [n_q_rows, Hq, d]        segment s's queries = its LAST q_len
 *                                     tokens, at rows q_off .. q_off+q_len-1
 *   K, V     packed: [num_kv_rows, Hkv, d], segment s's token j at row kv_off+j
 *   K cache  paged:  [num_blocks, Hkv, d/8, 16, 8]  (chunk-major: element
 *                    (slot t, dim c) of a block at [c/8][kslot(t)][c%8],
 *                    kslot(t) = t with bits 2 and 3 swapped, i.e.
 *                    (t & 3) | (t & 4) << 1 | (t & 8) >> 1; 8 consecutive
 *                    dims of a token are one piece, the 16 tokens' pieces of
 *                    one chunk are contiguous, and tokens {0-3, 8-11} and
 *                    {4-7, 12-15} each fill one 128-byte line per chunk)
 *   V cache  paged:  [num_blocks, Hkv, d, 16]  (d-major: the 16 tokens of a
 *                    block are contiguous for each d)
 *            segment s's token j lives in block block_table[kv_off + j/16],
 *            slot t = j%16, of both caches
 *   LSE      float32 [n_q_rows, Hq], natural log
 *   GQA      query head h reads KV head h / (Hq/Hkv)
 *   dtype    Q, K, V and O share one dtype (bf16 or fp32); accumulation is
 *            fp32; O is rounded to nearest-even.
 *
 * Ownership: the caller owns every buffer.  The library never allocates
 * device memory: it reports a workspace size and the caller passes a device
 * buffer of at least that size to each launch (padoc_branch_decode_no_alloc
 * instead uses a fixed array the library holds on each GPU).  A plan owns host memory only,
 * is immutable after creation and may be reused for any number of launches
 * with the same tree; destroy it only after the stream has passed the last
 * launch that used it.
 *
 * Errors: every call returns a padoc_status and never throws.  All tree and
 * shape validation happens in padoc_plan_create; launches check pointers and
 * workspace size first.  On any error nothing is enqueued and
 * padoc_last_error() (thread-local) describes the cause.  Launches are
 * asynchronous on the caller's stream; a device fault surfaces at the
 * caller's next synchronisation.  Two launches that share a workspace must be
 * ordered (same stream or explicit events).
 */
#ifndef PADOC_ATTN_H
#define PADOC_ATTN_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PADOC_OK = 0,
  PADOC_ERR_ARG = -1,        /* null pointer, bad enum value, negative count    */
  PADOC_ERR_TREE = -2,       /* parent / fork / len / q_len inconsistent        */
  PADOC_ERR_SHAPE = -3,      /* heads or head_dim unsupported                   */
  PADOC_ERR_DTYPE = -4,      /* dtype unsupported                               */
  PADOC_ERR_BOUNDS = -5,     /* offsets outside the buffers, overlapping query
                                rows, block id outside the pool                 */
  PADOC_ERR_WORKSPACE = -6,  /* workspace null or too small                     */
  PADOC_ERR_HIP = -7,        /* a HIP call failed (message has the HIP error)   */
  PADOC_ERR_MODE = -8        /* plan built for the other entry point            */
} padoc_status;

typedef enum { PADOC_F32 = 0, PADOC_BF16 = 1 } padoc_dtype;

/* One tree segment: a page prefix (root), a layout stream or a branch. */
typedef struct {
  int32_t parent;   /* -1 for a root (one page); else index < own index        */
  int32_t fork;     /* leading parent tokens visible, 0..len(parent); roots: 0 */
  int32_t len;      /* tokens (K/V rows) in this segment, including the query
                       tokens of a decode step (their K/V is already written)  */
  int32_t q_len;    /* queries = the last q_len tokens, 0..len                 */
  int64_t kv_off;   /* packed: first K/V row; paged: first block-table entry   */
  int64_t q_off;    /* first Q/O/LSE row of this segment's queries             */
} padoc_segment;

/* A document page as the paper's packed sample [prefix | stream | Y_1..Y_N]
   (App. C): the stream sees the whole prefix, branch k sees the first
   branch_fork[k] stream tokens (its branch-start token is its own position
   0, Sec. 3.2).  Arrays have n_branches entries and are read only during the
   call. */
typedef struct {
  int32_t prefix_len, prefix_q_len;
  int32_t stream_len, stream_q_len;
  int32_t n_branches;
  const int32_t* branch_fork;
  const int32_t* branch_len;
  const int32_t* branch_q_len;
} padoc_page;

typedef struct {
  int32_t n_seg;
  const padoc_segment* seg;      /* host memory, read during padoc_plan_create  */
  int32_t num_heads_q;           /* Hq > 0                                      */
  int32_t num_heads_kv;          /* Hkv > 0, Hq % Hkv == 0, Hq/Hkv <= 64
                                                                               */
  int32_t head_dim;              /* 64 or 128                                   */
  float softmax_scale;           /* > 0, finite; the paper uses 1/sqrt(d)       */
  padoc_dtype dtype;
  int32_t block_size;            /* 0: packed K/V (forward); 16: paged (decode) */
  int64_t num_kv_rows;           /* packed: rows of K/V; paged: blocks in pool  */
  int64_t num_q_rows;            /* rows of Q/O/LSE                             */
  const int32_t* block_table_host; /* paged, optional: host copy of the table,
                                    used only to check ids are in the pool     */
  int64_t block_table_len;       /* paged: entries in the block table           */
  int32_t max_chunk_keys;        /* decode: split keys into chunks of at most
                                    this many (multiple of 64, at most 8192);
                                    0 = automatic                           */
  int32_t target_workgroups;     /* decode chunk sizes (0 = 1024): shared keys
                                    are cut into the fewest chunks (128 to 8192
                                    keys) that keep the tile items (8
                                    wavefronts each) within 3/16 of this,
                                    private keys into about 2x this many
                                    wavefront items (chunks of 512 to 8192
                                    keys)                                    */
} padoc_tree_desc;

typedef struct padoc_plan padoc_plan;

/* Schedule export (tests and tools).  Pointers stay valid until the plan is
   destroyed.  A work item processes, for one KV head, the queries
   toks[tok_begin .. tok_begin+ntok) (Q row indices; column c of the task is
   token c/G, head c%G; the item computes columns col0 .. col0+ncol-1) against
   the key ranges ranges[rng_begin ..
   rng_begin+rng_count).  Token i of the item sees keys [0, lim) of a range
   where lim = n_keys if lim_off < 0, else lims[lim_off + i]; every token sees
   at least [0, min_lim).  Key j of a range is K/V row kv_start + j (packed) or
   block_table[kv_start + j/16] slot j%16 (paged); seg and key_begin name the
   segment and the first key of it the range starts at.  For range r,
   tile_class[tile_class_off[r] + kt] is 1 (full: every token sees all
   tile_keys keys, no mask) or 2 (partial: masked) for each key tile kt below
   ceil(n_keys / tile_keys); tiles past n_keys are never visited.  Work items
   of different KV heads share token and range records.  Forward plans: one
   workgroup per item.  Decode plans: the first n_work_shared items (shared
   prefix / stream keys, up to 256 columns) run one per 8-wavefront
   workgroup on matrix cores, the remaining items (a private branch's keys,
   16 columns) one per wavefront, all in one launch; every item writes the
   split partial of column c to slot out_base + c and the combine kernel
   merges the rows listed in comb_rows (every row with partials).  Decode
   plans write one partial result per (item, column) at slot out_base + column
   and combine, for Q row r and KV head g, the slots comb_slot[comb_ptr[r*Hkv+g]
   .. comb_ptr[r*Hkv+g+1]) (+ head within group) in that order. */
typedef struct {
  int32_t tok_begin, ntok, rng_begin, rng_count, kvh, out_base, cost;
  int32_t col0;  /* first column of the task this item computes              */
  int32_t ncol;  /* columns this item computes: col0 .. col0+ncol-1, clipped
                    to the task's ntok*G columns                             */
  int32_t direct[3]; /* decode private items with one range, one query token
                        and no per-token limits: the range's kv_start, its
                        n_keys and the token's Q row (the kernel then reads
                        neither the range nor the token record); -1, 0, 0 in
                        every other item                                      */
} padoc_work_view;

typedef struct {
  int64_t kv_start;
  int32_t n_keys, min_lim, lim_off, seg, key_begin, reserved;
} padoc_range_view;

/* Backward key-major item (packed bf16 plans): keys key_row0 .. +n_keys-1
   (K/V rows of one segment, n_keys <= 128) of KV head kvh against the query
   tokens btoks[tok_begin .. tok_begin+ntok) (Q rows), of which token i sees
   the item's keys [0, blims[lim_begin + i]) (relative to key_row0); the item
   computes columns col0 .. col0+ncol-1 (column c = token c/G, head c%G).  An
   item with all ntok*G columns stores its rows' dK/dV; the items of a key
   run split into column pieces (multiples of 32) add into the same rows. */
typedef struct {
  int64_t key_row0;
  int32_t n_keys, tok_begin, ntok, lim_begin, col0, ncol, kvh, cost;
} padoc_bwd_view;

typedef struct {
  int32_t kind;                  /* 0 = forward (final O), 1 = decode (partials) */
  int32_t tile_cols, tile_keys;  /* columns per work item, keys per key tile     */
  int32_t n_work;  const padoc_work_view* work;
  int32_t n_work_shared;
  int32_t n_range; const padoc_range_view* ranges;
  int32_t n_lim;   const int32_t* lims;
  int32_t n_tok;   const int32_t* toks;
  int64_t n_tile_class; const int8_t* tile_class; const int64_t* tile_class_off;
  int64_t n_comb_ptr; const int32_t* comb_ptr;
  int64_t n_comb;     const int32_t* comb_slot;
  int64_t n_comb_rows; const int32_t* comb_rows; /* (row*Hkv + kv head) merged
                                                    by the combine kernel     */
  int32_t n_bwd; const padoc_bwd_view* bwd;      /* backward items (packed bf16) */
  int64_t n_btok; const int32_t* btoks;
  int64_t n_blim; const int32_t* blims;
  int64_t n_slots;
  size_t workspace_bytes;
} padoc_schedule_view;

/* Lay out a list of pages as segments in packed order (A1 of the hot path):
   per page [prefix, stream, branch 1..N]; kv_off/q_off are filled as running
   sums (packed rows when block_size == 0, block-table entries of
   ceil(len/block_size) when block_size > 0).  Writes at most `capacity`
   segments; *n_out receives the number needed (also when it exceeds
   capacity, which returns PADOC_ERR_ARG). */
padoc_status padoc_tree_from_pages(const padoc_page* pages, int32_t n_pages, int32_t block_size,
                                   padoc_segment* out, int32_t capacity, int32_t* n_out);

/* Fill kv_off / q_off of n segments in place with the canonical packed
   layout (node order, running sums as above).  parent/fork/len/q_len are
   read, not checked (padoc_plan_create checks them). */
padoc_status padoc_tree_layout(padoc_segment* seg, int32_t n, int32_t block_size);

/* Decoding depths of each page (Sec. 3.1 sequential depth vs critical path;
   App. D forward steps), host only.  Roots are page inputs (prefilled, not
   decoded); every other segment is decoded one token per step.  For each
   root r: d_seq[r] = total length of the page's decoded segments (one
   stream after another); d_crit[r] = steps when all streams run
   concurrently and a segment starts as soon as its parent has produced the
   `fork` tokens it conditions on: start(s) = start(parent) + fork (0 for a
   child of a root), and the page ends at the largest start(s) + len(s).
   Entries of non-root segments are set to 0.  The per-page forward-step
   reduction is 1 - d_crit / d_seq.  Checks parent < own index and
   0 <= fork <= len(parent); PADOC_ERR_TREE otherwise. */
padoc_status padoc_tree_depths(const padoc_segment* seg, int32_t n, int64_t* d_seq, int64_t* d_crit);

/* Remaining critical path of every segment from a point in decoding
   (Sec. 3.1: the decoding depth of a page under ideal parallel scheduling is
   its longest layout-content dependency path), host only.  progress[s] =
   tokens segment s has produced so far (NULL: all 0; roots are page inputs,
   prefilled, and their entry is not read).  A child of a root starts with
   the page; a deeper segment starts once its parent has started and
   produced the `fork` tokens it conditions on.  Every started segment
   produces one token per step.  For a decoded segment s, remaining[s] =
   steps until s and the segments below it that have not started yet have
   produced all their tokens (counted from the step s starts in, if it has
   not started): the larger of len(s) - progress[s] and, over
   children c not started, fork(c) - progress[s] + remaining[c] (started
   children are counted on their own).  For a root, steps until the whole
   page has: the largest remaining[] of its started segments; with all
   progress 0 this is d_crit of padoc_tree_depths.  Use: the priority of an
   open stream when a step can take fewer rows than there are streams
   (padoc_session_select).  Tree checks as padoc_tree_depths
   (PADOC_ERR_TREE); PADOC_ERR_ARG when a progress lies outside [0, len] or
   a segment that has not started has progress. */
padoc_status padoc_tree_remaining(const padoc_segment* seg, int32_t n, const int32_t* progress,
                                  int64_t* remaining);

/* Validate the tree and build the schedule (host only; no HIP call).  The
   schedule lists, for every group of query columns, the key ranges their
   ancestor sets make visible (Sec. 3.2: a node's tokens see its ancestors
   and its own earlier tokens; App. C: a branch sees the layout stream up to
   its fork offset), so keys outside them are never visited.  Packed plans
   (block_size 0) serve padoc_tree_attn_fwd / _bwd, paged plans (16) the
   decode calls.  *out receives a plan the caller destroys; on error *out is
   NULL and padoc_last_error() names the offending segment or field. */
padoc_status padoc_plan_create(const padoc_tree_desc* desc, padoc_plan** out);
padoc_status padoc_plan_workspace_bytes(const padoc_plan* plan, size_t* bytes);
padoc_status padoc_plan_export(const padoc_plan* plan, padoc_schedule_view* out);
void padoc_plan_destroy(padoc_plan* plan);

/* Packed forward (App. C tree-varlen relation: the layout stream's queries
   against its own causal keys after the prefix, each branch's queries
   against the stream's first fork-offset tokens and its own causal keys;
   App. E Attn equation).  Needs a plan with block_size == 0.  q/k/v/o are
   device pointers in the plan's dtype, lse a device float pointer; workspace
   a device buffer of at least padoc_plan_workspace_bytes; stream may be NULL
   (the null stream).  Argument errors are returned before anything is
   enqueued. */
padoc_status padoc_tree_attn_fwd(const padoc_plan* plan, const void* q, const void* k,
                                 const void* v, void* o, float* lse, void* workspace,
                                 size_t workspace_bytes, hipStream_t stream);

/* Rewrite paged K/V blocks from row layout into the paged layouts above,
   for callers whose cache keeps each token's row contiguous: k_rows and
   v_rows are [num_blocks, Hkv, 16, head_dim] (block, KV head, slot,
   dimension; the layout a row-per-token paged cache uses), k_cache and
   v_cache receive the same blocks in the chunk-major K and d-major V
   layouts, block for block (so block ids and block tables are unchanged).
   The decode step (App. E) reads the cached rows wherever they are stored;
   this only changes where.  Device pointers, caller-owned, four distinct
   buffers (no conversion in place); dtype bf16 or fp32 for all four;
   head_dim 64 or 128.  Enqueued on `stream` (NULL: the null stream), no
   allocation; call it once for a whole cache, or for the blocks a step
   wrote by passing pointers to their first block and their count.
   PADOC_ERR_ARG / _SHAPE / _DTYPE / _BOUNDS before anything is enqueued. */
padoc_status padoc_cache_from_rows(const void* k_rows, const void* v_rows, void* k_cache, void* v_cache,
                                   int64_t num_blocks, int32_t num_heads_kv, int32_t head_dim,
                                   padoc_dtype dtype, hipStream_t stream);

/* Decode step over a paged cache.  Needs a plan with block_size == 16.
   k_cache / v_cache follow the paged layouts above (chunk-major K, d-major
   V).  block_table is the device copy of the table the plan was built for
   (block_table_len int32 entries, every id < num_kv_rows).  The call copies
   the schedule (with zeroed work-queue counters) into the workspace and
   then runs the kernels, all on `stream`: calls that overlap on one
   workspace race (give concurrent calls their own workspaces). */
padoc_status padoc_branch_decode(const padoc_plan* plan, const void* q, const void* k_cache,
                                 const void* v_cache, const int32_t* block_table, void* o,
                                 float* lse, void* workspace, size_t workspace_bytes,
                                 hipStream_t stream);

/* The decode step with the schedule kept in the workspace (App. E: every
   layer of a decode step attends over the same tree, so one upload of its
   schedule serves all of them).  padoc_plan_upload enqueues the copy of a
   decode plan's schedule (with zeroed work-queue counters) into `workspace`
   on `stream`; padoc_branch_decode_resident then runs the same kernels as
   padoc_branch_decode, with the same arguments and results, without the
   copy (each call leaves the counters at zero for the next).  Between the
   upload and a resident call, the workspace may be used only by resident
   calls of the same plan, ordered on one stream (or synchronised); the
   caller must not write it, and padoc_branch_decode of another plan on it
   needs a new upload.  A resident call on a workspace other than the one
   of the plan's last upload, or after the plan was rebuilt, returns
   PADOC_ERR_MODE and enqueues nothing.  The upload reads the plan's pinned
   host copy (made on the first upload of a build). */
padoc_status padoc_plan_upload(const padoc_plan* plan, void* workspace, size_t workspace_bytes,
                               hipStream_t stream);
padoc_status padoc_branch_decode_resident(const padoc_plan* plan, const void* q,
                                          const void* k_cache, const void* v_cache,
                                          const int32_t* block_table, void* o, float* lse,
                                          void* workspace, size_t workspace_bytes,
                                          hipStream_t stream);

/* padoc_branch_decode without a workspace argument, for callers that cannot
   allocate device memory (code under stream capture, serving loops that must
   not call the allocator, harnesses that forbid it).  Same plan, inputs,
   outputs, kernels and results as padoc_branch_decode; the workspace is a
   fixed array the library holds on each GPU it runs on, of
   PADOC_NO_ALLOC_WORKSPACE_BYTES (64 MiB; the decode workloads measured here
   need at most about 28 MiB), kept until the process ends.  Its device
   address is looked up on the first call made with that device current.
   The schedule is copied from the plan's host memory (no pinned copy is
   made) and that copy also zeroes the work-queue counters; every other
   scratch value is written before it is read, so nothing else must start
   at zero.  No device or pinned host memory is allocated.
   A plan whose workspace exceeds the array returns PADOC_ERR_WORKSPACE and
   enqueues nothing.  All calls on one GPU share that GPU's array and it
   keeps the last call's contents: calls that overlap on one GPU (different
   streams, or host threads without ordering) race; order them. */
#define PADOC_NO_ALLOC_WORKSPACE_BYTES ((size_t)64 << 20)
padoc_status padoc_branch_decode_no_alloc(const padoc_plan* plan, const void* q,
                                          const void* k_cache, const void* v_cache,
                                          const int32_t* block_table, void* o, float* lse,
                                          hipStream_t stream);

/* Backward of the packed forward (bf16 plans with block_size == 0).
   Given the forward's inputs q, k, v, its outputs o and lse, and the
   upstream gradient dout ([n_q, Hq, d], same dtype), writes dq [n_q, Hq, d]
   and dk, dv [num_kv_rows, Hkv, d] (bf16, rounded to nearest-even from fp32
   accumulation; rows that no query sees get zero).  The gradient is that of
   sum(dout * O) with O = softmax(scale * q K^T + mask) V.  Rows of dk/dv
   whose key run is split over several items (runs seen by more query
   columns than about one compute unit's share of the whole backward) sum the
   pieces in an order that depends on scheduling (fp32 rounding differences
   only); all other results are deterministic.
   workspace: a device buffer of at least padoc_plan_backward_workspace_bytes
   bytes (256-byte aligned); fp32 plans return PADOC_ERR_DTYPE. */
padoc_status padoc_plan_backward_workspace_bytes(const padoc_plan* plan, size_t* bytes);
padoc_status padoc_tree_attn_bwd(const padoc_plan* plan, const void* q, const void* k,
                                 const void* v, const void* o, const float* lse,
                                 const void* dout, void* dq, void* dk, void* dv,
                                 void* workspace, size_t workspace_bytes, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Decode session: the step loop of masked parallel decoding (App. E, the
 * algorithm "Masked parallel decoding": append one input per live stream,
 * decode every live stream with its mask row, open a content stream when the
 * layout stream closes a region, retire a stream at its end of sequence).
 *
 * A session keeps the token tree of every page being decoded and the
 * paged-cache blocks its streams occupy.  A stream is one tree segment:
 * padoc_session_open(parent, fork) starts one whose tokens see the first
 * `fork` tokens of `parent` (and, through it, what `parent` sees), as a fork
 * of the fused mask row would (the child's row is the parent's row with
 * only the first `fork` parent tokens); parent -1 starts a page root.  A
 * new stream holds no tokens; every step appends tokens to the open streams
 * and queries the newest of them, so a fork costs no copy of the parent's
 * cache and no re-prefill: the child reads the parent's blocks in place.
 *
 * Typical page: open a root, step once with the prefix as its new tokens
 * (no queries), open the layout stream (parent = root, fork = prefix
 * length), close the root (its blocks stay while a descendant is open),
 * then step with one new token and one query per open stream; when the
 * layout stream closes a region, open a content stream with parent = the
 * layout stream and fork = the layout stream's current length; close a
 * stream at its end of sequence.
 *
 * Each step is two calls.  padoc_session_prepare (host only) appends
 * n_new[i] tokens to open stream i (rows in ascending stream id), takes
 * blocks from the pool for them, and builds the step's attention schedule
 * for the last n_query[i] of them.  padoc_session_launch writes the new
 * tokens' K/V rows into the caches and updates the device block table, then
 * runs the attention of padoc_branch_decode on the step's tree, all on the
 * caller's stream.  Between a prepare and its launch (or
 * padoc_session_commit) no other session call may change the tree.
 *
 * Memory: the caller owns the paged K and V caches (layouts as for
 * padoc_branch_decode, num_blocks blocks) and a device int32 block table of
 * block_table_capacity entries; the session only writes into them.  The
 * session keeps a pinned host staging buffer for its uploads (two of them,
 * reused once the upload two launches back has completed).  A stream's
 * blocks return to the pool when it is closed and no stream below it is
 * still kept; its block-table entries live in a power-of-two region of the
 * table that moves (copied by the next launch) when the stream outgrows it.
 * A session is not thread-safe; a session's launches must be ordered on the
 * device (one stream, or events).
 * ------------------------------------------------------------------------- */
typedef struct padoc_session padoc_session;

typedef struct {
  int32_t num_heads_q, num_heads_kv, head_dim;  /* as in padoc_tree_desc      */
  float softmax_scale;
  padoc_dtype dtype;                 /* of the caches and the step's tensors   */
  int64_t num_blocks;                /* blocks in each cache (the pool)        */
  int64_t block_table_capacity;      /* int32 entries of the device block table */
  void* k_cache;                     /* device, may be NULL for host-only use  */
  void* v_cache;                     /* (then padoc_session_launch is refused) */
  int32_t* block_table;
  int32_t max_chunk_keys, target_workgroups;  /* decode schedule, as in
                                                 padoc_tree_desc               */
} padoc_session_desc;

/* The prepared step, for inspection and for callers that do the device work
   themselves.  Pointers stay valid until the next session call that changes
   the tree. */
typedef struct {
  int32_t n_seg;
  const padoc_segment* seg;     /* the step's tree: every kept stream in id
                                   order, parent as an index into seg,
                                   kv_off = first block-table entry, len after
                                   the step's appends, q_len = n_query       */
  const int32_t* seg_id;        /* stream id of each segment                 */
  int32_t n_rows;               /* open streams, ascending id                */
  const int32_t* row_id;
  const int32_t* new_off;       /* n_rows + 1: new K/V rows of row i are
                                   new_off[i] .. new_off[i+1]-1              */
  const int32_t* q_off;         /* n_rows + 1: Q/O/LSE rows, same form       */
  const int32_t* new_slot;      /* per new K/V row: (block id, slot) pairs   */
  int32_t n_patch;
  const int32_t* patch;         /* (block-table entry, block id) pairs the
                                   launch writes into the device table       */
  const int32_t* block_table;   /* host copy of the table after the patches
                                   (block_table_capacity entries; unused
                                   entries -1)                               */
  const padoc_plan* plan;       /* the step's schedule (num_q_rows = q_off
                                   [n_rows]); usable with padoc_branch_decode
                                   once the patches and K/V rows are written */
  int64_t free_blocks;          /* pool blocks free after the step           */
  size_t workspace_bytes;       /* for padoc_session_launch                  */
} padoc_session_view;

/* Create / destroy.  Destroy waits for nothing: call it after the stream
   has passed the session's last launch. */
padoc_status padoc_session_create(const padoc_session_desc* desc, padoc_session** out);
void padoc_session_destroy(padoc_session* session);

/* Open a stream under `parent` (a kept stream id, or -1 for a new page root)
   seeing its first `fork` tokens (0 <= fork <= the parent's current length;
   roots: 0).  *id receives the new stream's id (ids increase from 0). */
padoc_status padoc_session_open(padoc_session* session, int32_t parent, int32_t fork, int32_t* id);

/* Close (retire) an open stream: it takes part in no later step.  Closed
   streams with no kept descendant are released at once, with their blocks
   and block-table region; a closed stream's tokens stay visible to the
   streams below it until they are released. */
padoc_status padoc_session_close(padoc_session* session, int32_t id);

/* Choose the open streams that advance in the next step when at most
   max_rows rows fit in it (a serving loop's batch budget; 0 = no limit):
   fills n_new[i] = n_query[i] = 1 for the chosen rows and 0 for the others
   (one entry per open stream in ascending id, the arrays of
   padoc_session_prepare).  priority (one entry per open stream, or NULL):
   the rows with the largest priority are chosen, equal priorities in
   ascending id; NULL chooses the oldest streams (ascending id).  With the
   remaining critical paths of padoc_tree_remaining as priorities, the
   streams that gate the longest dependency chains (a layout stream whose
   later regions still have to open, long branches) go first.  Host only;
   reads the session, changes nothing. */
padoc_status padoc_session_select(const padoc_session* session, int32_t max_rows, const int64_t* priority,
                                  int32_t* n_new, int32_t* n_query);

/* Prepare the next step (host only).  n_new / n_query: one entry per open
   stream in ascending id (NULL = 1 each), 0 <= n_query[i] <= n_new[i].  On
   success *n_kv_rows / *n_q_rows receive the rows of the launch's k_new/v_new
   and q/o/lse, and *workspace_bytes the launch's workspace.  Fails with
   PADOC_ERR_BOUNDS, leaving the session as it was, when the pool or the
   block table cannot hold the step; with PADOC_ERR_MODE when a prepared
   step has not been launched or committed. */
padoc_status padoc_session_prepare(padoc_session* session, const int32_t* n_new, const int32_t* n_query,
                                   int32_t* n_kv_rows, int32_t* n_q_rows, size_t* workspace_bytes);

/* Run the prepared step: k_new, v_new [n_kv_rows, Hkv, d] (device, packed,
   the rows of open stream i at new_off[i].. in order), q [n_q_rows, Hq, d],
   o [n_q_rows, Hq, d], lse float [n_q_rows, Hq]; workspace: device, 256-byte
   aligned, at least workspace_bytes.  Appends the K/V rows to the caches,
   applies the block-table patches, then computes O and LSE of every query
   (as padoc_branch_decode).  On an argument or workspace error nothing is
   enqueued and the step stays prepared; once enqueueing has begun the step
   is complete on the host (a HIP error then leaves the caches undefined). */
padoc_status padoc_session_launch(padoc_session* session, const void* q, const void* k_new, const void* v_new,
                                  void* o, float* lse, void* workspace, size_t workspace_bytes,
                                  hipStream_t stream);

/* Complete the prepared step without device work, for callers that write
   the step's K/V rows and block-table patches themselves (from the view)
   and run padoc_branch_decode on the view's plan. */
padoc_status padoc_session_commit(padoc_session* session);

/* View of the prepared step (or, when none is prepared, of the tree as it
   stands: seg/block table only, plan NULL). */
padoc_status padoc_session_view_get(const padoc_session* session, padoc_session_view* out);

/* Thread-local description of the last error on this thread ("" if none). */
const char* padoc_last_error(void);

/* Profiling hook (thread-local): when both events are non-null, later calls
   on this thread record `before` just before their first kernel and `after`
   just after their last (every kernel of the call: attention kernels and,
   for decode plans, the combine), on the launch stream.  The events are owned
   by the caller and must outlive the calls.  Pass nulls to stop. */
padoc_status padoc_set_kernel_events(hipEvent_t before, hipEvent_t after);

/* Library version string. */
const char* padoc_version(void);

#ifdef __cplusplus
}
#endif
#endif /* PADOC_ATTN_H */
