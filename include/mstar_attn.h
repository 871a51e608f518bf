/*
 * mstar_attn.h - batched variable-length attention over a paged KV cache,
 * with a per-request segment mask, for AMD Instinct MI355X (gfx950).
 *
 * What is computed.  A launch serves many requests at once, each at its own
 * point of its own traversal of the model graph (the paper's requests are
 * series of Walks over one graph, Sec. 3.1, and one LLM replica is multiplexed
 * across requests of every Walk, Sec. 3.2).  For every request r, query head
 * h and query row i (position p = kv_len - q_len + i):
 *
 *   out[q_start+i][h][:] = sum_t softmax_t(s) * V_r[t][h / (Hq/Hkv)][:]
 *   lse[q_start+i][h]    = ln sum_t exp(s_t),    s_t = sm_scale * <q, K_r[t]>
 *
 * over the keys t the row may see.  K_r[t] / V_r[t] are read in place from a
 * shared page pool through the request's block table (paged attention inside
 * the KVCacheEngine, Sec. 3.3; several contexts as labels over one page pool
 * whose tables are read in place, Sec. 4.1; K rollout candidates over one
 * shared context, Sec. 4.4 and App. A).  The paper does not define the masks;
 * the segment model below is this library's stated reading.
 *
 * Mask model.  A request's keys [0, kv_len) are tiled, in order, by segments.
 * Walking them assigns each position a block id: CAUSAL makes every token its
 * own block, FULL makes the whole segment one block, BLOCKS(b) makes runs of
 * b tokens one block each (the last run may be short).  Key t is visible to
 * the row at position p iff block(t) <= block(p) and, when window W > 0,
 * p - t < W (exactly W keys ending at p, plus later keys of p's own block).
 * A row with no visible key gets out = 0 and lse = -inf.
 *
 * Memory layouts (all row-major, element type = params.dtype unless noted):
 *   q, out        [total_q][Hq][head_dim]
 *   lse           [total_q][Hq]  float32, natural log
 *   k_pages/v_pages [num_pages][page_size][Hkv][head_dim]   ("NHD")
 *   block_table   int32 [num_seqs][max_blocks_per_seq]
 *
 * Error convention.  Every int-returning call returns MSTAR_OK (0) or a
 * negative MSTAR_ERR_* code and never throws or aborts; mstar_last_error()
 * then gives a message for the calling thread.
 */
#ifndef MSTAR_ATTN_H
#define MSTAR_ATTN_H

#include <hip/hip_runtime_api.h> /* hipStream_t, hipEvent_t */
#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- codes -------------------------------------------------------------- */
#define MSTAR_OK 0
#define MSTAR_ERR_INVALID_ARG (-1) /* a descriptor or pointer violates this contract */
#define MSTAR_ERR_UNSUPPORTED (-2) /* head_dim, page_size or dtype not built        */
#define MSTAR_ERR_WORKSPACE (-3)   /* workspace missing or smaller than required    */
#define MSTAR_ERR_HIP (-4)         /* a HIP runtime call failed (message has it)    */
#define MSTAR_ERR_NOMEM (-5)       /* host or device allocation failed              */

#define MSTAR_SEG_CAUSAL 0 /* every token its own block                        */
#define MSTAR_SEG_FULL 1   /* the whole segment one block                      */
#define MSTAR_SEG_BLOCKS 2 /* consecutive blocks of `block` tokens             */

#define MSTAR_DTYPE_F32 0
#define MSTAR_DTYPE_BF16 1

#define MSTAR_FLAG_FORCE_SPLIT 1u /* split every key range into small chunks (exercises the merge) */
#define MSTAR_FLAG_NO_SPLIT 2u    /* never split key ranges                                      */
#define MSTAR_FLAG_HOST_ONLY 4u   /* plan on the host only: no device allocation or upload; for
                                     inspection (stats, items, key ranges) without a GPU; fwd
                                     rejects such a plan                                         */
#define MSTAR_FLAG_CASCADE_ALL 8u /* mstar_attn_plan_cascade: every group member joins the cascade,
                                     not only the decode-like ones                               */
#define MSTAR_FLAG_SERIAL 16u     /* fwd runs every kernel on the caller's stream, one after the
                                     other (no side stream)                                      */

/* Bits of the sticky device error word (see mstar_attn_check). */
#define MSTAR_DEVERR_PAGE_RANGE 1 /* a block-table entry was outside [0, num_pages) */

/* ---- descriptors ---------------------------------------------------------- */

/* One segment of a request's key range: positions [start, start+len). */
typedef struct {
    int32_t start;
    int32_t len;
    int32_t kind;  /* MSTAR_SEG_* */
    int32_t block; /* block length for MSTAR_SEG_BLOCKS (> 0); ignored otherwise */
} mstar_segment;

/* A request's mask: segments [seg_begin, seg_begin+seg_count) of the segment
 * array, which must tile [0, kv_len) in order; window = 0 means no window. */
typedef struct {
    int32_t seg_begin;
    int32_t seg_count;
    int32_t window;
} mstar_mask_spec;

/* A request: its queries are the last q_len of its kv_len positions (new
 * tokens are already in the paged cache); they occupy packed rows
 * [q_start, q_start+q_len) of q/out/lse.  Row ranges of different requests
 * must not overlap.  Several requests may reference the same physical pages. */
typedef struct {
    int32_t q_len;
    int32_t kv_len;
    int32_t q_start;
} mstar_seq_desc;

typedef struct {
    int32_t num_qo_heads;       /* Hq, a multiple of Hkv                          */
    int32_t num_kv_heads;       /* Hkv                                            */
    int32_t head_dim;           /* 64 or 128                                      */
    int32_t page_size;          /* 16                                             */
    int32_t dtype;              /* MSTAR_DTYPE_F32 or MSTAR_DTYPE_BF16            */
    int32_t max_blocks_per_seq; /* row stride of block_table; kv_len <= 16 * this */
    int32_t num_pages;          /* pages in the pool (bounds-checked on device)   */
    uint32_t flags;             /* MSTAR_FLAG_*                                   */
    float sm_scale;             /* score scale > 0, typically 1/sqrt(head_dim)    */
} mstar_attn_params;

/* A shared-prefix group (for mstar_attn_plan_cascade): the requests listed
 * in members[member_begin .. member_begin + member_count) of the member array
 * keep their first prefix_len keys (a positive multiple of 16) in the same
 * physical pages -- their block tables agree on the first prefix_len / 16
 * entries -- and every query row of each of them sees all of those keys.
 * Candidates of one batched forward over a shared context (App. A, V-JEPA 2
 * MPC Walk), or contexts stored as labels over one pool with a common prefix
 * (Sec. 4.1), are such groups. */
typedef struct {
    int32_t member_begin;
    int32_t member_count;
    int32_t prefix_len;
} mstar_prefix_group;

typedef struct mstar_plan mstar_plan_t;
typedef struct mstar_planner mstar_planner_t;

typedef struct {
    int64_t visible_pairs;   /* (row, key) pairs the rows may see, summed over query heads */
    int64_t prefill_items;   /* work items of the multi-row tile kernel                    */
    int64_t decode_items;    /* work items of the few-row (decode / chunk) kernel           */
    int64_t f32_items;       /* work items of the fp32 kernel                               */
    int64_t merge_rows;      /* (row, head) outputs assembled from split partials           */
    int64_t partial_slots;   /* fp32 partial rows in the workspace                          */
    int64_t total_q;         /* packed query rows (max q_start + q_len)                     */
    double plan_host_us;     /* host time spent building the plan                           */
    int64_t device_bytes;    /* bytes of the work list's device copy (host-only: would-be)   */
} mstar_plan_stats;

/* ---- entry points -------------------------------------------------------- */

/* Build the launch plan for one batch (host side; the attention plan the
 * paper's workers build off the critical path, Sec. 3.3).  Reads descriptors
 * only, never tensor data, and copies them, so the caller may free its arrays
 * on return; thread-safe, so it can run on a side thread while the previous
 * batch's fwd executes.  Derives each query row's visible key interval from
 * its mask, cuts the batch into work items (multi-row tiles for long query
 * spans, few-row items for decode-like requests, key ranges split into chunks
 * when there are too few items to fill the GPU), orders them longest first,
 * and uploads the work list with an async host-to-device copy enqueued on
 * `upload_stream` (NULL = default stream).  The caller must order that upload
 * before fwd (same stream, or synchronize).  The work list's device buffer,
 * its pinned staging copy and (for a plan whose fwd runs the few-row kernel
 * beside the tile kernel) a side stream come from a per-device pool that
 * destroyed plans return them to (the smallest free buffer that fits, the
 * most recently returned among equals): only the first plans of a process, or a
 * plan larger than every pooled buffer, allocate (hipMalloc, hipHostMalloc,
 * hipStreamCreate); steady-state planning allocates no device memory and
 * makes no device-synchronizing call.  A pooled buffer's upload first waits,
 * on `upload_stream`, for the work its previous plan enqueued.  The host-side
 * item lists are pooled too (up to 8 sets, none over 64 MB), so that a plan
 * writes into memory an earlier plan has already touched.  On success
 * *out is a new plan; on failure *out is NULL.
 * Errors: INVALID_ARG (null pointer, Hq % Hkv != 0, q_len > kv_len, segments
 * not tiling [0, kv_len), negative window, kv_len > 16 * max_blocks_per_seq,
 * overlapping row ranges, ...), UNSUPPORTED (head_dim, page_size, dtype),
 * NOMEM, HIP. */
int mstar_attn_plan(const mstar_attn_params* params, const mstar_seq_desc* seqs,
                    const mstar_mask_spec* masks, int32_t num_seqs, const mstar_segment* segments,
                    int32_t num_segs, hipStream_t upload_stream, mstar_plan_t** out);

/* mstar_attn_plan with shared-prefix groups (a cascade).  For each group the
 * prefix keys are attended once for the query rows of all members together
 * -- 128 rows (member, query row, query head) per tile against one copy of
 * each prefix K/V tile, read through the first member's block table -- and
 * each member's own keys [prefix_len, ...) separately; the two partial
 * results of every (row, head) are combined by their log-sum-exps.  Results
 * equal those of mstar_attn_plan up to rounding.  Only decode-like members
 * (query rows x (Hq / Hkv) <= 64, which mstar_attn_plan gives to the few-row
 * kernel, one pass over all of their keys per KV head) join the cascade: a
 * member with more rows already reads each prefix tile once per 128 rows, so
 * the cascade would only add the merge; such members are planned as by
 * mstar_attn_plan, unless MSTAR_FLAG_CASCADE_ALL is set.  A request may belong to at
 * most one group.  Errors as mstar_attn_plan, plus INVALID_ARG for a bad group
 * (member index out of range or repeated, prefix_len not a positive multiple
 * of 16 or longer than a member's kv_len, or a member query row that does not
 * see every prefix key) and UNSUPPORTED for the fp32 dtype.  The plan needs
 * a workspace (mstar_attn_workspace_bytes).  num_groups = 0 is mstar_attn_plan. */
int mstar_attn_plan_cascade(const mstar_attn_params* params, const mstar_seq_desc* seqs,
                            const mstar_mask_spec* masks, int32_t num_seqs, const mstar_segment* segments,
                            int32_t num_segs, const mstar_prefix_group* groups, int32_t num_groups,
                            const int32_t* members, int32_t num_members, hipStream_t upload_stream,
                            mstar_plan_t** out);

/* Bytes of device scratch fwd needs (fp32 partial outputs and their LSEs for
 * split key ranges); 0 if nothing is split.  Returns 0 for a NULL plan. */
size_t mstar_attn_workspace_bytes(const mstar_plan_t* plan);

/* Run the planned attention on `stream` (NULL = default stream): the
 * batched attention of one node execution, every request of the batch at its
 * own graph position with its own mask, over K/V read in place from the paged
 * pool (paged attention of the transformer engine, Sec. 3.3, Runtime; one
 * replica serving requests of every Walk in one batch, Sec. 3.2; labels and
 * rollout candidates over shared pages, Sec. 4.1 and 4.4).
 * q, k_pages, v_pages, block_table: caller-owned device memory, read only;
 * pages may be shared between requests.  out, lse: caller-owned device
 * memory, written for every row of every request (rows of no request are
 * untouched).  workspace: caller-owned device memory of at least
 * mstar_attn_workspace_bytes(plan) bytes (may be NULL if that is 0); fwd
 * overwrites it.  Enqueues the plan's kernels -- multi-row tiles, few-row
 * items, shared-prefix cascade items or fp32 items, then the merge of split
 * key ranges; at most four, three for a plan without prefix groups -- with no
 * allocation, no host synchronization and no host reads, so the call may be
 * captured in a HIP graph.  When a plan has both multi-row tile items and
 * few-row items, the few-row kernel runs beside the tile kernel on the plan's
 * side stream (default priority, made when the plan was built): `stream`
 * forks to it and joins back before the merge through two events of the
 * plan, so calls with one such plan must not overlap in time
 * (MSTAR_FLAG_SERIAL turns this off).  Outside graph capture fwd also records
 * an event of the plan on `stream` after its kernels (see
 * mstar_attn_plan_destroy).  The same plan may run with any tensors of the
 * planned shapes.  Two fwd calls that overlap in time must use different
 * workspaces.  Block-table entries outside [0, num_pages) are never
 * dereferenced: they read as zeros and set MSTAR_DEVERR_PAGE_RANGE in the
 * plan's device error word.
 * Errors: INVALID_ARG (null tensor pointer, misaligned pointer), WORKSPACE,
 * HIP (launch failure). */
int mstar_attn_fwd(const mstar_plan_t* plan, const void* q, const void* k_pages,
                   const void* v_pages, const int32_t* block_table, void* out, float* lse,
                   void* workspace, size_t workspace_bytes, hipStream_t stream);

/* mstar_attn_fwd, additionally recording caller-created HIP events right
 * before and right after each kernel it enqueues, on the
 * stream that kernel runs on (`stream`, or the side stream for a few-row
 * kernel beside multi-row work): index 0 = multi-row tile kernel, 1 = few-row kernel, 2 = fp32
 * kernel, 3 = merge kernel, 4 = shared-prefix cascade kernel (arrays of 5
 * entries).  Either array, and any entry, may be NULL; events
 * of kernels the plan does not launch are left untouched.  For per-kernel
 * timing (profiling); same contract and errors as mstar_attn_fwd. */
int mstar_attn_fwd_timed(const mstar_plan_t* plan, const void* q, const void* k_pages,
                         const void* v_pages, const int32_t* block_table, void* out, float* lse,
                         void* workspace, size_t workspace_bytes, hipStream_t stream,
                         const hipEvent_t* events_before, const hipEvent_t* events_after);

/* mstar_attn_fwd without a caller workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): the split-K partials go to a static
 * device array of MSTAR_NOALLOC_SCRATCH_BYTES held by the library on each GPU
 * it runs on until the process ends.  The call allocates nothing (no
 * hipMalloc, no allocating library routine); its first call on a device looks
 * up that device's array address once.  The caller still passes inputs and
 * outputs; plan, tensors, stream and errors as for mstar_attn_fwd.  Returns
 * MSTAR_ERR_WORKSPACE, without enqueuing anything, if the plan needs more
 * scratch than the array holds (mstar_attn_workspace_bytes(plan) >
 * MSTAR_NOALLOC_SCRATCH_BYTES).  Every call on one GPU shares that GPU's
 * array and leaves its contents behind: nothing in it needs to start at
 * zero (every partial a merge reads is written by the same call), but two
 * calls whose kernels overlap in time on one GPU (different streams, or
 * threads) race on it and must not be issued. */
#define MSTAR_NOALLOC_SCRATCH_BYTES (32u << 20)
int mstar_attn_fwd_noalloc(const mstar_plan_t* plan, const void* q, const void* k_pages,
                           const void* v_pages, const int32_t* block_table, void* out, float* lse,
                           hipStream_t stream);

/* Synchronize `stream`, then read and clear the plan's sticky device error
 * word into *error_bits (MSTAR_DEVERR_* bits; 0 = no error seen).  Returns
 * INVALID_ARG if a bit was set, OK otherwise, HIP on a runtime failure. */
int mstar_attn_check(mstar_plan_t* plan, hipStream_t stream, int32_t* error_bits);

/* Planner statistics (host side; no device access). */
int mstar_attn_plan_stats(const mstar_plan_t* plan, mstar_plan_stats* out);

/* Each request's union of visible keys as [lo, hi) pairs into lo_hi[2*num_seqs]
 * (0, 0 for a request without queries). */
int mstar_attn_plan_key_ranges(const mstar_plan_t* plan, int32_t* lo_hi, int32_t num_seqs);

/* Copy one host-side list of the plan (0 = multi-row tiles, 1 = few-row
 * items, 2 = fp32 items, 3 = rows merged by the merge kernel, 4 = cascade
 * items, 5 = cascade rows) into `items` as int32 records of 8 fields; *count
 * receives the number of records, and at most `capacity` records are written.
 * For inspection and tests.
 * Work record: seq, head (query head; KV head for classes 1 and 4; -1 for
 *              class 0, whose records serve every query head), row0, nrows,
 *              key_begin, key_end, partial_slot (-1 = final), head_stride
 *              (class 0 with a split key range or a cascade member: query head
 *              h, row r writes partial slot partial_slot + h * head_stride + r;
 *              otherwise -1).  A cascade item (class 4) reads keys through the
 *              block table of request `seq`, its rows are entries row0 ..
 *              row0 + nrows - 1 of the cascade rows, and row r writes partial
 *              slot partial_slot + r.
 * Merge record: packed_row, head, slot0, slot_stride, nslots, prefix_slot0,
 *              prefix_stride, prefix_nslots (the output combines the partials
 *              at slot0 + s * slot_stride, s < nslots, and at prefix_slot0 +
 *              s * prefix_stride, s < prefix_nslots).
 * Cascade row record: packed query row, query head, 0, 0, 0, 0, 0, 0. */
int mstar_attn_plan_items(const mstar_plan_t* plan, int32_t kind, int32_t* items,
                          int64_t capacity, int64_t* count);

/* Launch order of the multi-row kernel: *count receives the number of
 * workgroups (a multiple of 8) and at most `capacity` (tile item, query head)
 * int32 pairs are written to pairs[2*capacity]; (-1, -1) marks a padding
 * workgroup.  Workgroup b runs on XCD b % 8; the workgroups that read one
 * request's pages for one KV head run consecutively on one XCD, except that a
 * request whose work exceeds an eighth of the launch is cut into runs of
 * consecutive items spread over several XCDs.  For inspection and tests. */
int mstar_attn_plan_tile_order(const mstar_plan_t* plan, int32_t* pairs, int64_t capacity, int64_t* count);

/* The same for the cascade kernel: (cascade item, a query head of its KV
 * head) pairs; empty for a plan without cascade items. */
int mstar_attn_plan_cascade_order(const mstar_plan_t* plan, int32_t* pairs, int64_t capacity, int64_t* count);

/* Asynchronous, double-buffered planning.  The paper's workers build the
 * attention plan of the next batch on a separate thread and stream while the
 * current batch runs, since planning is often the heaviest CPU overhead of a
 * step (Sec. 3.3, Runtime).  A planner owns one worker thread and one HIP
 * stream (default priority) for the uploads.
 *
 * mstar_planner_create: `depth` (1..64, normally 2) is the number of plans
 *   that may be submitted and not yet taken.
 * mstar_planner_submit: copies the descriptors (same meaning and checks as
 *   mstar_attn_plan; the device is the calling thread's current one) and
 *   returns at once, unless `depth` plans are outstanding, in which case it
 *   waits until one is taken.  Plans are built in submission order.
 * mstar_planner_submit_cascade: the same for mstar_attn_plan_cascade (shared-
 *   prefix groups, copied like the descriptors).
 * mstar_planner_take: waits for the oldest outstanding plan, makes `stream`
 *   wait (on the device, no host sync) for its upload, and returns it; the
 *   caller owns it (mstar_attn_plan_destroy).  A planning error is returned
 *   here with its message.  MSTAR_ERR_INVALID_ARG if nothing is outstanding.
 * mstar_attn_plan_wait: makes `stream` wait for a planner-built plan's upload
 *   (a plan from mstar_attn_plan has none to wait for: its upload is ordered
 *   by the stream it was given).  Not for use inside graph capture.
 * mstar_planner_destroy: finishes queued work, destroys untaken plans and
 *   the stream.  Submit and take may be called from different threads; one
 *   planner must not be destroyed while another thread uses it. */
int mstar_planner_create(int32_t depth, mstar_planner_t** out);
int mstar_planner_submit(mstar_planner_t* planner, const mstar_attn_params* params, const mstar_seq_desc* seqs,
                         const mstar_mask_spec* masks, int32_t num_seqs, const mstar_segment* segments,
                         int32_t num_segs);
int mstar_planner_submit_cascade(mstar_planner_t* planner, const mstar_attn_params* params,
                                 const mstar_seq_desc* seqs, const mstar_mask_spec* masks, int32_t num_seqs,
                                 const mstar_segment* segments, int32_t num_segs, const mstar_prefix_group* groups,
                                 int32_t num_groups, const int32_t* members, int32_t num_members);
int mstar_planner_take(mstar_planner_t* planner, hipStream_t stream, mstar_plan_t** out);
int mstar_attn_plan_wait(const mstar_plan_t* plan, hipStream_t stream);
void mstar_planner_destroy(mstar_planner_t* planner);

/* Paged KV append: write the step's new key and value rows into their pages
 * before attention reads them.  Each node execution of the paper's
 * transformer engine stores the K/V of the tokens it processes in the paged
 * cache and then attends over it (Sec. 3.3, Runtime; Sec. 4.4: rollouts reuse
 * the paged cache instead of re-prefilling).
 *
 * For request r of the plan, packed row q_start + i of k_new / v_new
 * ([total_q][num_kv_heads][head_dim], the plan's dtype; the same row
 * numbering as q) holds the key / value of position kv_len - q_len + i, the
 * position of its query row; it is copied to page block_table[r][pos / 16],
 * slot pos % 16 of k_pages / v_pages (NHD layout as in mstar_attn_fwd).  No
 * other slot is written.  Two new rows must not target one slot (pages shared
 * between requests hold cached positions, not new ones); if they do, which one
 * lands is unspecified.  A target page outside [0, num_pages) is skipped and
 * sets MSTAR_DEVERR_PAGE_RANGE in the plan's error word (mstar_attn_check).
 *
 * All pointers are caller-owned device memory; k_new, v_new, k_pages and
 * v_pages must be 16-byte aligned.  Enqueued on `stream` with no allocation
 * and no host synchronisation; an attention call on the same stream afterwards
 * sees the new rows.  Returns MSTAR_OK (also when the plan has no new rows) or
 * a negative code. */
int mstar_kv_append(const mstar_plan_t* plan, const void* k_new, const void* v_new, const int32_t* block_table,
                    void* k_pages, void* v_pages, hipStream_t stream);

/* Release the plan: its host item lists go back to the host pool (or are
 * freed) and its device buffers, staging
 * copy, events and side stream go back to the per-device pool (no HIP call,
 * no device synchronization).  The work of the plan's last fwd or kv_append
 * call enqueued outside graph capture may still be running: a later plan that
 * takes the same buffers waits for it on the device before overwriting them.
 * Calls with the plan on other streams than the last one must have completed
 * (the caller orders them), and a graph that captured the plan's calls must
 * not be replayed after the plan is destroyed.  NULL is ignored. */
void mstar_attn_plan_destroy(mstar_plan_t* plan);

/* Message for the calling thread's last failing call ("" if none). */
const char* mstar_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* MSTAR_ATTN_H */
