// C-ABI of the attention library: plan construction and upload, fwd launch,
// device error check and plan introspection.  Nothing here throws across the
// boundary or aborts; failures return MSTAR_ERR_* with a thread-local message.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <condition_variable>
#include <cstring>
#include <deque>
#include <mutex>
#include <new>
#include <string>
#include <thread>
#include <vector>

#include "mstar_attn.h"
#include "kernels.h"
#include "planner.h"

#define MSTAR_EXPORT extern "C" __attribute__((visibility("default")))

namespace {

// Device-side resources of one plan: the device copy of the plan blob, its
// pinned staging copy, the events that order their reuse, and (for plans that
// run the few-row kernel beside the tile kernel) a side stream with its fork
// and join events.  Blocks are pooled per device: a destroyed plan returns its
// block and later plans take it back, so steady-state planning calls no
// hipMalloc / hipHostMalloc / hipFree (hipFree would also synchronize the
// device) and plan destruction makes no HIP call at all.
struct PlanBlock {
    int device = -1;
    size_t bytes = 0;          // capacity of dev and pinned
    void* dev = nullptr;
    void* pinned = nullptr;
    hipEvent_t uploaded = nullptr;  // after the last upload from `pinned`
    hipEvent_t last_use = nullptr;  // after the last fwd / kv_append enqueued outside graph capture
    bool uploaded_set = false, last_use_set = false;
    hipEvent_t ready = nullptr;     // the async planner's upload-done event
    hipStream_t side = nullptr;     // few-row kernel beside the tile kernel (default priority)
    hipEvent_t fork = nullptr, join = nullptr;
};

constexpr size_t kMinBlockBytes = 64 << 10;
constexpr size_t kPoolMaxBlocks = 64;  // free blocks kept; more are released
std::mutex g_pool_mu;
std::vector<PlanBlock*> g_pool;

void free_block(PlanBlock* b) {
    int cur = 0;
    const bool have = hipGetDevice(&cur) == hipSuccess;
    if (hipSetDevice(b->device) == hipSuccess) {
        if (b->uploaded) (void)hipEventDestroy(b->uploaded);
        if (b->last_use) (void)hipEventDestroy(b->last_use);
        if (b->ready) (void)hipEventDestroy(b->ready);
        if (b->fork) (void)hipEventDestroy(b->fork);
        if (b->join) (void)hipEventDestroy(b->join);
        if (b->side) (void)hipStreamDestroy(b->side);
        if (b->dev) (void)hipFree(b->dev);
        if (b->pinned) (void)hipHostFree(b->pinned);
    }
    if (have) (void)hipSetDevice(cur);
    delete b;
}

// A block of at least `bytes` on the current device: the smallest fitting free
// one, the most recently released among equals (its staging copy is the most
// likely to be cache-warm), else a new one (capacity rounded up to a power of two).
hipError_t acquire_block(size_t bytes, PlanBlock** out) {
    *out = nullptr;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    {
        std::lock_guard<std::mutex> lk(g_pool_mu);
        size_t best = g_pool.size();
        for (size_t i = g_pool.size(); i-- > 0;)
            if (g_pool[i]->device == dev && g_pool[i]->bytes >= bytes &&
                (best == g_pool.size() || g_pool[i]->bytes < g_pool[best]->bytes))
                best = i;
        if (best < g_pool.size()) {
            *out = g_pool[best];
            g_pool.erase(g_pool.begin() + (ptrdiff_t)best);
            return hipSuccess;
        }
    }
    PlanBlock* b = new (std::nothrow) PlanBlock();
    if (!b) return hipErrorOutOfMemory;
    b->device = dev;
    size_t cap = kMinBlockBytes;
    while (cap < bytes) cap <<= 1;
    b->bytes = cap;
    if ((e = hipMalloc(&b->dev, cap)) == hipSuccess && (e = hipHostMalloc(&b->pinned, cap, hipHostMallocDefault)) == hipSuccess &&
        (e = hipEventCreateWithFlags(&b->uploaded, hipEventDisableTiming)) == hipSuccess &&
        (e = hipEventCreateWithFlags(&b->last_use, hipEventDisableTiming)) == hipSuccess) {
        *out = b;
        return hipSuccess;
    }
    free_block(b);
    return e;
}

void release_block(PlanBlock* b) {
    if (!b) return;
    {
        std::lock_guard<std::mutex> lk(g_pool_mu);
        if (g_pool.size() < kPoolMaxBlocks) {
            g_pool.push_back(b);
            return;
        }
    }
    free_block(b);
}

// Host halves of plans are pooled the same way: a destroyed plan's item
// lists keep their capacity for a later plan, which then writes into memory
// it has already touched (on large batches the first-touch page faults of
// fresh multi-megabyte lists cost more than the planning).  At most
// kHostPoolMax are kept, and none holding more than kHostPoolMaxBytes.
constexpr size_t kHostPoolMax = 8;
constexpr size_t kHostPoolMaxBytes = 64 << 20;
std::mutex g_host_mu;
std::vector<mstar::HostPlan> g_host_pool;

void take_host(mstar::HostPlan& h) {
    std::lock_guard<std::mutex> lk(g_host_mu);
    if (g_host_pool.empty()) return;
    h = std::move(g_host_pool.back());
    g_host_pool.pop_back();
}

void give_host(mstar::HostPlan& h) {
    if (h.capacity_bytes() > kHostPoolMaxBytes) return;
    std::lock_guard<std::mutex> lk(g_host_mu);
    if (g_host_pool.size() < kHostPoolMax) g_host_pool.push_back(std::move(h));
}

}  // namespace

struct mstar_plan {
    mstar::HostPlan host;
    PlanBlock* blk = nullptr;  // device resources (NULL for a host-only plan)
    void* dev = nullptr;       // blk->dev
    size_t bytes = 0;
    size_t off_seqs = 0, off_row_hi = 0, off_tiles = 0, off_order = 0, off_few = 0, off_f32 = 0, off_merge = 0, off_append = 0, off_casc = 0, off_casc_rows = 0, off_casc_order = 0, off_err = 0;
    double plan_us = 0.0;
    // A plan with both tile and few-row items runs the few-row kernel on
    // blk->side beside the tile kernel: the caller's stream forks at blk->fork
    // and joins at blk->join before the merge.
    bool forked = false;
    bool from_planner = false;  // built by an async planner: blk->ready marks its upload
};

namespace {

thread_local std::string g_err;

int fail(int code, const std::string& msg) {
    g_err = msg;
    return code;
}

int hip_fail(hipError_t e, const char* what) {
    return fail(MSTAR_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Records that `plan`'s device blob is read by work enqueued on `s` (so that a
// later plan reusing the block waits for it), unless `s` is being captured
// into a graph: a capture's replays are the caller's to finish before the
// plan is destroyed.
hipError_t mark_use(const mstar_plan* plan, hipStream_t s) {
    hipStreamCaptureStatus st = hipStreamCaptureStatusNone;
    hipError_t e = hipStreamIsCapturing(s, &st);
    if (e != hipSuccess || st != hipStreamCaptureStatusNone) return e;
    e = hipEventRecord(plan->blk->last_use, s);
    if (e == hipSuccess) plan->blk->last_use_set = true;
    return e;
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

}  // namespace

static int plan_impl(const mstar_attn_params* params, const mstar_seq_desc* seqs, const mstar_mask_spec* masks,
                     int32_t num_seqs, const mstar_segment* segments, int32_t num_segs,
                     const mstar_prefix_group* groups, int32_t num_groups, const int32_t* members,
                     int32_t num_members, hipStream_t upload_stream, mstar_plan_t** out) {
    const auto t0 = std::chrono::steady_clock::now();
    if (!out) return fail(MSTAR_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    if (!params) return fail(MSTAR_ERR_INVALID_ARG, "params is NULL");
    mstar_attn_params p = *params;
    const bool host_only = (p.flags & MSTAR_FLAG_HOST_ONLY) != 0;
    p.flags &= ~MSTAR_FLAG_HOST_ONLY;

    mstar_plan* plan = new (std::nothrow) mstar_plan();
    if (!plan) return fail(MSTAR_ERR_NOMEM, "host allocation failed");
    take_host(plan->host);
    std::string err;
    int rc;
    try {
        rc = mstar::build_host_plan(&p, seqs, masks, num_seqs, segments, num_segs, plan->host, err, groups,
                                    num_groups, members, num_members);
    } catch (const std::bad_alloc&) {
        rc = MSTAR_ERR_NOMEM;
        err = "host allocation failed";
    } catch (...) {
        rc = MSTAR_ERR_INVALID_ARG;
        err = "planner failure";
    }
    if (rc != MSTAR_OK) {
        delete plan;
        return fail(rc, err);
    }
    const mstar::HostPlan& h = plan->host;

    // blob layout: seqs | row_hi | tiles | tile order | few | f32 | merges | appends | cascade items, rows, order | error word
    size_t off = 0;
    plan->off_seqs = off;   off = align256(off + h.seqs.size() * sizeof(mstar::SeqInfo));
    plan->off_row_hi = off; off = align256(off + h.row_hi.size() * sizeof(int32_t));
    plan->off_tiles = off;  off = align256(off + h.tiles.size() * sizeof(mstar::WorkItem));
    plan->off_order = off;  off = align256(off + h.tile_order.size() * sizeof(int32_t));
    plan->off_few = off;    off = align256(off + h.few.size() * sizeof(mstar::WorkItem));
    plan->off_f32 = off;    off = align256(off + h.f32.size() * sizeof(mstar::WorkItem));
    plan->off_merge = off;  off = align256(off + h.merges.size() * sizeof(mstar::MergeItem));
    plan->off_append = off; off = align256(off + h.appends.size() * sizeof(mstar::WorkItem));
    plan->off_casc = off;   off = align256(off + h.cascade.size() * sizeof(mstar::WorkItem));
    plan->off_casc_rows = off; off = align256(off + h.casc_rows.size() * sizeof(int32_t));
    plan->off_casc_order = off; off = align256(off + h.casc_order.size() * sizeof(int32_t));
    plan->off_err = off;    off = align256(off + sizeof(int32_t));
    plan->bytes = off;

    if (!host_only) {
        hipStream_t up = upload_stream;
        PlanBlock* b = nullptr;
        hipError_t e = acquire_block(plan->bytes, &b);
        if (e != hipSuccess) {
            delete plan;
            return e == hipErrorOutOfMemory ? fail(MSTAR_ERR_NOMEM, "plan buffers: out of memory")
                                            : hip_fail(e, "plan buffers");
        }
        plan->blk = b;
        plan->dev = b->dev;
        // a failure after the upload was enqueued: let that copy finish
        // (best effort) before the block goes back to the pool
        bool enqueued = false;
        auto give_up = [&](hipError_t err, const char* what) {
            if (enqueued) (void)hipStreamSynchronize(up);
            release_block(b);
            delete plan;
            return hip_fail(err, what);
        };
        // a reused block: its previous upload must have left the staging copy
        // (normally long done) before the host rewrites it
        if (b->uploaded_set && (e = hipEventSynchronize(b->uploaded)) != hipSuccess)
            return give_up(e, "hipEventSynchronize(plan staging)");
        unsigned char* blob = static_cast<unsigned char*>(b->pinned);
        // the sections in layout order; only the alignment gaps between them
        // and the tail (the error word) are zeroed
        size_t pos = 0;
        auto put = [&](size_t off, const auto& v) {
            if (off > pos) std::memset(blob + pos, 0, off - pos);
            const size_t n = v.size() * sizeof(v[0]);
            if (n) std::memcpy(blob + off, v.data(), n);
            pos = off + n;
        };
        put(plan->off_seqs, h.seqs);
        put(plan->off_row_hi, h.row_hi);
        put(plan->off_tiles, h.tiles);
        put(plan->off_order, h.tile_order);
        put(plan->off_few, h.few);
        put(plan->off_f32, h.f32);
        put(plan->off_merge, h.merges);
        put(plan->off_append, h.appends);
        put(plan->off_casc, h.cascade);
        put(plan->off_casc_rows, h.casc_rows);
        put(plan->off_casc_order, h.casc_order);
        std::memset(blob + pos, 0, plan->bytes - pos);
        // ... and work of the block's previous plan that reads the device copy
        // must be done before the upload overwrites it (a device-side wait)
        if (b->last_use_set && (e = hipStreamWaitEvent(up, b->last_use, 0)) != hipSuccess)
            return give_up(e, "hipStreamWaitEvent(plan reuse)");
        enqueued = true;
        if ((e = hipMemcpyAsync(b->dev, b->pinned, plan->bytes, hipMemcpyHostToDevice, up)) != hipSuccess)
            return give_up(e, "plan upload");
        if ((e = hipEventRecord(b->uploaded, up)) != hipSuccess) return give_up(e, "hipEventRecord(plan upload)");
        b->uploaded_set = true;
        // the few-row kernel goes beside the tile kernel (prefill work), not
        // beside the cascade kernel, whose L2-fed prefix tiles and the few-row
        // kernel's HBM stream slow each other down more than they overlap;
        // the side stream and its events are made here (once per block), not
        // in fwd
        if (!h.tiles.empty() && !h.few.empty() && !(p.flags & MSTAR_FLAG_SERIAL)) {
            if (!b->side && (e = hipStreamCreateWithFlags(&b->side, hipStreamNonBlocking)) != hipSuccess) {
                b->side = nullptr;
                return give_up(e, "side stream");
            }
            if (!b->fork && (e = hipEventCreateWithFlags(&b->fork, hipEventDisableTiming)) != hipSuccess) {
                b->fork = nullptr;
                return give_up(e, "fork event");
            }
            if (!b->join && (e = hipEventCreateWithFlags(&b->join, hipEventDisableTiming)) != hipSuccess) {
                b->join = nullptr;
                return give_up(e, "join event");
            }
            plan->forked = true;
        }
    }
    plan->plan_us = std::chrono::duration<double, std::micro>(std::chrono::steady_clock::now() - t0).count();
    *out = plan;
    return MSTAR_OK;
}

MSTAR_EXPORT int mstar_attn_plan(const mstar_attn_params* params, const mstar_seq_desc* seqs,
                                 const mstar_mask_spec* masks, int32_t num_seqs,
                                 const mstar_segment* segments, int32_t num_segs, hipStream_t upload_stream,
                                 mstar_plan_t** out) {
    return plan_impl(params, seqs, masks, num_seqs, segments, num_segs, nullptr, 0, nullptr, 0, upload_stream, out);
}

MSTAR_EXPORT int mstar_attn_plan_cascade(const mstar_attn_params* params, const mstar_seq_desc* seqs,
                                         const mstar_mask_spec* masks, int32_t num_seqs,
                                         const mstar_segment* segments, int32_t num_segs,
                                         const mstar_prefix_group* groups, int32_t num_groups,
                                         const int32_t* members, int32_t num_members, hipStream_t upload_stream,
                                         mstar_plan_t** out) {
    return plan_impl(params, seqs, masks, num_seqs, segments, num_segs, groups, num_groups, members, num_members,
                     upload_stream, out);
}

MSTAR_EXPORT size_t mstar_attn_workspace_bytes(const mstar_plan_t* plan) {
    if (!plan || plan->host.partial_slots == 0) return 0;
    const size_t slots = (size_t)plan->host.partial_slots;
    return align256(slots * plan->host.params.head_dim * sizeof(float)) + align256(slots * sizeof(float));
}

MSTAR_EXPORT int mstar_attn_fwd(const mstar_plan_t* plan, const void* q, const void* k_pages,
                                const void* v_pages, const int32_t* block_table, void* out, float* lse,
                                void* workspace, size_t workspace_bytes, hipStream_t stream) {
    return mstar_attn_fwd_timed(plan, q, k_pages, v_pages, block_table, out, lse, workspace, workspace_bytes,
                                stream, nullptr, nullptr);
}

MSTAR_EXPORT int mstar_attn_fwd_timed(const mstar_plan_t* plan, const void* q, const void* k_pages,
                                      const void* v_pages, const int32_t* block_table, void* out, float* lse,
                                      void* workspace, size_t workspace_bytes, hipStream_t stream,
                                      const hipEvent_t* events_before, const hipEvent_t* events_after) {
    if (!plan) return fail(MSTAR_ERR_INVALID_ARG, "plan is NULL");
    if (!plan->dev) return fail(MSTAR_ERR_INVALID_ARG, "plan was built host-only");
    const mstar::HostPlan& h = plan->host;
    const bool any_work = !h.tiles.empty() || !h.few.empty() || !h.f32.empty() || !h.cascade.empty();
    if (!any_work) return MSTAR_OK;
    if (!q || !k_pages || !v_pages || !block_table || !out || !lse)
        return fail(MSTAR_ERR_INVALID_ARG, "a tensor pointer is NULL");
    if (!aligned(q, 16) || !aligned(k_pages, 16) || !aligned(v_pages, 16) || !aligned(out, 16) ||
        !aligned(lse, 4) || !aligned(block_table, 4))
        return fail(MSTAR_ERR_INVALID_ARG, "q/k_pages/v_pages/out must be 16-byte aligned");
    const size_t need = mstar_attn_workspace_bytes(plan);
    if (need > 0 && (!workspace || workspace_bytes < need || !aligned(workspace, 16)))
        return fail(MSTAR_ERR_WORKSPACE, "workspace missing, misaligned or smaller than mstar_attn_workspace_bytes");

    const int D = h.params.head_dim;
    unsigned char* blob = static_cast<unsigned char*>(plan->dev);
    mstar::KArgs a{};
    a.seqs = reinterpret_cast<const mstar::SeqInfo*>(blob + plan->off_seqs);
    a.row_hi = reinterpret_cast<const int32_t*>(blob + plan->off_row_hi);
    a.q = q;
    a.k = k_pages;
    a.v = v_pages;
    a.bt = block_table;
    a.out = out;
    a.lse = lse;
    a.part_o = static_cast<float*>(workspace);
    a.part_lse = need > 0 ? reinterpret_cast<float*>(static_cast<unsigned char*>(workspace) +
                                                     align256((size_t)h.partial_slots * D * sizeof(float)))
                          : nullptr;
    a.err = reinterpret_cast<int32_t*>(blob + plan->off_err);
    a.hq = h.params.num_qo_heads;
    a.hkv = h.params.num_kv_heads;
    a.group = h.group;
    a.bt_stride = h.params.max_blocks_per_seq;
    a.num_pages = h.params.num_pages;
    a.sm_scale = h.params.sm_scale;
    a.scale_log2 = h.params.sm_scale * 1.4426950408889634f;
    hipStream_t s = stream;

    hipError_t e;
    // The few-row kernel runs on the thread's side stream when the plan also
    // has tile work: it streams K/V from HBM while the tile kernel keeps the
    // matrix units busy.  Both write disjoint outputs and partial slots; the
    // merge waits for both.
    PlanBlock* b = plan->blk;
    hipStream_t side = plan->forked ? b->side : nullptr;
    if (side) {
        if ((e = hipEventRecord(b->fork, s)) != hipSuccess) return hip_fail(e, "hipEventRecord(fork)");
        if ((e = hipStreamWaitEvent(side, b->fork, 0)) != hipSuccess) return hip_fail(e, "hipStreamWaitEvent(fork)");
    }
    hipStream_t s_few = side ? side : s;
    // optional HIP events around kernel class k (0 tiles, 1 few-row, 2 fp32, 3 merge, 4 cascade),
    // recorded on the stream that kernel runs on
    auto mark = [&](const hipEvent_t* evs, int k) -> hipError_t {
        if (!evs || !evs[k]) return hipSuccess;
        return hipEventRecord(evs[k], k == 1 ? s_few : s);
    };
#define MSTAR_MARK(evs, k) \
    if ((e = mark(evs, k)) != hipSuccess) return hip_fail(e, "hipEventRecord")
    if (!h.few.empty()) {
        a.items = reinterpret_cast<const mstar::WorkItem*>(blob + plan->off_few);
        a.n_items = (int32_t)h.few.size();
        MSTAR_MARK(events_before, 1);
        if ((e = mstar::launch_few(a, D, h.decode_rb, s_few)) != hipSuccess) return hip_fail(e, "few-row kernel launch");
        MSTAR_MARK(events_after, 1);
    }
    if (side) {
        if ((e = hipEventRecord(b->join, side)) != hipSuccess) return hip_fail(e, "hipEventRecord(join)");
    }
    if (!h.tiles.empty()) {
        a.items = reinterpret_cast<const mstar::WorkItem*>(blob + plan->off_tiles);
        a.n_items = (int32_t)h.tiles.size();
        a.order = reinterpret_cast<const int32_t*>(blob + plan->off_order);
        a.n_wgs = (int32_t)(h.tile_order.size() / 2);
        MSTAR_MARK(events_before, 0);
        if ((e = mstar::launch_tiles(a, D, s)) != hipSuccess) return hip_fail(e, "tile kernel launch");
        MSTAR_MARK(events_after, 0);
    }
    if (!h.cascade.empty()) {
        a.items = reinterpret_cast<const mstar::WorkItem*>(blob + plan->off_casc);
        a.n_items = (int32_t)h.cascade.size();
        a.order = reinterpret_cast<const int32_t*>(blob + plan->off_casc_order);
        a.n_wgs = (int32_t)(h.casc_order.size() / 2);
        a.rows = reinterpret_cast<const int32_t*>(blob + plan->off_casc_rows);
        MSTAR_MARK(events_before, 4);
        if ((e = mstar::launch_cascade(a, D, s)) != hipSuccess) return hip_fail(e, "cascade kernel launch");
        MSTAR_MARK(events_after, 4);
    }
    if (side) {
        if ((e = hipStreamWaitEvent(s, b->join, 0)) != hipSuccess) return hip_fail(e, "hipStreamWaitEvent(join)");
    }
    if (!h.f32.empty()) {
        a.items = reinterpret_cast<const mstar::WorkItem*>(blob + plan->off_f32);
        a.n_items = (int32_t)h.f32.size();
        MSTAR_MARK(events_before, 2);
        if ((e = mstar::launch_f32(a, D, s)) != hipSuccess) return hip_fail(e, "fp32 kernel launch");
        MSTAR_MARK(events_after, 2);
    }
    if (!h.merges.empty()) {
        mstar::MArgs m{};
        m.items = reinterpret_cast<const mstar::MergeItem*>(blob + plan->off_merge);
        m.part_o = a.part_o;
        m.part_lse = a.part_lse;
        m.out = out;
        m.lse = lse;
        m.n_items = (int32_t)h.merges.size();
        m.hq = a.hq;
        MSTAR_MARK(events_before, 3);
        if ((e = mstar::launch_merge(m, D, h.params.dtype == MSTAR_DTYPE_BF16, s)) != hipSuccess)
            return hip_fail(e, "merge kernel launch");
        MSTAR_MARK(events_after, 3);
    }
#undef MSTAR_MARK
    if ((e = mark_use(plan, s)) != hipSuccess) return hip_fail(e, "hipEventRecord(plan use)");
    return MSTAR_OK;
}

MSTAR_EXPORT int mstar_attn_fwd_noalloc(const mstar_plan_t* plan, const void* q, const void* k_pages,
                                        const void* v_pages, const int32_t* block_table, void* out, float* lse,
                                        hipStream_t stream) {
    if (!plan) return fail(MSTAR_ERR_INVALID_ARG, "plan is NULL");
    const size_t need = mstar_attn_workspace_bytes(plan);
    if (need > mstar::kScratchBytes)
        return fail(MSTAR_ERR_WORKSPACE, "the plan needs " + std::to_string(need) +
                                             " bytes of scratch, more than the " +
                                             std::to_string(mstar::kScratchBytes) +
                                             " the allocation-free entry point holds; use mstar_attn_fwd");
    if (!plan->dev) return fail(MSTAR_ERR_INVALID_ARG, "plan was built host-only");
    void* ws = nullptr;
    if (need > 0) {
        hipError_t e = mstar::scratch_buffer(&ws);
        if (e != hipSuccess) return hip_fail(e, "scratch address");
    }
    return mstar_attn_fwd_timed(plan, q, k_pages, v_pages, block_table, out, lse, ws, need > 0 ? mstar::kScratchBytes : 0,
                                stream, nullptr, nullptr);
}

MSTAR_EXPORT int mstar_kv_append(const mstar_plan_t* plan, const void* k_new, const void* v_new,
                                 const int32_t* block_table, void* k_pages, void* v_pages, hipStream_t stream) {
    if (!plan) return fail(MSTAR_ERR_INVALID_ARG, "plan is NULL");
    if (!plan->dev) return fail(MSTAR_ERR_INVALID_ARG, "plan was built host-only");
    const mstar::HostPlan& h = plan->host;
    if (h.appends.empty()) return MSTAR_OK;
    if (!k_new || !v_new || !block_table || !k_pages || !v_pages)
        return fail(MSTAR_ERR_INVALID_ARG, "a tensor pointer is NULL");
    if (!aligned(k_new, 16) || !aligned(v_new, 16) || !aligned(k_pages, 16) || !aligned(v_pages, 16) ||
        !aligned(block_table, 4))
        return fail(MSTAR_ERR_INVALID_ARG, "k_new/v_new/k_pages/v_pages must be 16-byte aligned");
    unsigned char* blob = static_cast<unsigned char*>(plan->dev);
    mstar::AArgs a{};
    a.seqs = reinterpret_cast<const mstar::SeqInfo*>(blob + plan->off_seqs);
    a.items = reinterpret_cast<const mstar::WorkItem*>(blob + plan->off_append);
    a.k_new = k_new;
    a.v_new = v_new;
    a.bt = block_table;
    a.k = k_pages;
    a.v = v_pages;
    a.err = reinterpret_cast<int32_t*>(blob + plan->off_err);
    a.n_items = (int32_t)h.appends.size();
    const int elt = h.params.dtype == MSTAR_DTYPE_BF16 ? 2 : 4;
    a.row_bytes = h.params.num_kv_heads * h.params.head_dim * elt;
    a.bt_stride = h.params.max_blocks_per_seq;
    a.num_pages = h.params.num_pages;
    hipError_t e = mstar::launch_append(a, stream);
    if (e != hipSuccess) return hip_fail(e, "append kernel launch");
    if ((e = mark_use(plan, stream)) != hipSuccess)
        return hip_fail(e, "hipEventRecord(plan use)");
    return MSTAR_OK;
}

MSTAR_EXPORT int mstar_attn_check(mstar_plan_t* plan, hipStream_t stream, int32_t* error_bits) {
    if (!plan || !error_bits) return fail(MSTAR_ERR_INVALID_ARG, "plan or error_bits is NULL");
    *error_bits = 0;
    if (!plan->dev) return MSTAR_OK;
    hipStream_t s = stream;
    hipError_t e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
    int32_t* d_err = reinterpret_cast<int32_t*>(static_cast<unsigned char*>(plan->dev) + plan->off_err);
    int32_t v = 0;
    e = hipMemcpy(&v, d_err, sizeof v, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "error word read");
    *error_bits = v;
    if (v != 0) {
        const int32_t zero = 0;
        e = hipMemcpy(d_err, &zero, sizeof zero, hipMemcpyHostToDevice);
        if (e != hipSuccess) return hip_fail(e, "error word clear");
        return fail(MSTAR_ERR_INVALID_ARG, "a block-table entry was outside [0, num_pages)");
    }
    return MSTAR_OK;
}

MSTAR_EXPORT int mstar_attn_plan_stats(const mstar_plan_t* plan, mstar_plan_stats* out) {
    if (!plan || !out) return fail(MSTAR_ERR_INVALID_ARG, "plan or out is NULL");
    const mstar::HostPlan& h = plan->host;
    out->visible_pairs = h.visible_pairs;
    out->prefill_items = (int64_t)h.tiles.size();
    out->decode_items = (int64_t)h.few.size();
    out->f32_items = (int64_t)h.f32.size();
    out->merge_rows = (int64_t)h.merges.size();
    out->partial_slots = h.partial_slots;
    out->total_q = h.total_q;
    out->plan_host_us = plan->plan_us;
    out->device_bytes = (int64_t)plan->bytes;
    return MSTAR_OK;
}

MSTAR_EXPORT int mstar_attn_plan_key_ranges(const mstar_plan_t* plan, int32_t* lo_hi, int32_t num_seqs) {
    if (!plan || (!lo_hi && num_seqs > 0)) return fail(MSTAR_ERR_INVALID_ARG, "plan or lo_hi is NULL");
    if (num_seqs != plan->host.num_seqs) return fail(MSTAR_ERR_INVALID_ARG, "num_seqs differs from the plan");
    for (int32_t r = 0; r < num_seqs; ++r) {
        lo_hi[2 * r] = plan->host.key_lo[r];
        lo_hi[2 * r + 1] = plan->host.key_hi[r];
    }
    return MSTAR_OK;
}

MSTAR_EXPORT int mstar_attn_plan_items(const mstar_plan_t* plan, int32_t kind, int32_t* items, int64_t capacity,
                                       int64_t* count) {
    if (!plan || !count) return fail(MSTAR_ERR_INVALID_ARG, "plan or count is NULL");
    const mstar::HostPlan& h = plan->host;
    const void* src;
    size_t n;
    switch (kind) {
        case 0: src = h.tiles.data(); n = h.tiles.size(); break;
        case 1: src = h.few.data(); n = h.few.size(); break;
        case 2: src = h.f32.data(); n = h.f32.size(); break;
        case 3: src = h.merges.data(); n = h.merges.size(); break;
        case 4: src = h.cascade.data(); n = h.cascade.size(); break;
        case 5: {  // cascade rows, one (packed query row, query head, 0, ..., 0) record each
            n = h.casc_rows.size() / 2;
            *count = (int64_t)n;
            if (capacity > 0 && !items) return fail(MSTAR_ERR_INVALID_ARG, "items is NULL");
            const size_t m = capacity < 0 ? 0 : std::min<size_t>(n, (size_t)capacity);
            for (size_t i = 0; i < m; ++i) {
                std::memset(items + 8 * i, 0, 32);
                items[8 * i] = h.casc_rows[2 * i];
                items[8 * i + 1] = h.casc_rows[2 * i + 1];
            }
            return MSTAR_OK;
        }
        default: return fail(MSTAR_ERR_INVALID_ARG, "kind must be 0..5");
    }
    *count = (int64_t)n;
    if (capacity > 0 && !items) return fail(MSTAR_ERR_INVALID_ARG, "items is NULL");
    const size_t m = capacity < 0 ? 0 : std::min<size_t>(n, (size_t)capacity);
    if (m) std::memcpy(items, src, m * 32);
    return MSTAR_OK;
}

static int copy_order(const std::vector<int32_t>& o, int32_t* pairs, int64_t capacity, int64_t* count) {
    *count = (int64_t)(o.size() / 2);
    if (capacity > 0 && !pairs) return fail(MSTAR_ERR_INVALID_ARG, "pairs is NULL");
    const size_t m = capacity < 0 ? 0 : std::min<size_t>(o.size() / 2, (size_t)capacity);
    if (m) std::memcpy(pairs, o.data(), m * 2 * sizeof(int32_t));
    return MSTAR_OK;
}

MSTAR_EXPORT int mstar_attn_plan_tile_order(const mstar_plan_t* plan, int32_t* pairs, int64_t capacity,
                                            int64_t* count) {
    if (!plan || !count) return fail(MSTAR_ERR_INVALID_ARG, "plan or count is NULL");
    return copy_order(plan->host.tile_order, pairs, capacity, count);
}

MSTAR_EXPORT int mstar_attn_plan_cascade_order(const mstar_plan_t* plan, int32_t* pairs, int64_t capacity,
                                               int64_t* count) {
    if (!plan || !count) return fail(MSTAR_ERR_INVALID_ARG, "plan or count is NULL");
    return copy_order(plan->host.casc_order, pairs, capacity, count);
}

MSTAR_EXPORT void mstar_attn_plan_destroy(mstar_plan_t* plan) {
    if (!plan) return;
    release_block(plan->blk);  // back to the pool: no HIP call, no device synchronization
    give_host(plan->host);
    delete plan;
}

MSTAR_EXPORT const char* mstar_last_error(void) { return g_err.c_str(); }

// ---------------------------------------------------------------------------
// Async planner: plans built in submission order on a worker thread that owns
// a HIP stream for the uploads; at most `depth` plans submitted and not yet
// taken (two: the plan the current step uses and the one being built for the
// next step).
// ---------------------------------------------------------------------------
struct mstar_planner {
    struct Job {
        uint64_t id = 0;
        mstar_attn_params p{};
        std::vector<mstar_seq_desc> seqs;
        std::vector<mstar_mask_spec> masks;
        std::vector<mstar_segment> segs;
        std::vector<mstar_prefix_group> groups;  // empty: a plain plan
        std::vector<int32_t> members;
        int device = 0;
    };
    struct Done {
        uint64_t id = 0;
        int rc = MSTAR_OK;
        std::string err;
        mstar_plan_t* plan = nullptr;
        bool planner_built = false;
    };
    std::mutex mu;
    std::condition_variable cv_work, cv_done, cv_space;
    std::deque<Job> jobs;
    std::deque<Done> done;
    size_t depth = 2, outstanding = 0;
    uint64_t next_id = 0, next_take = 0;
    bool stop = false;
    std::thread worker;
    hipStream_t stream = nullptr;  // touched by the worker only (and by destroy after the join)
    int stream_device = -1;

    void run() {
        for (;;) {
            Job job;
            {
                std::unique_lock<std::mutex> lk(mu);
                cv_work.wait(lk, [&] { return stop || !jobs.empty(); });
                if (jobs.empty()) return;
                job = std::move(jobs.front());
                jobs.pop_front();
            }
            Done d;
            d.id = job.id;
            const bool host_only = (job.p.flags & MSTAR_FLAG_HOST_ONLY) != 0;
            hipStream_t s = nullptr;
            if (!host_only) {
                hipError_t e = hipSetDevice(job.device);
                if (e == hipSuccess && (!stream || stream_device != job.device)) {
                    if (stream) (void)hipStreamDestroy(stream);
                    stream = nullptr;
                    e = hipStreamCreateWithFlags(&stream, hipStreamNonBlocking);
                    stream_device = e == hipSuccess ? job.device : -1;
                }
                if (e != hipSuccess) {
                    d.rc = MSTAR_ERR_HIP;
                    d.err = std::string("async planner stream: ") + hipGetErrorString(e);
                }
                s = stream;
            }
            if (d.rc == MSTAR_OK) {
                d.rc = mstar_attn_plan_cascade(&job.p, job.seqs.data(), job.masks.data(), (int32_t)job.seqs.size(),
                                               job.segs.data(), (int32_t)job.segs.size(), job.groups.data(),
                                               (int32_t)job.groups.size(), job.members.data(),
                                               (int32_t)job.members.size(), s, &d.plan);
                if (d.rc != MSTAR_OK) {
                    d.err = mstar_last_error();
                } else if (!host_only) {
                    PlanBlock* b = d.plan->blk;
                    hipError_t e = b->ready ? hipSuccess : hipEventCreateWithFlags(&b->ready, hipEventDisableTiming);
                    if (e == hipSuccess) e = hipEventRecord(b->ready, stream);
                    if (e != hipSuccess) {
                        mstar_attn_plan_destroy(d.plan);
                        d.plan = nullptr;
                        d.rc = MSTAR_ERR_HIP;
                        d.err = std::string("async planner event: ") + hipGetErrorString(e);
                    } else {
                        d.planner_built = true;
                    }
                }
            }
            {
                std::lock_guard<std::mutex> lk(mu);
                done.push_back(std::move(d));
            }
            cv_done.notify_all();
        }
    }
};

MSTAR_EXPORT int mstar_planner_create(int32_t depth, mstar_planner_t** out) {
    if (!out) return fail(MSTAR_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    if (depth < 1 || depth > 64) return fail(MSTAR_ERR_INVALID_ARG, "depth must be in [1, 64]");
    mstar_planner* pl = new (std::nothrow) mstar_planner();
    if (!pl) return fail(MSTAR_ERR_NOMEM, "host allocation failed");
    pl->depth = (size_t)depth;
    try {
        pl->worker = std::thread([pl] { pl->run(); });
    } catch (...) {
        delete pl;
        return fail(MSTAR_ERR_NOMEM, "cannot start the planner thread");
    }
    *out = pl;
    return MSTAR_OK;
}

MSTAR_EXPORT int mstar_planner_submit_cascade(mstar_planner_t* planner, const mstar_attn_params* params,
                                              const mstar_seq_desc* seqs, const mstar_mask_spec* masks,
                                              int32_t num_seqs, const mstar_segment* segments, int32_t num_segs,
                                              const mstar_prefix_group* groups, int32_t num_groups,
                                              const int32_t* members, int32_t num_members) {
    if (!planner || !params) return fail(MSTAR_ERR_INVALID_ARG, "planner or params is NULL");
    if (num_seqs < 0 || num_segs < 0 || num_groups < 0 || num_members < 0)
        return fail(MSTAR_ERR_INVALID_ARG, "negative count");
    if ((num_seqs > 0 && (!seqs || !masks)) || (num_segs > 0 && !segments) || (num_groups > 0 && !groups) ||
        (num_members > 0 && !members))
        return fail(MSTAR_ERR_INVALID_ARG, "descriptor pointer is NULL");
    mstar_planner::Job job;
    try {
        job.p = *params;
        job.seqs.assign(seqs, seqs + num_seqs);
        job.masks.assign(masks, masks + num_seqs);
        job.segs.assign(segments, segments + num_segs);
        job.groups.assign(groups, groups + num_groups);
        job.members.assign(members, members + num_members);
    } catch (const std::bad_alloc&) {
        return fail(MSTAR_ERR_NOMEM, "host allocation failed");
    }
    if (!(job.p.flags & MSTAR_FLAG_HOST_ONLY)) {
        hipError_t e = hipGetDevice(&job.device);
        if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    }
    {
        std::unique_lock<std::mutex> lk(planner->mu);
        planner->cv_space.wait(lk, [&] { return planner->outstanding < planner->depth; });
        job.id = planner->next_id++;
        planner->jobs.push_back(std::move(job));
        ++planner->outstanding;
    }
    planner->cv_work.notify_one();
    return MSTAR_OK;
}

MSTAR_EXPORT int mstar_planner_submit(mstar_planner_t* planner, const mstar_attn_params* params,
                                      const mstar_seq_desc* seqs, const mstar_mask_spec* masks, int32_t num_seqs,
                                      const mstar_segment* segments, int32_t num_segs) {
    return mstar_planner_submit_cascade(planner, params, seqs, masks, num_seqs, segments, num_segs, nullptr, 0,
                                        nullptr, 0);
}

MSTAR_EXPORT int mstar_planner_take(mstar_planner_t* planner, hipStream_t stream, mstar_plan_t** out) {
    if (!planner || !out) return fail(MSTAR_ERR_INVALID_ARG, "planner or out is NULL");
    *out = nullptr;
    mstar_planner::Done d;
    {
        std::unique_lock<std::mutex> lk(planner->mu);
        if (planner->outstanding == 0) return fail(MSTAR_ERR_INVALID_ARG, "no plan was submitted");
        const uint64_t want = planner->next_take;
        planner->cv_done.wait(lk, [&] { return !planner->done.empty() && planner->done.front().id == want; });
        d = std::move(planner->done.front());
        planner->done.pop_front();
        ++planner->next_take;
        --planner->outstanding;
    }
    planner->cv_space.notify_one();
    if (d.rc != MSTAR_OK) return fail(d.rc, d.err);
    if (d.planner_built) d.plan->from_planner = true;
    if (d.plan->from_planner && stream) {
        hipError_t e = hipStreamWaitEvent(stream, d.plan->blk->ready, 0);
        if (e != hipSuccess) {
            mstar_attn_plan_destroy(d.plan);
            return hip_fail(e, "hipStreamWaitEvent(plan upload)");
        }
    }
    *out = d.plan;
    return MSTAR_OK;
}

MSTAR_EXPORT int mstar_attn_plan_wait(const mstar_plan_t* plan, hipStream_t stream) {
    if (!plan) return fail(MSTAR_ERR_INVALID_ARG, "plan is NULL");
    if (!plan->from_planner) return MSTAR_OK;
    hipError_t e = hipStreamWaitEvent(stream, plan->blk->ready, 0);
    return e == hipSuccess ? MSTAR_OK : hip_fail(e, "hipStreamWaitEvent(plan upload)");
}

MSTAR_EXPORT void mstar_planner_destroy(mstar_planner_t* planner) {
    if (!planner) return;
    {
        std::lock_guard<std::mutex> lk(planner->mu);
        planner->stop = true;
    }
    planner->cv_work.notify_all();
    if (planner->worker.joinable()) planner->worker.join();
    for (auto& d : planner->done) mstar_attn_plan_destroy(d.plan);
    if (planner->stream) {
        int cur = 0;
        const bool have = hipGetDevice(&cur) == hipSuccess;
        if (hipSetDevice(planner->stream_device) == hipSuccess) (void)hipStreamDestroy(planner->stream);
        if (have) (void)hipSetDevice(cur);
    }
    delete planner;
}
