// Device-visible plan records shared by the host planner and the kernels.
// Every record is 32 bytes so the packed plan blob keeps 16-byte alignment.
#pragma once
#include <stdint.h>

namespace mstar {

constexpr int kPage = 16;          // keys per KV page
constexpr int kTileRows = 128;     // query rows per multi-row tile item
constexpr int kTileKeys = 64;      // keys per LDS tile in the multi-row kernel
constexpr int kDecodeMaxRows = 64; // (query row x head) rows a few-row item may hold
constexpr int kSubKeys = 32;       // keys per wave step in the few-row kernel
constexpr int kF32Rows = 4;        // query rows per fp32 item (one wave each)
constexpr int kAppendRows = 16;    // new K/V rows per KV-append item

// Per request.  Query row i sits at position kv_len - q_len + i; its visible
// keys are [lo(i), hi(i)) with hi(i) = row_hi[hi_off + i] and
// lo(i) = window ? max(0, position - window + 1) : 0.
struct SeqInfo {
    int32_t q_len, kv_len, q_start, window;
    int32_t hi_off, seq_index, pad0, pad1;
};

// A unit of work over key range [k_begin, k_end).
//  multi-row / fp32 items: `head` is a query head; rows row0 .. row0+nrows-1
//    are query rows of the request.
//  few-row items: `head` is a KV head; row r in [row0, row0+nrows) stands for
//    query row r / G and query head head*G + r % G (G = Hq / Hkv).
// part < 0: write the final out/lse; otherwise write fp32 partials to slots
// part + (r - row0), combined afterwards by the merge kernel.
// One work item.  Few-row and fp32 items name their (KV or query) head;
// multi-row tile items have head = -1 and serve every query head (the head
// comes from the launch grid), and for a split tile the partial slot of query
// head h and row r is part + h * head_stride + r.
struct WorkItem {
    int32_t seq, head, row0, nrows;
    int32_t k_begin, k_end, part, head_stride;  // head_stride: -1 unless a split tile
};

// Output (packed_row, head) assembled from nslots partials at
// slot0 + s * stride and pad2 partials at pad0 + s * pad1 (the chunks of a
// shared prefix, for cascade members; pad2 = 0 otherwise).
struct MergeItem {
    int32_t row, head, slot0, stride;
    int32_t nslots, pad0, pad1, pad2;
};

static_assert(sizeof(SeqInfo) == 32, "SeqInfo layout");
static_assert(sizeof(WorkItem) == 32, "WorkItem layout");
static_assert(sizeof(MergeItem) == 32, "MergeItem layout");

}  // namespace mstar
