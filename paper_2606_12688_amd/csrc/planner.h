// Host planner: mask descriptors -> per-row visible intervals -> work items.
// Pure C++ (no HIP); the C-ABI layer uploads what it produces.
#pragma once
#include <stdint.h>

#include <string>
#include <vector>

#include "mstar_attn.h"
#include "plan_types.h"

namespace mstar {

struct HostPlan {
    mstar_attn_params params{};
    int32_t num_seqs = 0;
    int32_t total_q = 0;
    int32_t group = 1;       // Hq / Hkv
    int32_t decode_rb = 1;   // 16-row blocks per few-row item (1, 2 or 4)
    std::vector<SeqInfo> seqs;
    std::vector<int32_t> row_hi;
    std::vector<int32_t> key_lo, key_hi;  // per request union of visible keys
    std::vector<WorkItem> tiles;          // multi-row kernel
    std::vector<int32_t> tile_order;      // (tile item, query head) of every multi-row workgroup, in launch order
    std::vector<WorkItem> few;            // few-row kernel
    std::vector<WorkItem> f32;            // fp32 kernel
    std::vector<MergeItem> merges;        // (row, head) outputs assembled from partials
    std::vector<WorkItem> appends;        // KV append: up to kAppendRows new rows of one request each
    // shared-prefix cascade: items over a group's prefix keys (seq = the first
    // member, head = KV head, rows row0 .. row0 + nrows - 1 of casc_rows), the
    // (packed query row, query head) of every row, and their launch order
    std::vector<WorkItem> cascade;
    std::vector<int32_t> casc_rows;
    std::vector<int32_t> casc_order;
    int64_t visible_pairs = 0;
    int64_t partial_slots = 0;

    // Back to the state of a new HostPlan, keeping the vectors' capacity (a
    // pooled plan then writes into memory it has already touched).  Every
    // member above is reset here.
    void reset() {
        params = mstar_attn_params{};
        num_seqs = total_q = 0;
        group = decode_rb = 1;
        for (auto* v : {&row_hi, &key_lo, &key_hi, &tile_order, &casc_rows, &casc_order}) v->clear();
        for (auto* v : {&tiles, &few, &f32, &appends, &cascade}) v->clear();
        seqs.clear();
        merges.clear();
        visible_pairs = partial_slots = 0;
    }
    // Bytes the vectors hold (their capacity).
    size_t capacity_bytes() const {
        size_t n = seqs.capacity() * sizeof(SeqInfo) + merges.capacity() * sizeof(MergeItem);
        for (auto* v : {&row_hi, &key_lo, &key_hi, &tile_order, &casc_rows, &casc_order}) n += v->capacity() * 4;
        for (auto* v : {&tiles, &few, &f32, &appends, &cascade}) n += v->capacity() * sizeof(WorkItem);
        return n;
    }
};

// Fills `plan` from the descriptors.  Returns MSTAR_OK or an MSTAR_ERR_* code
// with a message in `err`.
int build_host_plan(const mstar_attn_params* params, const mstar_seq_desc* seqs,
                    const mstar_mask_spec* masks, int32_t num_seqs, const mstar_segment* segs,
                    int32_t num_segs, HostPlan& plan, std::string& err,
                    const mstar_prefix_group* groups = nullptr, int32_t num_groups = 0,
                    const int32_t* members = nullptr, int32_t num_members = 0);

}  // namespace mstar
