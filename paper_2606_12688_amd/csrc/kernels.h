// Launch interface between the C-ABI layer and the HIP kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mstar_attn.h"
#include "plan_types.h"

namespace mstar {

struct KArgs {
    const SeqInfo* seqs;
    const int32_t* row_hi;
    const WorkItem* items;
    const int32_t* order;  // multi-row launch: (item, query head) per workgroup
    const int32_t* rows;   // cascade launch: (packed query row, query head) of every row
    const void* q;
    const void* k;
    const void* v;
    const int32_t* bt;
    void* out;
    float* lse;
    float* part_o;    // [partial_slots][head_dim] fp32
    float* part_lse;  // [partial_slots] fp32 natural log
    int32_t* err;     // sticky device error word
    int32_t n_items;
    int32_t n_wgs;         // multi-row launch: workgroups (a multiple of 8)
    int32_t hq, hkv, group, bt_stride, num_pages;
    float sm_scale;
    float scale_log2;  // sm_scale * log2(e)
};

struct MArgs {
    const MergeItem* items;
    const float* part_o;
    const float* part_lse;
    void* out;
    float* lse;
    int32_t n_items;
    int32_t hq;
};

struct AArgs {
    const SeqInfo* seqs;
    const WorkItem* items;  // KV append items: rows row0 .. row0 + nrows - 1 of request seq
    const void* k_new;      // [total_q][row_bytes]
    const void* v_new;
    const int32_t* bt;
    void* k;                // pages [num_pages][16][row_bytes]
    void* v;
    int32_t* err;           // sticky device error word
    int32_t n_items;
    int32_t row_bytes;      // Hkv * head_dim * element size (a multiple of 16)
    int32_t bt_stride, num_pages;
};

hipError_t launch_tiles(const KArgs& a, int head_dim, hipStream_t s);
hipError_t launch_cascade(const KArgs& a, int head_dim, hipStream_t s);
hipError_t launch_append(const AArgs& a, hipStream_t s);
hipError_t launch_few(const KArgs& a, int head_dim, int row_blocks, hipStream_t s);
hipError_t launch_f32(const KArgs& a, int head_dim, hipStream_t s);
hipError_t launch_merge(const MArgs& a, int head_dim, bool bf16_out, hipStream_t s);

// Device scratch for the allocation-free entry point (a static device array of
// kScratchBytes per GPU): its device address on the current device.
constexpr size_t kScratchBytes = MSTAR_NOALLOC_SCRATCH_BYTES;
hipError_t scratch_buffer(void** ptr);

}  // namespace mstar
