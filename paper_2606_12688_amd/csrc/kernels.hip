// HIP kernels for batched paged attention with per-row visible intervals,
// written for gfx950 (CDNA4): 64-lane waves, 16x16x32 bf16 MFMA, LDS
// transpose reads.
//
// Notation used throughout: a 16x16x32 MFMA computes D[16][16] += A[16][32] *
// B[32][16].  Lane l (group G = l / 16, index n = l % 16) supplies
// A[n][8G .. 8G+7] and B[8G .. 8G+7][n], and receives D[4G .. 4G+3][n].
//
// Scores are formed transposed, S^T = K * Q^T (A = 16 keys x 32 dims of K,
// B = 32 dims x 16 query rows of Q^T), so lane l owns query row n and keys
// 4G .. 4G+3 of every 16-key block.  The weighted value sum is likewise
// transposed, O^T = V^T * P^T: the B operand P^T needs exactly the score
// values lane l already holds (two 16-key blocks make one 32-key step), and the
// A operand V^T is read from LDS with ds_read_b64_tr_b16.  Row statistics
// (running max, running sum, rescale factor) are therefore per-lane scalars.
//
// The softmax runs in base 2: s2 = s * sm_scale * log2(e), p = 2^(s2 - m2),
// and lse = (m2 + log2 l) * ln 2 at the end.
#include <hip/hip_runtime.h>

#include <mutex>

#include "kernels.h"

// Device scratch of the allocation-free entry point: the split-K partials of
// one call (fp32 partial rows, then their log-sum-exps) live here instead of
// in a caller workspace.  One copy per GPU, held until the process ends.  In
// host code this name is a host-side stand-in, never a device address: the
// device address comes from hipGetSymbolAddress (scratch_buffer below).
static __device__ __align__(256) unsigned char scratch[mstar::kScratchBytes];

namespace mstar {
namespace {

typedef __bf16 bf16_t;
typedef bf16_t bf16x8 __attribute__((ext_vector_type(8)));
typedef bf16_t bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

constexpr float kLn2 = 0.6931471805599453f;
constexpr int MSTAR_DEVERR_PAGE_RANGE_BIT = 1;  // MSTAR_DEVERR_PAGE_RANGE
constexpr float kNegInf = -__builtin_inff();

__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Workgroup and work-item indices straight from the hardware.  The runtime
// library's blockIdx / threadIdx accessors are not inlined into functions built
// with the IEEE mode bit off (their attributes differ), so they would be real
// calls returning the indices in vector registers, and everything derived from
// the workgroup index (item, bounds, loop counts) would leave scalar registers.
__device__ __forceinline__ int wg_id() { return (int)__builtin_amdgcn_workgroup_id_x(); }
__device__ __forceinline__ int thread_id() { return (int)__builtin_amdgcn_workitem_id_x(); }

// Reductions over the four lanes l, l^16, l^32, l^48 that share a query row,
// with gfx950's permlane swaps (v_permlane32_swap exchanges the upper half-wave
// of one register with the lower half of another; with both operands the same
// value, the two results hold x[l] and x[l^32] in some order, and likewise
// for 16).  Sums are formed in the same order on all four lanes.
// IEEE maximumNumber: the hardware max instruction as is.  fmaxf also has to
// quiet signalling NaNs, which costs an extra instruction per operand whenever
// the compiler cannot prove an input is not one (e.g. after a masking select).
__device__ __forceinline__ float fmax_num(float a, float b) { return __builtin_elementwise_maximumnum(a, b); }

struct RowGroup {
    __device__ __forceinline__ static float max(float x) {
        const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
        x = fmax_num(__uint_as_float(a[0]), __uint_as_float(a[1]));
        const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
        return fmax_num(__uint_as_float(b[0]), __uint_as_float(b[1]));
    }
    __device__ __forceinline__ static float sum(float x) {
        const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
        x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
        const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
        return __uint_as_float(b[0]) + __uint_as_float(b[1]);
    }
};

__device__ __forceinline__ bf16x4 lds_read_tr16(const bf16_t* p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p));
}

__device__ __forceinline__ bf16x8 cat(bf16x4 a, bf16x4 b) {
    return bf16x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

__device__ __forceinline__ bf16x8 to_bf16x8(f32x4 a, f32x4 b) {
    return cat(__builtin_convertvector(a, bf16x4), __builtin_convertvector(b, bf16x4));
}

// K/V rows are read through a buffer resource per page: the page base lives in
// scalar registers (built with scalar ops from the wave-uniform page index) and
// each lane adds a 32-bit byte offset that does not change from tile to tile,
// so the loads cost no vector ALU work.  The resource's range is one page.
constexpr int kBufferDword3 = 0x00020000;  // gfx9 buffer resource word 3 (raw, no format)

__device__ __forceinline__ __amdgpu_buffer_rsrc_t page_rsrc(const char* base, size_t byte_ofs, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(base + byte_ofs), (short)0, (int)bytes,
                                             kBufferDword3);
}

__device__ __forceinline__ uint4 load16_at(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)byte_off, 0, 0));
}

__device__ __forceinline__ uint4 load16(const void* base, int64_t elem_off_bf16) {
    return *reinterpret_cast<const uint4*>(reinterpret_cast<const bf16_t*>(base) + elem_off_bf16);
}
// The same with the non-temporal hint: for data read once (a tile's Q rows),
// so that it does not push shared K/V lines out of the caches (text+latent
// launch: fetched bytes 527 -> 334 MB, of which 250 MB are Q).
__device__ __forceinline__ uint4 load16_nt(const void* base, int64_t elem_off_bf16) {
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    const u32x4 w =
        __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(reinterpret_cast<const bf16_t*>(base) + elem_off_bf16));
    return __builtin_bit_cast(uint4, w);
}

// Visible interval of query row i of a request, clipped to the item's keys.
__device__ __forceinline__ void row_interval(const KArgs& a, const SeqInfo& si, const WorkItem& it,
                                             int32_t i, int32_t& lo, int32_t& hi) {
    const int32_t pos = si.kv_len - si.q_len + i;
    int32_t l0 = si.window > 0 ? max(0, pos - si.window + 1) : 0;
    int32_t h0 = a.row_hi[si.hi_off + i];
    lo = max(l0, it.k_begin);
    hi = min(h0, it.k_end);
}

// Lazy reference threshold (base-2 units): the online softmax moves its
// reference max only when a row's max exceeds it by more than this, so
// probabilities taken against a stale reference stay below 2^kLazy.
constexpr float kLazy = 8.0f;

// Balanced reductions over the 4*NB score values a lane holds for one row.
// Three-input maximum (one v_max3_f32).
__device__ __forceinline__ float max3(float a, float b, float c) { return fmax_num(fmax_num(a, b), c); }
template <int NB>
__device__ __forceinline__ float tree_max(const f32x4 (&s)[NB]) {
    static_assert(NB == 2 || NB == 4, "tree shapes for 8 and 16 values");
    if constexpr (NB == 4) {  // 16 values: 5 + 2 three-input maxima and one pair
        const float a0 = max3(s[0][0], s[0][1], s[0][2]), a1 = max3(s[0][3], s[1][0], s[1][1]);
        const float a2 = max3(s[1][2], s[1][3], s[2][0]), a3 = max3(s[2][1], s[2][2], s[2][3]);
        const float a4 = max3(s[3][0], s[3][1], s[3][2]);
        return fmax_num(max3(a0, a1, a2), max3(a3, a4, s[3][3]));
    } else {  // 8 values: two three-input maxima and one more over the rest
        const float a0 = max3(s[0][0], s[0][1], s[0][2]), a1 = max3(s[0][3], s[1][0], s[1][1]);
        return max3(a0, a1, fmax_num(s[1][2], s[1][3]));
    }
}
template <int NB>
__device__ __forceinline__ float tree_sum(const f32x4 (&s)[NB]) {
    float v[NB];
#pragma unroll
    for (int kb = 0; kb < NB; ++kb) v[kb] = (s[kb][0] + s[kb][1]) + (s[kb][2] + s[kb][3]);
#pragma unroll
    for (int w = NB / 2; w >= 1; w /= 2)
#pragma unroll
        for (int kb = 0; kb < w; ++kb) v[kb] = v[kb] + v[kb + w];
    return v[0];
}

// Online-softmax update of all RB 16-row blocks a wave owns, each with NB
// 16-key blocks of raw scores (hidden keys already -inf).  m and l are kept
// in base-2 units of the scaled scores: c = sm_scale * log2(e) > 0, so
// max(c s) = c max(s) and every probability is one FMA and one exp2.  The row
// blocks are processed side by side and reductions are balanced trees, so the
// dependency chains stay short.
//
// The reference max m is refreshed lazily: only when some row of the wave
// sees its max grow by more than kLazy (or has no reference yet).  Otherwise
// probabilities are taken against the stale m, so they stay below 2^kLazy, and
// the rescale of the O accumulators (the most expensive VALU work per tile)
// is skipped.  The result is exact either way: out = O / l and
// lse = m + log2(l) use the same reference.  Returns true (wave-uniform) when
// every O block rb must be multiplied by alpha[rb].  Leaves the probabilities
// in s.
template <int RB, int NB>
__device__ __forceinline__ bool softmax_update(const RowGroup& rg, f32x4 (&s)[RB][NB], float c, float (&m)[RB],
                                               float (&l)[RB], float (&alpha)[RB]) {
    float mx[RB];
    bool grow = false;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) mx[rb] = tree_max<NB>(s[rb]);
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        mx[rb] = rg.max(mx[rb]) * c;
        grow |= mx[rb] > m[rb] + kLazy;  // false while both are -inf
    }
    const bool rescale = __builtin_amdgcn_ballot_w64(grow) != 0;
    float m_use[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        alpha[rb] = 1.0f;
        if (rescale) {
            const float m_new = fmax_num(m[rb], mx[rb]);
            alpha[rb] = fast_exp2(m[rb] - (m_new == kNegInf ? 0.0f : m_new));
            m[rb] = m_new;
        }
        m_use[rb] = m[rb] == kNegInf ? 0.0f : m[rb];
    }
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int kb = 0; kb < NB; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) s[rb][kb][i] = fast_exp2(fmaf(s[rb][kb][i], c, -m_use[rb]));
    // The sums are taken over the fp32 probabilities, not over their bf16
    // roundings that enter P.V: a row dominated by a few keys would otherwise
    // carry up to 2^-9 relative error into lse.
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        const float sum = tree_sum<NB>(s[rb]);  // per-lane partial; row total reduced at the end
        l[rb] = rescale ? l[rb] * alpha[rb] + sum : l[rb] + sum;
    }
    return rescale;
}

// Probabilities against a fixed per-row reference m: p = 2^(c s - m), with no
// maximum; hidden keys are -inf and give 0.  ts receives the lane's partial
// sums of the tile.
template <int RB, int NB>
__device__ __forceinline__ void softmax_fixed(f32x4 (&s)[RB][NB], float c, const float (&m)[RB], float (&ts)[RB]) {
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int kb = 0; kb < NB; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) s[rb][kb][i] = fast_exp2(fmaf(s[rb][kb][i], c, -m[rb]));
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) ts[rb] = tree_sum<NB>(s[rb]);
}
// Bound on a lane's partial sum of one tile under the fixed reference: below
// it every probability is below 2^32, far from overflow of the sums and the
// weighted values; at or above it (or inf / NaN) the tile is redone exactly.
constexpr float kFixedTileLimit = 4294967296.0f;  // 2^32

// ---------------------------------------------------------------------------
// Multi-row tile kernel: one workgroup = 64 * RBW query rows of one query head
// (4 waves x RBW blocks of 16 rows) against the item's key range, 64 keys per
// tile, K and V tiles double-buffered in LDS.
//
// K/V tiles go from HBM straight into LDS (buffer loads with the LDS bit: lane
// i of a wave writes bytes [16 i, 16 i + 16) after the wave's base address), so
// no VGPRs, no LDS store instructions and no wait for the data sit between a
// tile's load and its use.  Rows are stored unpadded (2 D bytes) and the
// 16-byte chunks of each row are XOR-permuted by a function of the row, chosen
// so that the lanes served together by the K fragment reads (16 rows, one
// chunk column) and by the transposing V reads (8 rows, 32 bytes each) hit
// distinct banks.  The permutation is applied on the load side: the lane that
// fills physical chunk p of row r fetches logical chunk p ^ swz(r).
// ---------------------------------------------------------------------------
template <int D>
__device__ __forceinline__ int k_swizzle(int row) {  // 16-byte chunk XOR for K rows
    return D == 128 ? (row & 15) : ((row >> 1) & 7);
}
template <int D>
__device__ __forceinline__ int v_swizzle(int row) {  // 16-byte chunk XOR for V rows (even: 32-byte pairs stay whole)
    return D == 128 ? ((row & 7) << 1) : (((row >> 1) & 3) << 1);
}

// 4-byte direct global -> LDS load of one wave: lane i writes LDS bytes
// [lds_addr + 4 i, +4).  Issued from assembly so that the compiler does not
// track it (a tracked load in the tile loop makes the compiler wait for every
// outstanding load before its result is first used); the kernel waits itself
// (dma_barrier) before reading the filled bytes.
__device__ __forceinline__ void lds_dma4(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t lds_addr) {
    // M0 holds the (wave-uniform) LDS address; the compiler reserves M0, so
    // the asm puts its previous value back instead of declaring it clobbered
    uint32_t saved;
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %3\n\t"
        "buffer_load_dword %1, %2, 0 offen lds\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "v"(voff), "s"(r), "s"(__builtin_amdgcn_readfirstlane(lds_addr))
        : "memory");
}
// Waits for this wave's direct loads and LDS reads, then for the workgroup.
__device__ __forceinline__ void dma_barrier() {
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
}
typedef __attribute__((address_space(3))) char lds_char;

// Waits until at most N vector memory operations of this wave are outstanding.
template <int N>
__device__ __forceinline__ void wait_vmem() {
    static_assert(N >= 0 && N < 16, "vmcnt immediate");
    // gfx9 s_waitcnt encoding: vmcnt[3:0] in bits 3:0, expcnt and lgkmcnt at
    // their no-wait maxima (7 in bits 6:4, 15 in bits 11:8)
    __builtin_amdgcn_s_waitcnt(N | (7 << 4) | (15 << 8));
}

// 16-byte direct global -> LDS load of one wave through the compiler's
// builtin (lane i writes bytes [16 i, 16 i + 16) after `lds`, which must be
// wave-uniform).  The compiler tracks it and waits for it before later LDS
// reads.  The load is marked non-temporal (the NT cache-policy bit): the few-row
// kernel reads each V row of a request once, so its lines go first when the
// caches need room (decode batch: 0.617 -> 0.676 of HBM peak; 16-token
// chunks: 0.593 -> 0.618).  Marking the K loads into registers as well was
// slower on the chunk batch (0.571).
constexpr int kCachePolicyNT = 2;
__device__ __forceinline__ void lds_load16_nt(__amdgpu_buffer_rsrc_t r, uint32_t voff, void* lds) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)(lds), 16, voff, 0, 0,
                                             kCachePolicyNT);
}
__device__ __forceinline__ uint32_t lds_address(const void* p) {
    return (uint32_t)(uintptr_t)(const lds_char*)(p);
}
// 16-byte direct load with a wave-uniform scalar byte offset added to the
// global address, issued from assembly with the LDS address in M0.  The
// compiler waits for a direct load it tracks before any later LDS read that
// it cannot prove disjoint, and without alias-scope information it proves
// none: through the builtin, the next tile's prefetch made every tile wait
// for that prefetch before its first K read (text+latent 1.790 -> 1.709 ms
// together with the page indices read a tile ahead).  This one is not
// tracked; the caller waits itself (dma_barrier) before anything reads the
// bytes it writes.
__device__ __forceinline__ void lds_dma16s(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff, uint32_t lds_addr) {
    asm volatile("buffer_load_dwordx4 %0, %1, %2 offen lds"
                 :
                 : "v"(voff), "s"(r), "s"(soff), "{m0}"(__builtin_amdgcn_readfirstlane(lds_addr))
                 : "memory");
}

// K/V of a pool that fits in 2 GB are read through one buffer resource per
// pool with the page's byte offset in the instruction's scalar offset, so a
// load costs no scalar work beyond one multiply per page.  Larger pools get a
// resource per page (SMALL = false).  The 2 GB resource range keeps every
// valid offset in range and pushes the marker offset below out of range.
constexpr uint32_t kSmallPoolBytes = 0x80000000u;

// Keys per tile of the d = 128 tile kernel: 32-key tiles (32 KB of LDS, 162
// VGPRs) run three workgroups per CU instead of two with 64-key tiles, which
// the extra barrier per 32 keys more than pays for (text+latent 1.788 ->
// 1.713 ms, CFG labels 2.120 -> 2.006 ms).  At d = 64 the 64-key tile stays:
// 32-key tiles at five workgroups per CU were 1.6% slower.
#ifndef MSTAR_TILE_KEYS_D128
#define MSTAR_TILE_KEYS_D128 32
#endif
constexpr int kTileKeysD128 = MSTAR_TILE_KEYS_D128;

// Occupancy: two workgroups per CU at d = 128 with 64-key tiles (64 KB of
// LDS and up to 256 VGPRs each), four at d = 64 (32 KB, at most 128 VGPRs: the
// softmax's vector work, which bounds d = 64, then has four waves per SIMD to
// draw from).  BN keys per tile: 64, or 32 (half the LDS and score registers
// for a third workgroup per CU at d = 128, with a barrier per 32 keys).
template <int D, int RBW, bool SMALL, bool CASC, int BN>
__global__ __launch_bounds__(256, D == 64 ? 4 : (BN == 32 ? 3 : 2)) void tile_kernel(KArgs a) {
    static_assert(BN == 32 || BN == 64, "tile sizes");
    constexpr int NW = 4;            // waves per workgroup (32 rows each)
    constexpr int NB = BN / 16;      // 16-key blocks of a tile
    constexpr int NC = BN / 32;      // 32-key steps of the value product
    constexpr int RBY = 2 * D;       // bytes per K/V row in LDS
    constexpr int CH = D / 8;        // 16-byte chunks per row
    constexpr int DS = D / 32;       // MFMA steps over the head dimension
    constexpr int DB = D / 16;       // 16-wide blocks of O^T
    constexpr int NLD = BN * CH / (64 * NW);  // direct loads per wave, matrix and tile
    constexpr int RPL = 64 / CH;     // rows filled by one wave-wide load
    constexpr int TB = BN * RBY;     // bytes of one K or V tile
    constexpr int PPT = BN / 16;     // pages per tile
    // two tile buffers: tile t + 1 loads into one while tile t is read from the other
    __shared__ __attribute__((aligned(1024))) char buf0[2][TB];  // [K, V] of even tiles
    __shared__ __attribute__((aligned(1024))) char buf1[2][TB];  // [K, V] of odd tiles
    __shared__ __attribute__((aligned(256))) int32_t page_ring[2][64];
    // each row's visible interval [lo, hi), read on partial tiles only (kept
    // out of the registers the tile loop carries)
    __shared__ __attribute__((aligned(16))) int2 row_lohi[NW][16 * RBW];

    // The planner's launch order names the (item, query head) of every
    // workgroup; it keeps the workgroups that read the same K/V pages on one
    // XCD.  Padding entries (item < 0) exit.
    const int item = a.order[2 * wg_id()], head = a.order[2 * wg_id() + 1];
    if (item < 0) return;
    const int kvh = head / a.group;
    const WorkItem it = a.items[item];
    const SeqInfo si = a.seqs[it.seq];
    // the wave index is wave-uniform; readfirstlane lets the compiler keep
    // everything derived from it (row bounds, loop decisions) in scalars
    const int tid = thread_id(), wave = __builtin_amdgcn_readfirstlane(tid >> 6) & (NW - 1), lane = tid & 63;
    const int n = lane & 15, grp = lane >> 4;
    const int32_t* bt_row = a.bt + (int64_t)it.seq * a.bt_stride;
    const RowGroup rg;

    // ---- rows owned by this lane ------------------------------------------
    // CASC (a shared-prefix cascade item): row r is entry row0 + r of the row
    // list, a (packed query row, query head) of some group member; every key
    // of the item is visible to it.
    int32_t lo[RBW], hi[RBW];  // written to row_lohi, read back on partial tiles
    bool valid[RBW];
    bf16x8 qf[RBW][DS];
#pragma unroll
    for (int rb = 0; rb < RBW; ++rb) {
        const int r = wave * 16 * RBW + rb * 16 + n;
        valid[rb] = r < it.nrows;
        lo[rb] = 0;
        hi[rb] = 0;
        int64_t qoff;
        if constexpr (CASC) {
            if (valid[rb]) hi[rb] = it.k_end;
            const int32_t e = valid[rb] ? it.row0 + r : it.row0;
            qoff = ((int64_t)a.rows[2 * e] * a.hq + a.rows[2 * e + 1]) * D;
        } else {
            if (valid[rb]) row_interval(a, si, it, it.row0 + r, lo[rb], hi[rb]);
            qoff = ((int64_t)(si.q_start + it.row0 + r) * a.hq + head) * D;
        }
#pragma unroll
        for (int s = 0; s < DS; ++s) {
            if (valid[rb]) {
                uint4 u = load16_nt(a.q, qoff + 32 * s + 8 * grp);
                qf[rb][s] = __builtin_bit_cast(bf16x8, u);
            } else {
                qf[rb][s] = bf16x8{};
            }
        }
    }
    if (grp == 0) {
#pragma unroll
        for (int rb = 0; rb < RBW; ++rb) row_lohi[wave][rb * 16 + n] = make_int2(lo[rb], hi[rb]);
    }
    // wave-uniform bounds: intervals never shrink from one row to the next
    const int wr0 = wave * 16 * RBW;
    const int wr1 = min(wr0 + 16 * RBW - 1, it.nrows - 1);
    const bool wave_active = wr0 < it.nrows;
    int32_t w_lo_min = 0, w_lo_max = 0, w_hi_min = 0, w_hi_max = 0;
    if (wave_active) {
        if constexpr (CASC) {
            w_hi_min = w_hi_max = it.k_end;  // lo = 0 for every row
        } else {
            row_interval(a, si, it, it.row0 + wr0, w_lo_min, w_hi_min);
            row_interval(a, si, it, it.row0 + wr1, w_lo_max, w_hi_max);
        }
    }

    float m[RBW], l[RBW];
    f32x4 o[RBW][DB];
#pragma unroll
    for (int rb = 0; rb < RBW; ++rb)
#pragma unroll
        for (int db = 0; db < DB; ++db) o[rb][db] = f32x4{0, 0, 0, 0};
    // Rows past the item's end (never stored) start with reference 0, so that
    // the fixed mode below never meets an infinite reference.
#pragma unroll
    for (int rb = 0; rb < RBW; ++rb) {
        m[rb] = valid[rb] ? kNegInf : 0.0f;
        l[rb] = 0.0f;
    }

    // ---- LDS read offsets (per lane, the same for every tile) ----------------
    // K fragment (kb, s): row kb*16 + n, logical chunk 4 s + grp.
    uint32_t koff[DS];
    {
        const int sw = k_swizzle<D>(n);
#pragma unroll
        for (int s = 0; s < DS; ++s) koff[s] = n * RBY + (((4 * s + grp) ^ sw) << 4);
    }
    // V^T fragment (c, db, half h): row 32 c + 16 h + 4 grp + n / 4, bf16
    // column 16 db + 4 (n & 3), i.e. logical chunk 2 db + (n & 3) / 2.
    uint32_t voff[DB];
    {
        const int vr = 4 * grp + (n >> 2);
        const int vh = v_swizzle<D>(vr) >> 1;
        const uint32_t base = vr * RBY + (((n & 3) >> 1) << 4) + ((n & 1) << 3);
#pragma unroll
        for (int db = 0; db < DB; ++db) voff[db] = base + ((db ^ vh) << 5);
    }

    // ---- direct K/V loads ---------------------------------------------------
    // The item's page indices pass through a two-window LDS ring (64 pages =
    // 16 tiles per window).  Wave 0 fills a window with one direct-to-LDS dword
    // load (lane i writes page 64 w + i at ring[w & 1][i]) a whole window ahead
    // of its use; like the K/V loads it is covered by the wait at the top of
    // every tile.  Keeping the page indices out of compiler-tracked registers
    // matters: a tracked load in the loop makes the compiler wait for every
    // outstanding load (the just-issued K/V prefetch included) before its
    // result is first moved.  Load j of wave w fills rows (NW j + w) RPL ..
    // +RPL of the tile, which lie in one page; a thread's slot inside that
    // page and its logical chunk are the same for every tile and every j.
    const int32_t page0 = it.k_begin >> 4;
    const int32_t n_pages = ((it.k_end + 15) >> 4) - page0;
    const int n_tiles = (it.k_end - it.k_begin + BN - 1) / BN;
    const int32_t* bt_item = bt_row + page0;
    // window w of the item's pages: zeros past the last page (range check)
    auto load_window = [&](int w) {
        if (wave == 0 && 64 * w < n_pages) {
            // the pointer and size are wave-uniform; readfirstlane puts them in
            // scalar registers, where a buffer resource must live
            const uint64_t base = reinterpret_cast<uint64_t>(bt_item);
            const uint32_t lo32 = __builtin_amdgcn_readfirstlane((uint32_t)base);
            const uint32_t hi32 = __builtin_amdgcn_readfirstlane((uint32_t)(base >> 32));
            const __amdgpu_buffer_rsrc_t r =
                page_rsrc(reinterpret_cast<const char*>(((uint64_t)hi32 << 32) | lo32), 0,
                          (uint32_t)__builtin_amdgcn_readfirstlane(n_pages * 4));
            lds_dma4(r, (uint32_t)(64 * w + lane) * 4u, lds_address(&page_ring[w & 1][0]));
        }
    };
    bool page_err = false;
    const int64_t slot_stride = (int64_t)a.hkv * D;
    const uint32_t page_bytes = (uint32_t)(16 * slot_stride * sizeof(bf16_t));
    const int lrow0 = wave * RPL + lane / CH;  // tile row of load j = 0
    const int pch = lane % CH;                 // physical chunk this lane fills
    const uint32_t slot_off = (uint32_t)(((lrow0 & 15) * slot_stride + (int64_t)kvh * D) * sizeof(bf16_t));
    const uint32_t gk = slot_off + ((pch ^ k_swizzle<D>(lrow0)) << 4);
    const uint32_t gv = slot_off + ((pch ^ v_swizzle<D>(lrow0)) << 4);
    const char* kbase = reinterpret_cast<const char*>(a.k);
    const char* vbase = reinterpret_cast<const char*>(a.v);
    const __amdgpu_buffer_rsrc_t kpool = page_rsrc(kbase, 0, kSmallPoolBytes);
    const __amdgpu_buffer_rsrc_t vpool = page_rsrc(vbase, 0, kSmallPoolBytes);
    // Rows past the item's end read zeros through the buffer range check (their
    // offset is pushed out of range), and so does every row of a page outside
    // the pool: no access outside the pool, and zeros in LDS.
    constexpr uint32_t kOutOfRange = 0x80000000u;
    // LDS addresses of the two tile buffers (K at +0, V at +TB)
    const uint32_t lds_buf0 = __builtin_amdgcn_readfirstlane(lds_address(&buf0[0][0]));
    const uint32_t lds_buf1 = __builtin_amdgcn_readfirstlane(lds_address(&buf1[0][0]));
    // Page indices of tile tix for this wave's loads, read from the ring.
    // Load j of wave w fills tile rows (NW j + w) RPL .. +RPL, which lie in
    // page (NW j + w) RPL / 16 of the tile.  With four waves and RPL = 4
    // (d = 128) that page is j for every wave: one 8- or 16-byte LDS read
    // holds them.  Otherwise each wave reads its own indices at a
    // wave-uniform LDS address, with no per-lane selection.
    auto read_pages = [&](int tix, int32_t (&pv)[NLD]) {
        const int rel0 = tix * PPT;
        const int32_t* ring = &page_ring[(rel0 >> 6) & 1][rel0 & 63];
        if constexpr (NW == 4 && RPL == 4 && NLD == 4) {
            const int4 pq = *reinterpret_cast<const int4*>(ring);
            pv[0] = pq.x; pv[1] = pq.y; pv[2] = pq.z; pv[3] = pq.w;
        } else if constexpr (NW == 4 && RPL == 4 && NLD == 2) {
            const int2 pq = *reinterpret_cast<const int2*>(ring);
            pv[0] = pq.x; pv[1] = pq.y;
        } else {
#pragma unroll
            for (int j = 0; j < NLD; ++j) pv[j] = ring[((NW * j + wave) * RPL) >> 4];
        }
    };
    // Loads of tile tix into the buffer at LDS address `dst` ([K, V]), with
    // the page indices `pv` read one tile earlier (so that the LDS round trip
    // of the read overlaps a tile's compute); then the indices of tile tix + 1.
    int32_t pv[NLD];
    auto issue_tile = [&](int tix, uint32_t dst) {
        const int rel0 = tix * PPT;
        uint32_t page[NLD];
#pragma unroll
        for (int j = 0; j < NLD; ++j) page[j] = (uint32_t)__builtin_amdgcn_readfirstlane(pv[j]);
        // first tile of window w >= 1: every wave is past its last read of
        // window w - 1, so its ring slot can take window w + 1 (tile tix + 1
        // lies in window w, or in w + 1 only if tix ends window w, whose
        // successor has landed long before)
        if (tix > 0 && (rel0 & 63) == 0) load_window((rel0 >> 6) + 1);
        if (tix + 1 < n_tiles) read_pages(tix + 1, pv);
        bool all_ok = true;
#pragma unroll
        for (int j = 0; j < NLD; ++j) all_ok &= page[j] < (uint32_t)a.num_pages;
        const int32_t k0 = it.k_begin + tix * BN;
        const bool tail = k0 + BN > it.k_end;
        if (__builtin_expect(SMALL && all_ok && !tail, 1)) {
            // common case: only the page offsets change from tile to tile
#pragma unroll
            for (int j = 0; j < NLD; ++j) {
                const uint32_t soff = page[j] * page_bytes;
                lds_dma16s(kpool, gk, soff, dst + (NW * j + wave) * 1024);
                lds_dma16s(vpool, gv, soff, dst + TB + (NW * j + wave) * 1024);
            }
        } else {
#pragma unroll
            for (int j = 0; j < NLD; ++j) {
                const int pg = ((NW * j + wave) * RPL) >> 4;  // page of this load within the tile
                const bool ok = page[j] < (uint32_t)a.num_pages;
                page_err |= !ok && k0 + 16 * pg < it.k_end;
                const bool live = ok && (!tail || k0 + lrow0 + NW * j * RPL < it.k_end);
                if (SMALL) {
                    const uint32_t soff = ok ? page[j] * page_bytes : 0u;
                    lds_dma16s(kpool, live ? gk : kOutOfRange, soff, dst + (NW * j + wave) * 1024);
                    lds_dma16s(vpool, live ? gv : kOutOfRange, soff, dst + TB + (NW * j + wave) * 1024);
                } else {
                    const size_t pofs = ok ? (size_t)page[j] * page_bytes : 0;
                    const uint32_t nrec = ok ? page_bytes : 0u;
                    lds_dma16s(page_rsrc(kbase, pofs, nrec), live ? gk : kOutOfRange, 0u,
                               dst + (NW * j + wave) * 1024);
                    lds_dma16s(page_rsrc(vbase, pofs, nrec), live ? gv : kOutOfRange, 0u,
                               dst + TB + (NW * j + wave) * 1024);
                }
            }
        }
    };

    // ---- one tile: scores, mask, online softmax, weighted values ---------------
    const float c2 = a.scale_log2;
    auto scores = [&](const char* kl, f32x4 (&sc)[RBW][NB]) {
#pragma unroll
        for (int kb = 0; kb < NB; ++kb) {
            bf16x8 kf[DS];
#pragma unroll
            for (int s = 0; s < DS; ++s) kf[s] = *reinterpret_cast<const bf16x8*>(kl + kb * 16 * RBY + koff[s]);
#pragma unroll
            for (int rb = 0; rb < RBW; ++rb) sc[rb][kb] = mfma16(kf[0], qf[rb][0], f32x4{0, 0, 0, 0});
#pragma unroll
            for (int s = 1; s < DS; ++s)
#pragma unroll
                for (int rb = 0; rb < RBW; ++rb) sc[rb][kb] = mfma16(kf[s], qf[rb][s], sc[rb][kb]);
        }
    };
    auto mask = [&](int32_t k0, f32x4 (&sc)[RBW][NB]) {
#pragma unroll
        for (int rb = 0; rb < RBW; ++rb) {
            // key k0 + 4 grp + c is visible iff lo <= key < hi
            const int2 lh = row_lohi[wave][rb * 16 + n];
            const int32_t lo_r = lh.x - (k0 + 4 * grp), hi_r = lh.y - (k0 + 4 * grp);
#pragma unroll
            for (int kb = 0; kb < NB; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int c = kb * 16 + i;
                    if (!(c >= lo_r && c < hi_r)) sc[rb][kb][i] = kNegInf;
                }
        }
    };
    // probabilities as the bf16 B operands of the value product (32-key halves)
    auto pack = [&](const f32x4 (&sc)[RBW][NB], bf16x8 (&pf)[NC][RBW]) {
#pragma unroll
        for (int c = 0; c < NC; ++c)
#pragma unroll
            for (int rb = 0; rb < RBW; ++rb) pf[c][rb] = to_bf16x8(sc[rb][2 * c], sc[rb][2 * c + 1]);
    };
    auto values = [&](const char* vl, const bf16x8 (&pf)[NC][RBW]) {
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            bf16x8 vf[DB];
#pragma unroll
            for (int db = 0; db < DB; ++db) {
                const bf16_t* base = reinterpret_cast<const bf16_t*>(vl + 32 * c * RBY + voff[db]);
                vf[db] = cat(lds_read_tr16(base), lds_read_tr16(base + 16 * D));
            }
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
                for (int rb = 0; rb < RBW; ++rb) o[rb][db] = mfma16(vf[db], pf[c][rb], o[rb][db]);
        }
    };
    // Two softmax modes.  Exact: the tile's row maxima are taken and the
    // reference moved lazily (softmax_update); used on a wave's tiles until
    // every valid row of the wave has a reference.  Fixed: probabilities
    // against each row's reference as it stands, with no maximum at all (an
    // fma, an exp2 and a sum per score), which takes the reductions and the
    // cross-lane exchange out of the tile.  Both are exact (out = O / l and
    // lse = m + log2 l share the reference).  A fixed-mode tile whose sums
    // reach kFixedTileLimit (scores far above the reference) is redone in exact
    // mode from its scores, recomputed from the K tile still in LDS.
    bool need_ref = true;  // wave-uniform: some valid row of the wave has no reference yet
    auto exact_update = [&](f32x4 (&sc)[RBW][NB]) {
        float alpha[RBW];
        if (softmax_update<RBW, NB>(rg, sc, c2, m, l, alpha)) {
#pragma unroll
            for (int rb = 0; rb < RBW; ++rb)
#pragma unroll
                for (int db = 0; db < DB; ++db) o[rb][db] *= alpha[rb];
        }
    };
    auto compute_tile = [&](int tix, const char (&cur)[2][TB]) {
        const int32_t k0 = it.k_begin + tix * BN;
        if (!(wave_active && k0 < w_hi_max && k0 + BN > w_lo_min)) return;
        // the compiler's interleaving strategy for LDS reads among MFMAs
        // (1-2% at d = 128, neutral at d = 64)
        __builtin_amdgcn_iglp_opt(0);
        const char* kl = &cur[0][0];
        const char* vl = &cur[1][0];
        const bool full = k0 >= w_lo_max && k0 + BN <= w_hi_min;
        f32x4 sc[RBW][NB];
        bf16x8 pf[NC][RBW];
        scores(kl, sc);
        if (!full) mask(k0, sc);
        bool exact = need_ref;
        if (!need_ref) {
            float ts[RBW];
            softmax_fixed<RBW, NB>(sc, c2, m, ts);
            bool over = false;
#pragma unroll
            for (int rb = 0; rb < RBW; ++rb) over |= !(ts[rb] < kFixedTileLimit);
            exact = __builtin_amdgcn_ballot_w64(over) != 0;
            if (!exact) {
#pragma unroll
                for (int rb = 0; rb < RBW; ++rb) l[rb] += ts[rb];
                pack(sc, pf);
            }
        }
        if (exact) {
            if (!need_ref) {
                // a fixed-mode tile out of range: its scores again, from an
                // opaque copy of the K tile's address so that the compiler
                // loads the fragments anew instead of keeping the first ones
                // (and the raw scores) alive through the softmax
                uint32_t ka = lds_address(kl);
                asm volatile("" : "+s"(ka));
                scores((const char*)((const lds_char*)(uintptr_t)ka), sc);
                if (!full) mask(k0, sc);
            }
            exact_update(sc);
            bool missing = false;
#pragma unroll
            for (int rb = 0; rb < RBW; ++rb) missing |= m[rb] == kNegInf;
            need_ref = __builtin_amdgcn_ballot_w64(missing) != 0;
            pack(sc, pf);
        }
        values(vl, pf);
    };

    if (n_tiles > 0) {
        load_window(0);
        load_window(1);
        // The Q fragments are consumed here, so the compiler's wait for their
        // loads sits before any K/V load is in flight.
#pragma unroll
        for (int rb = 0; rb < RBW; ++rb)
#pragma unroll
            for (int s = 0; s < DS; ++s) asm volatile("" ::"v"(qf[rb][s]));
        dma_barrier();  // windows 0 and 1 of the page ring have landed
        read_pages(0, pv);
        issue_tile(0, lds_buf0);
        // Tile tix is in buf[tix & 1].  At the top of each tile every wave has
        // its own loads of the tile done (vmcnt) and every wave is done with
        // the other buffer (barrier), which the next tile's loads then take.
        for (int tix = 0; tix < n_tiles; tix += 2) {
            dma_barrier();
            if (tix + 1 < n_tiles) issue_tile(tix + 1, lds_buf1);
            compute_tile(tix, buf0);
            if (tix + 1 < n_tiles) {
                dma_barrier();
                if (tix + 2 < n_tiles) issue_tile(tix + 2, lds_buf0);
                compute_tile(tix + 1, buf1);
            }
        }
    }
    if (page_err && lane == 0) atomicOr(a.err, MSTAR_DEVERR_PAGE_RANGE_BIT);

    // ---- epilogue -------------------------------------------------------------
#pragma unroll
    for (int rb = 0; rb < RBW; ++rb) {
        const float lt = rg.sum(l[rb]);
        if (!valid[rb]) continue;
        const int r = wave * 16 * RBW + rb * 16 + n;
        const float inv = lt > 0.0f ? 1.0f / lt : 0.0f;
        const float lse = lt > 0.0f ? (m[rb] + __log2f(lt)) * kLn2 : kNegInf;
        if constexpr (CASC) {
            const int64_t slot = it.part + r;  // cascade items always write partials
            float* po = a.part_o + slot * D;
#pragma unroll
            for (int db = 0; db < DB; ++db)
                *reinterpret_cast<f32x4*>(po + db * 16 + 4 * grp) = o[rb][db] * inv;
            if (grp == 0) a.part_lse[slot] = lse;
        } else if (it.part < 0) {
            const int64_t row = (int64_t)(si.q_start + it.row0 + r) * a.hq + head;
            bf16_t* out = reinterpret_cast<bf16_t*>(a.out) + row * D;
#pragma unroll
            for (int db = 0; db < DB; ++db) {
                const bf16x4 v = __builtin_convertvector(o[rb][db] * inv, bf16x4);
                *reinterpret_cast<bf16x4*>(out + db * 16 + 4 * grp) = v;
            }
            if (grp == 0) a.lse[row] = lse;
        } else {
            const int64_t slot = it.part + (int64_t)head * it.head_stride + r;
            float* po = a.part_o + slot * D;
#pragma unroll
            for (int db = 0; db < DB; ++db)
                *reinterpret_cast<f32x4*>(po + db * 16 + 4 * grp) = o[rb][db] * inv;
            if (grp == 0) a.part_lse[slot] = lse;
        }
    }
}

// ---------------------------------------------------------------------------
// Few-row kernel: one workgroup = up to 16*RB rows (query rows x the query
// heads of one KV head) against the item's key range.  The four waves take
// interleaved 32-key steps; K goes straight from HBM into MFMA operand
// registers, V is staged through a wave-private LDS slice for the transpose
// read, and the next step's loads are in flight while the current one is
// computed.  The four waves' partial results are combined through LDS.
// ---------------------------------------------------------------------------
template <int D, int RB>
__global__ __launch_bounds__(256, RB == 4 ? 1 : 2) void few_kernel(KArgs a) {
    constexpr int SK = kSubKeys;
    constexpr int RBY = 2 * D;        // bytes per V row in LDS
    constexpr int DS = D / 32, DB = D / 16, CH = D / 8;
    constexpr int VL = SK * CH / 64;  // direct V loads per wave and step
    constexpr int RPL = 64 / CH;      // V rows filled by one wave-wide load
    constexpr int SB = SK * RBY;      // bytes of one wave's V slot
    static_assert(RB * 16 * D * 4 <= 4 * SB, "combine buffer must fit in one set of V slots");
    // V of the steps held in register buffers A and B goes straight from HBM
    // into wave-private LDS slots, one array per buffer (the wave waits for
    // all of its loads before each step; see compute_step).
    __shared__ __attribute__((aligned(1024))) char v_slot_a[4][SB];
    __shared__ __attribute__((aligned(1024))) char v_slot_b[4][SB];
    __shared__ float ml_lds[4][2][RB * 16];
    __shared__ float fin_lds[2][RB * 16];

    const WorkItem it = a.items[wg_id()];
    const SeqInfo si = a.seqs[it.seq];
    const int tid = thread_id(), wave = __builtin_amdgcn_readfirstlane(tid >> 6) & 3, lane = tid & 63;
    const int n = lane & 15, grp = lane >> 4;
    const int G = a.group;
    const int kvh = it.head;
    const int32_t* bt_row = a.bt + (int64_t)it.seq * a.bt_stride;
    const RowGroup rg;

    int32_t lo[RB], hi[RB];
    bool valid[RB];
    bf16x8 qf[RB][DS];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        const int r = rb * 16 + n;
        valid[rb] = r < it.nrows;
        const int rr = it.row0 + r;
        const int qi = rr / G, h = kvh * G + rr % G;
        lo[rb] = 0;
        hi[rb] = 0;
        if (valid[rb]) row_interval(a, si, it, qi, lo[rb], hi[rb]);
        const int64_t qoff = ((int64_t)(si.q_start + qi) * a.hq + h) * D;
#pragma unroll
        for (int s = 0; s < DS; ++s) {
            if (valid[rb]) {
                qf[rb][s] = __builtin_bit_cast(bf16x8, load16(a.q, qoff + 32 * s + 8 * grp));
            } else {
                qf[rb][s] = bf16x8{};
            }
        }
    }
    int32_t lo_max, hi_min, dummy;
    {
        const int q_first = it.row0 / G, q_last = (it.row0 + it.nrows - 1) / G;
        row_interval(a, si, it, q_first, dummy, hi_min);
        row_interval(a, si, it, q_last, lo_max, dummy);
    }

    float m[RB], l[RB];
    f32x4 o[RB][DB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        m[rb] = kNegInf;
        l[rb] = 0.0f;
#pragma unroll
        for (int db = 0; db < DB; ++db) o[rb][db] = f32x4{0, 0, 0, 0};
    }

    // Wave w takes steps w, w+4, w+8, ... of 32 keys; its i-th step starts at
    // key k_begin + 32 * (w + 4 i) and spans exactly two pages (k_begin is page
    // aligned).  The page indices of 32 consecutive steps live in one register
    // (lane 2i+h holds half h of step i) and are read back with readlane, so no
    // block-table load sits between a step and its K/V loads.
    const int n_steps = (it.k_end - it.k_begin + SK - 1) / SK;
    const int my_steps = wave < n_steps ? (n_steps - wave + 3) / 4 : 0;
    const int32_t page0 = it.k_begin >> 4;
    const int32_t n_pages = ((it.k_end + 15) >> 4) - page0;
    auto load_pages = [&](int first_step) {
        const int pg = 2 * (wave + 4 * (first_step + (lane >> 1))) + (lane & 1);
        return pg < n_pages ? bt_row[page0 + pg] : 0;
    };
    int32_t pw_cur = load_pages(0), pw_next = my_steps > 32 ? load_pages(32) : 0;
    const int64_t slot_stride = (int64_t)a.hkv * D;

    // K of one step, straight into MFMA operand registers
    struct Step {
        uint4 k[2][DS];
    };
    // Byte offsets of this lane's K and V chunks inside their page, the same
    // for every step; the page (wave-uniform) supplies a scalar base.  Rows past
    // the item's end read zeros through the buffer range check and a page
    // outside the pool gets an empty range, so the data needs no selects.
    constexpr uint32_t kOutOfRange = 0x80000000u;
    const size_t page_bytes = (size_t)16 * slot_stride * sizeof(bf16_t);
    uint32_t koff[DS];
#pragma unroll
    for (int s = 0; s < DS; ++s)
        koff[s] = (uint32_t)((n * slot_stride + (int64_t)kvh * D + 32 * s + 8 * grp) * sizeof(bf16_t));
    // V load j fills rows j RPL .. j RPL + RPL - 1 of the step; the lane writes
    // physical chunk lane % CH of its row and fetches the logical chunk that the
    // row's swizzle puts there.  The in-page slot and the swizzle repeat every
    // 16 / RPL loads.
    constexpr int VJ = 16 / RPL;
    uint32_t voff[VJ];
#pragma unroll
    for (int j = 0; j < VJ; ++j) {
        const int row = j * RPL + lane / CH;
        const int chunk = (lane % CH) ^ v_swizzle<D>(row);
        voff[j] = (uint32_t)(((row & 15) * slot_stride + (int64_t)kvh * D + 8 * chunk) * sizeof(bf16_t));
    }
    // transposing V reads: rows 4 grp + n / 4 (+16), bf16 columns 16 db + 4 (n & 3)
    uint32_t vrd[DB];
    {
        const int vr = 4 * grp + (n >> 2);
        const int vh = v_swizzle<D>(vr) >> 1;
        const uint32_t base = vr * RBY + (((n & 3) >> 1) << 4) + ((n & 1) << 3);
#pragma unroll
        for (int db = 0; db < DB; ++db) vrd[db] = base + ((db ^ vh) << 5);
    }
    const int wave_u = __builtin_amdgcn_readfirstlane(wave);
    const char* kbase = reinterpret_cast<const char*>(a.k);
    const char* vbase = reinterpret_cast<const char*>(a.v);
    bool page_err = false;
    auto load_step = [&](Step& st, char (&vs)[4][SB], int i) {
        if (i > 0 && (i & 31) == 0) {  // next window of page indices
            pw_cur = pw_next;
            pw_next = i + 32 < my_steps ? load_pages(i + 32) : 0;
        }
        const int32_t k0 = it.k_begin + SK * (wave + 4 * i);
        const bool tail = k0 + SK > it.k_end;
        __amdgpu_buffer_rsrc_t rk[2], rv[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int32_t page = __builtin_amdgcn_readlane(pw_cur, 2 * (i & 31) + h);
            const bool ok = (uint32_t)page < (uint32_t)a.num_pages;
            page_err |= !ok && k0 + 16 * h < it.k_end;
            const size_t pofs = ok ? (size_t)page * page_bytes : 0;
            const uint32_t nrec = ok ? (uint32_t)page_bytes : 0u;
            rk[h] = page_rsrc(kbase, pofs, nrec);
            rv[h] = page_rsrc(vbase, pofs, nrec);
        }
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            const bool live = !tail || k0 + kb * 16 + n < it.k_end;
#pragma unroll
            for (int s = 0; s < DS; ++s) st.k[kb][s] = load16_at(rk[kb], live ? koff[s] : kOutOfRange);
        }
#pragma unroll
        for (int j = 0; j < VL; ++j) {
            const int row = j * RPL + lane / CH;
            const int h = (j * RPL) >> 4;  // page half of the load's rows: the same across the wave
            const bool live = !tail || k0 + row < it.k_end;
            lds_load16_nt(rv[h], live ? voff[j % VJ] : kOutOfRange, &vs[wave_u][j * 1024]);
        }
    };

    auto compute_step = [&](Step& cur, const char (&vs)[4][SB], int i) {
        // Wait for every outstanding load of this wave, K registers and V
        // slots alike, before the step.  A partial wait that counts the next
        // step's loads as younger (what the compiler emits, and tighter forms
        // of it) has produced stale V on this hardware when direct-to-LDS
        // loads and loads into registers are in flight together, so the
        // kernel does not rely on their relative completion order.  With
        // eight waves per CU streaming, the shallower prefetch this leaves
        // costs about 1% on the decode batch.
        wait_vmem<0>();
        const int32_t k0 = it.k_begin + SK * (wave + 4 * i);
        f32x4 sc[RB][2];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int s = 0; s < DS; ++s) {
                const bf16x8 kf = __builtin_bit_cast(bf16x8, cur.k[kb][s]);
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
                    sc[rb][kb] = mfma16(kf, qf[rb][s], s == 0 ? f32x4{0, 0, 0, 0} : sc[rb][kb]);
            }

        const bool full = k0 >= lo_max && k0 + SK <= hi_min;
        if (!full) {
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) {
                const int32_t lo_r = lo[rb] - (k0 + 4 * grp), hi_r = hi[rb] - (k0 + 4 * grp);
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int c = kb * 16 + e;
                        if (!(c >= lo_r && c < hi_r)) sc[rb][kb][e] = kNegInf;
                    }
            }
        }
        float alpha[RB];
        if (softmax_update<RB, 2>(rg, sc, a.scale_log2, m, l, alpha)) {
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                for (int db = 0; db < DB; ++db) o[rb][db] *= alpha[rb];
        }
        bf16x8 pf[RB];
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) pf[rb] = to_bf16x8(sc[rb][0], sc[rb][1]);
#pragma unroll
        for (int db = 0; db < DB; ++db) {
            const bf16_t* base = reinterpret_cast<const bf16_t*>(&vs[wave][vrd[db]]);
            const bf16x8 vf = cat(lds_read_tr16(base), lds_read_tr16(base + 16 * D));
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) o[rb][db] = mfma16(vf, pf[rb], o[rb][db]);
        }
        asm volatile("" ::: "memory");
    };

    // Two register buffers: step i computes while step i+1 (and then i+2) is in
    // flight.  The steady-state loop always issues both loads, so every path
    // into it has the same loads pending and the compiler waits only for the
    // buffer it is about to use; the last two or three steps are peeled.
    Step sa, sb;
    int i = 0;
    if (my_steps >= 4) {
        load_step(sa, v_slot_a, 0);
        load_step(sb, v_slot_b, 1);
        do {
            compute_step(sa, v_slot_a, i);
            load_step(sa, v_slot_a, i + 2);
            compute_step(sb, v_slot_b, i + 1);
            load_step(sb, v_slot_b, i + 3);
            i += 2;
        } while (i + 3 < my_steps);
    } else {
        if (my_steps > 0) load_step(sa, v_slot_a, 0);
        if (my_steps > 1) load_step(sb, v_slot_b, 1);
    }
    if (i < my_steps) {
        compute_step(sa, v_slot_a, i);
        if (i + 2 < my_steps) load_step(sa, v_slot_a, i + 2);
    }
    if (i + 1 < my_steps) compute_step(sb, v_slot_b, i + 1);
    if (i + 2 < my_steps) compute_step(sa, v_slot_a, i + 2);

    if (page_err && lane == 0) atomicOr(a.err, MSTAR_DEVERR_PAGE_RANGE_BIT);

    // ---- combine the four waves -------------------------------------------------
    float lt[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) lt[rb] = rg.sum(l[rb]);
    __syncthreads();  // every wave is done with its V slots
    if (grp == 0) {
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
            ml_lds[wave][0][rb * 16 + n] = m[rb];
            ml_lds[wave][1][rb * 16 + n] = lt[rb];
        }
    }
    __syncthreads();
    float* obuf = reinterpret_cast<float*>(&v_slot_a[0][0]);
    float scale_own[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        const int row = rb * 16 + n;
        float mstar = kNegInf;
#pragma unroll
        for (int w = 0; w < 4; ++w) mstar = fmaxf(mstar, ml_lds[w][0][row]);
        const float mu = mstar == kNegInf ? 0.0f : mstar;
        float L = 0.0f;
#pragma unroll
        for (int w = 0; w < 4; ++w) L += fast_exp2(ml_lds[w][0][row] - mu) * ml_lds[w][1][row];
        scale_own[rb] = fast_exp2(m[rb] - mu);
        if (wave == 0 && grp == 0) {
            fin_lds[0][row] = mstar;
            fin_lds[1][row] = L;
        }
    }
    for (int w = 0; w < 4; ++w) {
        if (wave == w) {
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                for (int db = 0; db < DB; ++db) {
                    f32x4* dst = reinterpret_cast<f32x4*>(&obuf[(rb * 16 + n) * D + db * 16 + 4 * grp]);
                    const f32x4 val = o[rb][db] * scale_own[rb];
                    *dst = (w == 0) ? val : *dst + val;
                }
        }
        __syncthreads();
    }
    constexpr int NV = RB * 16 * D / 4;  // float4 elements of the combined block
    for (int e = tid; e < NV; e += 256) {
        const int row = e / (D / 4), d4 = (e % (D / 4)) * 4;
        if (row >= it.nrows) continue;
        const float mstar = fin_lds[0][row], L = fin_lds[1][row];
        const float inv = L > 0.0f ? 1.0f / L : 0.0f;
        const float lse = L > 0.0f ? (mstar + __log2f(L)) * kLn2 : kNegInf;
        const f32x4 val = *reinterpret_cast<const f32x4*>(&obuf[row * D + d4]) * inv;
        const int rr = it.row0 + row;
        if (it.part < 0) {
            const int64_t orow = (int64_t)(si.q_start + rr / G) * a.hq + kvh * G + rr % G;
            *reinterpret_cast<bf16x4*>(reinterpret_cast<bf16_t*>(a.out) + orow * D + d4) =
                __builtin_convertvector(val, bf16x4);
            if (d4 == 0) a.lse[orow] = lse;
        } else {
            const int64_t slot = it.part + row;
            *reinterpret_cast<f32x4*>(a.part_o + slot * D + d4) = val;
            if (d4 == 0) a.part_lse[slot] = lse;
        }
    }
}

// ---------------------------------------------------------------------------
// fp32 kernel: one wave per (query row, head); lanes take 64 keys at a time
// for the scores and the head dimension for the weighted value sum.  All
// arithmetic in fp32 with the accurate exp/log.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void f32_kernel(KArgs a) {
    constexpr int E = D / 64;
    __shared__ float q_lds[4][D];
    const WorkItem it = a.items[wg_id()];
    const SeqInfo si = a.seqs[it.seq];
    const int wave = thread_id() >> 6, lane = thread_id() & 63;
    const int r = wave;
    if (r >= it.nrows) return;
    const int i = it.row0 + r;
    int32_t lo, hi;
    row_interval(a, si, it, i, lo, hi);
    const int kvh = it.head / a.group;
    const int32_t* bt_row = a.bt + (int64_t)it.seq * a.bt_stride;
    const float* qg = reinterpret_cast<const float*>(a.q) + ((int64_t)(si.q_start + i) * a.hq + it.head) * D;
    const float* kg = reinterpret_cast<const float*>(a.k);
    const float* vg = reinterpret_cast<const float*>(a.v);
#pragma unroll
    for (int e = 0; e < E; ++e) q_lds[wave][lane + 64 * e] = qg[lane + 64 * e];
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_wave_barrier();

    float m = kNegInf, l = 0.0f, acc[E];
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = 0.0f;
    for (int32_t kb = lo; kb < hi; kb += 64) {
        const int32_t t = kb + lane;
        float s = kNegInf;
        // this lane's key: its V row (page 0 for a bad page, whose key reads as zeros)
        int32_t vrow = 0;
        bool vok = false;
        if (t < hi) {
            const int32_t page = bt_row[t >> 4];
            vok = (uint32_t)page < (uint32_t)a.num_pages;
            vrow = vok ? (page * 16 + (t & 15)) : 0;
            if (vok) {
                const float* kr = kg + (((int64_t)page * 16 + (t & 15)) * a.hkv + kvh) * D;
                float dot = 0.0f;
                for (int d = 0; d < D; d += 4) {
                    const float4 kv = *reinterpret_cast<const float4*>(kr + d);
                    dot = fmaf(q_lds[wave][d], kv.x, dot);
                    dot = fmaf(q_lds[wave][d + 1], kv.y, dot);
                    dot = fmaf(q_lds[wave][d + 2], kv.z, dot);
                    dot = fmaf(q_lds[wave][d + 3], kv.w, dot);
                }
                s = dot * a.sm_scale;
            } else {
                atomicOr(a.err, 1);
                s = 0.0f;  // the key reads as zeros
            }
        }
        float cm = s;
        for (int off = 32; off > 0; off >>= 1) cm = fmaxf(cm, __shfl_xor(cm, off, 64));
        const float m_new = fmaxf(m, cm);
        const float alpha = m == kNegInf ? 0.0f : expf(m - m_new);
        const float p = t < hi ? expf(s - m_new) : 0.0f;
        float ps = p;
        for (int off = 32; off > 0; off >>= 1) ps += __shfl_xor(ps, off, 64);
        l = l * alpha + ps;
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] *= alpha;
        // weighted V rows: key j's probability and row come from lane j (a
        // bad page's key contributes its probability to l and zeros to acc)
        // (lanes past the last key hold probability 0 and row 0, so the keys
        // go in groups of eight, whose loads are all in flight together)
        const float pv = vok ? p : 0.0f;
        const int nk = min(64, hi - kb);
        for (int j0 = 0; j0 < nk; j0 += 8) {
            float vv[8][E], pj[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                pj[u] = __shfl(pv, j0 + u, 64);
                const int32_t rj = __shfl(vrow, j0 + u, 64);
                const float* vr = vg + ((int64_t)rj * a.hkv + kvh) * D;
#pragma unroll
                for (int e = 0; e < E; ++e) vv[u][e] = vr[lane + 64 * e];
            }
#pragma unroll
            for (int u = 0; u < 8; ++u)
#pragma unroll
                for (int e = 0; e < E; ++e) acc[e] = fmaf(pj[u], vv[u][e], acc[e]);
        }
        m = m_new;
    }
    const int64_t row = (int64_t)(si.q_start + i) * a.hq + it.head;
    float* out = reinterpret_cast<float*>(a.out) + row * D;
    const float inv = l > 0.0f ? 1.0f / l : 0.0f;
#pragma unroll
    for (int e = 0; e < E; ++e) out[lane + 64 * e] = acc[e] * inv;
    if (lane == 0) a.lse[row] = l > 0.0f ? m + logf(l) : kNegInf;
}

// ---------------------------------------------------------------------------
// Merge kernel: one wave per (row, head); combines the partial results of
// split key ranges (and of a shared prefix, for cascade members) by their
// log-sum-exps (lanes over the head dimension).
// ---------------------------------------------------------------------------
template <int D, bool BF16>
__global__ __launch_bounds__(256) void merge_kernel(MArgs a) {
    constexpr int E = D / 64;
    // one row per wave; the wave index is made scalar so that the item is
    // read with scalar loads
    const int idx = wg_id() * 4 + (__builtin_amdgcn_readfirstlane(thread_id() >> 6) & 3);
    const int lane = thread_id() & 63;
    if (idx >= a.n_items) return;
    const MergeItem mi = a.items[idx];
    // slot set 1: slot0 + s * stride, s < nslots (split key ranges of the row's
    // own keys); slot set 2: pad0 + s * pad1, s < pad2 (the chunks of a shared
    // prefix, for cascade members; empty otherwise)
    auto slot_of = [&](int s) -> int64_t {
        return s < mi.nslots ? mi.slot0 + (int64_t)s * mi.stride : mi.pad0 + (int64_t)(s - mi.nslots) * mi.pad1;
    };
    const int n = mi.nslots + mi.pad2;
    // The rows of the first four slots are requested together with the LSEs
    // (their addresses need only the item), so a row with few slots waits for
    // one round trip to memory instead of three.
    float v0[4][E];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int64_t slot = slot_of(u < n ? u : 0);
#pragma unroll
        for (int e = 0; e < E; ++e) v0[u][e] = u < n ? a.part_o[slot * D + lane + 64 * e] : 0.0f;
    }
    // the slots' LSEs are read across the lanes, 64 at a time, and reduced
    // over the wave (a fixed order: the result does not depend on timing)
    float mstar = kNegInf, x0 = kNegInf;
    for (int s0 = 0; s0 < n; s0 += 64) {
        float x = s0 + lane < n ? a.part_lse[slot_of(s0 + lane)] : kNegInf;
        if (s0 == 0) x0 = x;
        for (int off = 32; off > 0; off >>= 1) x = fmaxf(x, __shfl_xor(x, off, 64));
        mstar = fmaxf(mstar, x);
    }
    float acc[E], tot = 0.0f;
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = 0.0f;
    if (mstar != kNegInf) {
        for (int s0 = 0; s0 < n; s0 += 64) {
            const int cnt = min(64, n - s0);
            // lane j holds the weight of slot s0 + j (the first 64 LSEs are
            // still in registers)
            const float xl = s0 == 0 ? x0 : (lane < cnt ? a.part_lse[slot_of(s0 + lane)] : kNegInf);
            float w = lane < cnt ? expf(xl - mstar) : 0.0f;
            float ws = w;
            for (int off = 32; off > 0; off >>= 1) ws += __shfl_xor(ws, off, 64);
            tot += ws;
            // slots in order; four rows loaded together
            int j = 0;
            if (s0 == 0) {
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const float wj = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(w), u));
#pragma unroll
                    for (int e = 0; e < E; ++e)
                        if (u < cnt) acc[e] = fmaf(wj, v0[u][e], acc[e]);
                }
                j = 4;
            }
            for (; j + 4 <= cnt; j += 4) {
                float v[4][E];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int64_t slot = slot_of(s0 + j + u);
#pragma unroll
                    for (int e = 0; e < E; ++e) v[u][e] = a.part_o[slot * D + lane + 64 * e];
                }
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const float wj = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(w), j + u));
#pragma unroll
                    for (int e = 0; e < E; ++e) acc[e] = fmaf(wj, v[u][e], acc[e]);
                }
            }
            for (; j < cnt; ++j) {
                const int64_t slot = slot_of(s0 + j);
                const float wj = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(w), j));
#pragma unroll
                for (int e = 0; e < E; ++e) acc[e] = fmaf(wj, a.part_o[slot * D + lane + 64 * e], acc[e]);
            }
        }
    }
    const float inv = tot > 0.0f ? 1.0f / tot : 0.0f;
    const int64_t row = (int64_t)mi.row * a.hq + mi.head;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const float v = acc[e] * inv;
        if (BF16)
            reinterpret_cast<bf16_t*>(a.out)[row * D + lane + 64 * e] = (bf16_t)v;
        else
            reinterpret_cast<float*>(a.out)[row * D + lane + 64 * e] = v;
    }
    if (lane == 0) a.lse[row] = tot > 0.0f ? mstar + logf(tot) : kNegInf;
}

// ---------------------------------------------------------------------------
// KV append: one workgroup per item of up to 16 new rows of one request; wave
// w copies rows w, w + 4, ...  A row is one token's keys (or values) for
// every KV head, contiguous in both the packed input and the page slot, so
// lanes copy it in 16-byte pieces.  A target page outside the pool is
// skipped and sets the error word.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void append_kernel(AArgs a) {
    const WorkItem it = a.items[wg_id()];
    const SeqInfo si = a.seqs[it.seq];
    const int wave = __builtin_amdgcn_readfirstlane(thread_id() >> 6) & 3, lane = thread_id() & 63;
    const int chunks = a.row_bytes >> 4;
    const int32_t* bt_row = a.bt + (int64_t)it.seq * a.bt_stride;
    bool bad = false;
    for (int r = wave; r < it.nrows; r += 4) {
        const int32_t i = it.row0 + r;                 // new row within the request
        const int32_t pos = si.kv_len - si.q_len + i;  // its position in the cache
        const int32_t page = bt_row[pos >> 4];
        if ((uint32_t)page >= (uint32_t)a.num_pages) {
            bad = true;
            continue;
        }
        const int64_t src = (int64_t)(si.q_start + i) * a.row_bytes;
        const int64_t dst = ((int64_t)page * 16 + (pos & 15)) * a.row_bytes;
        const uint4* ks = reinterpret_cast<const uint4*>(static_cast<const char*>(a.k_new) + src);
        const uint4* vs = reinterpret_cast<const uint4*>(static_cast<const char*>(a.v_new) + src);
        uint4* kd = reinterpret_cast<uint4*>(static_cast<char*>(a.k) + dst);
        uint4* vd = reinterpret_cast<uint4*>(static_cast<char*>(a.v) + dst);
        for (int c = lane; c < chunks; c += 64) {
            const uint4 kx = ks[c], vx = vs[c];
            kd[c] = kx;
            vd[c] = vx;
        }
    }
    if (bad && lane == 0) atomicOr(a.err, MSTAR_DEVERR_PAGE_RANGE_BIT);
}

}  // namespace

hipError_t launch_append(const AArgs& a, hipStream_t s) {
    if (a.n_items == 0) return hipSuccess;
    hipLaunchKernelGGL(append_kernel, dim3(a.n_items), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_tiles(const KArgs& a, int head_dim, hipStream_t s) {
    if (a.n_items == 0) return hipSuccess;
    const dim3 g((unsigned)a.n_wgs), b(256);
    // both pools within the range of one buffer resource
    const uint64_t pool_bytes = (uint64_t)a.num_pages * 16 * a.hkv * head_dim * 2;
    const bool small = pool_bytes <= kSmallPoolBytes;
    if (head_dim == 64) {
        if (small) hipLaunchKernelGGL((tile_kernel<64, 2, true, false, 64>), g, b, 0, s, a);
        else hipLaunchKernelGGL((tile_kernel<64, 2, false, false, 64>), g, b, 0, s, a);
    } else {
        if (small) hipLaunchKernelGGL((tile_kernel<128, 2, true, false, kTileKeysD128>), g, b, 0, s, a);
        else hipLaunchKernelGGL((tile_kernel<128, 2, false, false, kTileKeysD128>), g, b, 0, s, a);
    }
    return hipGetLastError();
}

hipError_t launch_cascade(const KArgs& a, int head_dim, hipStream_t s) {
    if (a.n_items == 0) return hipSuccess;
    const dim3 g((unsigned)a.n_wgs), b(256);
    const uint64_t pool_bytes = (uint64_t)a.num_pages * 16 * a.hkv * head_dim * 2;
    const bool small = pool_bytes <= kSmallPoolBytes;
    if (head_dim == 64) {
        if (small) hipLaunchKernelGGL((tile_kernel<64, 2, true, true, 64>), g, b, 0, s, a);
        else hipLaunchKernelGGL((tile_kernel<64, 2, false, true, 64>), g, b, 0, s, a);
    } else {
        if (small) hipLaunchKernelGGL((tile_kernel<128, 2, true, true, kTileKeysD128>), g, b, 0, s, a);
        else hipLaunchKernelGGL((tile_kernel<128, 2, false, true, kTileKeysD128>), g, b, 0, s, a);
    }
    return hipGetLastError();
}

hipError_t launch_few(const KArgs& a, int head_dim, int rb, hipStream_t s) {
    if (a.n_items == 0) return hipSuccess;
    const dim3 g(a.n_items), b(256);
    if (head_dim == 64) {
        if (rb == 1) hipLaunchKernelGGL((few_kernel<64, 1>), g, b, 0, s, a);
        else if (rb == 2) hipLaunchKernelGGL((few_kernel<64, 2>), g, b, 0, s, a);
        else hipLaunchKernelGGL((few_kernel<64, 4>), g, b, 0, s, a);
    } else {  // the planner gives d = 128 units at most 32 rows
        if (rb == 1) hipLaunchKernelGGL((few_kernel<128, 1>), g, b, 0, s, a);
        else hipLaunchKernelGGL((few_kernel<128, 2>), g, b, 0, s, a);
    }
    return hipGetLastError();
}

hipError_t launch_f32(const KArgs& a, int head_dim, hipStream_t s) {
    if (a.n_items == 0) return hipSuccess;
    if (head_dim == 64)
        hipLaunchKernelGGL(f32_kernel<64>, dim3(a.n_items), dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL(f32_kernel<128>, dim3(a.n_items), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t scratch_buffer(void** ptr) {
    // the array's device address, looked up once per device with that device
    // current (each GPU holds its own copy at its own address)
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static void* addr[kMaxDevices] = {};
    *ptr = nullptr;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(mu);
    if (!addr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        addr[dev] = p;
    }
    *ptr = addr[dev];
    return hipSuccess;
}

hipError_t launch_merge(const MArgs& a, int head_dim, bool bf16_out, hipStream_t s) {
    if (a.n_items == 0) return hipSuccess;
    const dim3 g((a.n_items + 3) / 4), b(256);
    if (head_dim == 64) {
        if (bf16_out) hipLaunchKernelGGL((merge_kernel<64, true>), g, b, 0, s, a);
        else hipLaunchKernelGGL((merge_kernel<64, false>), g, b, 0, s, a);
    } else {
        if (bf16_out) hipLaunchKernelGGL((merge_kernel<128, true>), g, b, 0, s, a);
        else hipLaunchKernelGGL((merge_kernel<128, false>), g, b, 0, s, a);
    }
    return hipGetLastError();
}

}  // namespace mstar
