// Host planner for batched paged attention with per-request segment masks.
//
// The paper's workers build the attention plan for the next batch on a side
// thread while the current batch runs, and name plan construction as the
// heaviest CPU overhead of a step (Sec. 3.3, Runtime).  This planner therefore
// reads only descriptors (never tensor data), is re-entrant, and does work
// linear in the number of query rows.
//
// Steps:
//  1. validate descriptors;
//  2. turn each request's segments + window into one visible key interval
//     [lo, hi) per query row (block ids never decrease along a request, so a
//     row sees every key up to the end of its own block, and a window only
//     cuts keys off from below);
//  3. cut the batch into work items: few-row items (decode-like requests whose
//     query rows times grouped heads fit one 64-row item, at most 32 rows per
//     item at head_dim 128; all query heads of a KV head share one stream of
//     K/V) and 128-row tiles of one query head for everything else; with
//     shared-prefix groups (a cascade), the prefix of each group is cut into
//     128-row items over the decode-like members' (row, head) list and the
//     members' own items start at the prefix end;
//  4. split key ranges into chunks when there are too few items to fill the
//     GPU (partials are merged by their log-sum-exps afterwards);
//  5. order every list longest first so that the hardware dispatcher, which
//     starts workgroups in order as slots free up, ends with short items;
//  6. lay out the multi-row workgroups (tiles, cascade items) so that the
//     readers of one request's pages for one KV head share an XCD and its L2;
//  7. the KV-append items: the step's new rows of each request, 16 per item.
#include "planner.h"

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdio>

// Few-row key pieces are sized to total_keys / MSTAR_FEW_TARGET_ITEMS (at least
// 256 keys): one round of the 512 workgroup slots of 256 CUs, plus one shorter
// remainder per unit.  Every split item costs an fp32 partial write and
// read-back in the merge kernel, so fewer is better once the GPU is full
// (measured on the decode batch: 512 beats 1024 and 2048).
#ifndef MSTAR_FEW_TARGET_ITEMS
#define MSTAR_FEW_TARGET_ITEMS 512
#endif
// Cascade items: the shared prefix is cut into chunks until the items reach
// about this many workgroups.  Every chunk adds an fp32 partial per member row
// to write and merge (shared-prefix decode: 256 beat 128, 512 and 1024).
#ifndef MSTAR_CASCADE_TARGET_WGS
#define MSTAR_CASCADE_TARGET_WGS 256
#endif

namespace mstar {
namespace {

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// The visible interval [lo(i), hi(i)) of every query row of one request: hi
// as stored in the plan's row_hi, lo from the window (a row at key position p
// sees keys from p - window + 1 on; from 0 without a window).
struct RowIntervals {
    const int32_t* hi_ = nullptr;
    int64_t p0 = 0;  // key position of query row 0: kv_len - q_len
    int32_t window = 0;

    int32_t hi(int32_t i) const { return hi_[i]; }
    int32_t lo(int32_t i) const { return window > 0 ? (int32_t)std::max<int64_t>(0, p0 + i - window + 1) : 0; }

    // Visible (row, key) pairs of rows [r0, r1) inside keys [kb, ke): the sum
    // over rows of max(0, min(hi, ke) - max(lo, kb)).  Items hold at most 128
    // rows, so the direct sum is cheap.
    int64_t pairs(int32_t r0, int32_t r1, int32_t kb, int32_t ke) const {
        if (r1 <= r0 || ke <= kb) return 0;
        // hi and lo never decrease from one row to the next: when the first row
        // reaches ke and the last starts at or below kb, every row sees [kb, ke)
        if (hi_[r0] >= ke && lo(r1 - 1) <= kb) return (int64_t)(r1 - r0) * (ke - kb);
        int64_t n = 0;
        if (window <= 0) {  // lo = 0 <= kb
            for (int32_t i = r0; i < r1; ++i) n += std::max(0, std::min(hi_[i], ke) - kb);
        } else {
            for (int32_t i = r0; i < r1; ++i) n += std::max(0, std::min(hi_[i], ke) - std::max(lo(i), kb));
        }
        return n;
    }
};

// Writes hi of every query row of one request to hi_out[0, q_len) and the
// request's visible (row, key) pairs to pairs.  Returns false (with a
// message) if the segments do not tile [0, kv_len) in order.
bool row_intervals(const mstar_seq_desc& s, const mstar_mask_spec& m, const mstar_segment* segs, int32_t* hi_out,
                   int64_t& pairs, std::string& err) {
    // validate the tiling first
    int64_t pos = 0;
    for (int32_t k = 0; k < m.seg_count; ++k) {
        const mstar_segment& g = segs[m.seg_begin + k];
        if (g.start != pos || g.len < 0) {
            err = "segments must tile [0, kv_len) in order";
            return false;
        }
        if (g.kind != MSTAR_SEG_CAUSAL && g.kind != MSTAR_SEG_FULL && g.kind != MSTAR_SEG_BLOCKS) {
            err = "unknown segment kind";
            return false;
        }
        if (g.kind == MSTAR_SEG_BLOCKS && g.block <= 0) {
            err = "BLOCKS segment needs block > 0";
            return false;
        }
        pos += g.len;
    }
    if (pos != s.kv_len) {
        err = "segments must tile [0, kv_len) in order";
        return false;
    }
    // Rows come in runs over which hi is constant (a FULL segment, one block
    // of a BLOCKS segment) or grows by one per row (CAUSAL): each run is
    // filled in one pass and its pair count summed in closed form.
    pairs = 0;
    const int64_t p0 = (int64_t)s.kv_len - s.q_len;  // key position of query row 0
    const int64_t W = m.window;
    // sum over positions p in [pa, pb) of lo(p) = max(0, p - W + 1) (0 without a window)
    auto lo_sum = [&](int64_t pa, int64_t pb) -> int64_t {
        if (W <= 0) return 0;
        const int64_t a = std::max(pa, W - 1);
        if (a >= pb) return 0;
        const int64_t first = a - W + 1, last = pb - W;  // lo of positions a and pb - 1
        return (first + last) * (pb - a) / 2;
    };
    int32_t k = 0;
    int32_t i = 0;
    while (i < s.q_len) {
        const int64_t p = p0 + i;
        while ((int64_t)segs[m.seg_begin + k].start + segs[m.seg_begin + k].len <= p) ++k;  // segment holding p
        const mstar_segment& g = segs[m.seg_begin + k];
        const int64_t seg_end = (int64_t)g.start + g.len;
        int64_t run_end = seg_end;  // position after the run
        if (g.kind == MSTAR_SEG_BLOCKS)
            run_end = std::min<int64_t>(g.start + ((p - g.start) / g.block + 1) * (int64_t)g.block, seg_end);
        const int32_t n = (int32_t)std::min<int64_t>(run_end - p, (int64_t)s.q_len - i);
        if (g.kind == MSTAR_SEG_CAUSAL) {
            for (int32_t r = 0; r < n; ++r) hi_out[i + r] = (int32_t)(p + 1 + r);  // hi = p + 1
            pairs += (2 * (p + 1) + n - 1) * n / 2;
        } else {
            std::fill(hi_out + i, hi_out + i + n, (int32_t)run_end);  // the end of the block or segment
            pairs += run_end * n;
        }
        pairs -= lo_sum(p, p + n);
        i += n;
    }
    return true;
}

int32_t align_down16(int32_t x) { return x & ~(kPage - 1); }

struct Unit {  // a few-row unit or a tile before key splitting
    int32_t seq, head, row0, nrows, k_begin, k_end;
    int64_t cost;
    bool partial = false;  // write partials even when the key range is not split (cascade members)
};

}  // namespace

int build_host_plan(const mstar_attn_params* params, const mstar_seq_desc* seqs,
                    const mstar_mask_spec* masks, int32_t num_seqs, const mstar_segment* segs,
                    int32_t num_segs, HostPlan& plan, std::string& err, const mstar_prefix_group* groups,
                    int32_t num_groups, const int32_t* members, int32_t num_members) {
    if (!params) { err = "params is NULL"; return MSTAR_ERR_INVALID_ARG; }
    if (num_seqs < 0 || num_segs < 0) { err = "negative count"; return MSTAR_ERR_INVALID_ARG; }
    if (num_seqs > 0 && (!seqs || !masks)) { err = "seqs/masks is NULL"; return MSTAR_ERR_INVALID_ARG; }
    if (num_segs > 0 && !segs) { err = "segments is NULL"; return MSTAR_ERR_INVALID_ARG; }
    const mstar_attn_params& P = *params;
    if (P.num_qo_heads <= 0 || P.num_kv_heads <= 0 || P.num_qo_heads % P.num_kv_heads != 0) {
        err = "num_qo_heads must be a positive multiple of num_kv_heads";
        return MSTAR_ERR_INVALID_ARG;
    }
    if (P.head_dim != 64 && P.head_dim != 128) { err = "head_dim must be 64 or 128"; return MSTAR_ERR_UNSUPPORTED; }
    if (P.page_size != kPage) { err = "page_size must be 16"; return MSTAR_ERR_UNSUPPORTED; }
    if (P.dtype != MSTAR_DTYPE_F32 && P.dtype != MSTAR_DTYPE_BF16) { err = "dtype must be F32 or BF16"; return MSTAR_ERR_UNSUPPORTED; }
    if (P.max_blocks_per_seq <= 0 || P.num_pages <= 0) {
        err = "max_blocks_per_seq and num_pages must be positive";
        return MSTAR_ERR_INVALID_ARG;
    }
    if (!std::isfinite(P.sm_scale) || !(P.sm_scale > 0.0f)) {
        err = "sm_scale must be finite and positive";
        return MSTAR_ERR_INVALID_ARG;
    }
    if ((P.flags & MSTAR_FLAG_FORCE_SPLIT) && (P.flags & MSTAR_FLAG_NO_SPLIT)) {
        err = "FORCE_SPLIT and NO_SPLIT are exclusive";
        return MSTAR_ERR_INVALID_ARG;
    }
    if (P.flags & ~(MSTAR_FLAG_FORCE_SPLIT | MSTAR_FLAG_NO_SPLIT | MSTAR_FLAG_CASCADE_ALL | MSTAR_FLAG_SERIAL)) {
        err = "unknown flag";
        return MSTAR_ERR_INVALID_ARG;
    }

    plan.reset();
    plan.params = P;
    plan.num_seqs = num_seqs;
    const int32_t G = P.num_qo_heads / P.num_kv_heads;
    plan.group = G;
    const int64_t max_kv = (int64_t)P.max_blocks_per_seq * kPage;

    // ---- 1. validate requests, 2. row intervals --------------------------
    std::vector<std::pair<int64_t, int64_t>> ranges;
    int64_t total_q = 0;
    for (int32_t r = 0; r < num_seqs; ++r) {
        const mstar_seq_desc& s = seqs[r];
        const mstar_mask_spec& m = masks[r];
        char buf[160];
        if (s.q_len < 0 || s.kv_len < s.q_len || s.q_start < 0) {
            snprintf(buf, sizeof buf, "request %d: need 0 <= q_len <= kv_len and q_start >= 0", r);
            err = buf;
            return MSTAR_ERR_INVALID_ARG;
        }
        if (s.kv_len > max_kv) {
            snprintf(buf, sizeof buf, "request %d: kv_len exceeds 16 * max_blocks_per_seq", r);
            err = buf;
            return MSTAR_ERR_INVALID_ARG;
        }
        if (m.window < 0 || m.seg_begin < 0 || m.seg_count < 0 || (int64_t)m.seg_begin + m.seg_count > num_segs) {
            snprintf(buf, sizeof buf, "request %d: bad mask spec (window < 0 or segment range)", r);
            err = buf;
            return MSTAR_ERR_INVALID_ARG;
        }
        if ((int64_t)s.q_start + s.q_len > INT32_MAX / P.num_qo_heads) {
            snprintf(buf, sizeof buf, "request %d: too many query rows", r);
            err = buf;
            return MSTAR_ERR_INVALID_ARG;
        }
        if (s.q_len > 0) ranges.push_back({s.q_start, (int64_t)s.q_start + s.q_len});
        total_q = std::max<int64_t>(total_q, (int64_t)s.q_start + s.q_len);
    }
    std::sort(ranges.begin(), ranges.end());
    for (size_t i = 1; i < ranges.size(); ++i) {
        if (ranges[i].first < ranges[i - 1].second) {
            err = "query row ranges of two requests overlap";
            return MSTAR_ERR_INVALID_ARG;
        }
    }
    plan.total_q = (int32_t)total_q;

    // every request's rows (disjoint ranges below INT32_MAX / Hq): hi goes
    // straight into row_hi, whose capacity is fixed here so the views stay valid
    std::vector<RowIntervals> iv(num_seqs);
    plan.seqs.resize(num_seqs);
    {
        int64_t rows = 0;
        for (int32_t r = 0; r < num_seqs; ++r) rows += seqs[r].q_len;
        plan.row_hi.reserve((size_t)rows + 8);
        plan.appends.reserve((size_t)(rows / kAppendRows + num_seqs));
    }
    plan.key_lo.assign(num_seqs, 0);
    plan.key_hi.assign(num_seqs, 0);
    for (int32_t r = 0; r < num_seqs; ++r) {
        const mstar_seq_desc& s = seqs[r];
        SeqInfo& si = plan.seqs[r];
        si.q_len = s.q_len;
        si.kv_len = s.kv_len;
        si.q_start = s.q_start;
        si.window = masks[r].window;
        si.hi_off = (int32_t)plan.row_hi.size();
        si.seq_index = r;
        si.pad0 = si.pad1 = 0;
        plan.row_hi.resize(plan.row_hi.size() + s.q_len);
        int32_t* hi = plan.row_hi.data() + si.hi_off;
        int64_t pairs = 0;
        std::string e2;
        if (!row_intervals(s, masks[r], segs, hi, pairs, e2)) {
            char buf[48];
            snprintf(buf, sizeof buf, "request %d: ", r);
            err = buf + e2;
            return MSTAR_ERR_INVALID_ARG;
        }
        iv[r] = RowIntervals{hi, (int64_t)s.kv_len - s.q_len, masks[r].window};
        plan.visible_pairs += pairs;
        if (s.q_len > 0) {
            plan.key_lo[r] = iv[r].lo(0);
            plan.key_hi[r] = iv[r].hi(s.q_len - 1);
        }
    }
    plan.visible_pairs *= P.num_qo_heads;
    while (plan.row_hi.size() % 8) plan.row_hi.push_back(0);

    // ---- shared-prefix groups (cascade) ------------------------------------
    // group_of[r]: the group of request r or -1; member_rows[r]: query rows of
    // the group's members before r (its rows start there in the group's list)
    std::vector<int32_t> group_of(num_seqs, -1);
    std::vector<int64_t> member_rows(num_seqs, 0);
    std::vector<int64_t> group_rows(std::max(num_groups, 0), 0);
    std::vector<std::vector<int32_t>> joined(std::max(num_groups, 0));  // members in the cascade
    std::vector<char> listed(num_seqs, 0);
    if (num_groups < 0 || num_members < 0) { err = "negative group count"; return MSTAR_ERR_INVALID_ARG; }
    if ((num_groups > 0 && !groups) || (num_members > 0 && !members)) {
        err = "groups/members is NULL";
        return MSTAR_ERR_INVALID_ARG;
    }
    if (num_groups > 0 && P.dtype == MSTAR_DTYPE_F32) { err = "prefix groups need the bf16 dtype"; return MSTAR_ERR_UNSUPPORTED; }
    for (int32_t g = 0; g < num_groups; ++g) {
        const mstar_prefix_group& gr = groups[g];
        char buf[160];
        if (gr.member_count < 1 || gr.member_begin < 0 || (int64_t)gr.member_begin + gr.member_count > num_members ||
            gr.prefix_len <= 0 || gr.prefix_len % kPage != 0) {
            snprintf(buf, sizeof buf, "prefix group %d: bad member range or prefix_len (a positive multiple of 16)", g);
            err = buf;
            return MSTAR_ERR_INVALID_ARG;
        }
        for (int32_t k = 0; k < gr.member_count; ++k) {
            const int32_t r = members[gr.member_begin + k];
            if (r < 0 || r >= num_seqs || listed[r]) {
                snprintf(buf, sizeof buf, "prefix group %d: member %d out of range or in two groups", g, r);
                err = buf;
                return MSTAR_ERR_INVALID_ARG;
            }
            listed[r] = 1;
            const mstar_seq_desc& s = seqs[r];
            // intervals never shrink from one row to the next: the first row
            // decides hi >= prefix_len, the last one lo == 0
            if (s.kv_len < gr.prefix_len ||
                (s.q_len > 0 && (iv[r].hi(0) < gr.prefix_len || iv[r].lo(s.q_len - 1) != 0))) {
                snprintf(buf, sizeof buf, "prefix group %d: a query row of request %d does not see the whole prefix",
                         g, r);
                err = buf;
                return MSTAR_ERR_INVALID_ARG;
            }
            // a member whose rows fill tiles already reads each prefix tile
            // once per 128 rows: the cascade would only add the merge
            if (!(P.flags & MSTAR_FLAG_CASCADE_ALL) && (int64_t)s.q_len * G > kDecodeMaxRows) continue;
            group_of[r] = g;
            member_rows[r] = group_rows[g];
            group_rows[g] += s.q_len;
            joined[g].push_back(r);
        }
    }

    // ---- 3. work units ----------------------------------------------------
    std::vector<Unit> few_units, tile_units;
    // (request, first row, rows) of member row tiles whose rows see no key past
    // the shared prefix: their outputs come from the prefix partials alone
    struct RowRun { int32_t seq, row0, nrows; };
    std::vector<RowRun> prefix_only;
    for (int32_t r = 0; r < num_seqs; ++r) {
        const mstar_seq_desc& s = seqs[r];
        if (s.q_len == 0) continue;
        const RowIntervals& v = iv[r];
        if (P.dtype == MSTAR_DTYPE_F32) {
            for (int32_t h = 0; h < P.num_qo_heads; ++h) {
                for (int32_t row0 = 0; row0 < s.q_len; row0 += kF32Rows) {
                    const int32_t nr = std::min(kF32Rows, s.q_len - row0);
                    WorkItem w{r, h, row0, nr, align_down16(v.lo(row0)), v.hi(row0 + nr - 1), -1, -1};
                    plan.f32.push_back(w);
                }
            }
            continue;
        }
        const int64_t R = (int64_t)s.q_len * G;
        // a cascade member's own work covers the keys after the shared prefix
        const bool member = group_of[r] >= 0;
        const int32_t own0 = member ? groups[group_of[r]].prefix_len : 0;
        if (member && v.hi(s.q_len - 1) <= own0) continue;  // the prefix is all it sees
        if (R <= kDecodeMaxRows) {
            // at d = 128 a unit holds at most 32 rows: the 64-row instance of
            // the few-row kernel does not fit its registers
            const int32_t span = P.head_dim == 128 ? 32 : kDecodeMaxRows;
            for (int32_t kvh = 0; kvh < P.num_kv_heads; ++kvh) {
                for (int32_t rr0 = 0; rr0 < R; rr0 += span) {
                    const int32_t nr = std::min<int32_t>(span, (int32_t)R - rr0);
                    const int32_t q0 = rr0 / G, q1 = (rr0 + nr - 1) / G;
                    Unit u{r, kvh, rr0, nr, member ? own0 : align_down16(v.lo(q0)), v.hi(q1), 0};
                    // a member unit whose rows see only the prefix keeps an
                    // empty own range (it writes empty partials for the merge)
                    u.k_end = std::max(u.k_end, u.k_begin);
                    u.cost = (int64_t)(u.k_end - u.k_begin);
                    u.partial = member;
                    few_units.push_back(u);
                    plan.decode_rb = std::max<int32_t>(plan.decode_rb, nr <= 16 ? 1 : nr <= 32 ? 2 : 4);
                }
            }
        } else {
            // one unit per row tile, shared by every query head
            for (int32_t row0 = 0; row0 < s.q_len; row0 += kTileRows) {
                const int32_t nr = std::min(kTileRows, s.q_len - row0);
                const int32_t kb = member ? own0 : align_down16(v.lo(row0));
                const int32_t ke = v.hi(row0 + nr - 1);
                if (ke <= kb) {  // rows that see only the prefix (members only: kb = 0 otherwise)
                    if (member) prefix_only.push_back({r, row0, nr});
                    continue;
                }
                Unit u{r, -1, row0, nr, kb, ke, 0};
                u.partial = member;
                tile_units.push_back(u);
            }
        }
    }

    // KV append items: the new rows of each request in chunks of kAppendRows
    {
        size_t n_app = 0;
        for (int32_t r = 0; r < num_seqs; ++r) n_app += (size_t)ceil_div(seqs[r].q_len, kAppendRows);
        plan.appends.resize(n_app);
        WorkItem* w = plan.appends.data();
        for (int32_t r = 0; r < num_seqs; ++r) {
            const mstar_seq_desc& s = seqs[r];
            const int32_t p0 = s.kv_len - s.q_len;
            for (int32_t row0 = 0; row0 < s.q_len; row0 += kAppendRows) {
                const int32_t nr = std::min(kAppendRows, s.q_len - row0);
                *w++ = WorkItem{r, -1, row0, nr, p0 + row0, p0 + row0 + nr, -1, -1};
            }
        }
    }

    // ---- 4. key splitting ---------------------------------------------------
    int64_t slot = 0;
    // Cascade: per (group, KV head) a row list of (member, query row, query
    // head) in member order, cut into 128-row items over the prefix keys, the
    // prefix cut into equal chunks when the items alone cannot fill the GPU.
    // The partial of chunk c, list row j sits at slot base + c * R + j.
    struct CascSlots { int64_t base = 0, rows = 0, chunks = 1; };
    std::vector<CascSlots> casc((size_t)std::max(num_groups, 0) * P.num_kv_heads);
    if (num_groups > 0) {
        int64_t tiles = 0;
        for (int32_t g = 0; g < num_groups; ++g) tiles += ceil_div(group_rows[g] * G, kTileRows) * P.num_kv_heads;
        for (int32_t g = 0; g < num_groups; ++g) {
            const mstar_prefix_group& gr = groups[g];
            const int64_t R = group_rows[g] * G;
            if (R == 0) continue;  // no member joined, or none has a query row
            int64_t nch = 1;
            if (!(P.flags & MSTAR_FLAG_NO_SPLIT) && tiles > 0 && tiles < MSTAR_CASCADE_TARGET_WGS)
                nch = ceil_div(MSTAR_CASCADE_TARGET_WGS, tiles);
            if (P.flags & MSTAR_FLAG_FORCE_SPLIT) nch = 3;
            nch = std::max<int64_t>(1, std::min<int64_t>(nch, gr.prefix_len / (2 * kTileKeys)));
            const int64_t cs = ceil_div(ceil_div(gr.prefix_len, nch), kTileKeys) * kTileKeys;
            nch = ceil_div(gr.prefix_len, cs);
            for (int32_t kvh = 0; kvh < P.num_kv_heads; ++kvh) {
                CascSlots& cslot = casc[(size_t)g * P.num_kv_heads + kvh];
                cslot.base = slot;
                cslot.rows = R;
                cslot.chunks = nch;
                const int64_t row_off = (int64_t)plan.casc_rows.size() / 2;
                for (const int32_t r : joined[g]) {
                    for (int32_t i = 0; i < seqs[r].q_len; ++i)
                        for (int32_t h = kvh * G; h < (kvh + 1) * G; ++h) {
                            plan.casc_rows.push_back(seqs[r].q_start + i);
                            plan.casc_rows.push_back(h);
                        }
                }
                for (int64_t c = 0; c < nch; ++c)
                    for (int64_t b0 = 0; b0 < R; b0 += kTileRows) {
                        WorkItem w;
                        w.seq = joined[g][0];
                        w.head = kvh;
                        w.row0 = (int32_t)(row_off + b0);
                        w.nrows = (int32_t)std::min<int64_t>(kTileRows, R - b0);
                        w.k_begin = (int32_t)(c * cs);
                        w.k_end = (int32_t)std::min<int64_t>((c + 1) * cs, gr.prefix_len);
                        w.part = (int32_t)(slot + c * R + b0);
                        w.head_stride = -1;
                        plan.cascade.push_back(w);
                    }
                slot += nch * R;
            }
        }
        if (plan.casc_rows.size() / 2 > (size_t)INT32_MAX) { err = "too many cascade rows"; return MSTAR_ERR_INVALID_ARG; }
    }
    // prefix slot set of (request r, its query row i, query head h)
    auto prefix_slots = [&](MergeItem& m, int32_t r, int32_t i, int32_t h) {
        if (group_of[r] < 0) {
            m.pad0 = m.pad1 = m.pad2 = 0;
            return;
        }
        const int32_t kvh = h / G;
        const CascSlots& cslot = casc[(size_t)group_of[r] * P.num_kv_heads + kvh];
        m.pad0 = (int32_t)(cslot.base + (member_rows[r] + i) * G + (h - kvh * G));
        m.pad1 = (int32_t)cslot.rows;
        m.pad2 = (int32_t)cslot.chunks;
    };
    // member rows that see nothing past the prefix (a whole request, or the
    // row tiles of one whose first rows sit inside the prefix's block): the
    // merge reads the prefix partials alone
    auto prefix_only_rows = [&](int32_t r, int32_t i0, int32_t i1) {
        for (int32_t i = i0; i < i1; ++i)
            for (int32_t h = 0; h < P.num_qo_heads; ++h) {
                MergeItem m;
                m.row = seqs[r].q_start + i;
                m.head = h;
                m.slot0 = 0;
                m.stride = 0;
                m.nslots = 0;
                prefix_slots(m, r, i, h);
                plan.merges.push_back(m);
            }
    };
    for (int32_t r = 0; r < num_seqs; ++r) {
        if (group_of[r] < 0 || seqs[r].q_len == 0) continue;
        if (iv[r].hi(seqs[r].q_len - 1) > groups[group_of[r]].prefix_len) continue;
        prefix_only_rows(r, 0, seqs[r].q_len);
    }
    for (const RowRun& run : prefix_only) prefix_only_rows(run.seq, run.row0, run.row0 + run.nrows);
    // Few-row units are cut into pieces of exactly `chunk` keys plus one shorter
    // remainder: with longest-first order the equal pieces fill every CU evenly
    // and the remainders fill the gaps (a simulation of the decode batch on 256
    // CUs sharing HBM bandwidth puts this within ~7% of a perfect split, against
    // ~17% for splitting each unit into equal parts).  Tiles are split into
    // equal parts.
    auto emit = [&](const Unit& u, int32_t chunk, int32_t align, std::vector<WorkItem>& dst, bool few) {
        const int64_t n = (int64_t)u.k_end - u.k_begin;
        int64_t nch = 1, cs = n;
        if (chunk > 0 && n > chunk) {
            if (few) {
                cs = chunk;
            } else {
                nch = ceil_div(n, chunk);
                cs = ceil_div(ceil_div(n, nch), align) * align;
            }
            nch = ceil_div(n, cs);
        }
        // partial slots of a split unit: few-row units [chunk][row]; tile units
        // [query head][chunk][row]
        const int64_t heads = few ? 1 : P.num_qo_heads;
        for (int64_t c = 0; c < nch; ++c) {
            WorkItem w;
            w.seq = u.seq;
            w.head = u.head;
            w.row0 = u.row0;
            w.nrows = u.nrows;
            w.k_begin = (int32_t)(u.k_begin + c * cs);
            w.k_end = (int32_t)std::min<int64_t>(u.k_begin + (c + 1) * cs, u.k_end);
            const bool partial = nch > 1 || u.partial;
            w.part = partial ? (int32_t)(slot + c * u.nrows) : -1;
            w.head_stride = (partial && !few) ? (int32_t)(nch * u.nrows) : -1;
            dst.push_back(w);
        }
        if (nch > 1 || u.partial) {
            const SeqInfo& si = plan.seqs[u.seq];
            for (int64_t h = 0; h < heads; ++h) {
                for (int32_t r = 0; r < u.nrows; ++r) {
                    MergeItem m;
                    const int32_t rr = u.row0 + r;
                    m.row = si.q_start + (few ? rr / G : rr);
                    m.head = few ? u.head * G + rr % G : (int32_t)h;
                    m.slot0 = (int32_t)(slot + h * nch * u.nrows + r);
                    m.stride = u.nrows;
                    m.nslots = (int32_t)nch;
                    prefix_slots(m, u.seq, few ? rr / G : rr, m.head);
                    plan.merges.push_back(m);
                }
            }
            slot += nch * u.nrows * heads;
        }
    };

    {  // few-row units: enough items to keep every CU streaming K/V
        int64_t total = 0, longest = 0;
        for (const Unit& u : few_units) {
            total += u.k_end - u.k_begin;
            longest = std::max<int64_t>(longest, u.k_end - u.k_begin);
        }
        int32_t chunk = 0;
        if (P.flags & MSTAR_FLAG_FORCE_SPLIT) {
            chunk = kSubKeys * 2;
        } else if (!(P.flags & MSTAR_FLAG_NO_SPLIT)) {
            const int64_t target_items = MSTAR_FEW_TARGET_ITEMS;
            int64_t c = std::max<int64_t>(256, ceil_div(total, target_items));
            chunk = (int32_t)std::min<int64_t>(ceil_div(c, 128) * 128, INT32_MAX / 2);
            // Units that already fill every slot and are within a quarter of
            // one piece of each other stay whole: splitting would only add a
            // merge launch (shared-prefix decode without the cascade: 512
            // units of 4.1-5.1k keys, step 129 -> 120 us).
            if ((int64_t)few_units.size() >= target_items && longest * 4 <= (int64_t)chunk * 5) chunk = 0;
        }
        for (const Unit& u : few_units) emit(u, chunk, kSubKeys, plan.few, true);
    }
    {  // multi-row tiles: split only when the tiles alone cannot fill the GPU
        int64_t total = 0;
        for (const Unit& u : tile_units) total += u.k_end - u.k_begin;
        int32_t chunk = 0;
        if (P.flags & MSTAR_FLAG_FORCE_SPLIT) {
            chunk = kTileKeys * 2;
        } else if (!(P.flags & MSTAR_FLAG_NO_SPLIT) && (int64_t)tile_units.size() * P.num_qo_heads < 512 &&
                   !tile_units.empty()) {
            int64_t c = std::max<int64_t>(1024, ceil_div(total, 1024));
            chunk = (int32_t)std::min<int64_t>(ceil_div(c, kTileKeys) * kTileKeys, INT32_MAX / 2);
        }
        for (const Unit& u : tile_units) emit(u, chunk, kTileKeys, plan.tiles, false);
    }
    plan.partial_slots = slot;
    if (slot > INT32_MAX) { err = "too many partial rows"; return MSTAR_ERR_INVALID_ARG; }

    // ---- 5. longest first ------------------------------------------------------
    auto visible_in = [&](const WorkItem& w) -> int64_t {
        return iv[w.seq].pairs(w.row0, w.row0 + w.nrows, w.k_begin, w.k_end);
    };
    // sorts items by decreasing key; `keys` (if given) receives the keys in the new order
    auto lpt = [&](std::vector<WorkItem>& items, bool by_pairs, std::vector<int64_t>* keys) {
        std::vector<std::pair<int64_t, int32_t>> key(items.size());
        for (size_t i = 0; i < items.size(); ++i)
            key[i] = {by_pairs ? visible_in(items[i]) : (int64_t)(items[i].k_end - items[i].k_begin), (int32_t)i};
        // decreasing key, equal keys in their original order (no merge buffer, unlike a stable sort)
        std::sort(key.begin(), key.end(),
                  [](const auto& a, const auto& b) { return a.first != b.first ? a.first > b.first : a.second < b.second; });
        std::vector<WorkItem> sorted(items.size());
        for (size_t i = 0; i < items.size(); ++i) sorted[i] = items[key[i].second];
        std::copy(sorted.begin(), sorted.end(), items.begin());  // items keeps its buffer
        if (keys) {
            keys->resize(key.size());
            for (size_t i = 0; i < key.size(); ++i) (*keys)[i] = key[i].first;
        }
    };
    std::vector<int64_t> tile_pairs;  // visible pairs of each tile item, for the launch order
    lpt(plan.tiles, true, &tile_pairs);
    lpt(plan.few, false, nullptr);
    lpt(plan.f32, true, nullptr);

    // ---- 6. launch order of the multi-row workgroups ----------------------------
    // One workgroup per (tile item, query head); one per cascade item (its rows
    // name their heads; the order entry carries a head of its KV head).  The
    // hardware deals workgroup b to XCD b % 8, and each XCD has its own L2.
    // Every workgroup that reads the same K/V pages -- the items of one
    // request and the G query heads of one KV head -- goes to the same XCD,
    // consecutively, so they run together and read each K/V tile from that
    // L2.  A group costlier than an even share of one XCD is cut into
    // consecutive runs of items (one such group alone would otherwise leave
    // the other XCDs idle).  Groups go to the least-loaded XCD, largest first;
    // inside a group the items keep their order.
    auto launch_order = [&](const std::vector<WorkItem>& items, bool per_head, const std::vector<int64_t>* pairs_of,
                            std::vector<int32_t>& order) {
        // groups in order of first appearance; members flat, by group (a counting sort)
        std::vector<int32_t> gid_of((size_t)num_seqs * P.num_kv_heads, -1);
        std::vector<int32_t> g_kvh, g_count;
        std::vector<int64_t> g_cost, item_cost(items.size());
        int64_t total = 0;
        auto heads_of = [&](const WorkItem& w, int32_t& k0, int32_t& k1) {
            k0 = per_head ? 0 : w.head;
            k1 = per_head ? P.num_kv_heads : w.head + 1;
        };
        for (size_t i = 0; i < items.size(); ++i) {
            const WorkItem& w = items[i];
            const int64_t pairs = per_head ? (*pairs_of)[i] * G : (int64_t)w.nrows * (w.k_end - w.k_begin);
            item_cost[i] = pairs + 1;  // +1: an empty item still costs a workgroup
            int32_t k0, k1;
            heads_of(w, k0, k1);
            for (int32_t kvh = k0; kvh < k1; ++kvh) {
                int32_t& gi = gid_of[(size_t)w.seq * P.num_kv_heads + kvh];
                if (gi < 0) {
                    gi = (int32_t)g_kvh.size();
                    g_kvh.push_back(kvh);
                    g_count.push_back(0);
                    g_cost.push_back(0);
                }
                ++g_count[gi];
                g_cost[gi] += pairs + 1;
                total += pairs + 1;
            }
        }
        const size_t ng = g_kvh.size();
        std::vector<int64_t> g_off(ng + 1, 0);
        for (size_t g = 0; g < ng; ++g) g_off[g + 1] = g_off[g] + g_count[g];
        std::vector<int32_t> members((size_t)g_off[ng]);
        {
            std::vector<int64_t> fill(g_off.begin(), g_off.end() - 1);
            for (size_t i = 0; i < items.size(); ++i) {
                int32_t k0, k1;
                heads_of(items[i], k0, k1);
                for (int32_t kvh = k0; kvh < k1; ++kvh)
                    members[(size_t)fill[gid_of[(size_t)items[i].seq * P.num_kv_heads + kvh]]++] = (int32_t)i;
            }
        }
        // pieces: whole groups, or consecutive runs of a group costlier than an
        // even share of one XCD
        constexpr int kXcds = 8;
        const int64_t share = ceil_div(total, kXcds);
        struct Piece { int64_t cost, begin, end; int32_t kvh; };
        std::vector<Piece> pieces;
        pieces.reserve(ng);
        for (size_t g = 0; g < ng; ++g) {
            if (g_cost[g] <= share) {
                pieces.push_back({g_cost[g], g_off[g], g_off[g + 1], g_kvh[g]});
                continue;
            }
            Piece pc{0, g_off[g], g_off[g], g_kvh[g]};
            for (int64_t k = g_off[g]; k < g_off[g + 1]; ++k) {
                const int64_t c = item_cost[(size_t)members[(size_t)k]];
                if (pc.end > pc.begin && pc.cost + c > share) {
                    pieces.push_back(pc);
                    pc = Piece{0, k, k, g_kvh[g]};
                }
                pc.end = k + 1;
                pc.cost += c;
            }
            pieces.push_back(pc);
        }
        // costliest first, equal costs in creation order (begin grows with it)
        std::sort(pieces.begin(), pieces.end(), [](const Piece& x, const Piece& y) {
            return x.cost != y.cost ? x.cost > y.cost : x.begin < y.begin;
        });
        // each piece to the least-loaded XCD, then workgroup b of XCD x at launch slot 8 b + x
        const int32_t hpi = per_head ? G : 1;  // workgroups per (item, KV head): its query heads, or the item
        std::vector<int8_t> xcd_of(pieces.size());
        int64_t load[kXcds] = {0, 0, 0, 0, 0, 0, 0, 0};
        size_t count[kXcds] = {0, 0, 0, 0, 0, 0, 0, 0};
        for (size_t q = 0; q < pieces.size(); ++q) {
            int x = 0;
            for (int k = 1; k < kXcds; ++k)
                if (load[k] < load[x]) x = k;
            load[x] += pieces[q].cost;
            count[x] += (size_t)(pieces[q].end - pieces[q].begin) * hpi;
            xcd_of[q] = (int8_t)x;
        }
        size_t slots = 0;
        for (int x = 0; x < kXcds; ++x) slots = std::max(slots, count[x]);
        if (slots * kXcds > (size_t)INT32_MAX / 2) return false;
        order.assign(2 * slots * kXcds, -1);  // padding workgroups exit at once
        size_t pos[kXcds] = {0, 0, 0, 0, 0, 0, 0, 0};
        for (size_t q = 0; q < pieces.size(); ++q) {
            const int x = xcd_of[q];
            const int32_t h0 = pieces[q].kvh * G;  // a cascade item's entry names the KV head's first query head
            for (int64_t k = pieces[q].begin; k < pieces[q].end; ++k)
                for (int32_t h = h0; h < h0 + hpi; ++h) {
                    const size_t b = pos[x]++ * kXcds + x;
                    order[2 * b] = members[(size_t)k];
                    order[2 * b + 1] = h;
                }
        }
        return true;
    };
    if (!launch_order(plan.tiles, true, &tile_pairs, plan.tile_order) ||
        !launch_order(plan.cascade, false, nullptr, plan.casc_order)) {
        err = "too many tile workgroups";
        return MSTAR_ERR_INVALID_ARG;
    }
    return MSTAR_OK;
}

}  // namespace mstar
