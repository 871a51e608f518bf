// Seeded random descriptors through the host planner, built with AddressSanitizer
// and UndefinedBehaviorSanitizer by tests/test_host_sanitizers.py (CPU only).
//
//   planner_fuzz <seed> <iterations>
//
// Each iteration draws a batch: head layout, dtype, flags, requests (lengths,
// packed rows), segment lists, windows and shared-prefix groups.  Most draws
// are valid; the rest break one rule (a gap between segments, a bad kind or
// block, q_len > kv_len, overlapping rows, a window < 0, a kv_len past the block
// table, a prefix group that is not shared or not seen, an unknown flag, a bad
// scale).  A valid plan must satisfy the invariants checked below; an invalid
// one must be rejected with a message.  Any sanitizer report, failed invariant
// or accepted invalid batch ends the run with a non-zero status.
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <string>
#include <vector>

#include "planner.h"

namespace {

int g_fail = 0;
long g_accepted = 0, g_rejected = 0, g_cascade = 0, g_merged = 0, g_tiles = 0, g_few = 0;

#define CHECK(cond, ...)                                              \
    do {                                                              \
        if (!(cond)) {                                                \
            std::fprintf(stderr, "iteration %d: check failed: %s: ", it, #cond); \
            std::fprintf(stderr, __VA_ARGS__);                        \
            std::fprintf(stderr, "\n");                               \
            ++g_fail;                                                 \
            return;                                                   \
        }                                                             \
    } while (0)

struct Rng {
    std::mt19937_64 g;
    explicit Rng(uint64_t s) : g(s) {}
    int64_t uni(int64_t lo, int64_t hi) { return std::uniform_int_distribution<int64_t>(lo, hi)(g); }
    bool coin(double p) { return std::uniform_real_distribution<double>(0, 1)(g) < p; }
};

void one(Rng& R, int it) {
    mstar_attn_params P{};
    const int divs[] = {1, 2, 4, 7, 8};
    P.num_kv_heads = (int32_t)R.uni(1, 8);
    P.num_qo_heads = P.num_kv_heads * divs[R.uni(0, 4)];
    P.head_dim = R.coin(0.5) ? 64 : 128;
    P.page_size = 16;
    P.dtype = R.coin(0.85) ? MSTAR_DTYPE_BF16 : MSTAR_DTYPE_F32;
    P.max_blocks_per_seq = (int32_t)R.uni(1, 700);
    P.num_pages = (int32_t)R.uni(1, 1 << 20);
    P.flags = 0;
    if (R.coin(0.2)) P.flags |= MSTAR_FLAG_FORCE_SPLIT;
    else if (R.coin(0.2)) P.flags |= MSTAR_FLAG_NO_SPLIT;
    if (R.coin(0.3)) P.flags |= MSTAR_FLAG_CASCADE_ALL;
    if (R.coin(0.2)) P.flags |= MSTAR_FLAG_SERIAL;
    P.sm_scale = 1.0f / std::sqrt((float)P.head_dim);

    const int n = (int)R.uni(0, 14);
    std::vector<mstar_seq_desc> seqs(n);
    std::vector<mstar_mask_spec> masks(n);
    std::vector<mstar_segment> segs;
    const int64_t max_kv = (int64_t)P.max_blocks_per_seq * 16;
    int32_t qs = (int32_t)R.uni(0, 5);
    for (int r = 0; r < n; ++r) {
        const int32_t L = (int32_t)R.uni(0, std::min<int64_t>(max_kv, 9000));
        const int32_t q = R.coin(0.3) ? (L > 0 ? 1 : 0) : (int32_t)R.uni(0, std::min<int32_t>(L, 600));
        seqs[r] = {q, L, qs};
        qs += q + (int32_t)R.uni(0, 3);
        masks[r].seg_begin = (int32_t)segs.size();
        int32_t pos = 0;
        int cnt = 0;
        while (pos < L || cnt == 0) {
            const int32_t len = std::min<int32_t>(L - pos, R.coin(0.3) ? L - pos : (int32_t)R.uni(0, L - pos + 1));
            const int kind = (int)R.uni(0, 2);
            segs.push_back({pos, len, kind, kind == MSTAR_SEG_BLOCKS ? (int32_t)R.uni(1, 300) : 0});
            pos += len;
            ++cnt;
            if (L == 0) break;
        }
        masks[r].seg_count = cnt;
        masks[r].window = R.coin(0.6) ? 0 : (int32_t)R.uni(1, 2 * std::max<int32_t>(L, 1));
    }
    // shared-prefix groups: members whose rows all see their first prefix_len keys
    std::vector<mstar_prefix_group> groups;
    std::vector<int32_t> members;
    if (n > 0 && R.coin(0.4)) {
        const int32_t plen = 16 * (int32_t)R.uni(1, 40);
        std::vector<int32_t> mem;
        for (int r = 0; r < n; ++r)
            if (R.coin(0.6)) mem.push_back(r);
        if (!mem.empty()) {
            for (int32_t r : mem) {  // make the prefix a FULL first segment every row sees
                mstar_seq_desc& s = seqs[r];
                if (s.kv_len < plen + 1) s.kv_len = std::min<int32_t>(plen + (int32_t)R.uni(1, 500), (int32_t)max_kv);
                if (s.kv_len <= plen) { s.kv_len = plen; }
                s.q_len = std::min<int32_t>(s.q_len, s.kv_len);
                masks[r].seg_begin = (int32_t)segs.size();
                masks[r].window = 0;
                segs.push_back({0, plen, MSTAR_SEG_FULL, 0});
                if (s.kv_len > plen) {
                    segs.push_back({plen, s.kv_len - plen, MSTAR_SEG_CAUSAL, 0});
                    masks[r].seg_count = 2;
                } else {
                    masks[r].seg_count = 1;
                }
            }
            // re-pack query rows after the length changes
            int32_t q0 = 0;
            for (int r = 0; r < n; ++r) {
                seqs[r].q_start = q0;
                q0 += seqs[r].q_len;
            }
            bool fits = true;
            for (int32_t r : mem) fits &= (int64_t)seqs[r].kv_len <= max_kv && seqs[r].kv_len >= plen;
            if (fits && P.dtype == MSTAR_DTYPE_BF16) {
                groups.push_back({0, (int32_t)mem.size(), plen});
                members = mem;
            }
        }
    }

    // one rule broken in about a quarter of the draws
    bool broken = false;
    if (R.coin(0.25) && n > 0) {
        const int r = (int)R.uni(0, n - 1);
        broken = true;
        switch (R.uni(0, 9)) {
            case 0: seqs[r].q_len = seqs[r].kv_len + 1; break;
            case 1: seqs[r].kv_len = (int32_t)max_kv + 16; break;
            case 2: masks[r].window = -1; break;
            case 3: segs[masks[r].seg_begin].start += 1; break;
            case 4: segs[masks[r].seg_begin].kind = 7; break;
            case 5:
                segs[masks[r].seg_begin].kind = MSTAR_SEG_BLOCKS;
                segs[masks[r].seg_begin].block = 0;
                break;
            case 6: masks[r].seg_count = (int32_t)segs.size() + 3; break;
            case 7:
                if (n > 1 && seqs[0].q_len > 0 && seqs[1].q_len > 0) seqs[1].q_start = seqs[0].q_start;
                else broken = false;
                break;
            case 8: P.flags |= 1u << 20; break;
            default: P.sm_scale = R.coin(0.5) ? -1.0f : NAN; break;
        }
    }
    if (!broken && !groups.empty() && R.coin(0.1)) {
        groups[0].prefix_len += 8;  // not a multiple of 16
        broken = true;
    }

    mstar::HostPlan plan;
    std::string err;
    const int rc = mstar::build_host_plan(&P, seqs.data(), masks.data(), n, segs.data(), (int32_t)segs.size(), plan,
                                          err, groups.data(), (int32_t)groups.size(), members.data(),
                                          (int32_t)members.size());
    if (broken) {
        CHECK(rc != MSTAR_OK, "a batch breaking a rule was accepted");
        CHECK(!err.empty(), "rejection without a message");
        ++g_rejected;
        return;
    }
    if (rc != MSTAR_OK) {
        CHECK(!err.empty(), "rejection without a message (rc %d)", rc);
        ++g_rejected;
        return;
    }
    ++g_accepted;
    g_cascade += !plan.cascade.empty();
    g_merged += !plan.merges.empty();
    g_tiles += !plan.tiles.empty();
    g_few += !plan.few.empty();
    // ---- invariants of an accepted plan
    const int64_t slots = plan.partial_slots;
    auto item_ok = [&](const mstar::WorkItem& w) {
        return w.seq >= 0 && w.seq < n && w.k_begin >= 0 && w.k_begin <= w.k_end && w.k_end <= seqs[w.seq].kv_len &&
               w.nrows > 0 && w.row0 >= 0;
    };
    for (const auto& w : plan.tiles) {
        CHECK(item_ok(w), "tile item seq %d keys [%d, %d)", w.seq, w.k_begin, w.k_end);
        CHECK(w.row0 + w.nrows <= seqs[w.seq].q_len, "tile rows past q_len");
        if (w.part >= 0)
            CHECK((int64_t)w.part + (int64_t)(P.num_qo_heads - 1) * w.head_stride + w.nrows <= slots,
                  "tile partial slots past the workspace");
    }
    const int32_t G = P.num_qo_heads / P.num_kv_heads;
    for (const auto& w : plan.few) {
        CHECK(item_ok(w), "few item seq %d keys [%d, %d)", w.seq, w.k_begin, w.k_end);
        CHECK(w.head >= 0 && w.head < P.num_kv_heads, "few item head");
        CHECK((int64_t)w.row0 + w.nrows <= (int64_t)seqs[w.seq].q_len * G, "few rows past q_len x group");
        if (w.part >= 0) CHECK((int64_t)w.part + w.nrows <= slots, "few partial slots past the workspace");
    }
    for (const auto& w : plan.f32) CHECK(item_ok(w), "f32 item");
    for (size_t i = 0; i + 1 < plan.tile_order.size(); i += 2) {
        const int32_t item = plan.tile_order[i], h = plan.tile_order[i + 1];
        CHECK(item >= -1 && item < (int32_t)plan.tiles.size(), "launch order item %d", item);
        CHECK(item < 0 || (h >= 0 && h < P.num_qo_heads), "launch order head %d", h);
    }
    CHECK(plan.tile_order.size() % 16 == 0, "launch order not a multiple of 8 workgroups");
    for (const auto& m : plan.merges) {
        CHECK(m.row >= 0 && m.row < plan.total_q && m.head >= 0 && m.head < P.num_qo_heads, "merge row/head");
        CHECK(m.nslots >= 0 && m.pad2 >= 0 && m.nslots + m.pad2 > 0, "merge with no slot");
        if (m.nslots > 0) CHECK((int64_t)m.slot0 + (int64_t)(m.nslots - 1) * m.stride < slots, "merge slot");
        if (m.pad2 > 0) CHECK((int64_t)m.pad0 + (int64_t)(m.pad2 - 1) * m.pad1 < slots, "merge prefix slot");
    }
    for (const auto& w : plan.cascade) {
        CHECK(w.head >= 0 && w.head < P.num_kv_heads && w.k_begin >= 0 && w.k_begin < w.k_end, "cascade item");
        CHECK((int64_t)w.row0 + w.nrows <= (int64_t)plan.casc_rows.size() / 2, "cascade rows");
        CHECK((int64_t)w.part + w.nrows <= slots, "cascade slots");
    }
    for (size_t i = 0; i + 1 < plan.casc_rows.size(); i += 2)
        CHECK(plan.casc_rows[i] >= 0 && plan.casc_rows[i] < plan.total_q && plan.casc_rows[i + 1] >= 0 &&
                  plan.casc_rows[i + 1] < P.num_qo_heads,
              "cascade row entry");
    for (const auto& w : plan.appends) CHECK(item_ok(w), "append item");
}

}  // namespace

int main(int argc, char** argv) {
    const uint64_t seed = argc > 1 ? std::strtoull(argv[1], nullptr, 10) : 1;
    const int iters = argc > 2 ? std::atoi(argv[2]) : 3000;
    Rng R(seed);
    for (int it = 0; it < iters && g_fail == 0; ++it) one(R, it);
    std::printf("planner_fuzz seed %llu: %d iterations (%ld accepted: %ld with tiles, %ld with few-row items, "
                "%ld with merges, %ld with cascade items; %ld rejected), %d failures\n",
                (unsigned long long)seed, iters, g_accepted, g_tiles, g_few, g_merged, g_cascade, g_rejected, g_fail);
    return g_fail ? 1 : 0;
}
