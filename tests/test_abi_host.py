"""Host-side tests of the C-ABI library (no GPU needed): exported symbols,
planner coverage, planner statistics and error paths."""
import os
import re

import numpy as np
import pytest

import workloads as W
from oracle import block_ids, useful_work, visible_matrix
from paper_2606_12688_amd import attn
from tests.helpers import plan_for

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_library_exports_every_declared_symbol():
    import ctypes

    hdr = open(os.path.join(ROOT, "include", "mstar_attn.h")).read()
    declared = set(re.findall(r"^\s*(?:int|size_t|void|const char\*)\s+(mstar_\w+)\s*\(", hdr, re.M))
    assert declared == set(attn.EXPORTS)
    L = ctypes.CDLL(attn.LIB_PATH)
    for name in declared:
        assert hasattr(L, name), name


WORKLOADS = ["tiny_causal_f32", "decode_bf16", "text_latent_bf16", "stream_window_bf16", "rollout_bf16",
             "cfg_labels_bf16", "serving_mix_bf16", "mixed"]


def _coverage(b, flags):
    pl = plan_for(b, flags | attn.FLAG_HOST_ONLY)
    G = b.num_qo_heads // b.num_kv_heads
    cover = {}  # (request, query_row, head) -> list of (k_begin, k_end)
    slots = {}
    for kind in (0, 1, 2):
        for seq, head, row0, nrows, kb, ke, part, head_stride in pl.items(kind):
            assert ke > kb
            # multi-row tile records serve every query head
            heads = range(b.num_qo_heads) if kind == 0 else [head]
            assert (head == -1) == (kind == 0)
            assert head_stride == -1 or (kind == 0 and part >= 0 and head_stride >= nrows)
            for h in heads:
                for r in range(nrows):
                    rr = row0 + r
                    if kind == 1:
                        key = (seq, rr // G, h * G + rr % G)
                    else:
                        key = (seq, rr, h)
                    cover.setdefault(key, []).append((kb, ke))
                    if part >= 0:
                        s = part + r + (h * head_stride if kind == 0 else 0)
                        assert s not in slots
                        slots[s] = key
    merges = pl.items(3)
    for row, head, slot0, stride, nslots, *_ in merges:
        keys = {slots[slot0 + s * stride] for s in range(nslots)}
        assert len(keys) == 1
        seq, i, h = keys.pop()
        assert h == head and row == b.seqs[seq, 2] + i
        assert len(cover[(seq, i, h)]) == nslots
    st = pl.stats()
    assert st["merge_rows"] == len(merges)
    pl.destroy()
    return cover, st, len(merges)


@pytest.mark.parametrize("name", WORKLOADS)
@pytest.mark.parametrize("flags", [0, attn.FLAG_FORCE_SPLIT, attn.FLAG_NO_SPLIT])
def test_planner_covers_each_visible_pair_exactly_once(name, flags):
    b = W.reduced(name)
    cover, st, n_merge = _coverage(b, flags)
    n_rows_heads = 0
    for r in range(b.num_seqs):
        q_len, L, _ = (int(x) for x in b.seqs[r])
        vis = visible_matrix(q_len, L, block_ids(b.seq_segments(r), L), int(b.masks[r, 2]))
        any_vis = np.nonzero(vis.any(axis=0))[0] if q_len else np.zeros(0, dtype=int)
        for i in range(q_len):
            keys = np.nonzero(vis[i])[0]
            for h in range(b.num_qo_heads):
                n_rows_heads += 1
                ranges = sorted(cover[(r, i, h)])
                # disjoint ranges ...
                for (a0, a1), (b0, b1) in zip(ranges[:-1], ranges[1:]):
                    assert a1 <= b0
                covered = np.zeros(L, dtype=bool)
                for a0, a1 in ranges:
                    assert 0 <= a0 and a1 <= L
                    covered[a0:a1] = True
                # ... whose union holds every visible key and stays inside the
                # page-aligned union of the request's visible keys
                assert covered[keys].all()
                assert ranges[0][0] >= (any_vis.min() // 16) * 16
                assert ranges[-1][1] <= any_vis.max() + 1
    assert len(cover) == n_rows_heads
    assert st["visible_pairs"] == useful_work(b)["pairs"]
    if flags == attn.FLAG_NO_SPLIT:
        assert n_merge == 0 and st["partial_slots"] == 0
    if flags == attn.FLAG_FORCE_SPLIT and b.dtype == "bf16":
        assert n_merge > 0


@pytest.mark.parametrize("name", ["decode_bf16", "text_latent_bf16", "stream_window_bf16", "rollout_bf16"])
def test_full_size_plans(name):
    b = W.FULL_SIZE[name]()
    pl = plan_for(b, attn.FLAG_HOST_ONLY)
    st = pl.stats()
    assert st["visible_pairs"] == useful_work(b)["pairs"]
    kr = pl.key_ranges()
    for r in range(b.num_seqs):
        q_len, L, _ = (int(x) for x in b.seqs[r])
        if name == "stream_window_bf16":
            assert (kr[r] == (L - 16 - 1023, L)).all()
        else:
            assert kr[r, 1] == L
    if name in ("text_latent_bf16", "rollout_bf16"):
        assert st["decode_items"] == 0 and st["prefill_items"] > 0
    else:
        assert st["prefill_items"] == 0 and st["decode_items"] > 0
    assert st["plan_host_us"] < 5e5
    # the work list: request records, per-row bounds and the 32-byte items, each section 256-aligned
    assert st["device_bytes"] % 256 == 0
    assert st["device_bytes"] >= 4 * st["total_q"] + 32 * (st["prefill_items"] + st["decode_items"] + st["f32_items"])
    pl.destroy()


def _params(**kw):
    base = dict(num_qo_heads=4, num_kv_heads=2, head_dim=64, dtype="bf16", seqs=[[3, 10, 0]], masks=[[0, 1, 0]],
                segments=[[0, 10, 0, 0]], max_blocks_per_seq=4, num_pages=8, flags=attn.FLAG_HOST_ONLY)
    base.update(kw)
    return base


@pytest.mark.parametrize("kw,code", [
    (dict(num_qo_heads=5), attn.ERR_INVALID_ARG),
    (dict(num_kv_heads=0), attn.ERR_INVALID_ARG),
    (dict(head_dim=96), attn.ERR_UNSUPPORTED),
    (dict(page_size=32), attn.ERR_UNSUPPORTED),
    (dict(dtype=7), attn.ERR_UNSUPPORTED),
    (dict(seqs=[[11, 10, 0]]), attn.ERR_INVALID_ARG),          # q_len > kv_len
    (dict(seqs=[[3, 10, -1]]), attn.ERR_INVALID_ARG),          # negative q_start
    (dict(segments=[[0, 9, 0, 0]]), attn.ERR_INVALID_ARG),     # does not tile [0, kv_len)
    (dict(segments=[[1, 10, 0, 0]]), attn.ERR_INVALID_ARG),    # does not start at 0
    (dict(segments=[[0, 10, 2, 0]]), attn.ERR_INVALID_ARG),    # BLOCKS without block size
    (dict(segments=[[0, 10, 9, 0]]), attn.ERR_INVALID_ARG),    # unknown kind
    (dict(masks=[[0, 1, -3]]), attn.ERR_INVALID_ARG),          # negative window
    (dict(masks=[[0, 2, 0]]), attn.ERR_INVALID_ARG),           # segment range past the array
    (dict(max_blocks_per_seq=0), attn.ERR_INVALID_ARG),
    (dict(sm_scale=0.0), attn.ERR_INVALID_ARG),
    (dict(sm_scale=-0.5), attn.ERR_INVALID_ARG),
    (dict(sm_scale=float("nan")), attn.ERR_INVALID_ARG),
    (dict(seqs=[[3, 70, 0]], segments=[[0, 70, 0, 0]]), attn.ERR_INVALID_ARG),  # kv_len > 16 * max_blocks
    (dict(seqs=[[3, 10, 0], [3, 10, 2]], masks=[[0, 1, 0], [0, 1, 0]]), attn.ERR_INVALID_ARG),  # rows overlap
    (dict(flags=attn.FLAG_HOST_ONLY | attn.FLAG_FORCE_SPLIT | attn.FLAG_NO_SPLIT), attn.ERR_INVALID_ARG),
    (dict(flags=attn.FLAG_HOST_ONLY | 64), attn.ERR_INVALID_ARG),
])
def test_plan_error_codes(kw, code):
    with pytest.raises(attn.MStarError) as ei:
        attn.plan(**_params(**kw))
    assert ei.value.code == code
    assert attn.last_error()


def test_null_pointers_and_host_only_fwd_are_rejected():
    import ctypes

    L = attn.lib()
    h = ctypes.c_void_p(None)
    assert L.mstar_attn_plan(None, None, None, 0, None, 0, None, ctypes.byref(h)) == attn.ERR_INVALID_ARG
    assert L.mstar_attn_plan(None, None, None, 0, None, 0, None, None) == attn.ERR_INVALID_ARG
    pl = attn.plan(**_params())
    rc = L.mstar_attn_fwd(pl.handle, None, None, None, None, None, None, None, 0, None)
    assert rc == attn.ERR_INVALID_ARG
    assert L.mstar_attn_fwd(None, None, None, None, None, None, None, None, 0, None) == attn.ERR_INVALID_ARG
    assert L.mstar_attn_workspace_bytes(None) == 0
    L.mstar_attn_plan_destroy(None)
    pl.destroy()


def test_empty_batch_and_zero_query_requests():
    pl = attn.plan(**_params(seqs=[[0, 10, 0]]))
    st = pl.stats()
    assert st["visible_pairs"] == 0 and st["decode_items"] == 0 and st["prefill_items"] == 0
    pl.destroy()
    pl = attn.plan(**_params(seqs=np.zeros((0, 3)), masks=np.zeros((0, 3)), segments=np.zeros((0, 4))))
    assert pl.stats()["total_q"] == 0
    pl.destroy()


@pytest.mark.parametrize("name", ["text_latent_bf16", "rollout_bf16", "cfg_labels_bf16", "mixed"])
def test_tile_launch_order_groups_kv_readers_on_one_xcd(name):
    """Every (tile item, query head) is launched exactly once; all workgroups
    reading one request's pages for one KV head sit on one XCD (workgroup b
    runs on XCD b % 8), consecutively; XCD loads differ by at most one group."""
    b = W.reduced(name) if name == "mixed" else W.FULL_SIZE[name]()
    pl = plan_for(b, attn.FLAG_HOST_ONLY)
    items = pl.items(0)
    order = pl.tile_order()
    G = b.num_qo_heads // b.num_kv_heads
    assert len(order) % 8 == 0
    real = [(i, h) for i, h in order.tolist() if i >= 0]
    assert all(i == -1 and h == -1 for i, h in order.tolist() if i < 0)
    assert sorted(real) == sorted((i, h) for i in range(len(items)) for h in range(b.num_qo_heads))
    _check_xcd_runs(order, items, G, balanced=name != "mixed")
    pl.destroy()


def _check_xcd_runs(order, items, G, balanced):
    """Each (request, KV head) group's workgroups are consecutive on an XCD;
    a group on several XCDs holds a run of consecutive items on each."""
    runs = {}  # group -> {xcd: [items]}
    lists = {x: [] for x in range(8)}
    for wg, (i, h) in enumerate(order.tolist()):
        if i < 0:
            continue
        grp = (int(items[i][0]), h // G)
        lst = runs.setdefault(grp, {}).setdefault(wg % 8, [])
        if not lst or lst[-1] != i:
            lst.append(i)
        lists[wg % 8].append(grp)
    for x, seq in lists.items():  # a group's workgroups are consecutive on its XCD
        seen = []
        for grp in seq:
            if not seen or seen[-1] != grp:
                assert grp not in seen, (x, grp)
                seen.append(grp)
    for grp, per_xcd in runs.items():
        pieces = sorted(per_xcd.values())
        flat = [i for p in pieces for i in p]
        assert flat == sorted(flat) and len(set(flat)) == len(flat)  # consecutive runs of the group's items
    sizes = {}
    for seq in lists.values():
        for grp in seq:
            sizes[grp] = sizes.get(grp, 0) + 1
    counts = [len(seq) for seq in lists.values()]
    if balanced:  # equal groups: workgroup counts per XCD within one group
        assert max(counts) - min(counts) <= max(sizes.values())
    return counts


def test_cascade_launch_order_spreads_one_group_over_every_xcd():
    """The shared-prefix decode has one cascade group per KV head (4 groups of
    equal cost): each is cut into runs so that all 8 XCDs get work of about
    equal size."""
    b = W.FULL_SIZE["shared_prefix_decode_bf16"]()
    pl = plan_for(b, attn.FLAG_HOST_ONLY, cascade=True)
    items = pl.items(4)
    order = pl.tile_order(cascade=True)
    G = b.num_qo_heads // b.num_kv_heads
    real = sorted(i for i, _ in order.tolist() if i >= 0)
    assert real == list(range(len(items)))
    for i, h in order.tolist():
        if i >= 0:
            assert h // G == items[i][1]
    counts = _check_xcd_runs(order, items, G, balanced=True)
    assert min(counts) > 0, counts
    # the work (rows x keys) per XCD differs by at most one item's
    load = [0] * 8
    for wg, (i, _) in enumerate(order.tolist()):
        if i >= 0:
            load[wg % 8] += int(items[i][3]) * (int(items[i][5]) - int(items[i][4]))
    biggest = max(int(w[3]) * (int(w[5]) - int(w[4])) for w in items)
    assert max(load) - min(load) <= biggest, load
    pl.destroy()


CASCADE = ["rollout_bf16", "cfg_labels_bf16", "mixed", "shared_prefix_decode_bf16", "serving_mix_bf16",
           "queried_prefix_bf16"]


@pytest.mark.parametrize("name", CASCADE)
@pytest.mark.parametrize("flags", [0, attn.FLAG_FORCE_SPLIT, attn.FLAG_NO_SPLIT])
def test_cascade_plan_covers_each_visible_pair_once_and_merges_read_written_slots(name, flags):
    """A cascade plan: cascade items cover the group's prefix keys for every
    member row and head, the members' own items the rest; every visible
    (row, key, head) exactly once; each merge record reads exactly the partial
    slots written for its (row, head)."""
    b = W.reduced(name)
    pl = plan_for(b, flags | attn.FLAG_HOST_ONLY | attn.FLAG_CASCADE_ALL, cascade=True)
    G = b.num_qo_heads // b.num_kv_heads
    req_of_row = {}
    for r in range(b.num_seqs):
        q_len, _, qs = (int(x) for x in b.seqs[r])
        for i in range(q_len):
            req_of_row[qs + i] = (r, i)
    cover, written = {}, {}

    def add(key, kb, ke, slot):
        cover.setdefault(key, []).append((kb, ke))
        if slot >= 0:
            assert slot not in written
            written[slot] = key

    for kind in (0, 1):
        for seq, head, row0, nrows, kb, ke, part, hs in pl.items(kind):
            for h in (range(b.num_qo_heads) if kind == 0 else [head]):
                for r in range(nrows):
                    rr = row0 + r
                    key = (seq, rr // G, h * G + rr % G) if kind == 1 else (seq, rr, h)
                    slot = -1 if part < 0 else part + r + (h * hs if kind == 0 else 0)
                    add(key, kb, ke, slot)
    rows = pl.items(5)
    members = {r for mem, _ in b.prefix_groups for r in mem}
    for seq, kvh, row0, nrows, kb, ke, part, _ in pl.items(4):
        assert seq in members and part >= 0
        for r in range(nrows):
            qrow, h = int(rows[row0 + r][0]), int(rows[row0 + r][1])
            assert h // G == kvh
            req, i = req_of_row[qrow]
            assert req in members
            add((req, i, h), kb, ke, part + r)
    for r in range(b.num_seqs):
        q_len, L, _ = (int(x) for x in b.seqs[r])
        vis = visible_matrix(q_len, L, block_ids(b.seq_segments(r), L), int(b.masks[r, 2]))
        for i in range(q_len):
            for h in range(b.num_qo_heads):
                ranges = sorted(cover[(r, i, h)])
                for (a0, a1), (c0, c1) in zip(ranges[:-1], ranges[1:]):
                    assert a1 <= c0
                covered = np.zeros(L, dtype=bool)
                for a0, a1 in ranges:
                    covered[a0:a1] = True
                assert covered[np.nonzero(vis[i])[0]].all()
    slots_cap = pl.stats()["partial_slots"]
    assert written and max(written) < slots_cap and min(written) >= 0
    merged = set()
    n_written = {}
    for k in written.values():
        n_written[k] = n_written.get(k, 0) + 1
    for row, head, s0, st, ns, p0, pst, pns in pl.items(3):
        slots = [s0 + k * st for k in range(ns)] + [p0 + k * pst for k in range(pns)]
        req, i = req_of_row[int(row)]
        assert {written[s] for s in slots} == {(req, i, int(head))}
        assert len(slots) == n_written[(req, i, int(head))]
        merged.add((req, i, int(head)))
    for (req, i, h) in cover:  # every member output is merged
        if req in members:
            assert (req, i, h) in merged
    # every output has exactly one writer: a final item or a merge record
    finals = set()
    for kind in (0, 1):
        for seq, head, row0, nrows, kb, ke, part, hs in pl.items(kind):
            if part >= 0:
                continue
            for h in (range(b.num_qo_heads) if kind == 0 else [head]):
                for r in range(nrows):
                    rr = row0 + r
                    finals.add((seq, rr // G, h * G + rr % G) if kind == 1 else (seq, rr, h))
    for r in range(b.num_seqs):
        for i in range(int(b.seqs[r, 0])):
            for h in range(b.num_qo_heads):
                assert ((r, i, h) in finals) != ((r, i, h) in merged), (r, i, h)
    pl.destroy()


@pytest.mark.parametrize("name", CASCADE)
def test_cascade_takes_only_decode_like_members_by_default(name):
    """Without FLAG_CASCADE_ALL only members with query rows x group size
    <= 64 join; a plan whose members all fill tiles equals the plain plan."""
    b = W.reduced(name)
    G = b.num_qo_heads // b.num_kv_heads
    pl = plan_for(b, attn.FLAG_HOST_ONLY, cascade=True)
    plain = plan_for(b, attn.FLAG_HOST_ONLY)
    rows = pl.items(5)
    joined = {int(r) for mem, _ in b.prefix_groups for r in mem if int(b.seqs[r, 0]) * G <= 64}
    qrow_req = {int(b.seqs[r, 2]) + i: r for r in range(b.num_seqs) for i in range(int(b.seqs[r, 0]))}
    assert {qrow_req[int(x[0])] for x in rows} == {r for r in joined if b.seqs[r, 0] > 0}
    if not joined:
        for kind in (0, 1, 3):
            assert np.array_equal(pl.items(kind), plain.items(kind))
        assert len(pl.items(4)) == 0
    pl.destroy()
    plain.destroy()


def test_cascade_rejects_bad_groups():
    b = W.reduced("rollout_bf16")
    args = (b.num_qo_heads, b.num_kv_heads, b.head_dim, b.dtype, b.seqs, b.masks, b.segments,
            b.block_table.shape[1], b.num_pages, b.sm_scale, attn.FLAG_HOST_ONLY)
    for groups in ([([0, 1], 30)],            # prefix not a multiple of 16
                   [([0, 0], 64)],            # repeated member
                   [([0, 99], 64)],           # member out of range
                   [([0, 1], 0)],             # empty prefix
                   [([0, 1], 512)]):          # longer than the members' kv_len
        with pytest.raises(attn.MStarError):
            attn.plan(*args, prefix_groups=groups).destroy()
    # a member query row that does not see the whole prefix: causal decode rows inside the prefix
    c = W.reduced("text_latent_bf16")  # text rows are causal: row 0 sees one key
    with pytest.raises(attn.MStarError) as ei:
        attn.plan(c.num_qo_heads, c.num_kv_heads, c.head_dim, c.dtype, c.seqs, c.masks, c.segments,
                  c.block_table.shape[1], c.num_pages, c.sm_scale, attn.FLAG_HOST_ONLY,
                  prefix_groups=[([0, 1], 32)]).destroy()
    assert "whole prefix" in str(ei.value)
    f = W.reduced("tiny_causal_f32")
    with pytest.raises(attn.MStarError) as ei:
        attn.plan(f.num_qo_heads, f.num_kv_heads, f.head_dim, f.dtype, f.seqs, f.masks, f.segments,
                  f.block_table.shape[1], f.num_pages, f.sm_scale, attn.FLAG_HOST_ONLY,
                  prefix_groups=[([0, 1], 16)]).destroy()
    assert ei.value.code == attn.ERR_UNSUPPORTED


@pytest.mark.parametrize("d,limit", [(128, 32), (64, 64)])
def test_few_row_items_hold_at_most_32_rows_at_d128(d, limit):
    """At d = 128 a decode-like request with 33..64 (query row, head) rows is
    cut into units of at most 32 rows (the 64-row few-row instance does not
    fit its registers there); at d = 64 one unit takes all 64."""
    b = W.mixed(seed=3, hq=8, hkv=2, d=d)
    G = b.num_qo_heads // b.num_kv_heads
    assert 64 in {int(x) * G for x in b.seqs[:, 0]}
    pl = plan_for(b, attn.FLAG_HOST_ONLY)
    rows = [int(x[3]) for x in pl.items(1)]
    assert rows and max(rows) == limit
    pl.destroy()


def test_near_equal_units_that_fill_the_gpu_stay_whole():
    """Decode units that already number at least one per workgroup slot and
    differ by less than a quarter of a piece are not split (no merge launch);
    one much longer unit among them brings the splitting back."""
    b = W.decode_bf16(seed=5, n=128, lmin=4096, lmax=4600, hq=28, hkv=4, pool_pages=None)
    pl = plan_for(b, attn.FLAG_HOST_ONLY)
    st = pl.stats()
    assert st["decode_items"] == 128 * 4 and st["merge_rows"] == 0
    assert all(int(x[6]) < 0 for x in pl.items(1))
    pl.destroy()
    b = W.decode_bf16(seed=5, n=128, lmin=4096, lmax=16384, hq=28, hkv=4, pool_pages=None)
    pl = plan_for(b, attn.FLAG_HOST_ONLY)
    assert pl.stats()["merge_rows"] > 0
    pl.destroy()


def test_noalloc_entry_point_refuses_plans_beyond_its_scratch_on_the_host():
    """The size check of mstar_attn_fwd_noalloc happens on the host before
    anything else: a host-only plan needing more than the static scratch is
    refused with MSTAR_ERR_WORKSPACE (nothing is dereferenced), one within it
    reaches the usual host-only refusal."""
    b = W.FULL_SIZE["decode_bf16"]()
    L = attn.lib()
    pl = plan_for(b, attn.FLAG_FORCE_SPLIT | attn.FLAG_HOST_ONLY)
    assert pl.workspace_bytes > 32 << 20
    assert L.mstar_attn_fwd_noalloc(pl.handle, 16, 16, 16, 16, 16, 16, None) == attn.ERR_WORKSPACE
    assert "scratch" in attn.last_error()
    pl.destroy()
    pl = plan_for(b, attn.FLAG_HOST_ONLY)
    assert 0 < pl.workspace_bytes <= 32 << 20
    assert L.mstar_attn_fwd_noalloc(pl.handle, 16, 16, 16, 16, 16, 16, None) == attn.ERR_INVALID_ARG
    assert "host-only" in attn.last_error()
    pl.destroy()


def _plan_record(pl):
    st = pl.stats()
    st.pop("plan_host_us")
    return (sorted(st.items()), [pl.items(k).tolist() for k in range(6)], pl.tile_order().tolist(),
            pl.tile_order(True).tolist(), pl.key_ranges().tolist())


def test_plans_built_on_recycled_host_lists_equal_fresh_ones():
    """Destroyed plans hand their host lists (capacity kept) to later plans:
    a plan built on the lists of a larger or different plan (tiles, few-row
    items, fp32 items, merges, a cascade) equals the same plan built while
    those lists were held by live plans."""
    batches = [(W.reduced("rollout_bf16"), 0, False), (W.reduced("mixed"), attn.FLAG_FORCE_SPLIT, False),
               (W.reduced("decode_bf16"), 0, False), (W.reduced("tiny_causal_f32"), 0, False),
               (W.reduced("shared_prefix_decode_bf16"), 0, True)]
    # reference records while every plan stays alive (no list is recycled between them)
    live = [plan_for(b, f | attn.FLAG_HOST_ONLY, cascade=c) for b, f, c in batches]
    ref = [_plan_record(p) for p in live]
    for p in live:
        p.destroy()
    for order in (range(len(batches)), reversed(range(len(batches)))):
        for i in order:
            b, f, c = batches[i]
            pl = plan_for(b, f | attn.FLAG_HOST_ONLY, cascade=c)
            assert _plan_record(pl) == ref[i], b.name
            pl.destroy()  # its lists go to the next plan
