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
             "cfg_labels_bf16", "mixed"]


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
    xcd_of, pos = {}, {}
    lists = {x: [] for x in range(8)}
    for wg, (i, h) in enumerate(order.tolist()):
        if i < 0:
            continue
        grp = (int(items[i][0]), h // G)
        assert xcd_of.setdefault(grp, wg % 8) == wg % 8
        lists[wg % 8].append(grp)
    for x, seq in lists.items():  # a group's workgroups are consecutive on its XCD
        seen = []
        for grp in seq:
            if not seen or seen[-1] != grp:
                assert grp not in seen, (x, grp)
                seen.append(grp)
    sizes = {}
    for seq in lists.values():
        for grp in seq:
            sizes[grp] = sizes.get(grp, 0) + 1
    counts = [len(seq) for seq in lists.values()]
    if name != "mixed":  # equal groups: workgroup counts per XCD within one group
        assert max(counts) - min(counts) <= max(sizes.values())
    pl.destroy()
