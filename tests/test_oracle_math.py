"""Pins of the oracle's softmax-attention arithmetic and paging: torch's CPU
float64 scaled_dot_product_attention on special cases, closed forms,
invariants, an independent scalar oracle, and the split/merge identity."""
import json
import math
import os

import numpy as np
import pytest
import torch

import workloads as W
from oracle import attend, block_ids, merge_partials, oracle_attention, oracle_rows, visible_matrix
from oracle.scalar import scalar_attention

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _one_request(q_len, kv_len, segs, window=0, hq=2, hkv=2, d=16, identity=True, seed=0, extra_pages=0):
    n_pages = (kv_len + 15) // 16 + extra_pages
    rng = np.random.default_rng(seed)
    order = np.arange(n_pages, dtype=np.int32) if identity else rng.permutation(n_pages).astype(np.int32)
    bt = order[None, : (kv_len + 15) // 16].copy()
    return W._finish("t", hq, hkv, d, "f32", [q_len], [kv_len], [segs], [window], bt, n_pages, seed)


def _contiguous(b, t, r=0):
    """K/V of request r as contiguous [Hkv, kv_len, d] read with a plain loop
    over the block table (test-side, independent of the oracle's gather)."""
    L = int(b.seqs[r, 1])
    K = np.zeros((b.num_kv_heads, L, b.head_dim))
    V = np.zeros_like(K)
    for tok in range(L):
        page = int(b.block_table[r, tok // 16])
        K[:, tok, :] = t["k_pages"][page, tok % 16]
        V[:, tok, :] = t["v_pages"][page, tok % 16]
    return K, V


def _sdpa(q, K, V, scale, mask=None, causal=False, gqa=False):
    qt = torch.from_numpy(np.ascontiguousarray(q.transpose(1, 0, 2)))[None]
    kt = torch.from_numpy(K)[None]
    vt = torch.from_numpy(V)[None]
    m = None if mask is None else torch.from_numpy(mask)
    o = torch.nn.functional.scaled_dot_product_attention(
        qt, kt, vt, attn_mask=m, is_causal=causal, scale=scale, enable_gqa=gqa)
    g = qt.shape[1] // kt.shape[1]
    kr = kt.repeat_interleave(g, dim=1)
    s = (qt @ kr.transpose(-1, -2)) * scale
    if m is not None:
        s = s.masked_fill(~m, float("-inf"))
    if causal:
        L = s.shape[-1]
        s = s.masked_fill(~torch.ones(L, L, dtype=torch.bool).tril(), float("-inf"))
    lse = torch.logsumexp(s, dim=-1)
    return o[0].numpy().transpose(1, 0, 2), lse[0].numpy().T


def test_causal_prefill_equals_sdpa_is_causal():
    b = _one_request(70, 70, [(0, 70, 0, 0)])
    t = W.make_tensors_numpy(b)
    out, lse = oracle_attention(b, t["q"], t["k_pages"], t["v_pages"])
    K, V = _contiguous(b, t)
    o_ref, l_ref = _sdpa(t["q"].astype(np.float64), K, V, b.sm_scale, causal=True)
    np.testing.assert_allclose(out, o_ref, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, l_ref, rtol=0, atol=1e-12)


def test_full_block_equals_unmasked_sdpa_with_gqa():
    b = _one_request(45, 45, [(0, 45, 1, 0)], hq=6, hkv=2)
    t = W.make_tensors_numpy(b)
    out, lse = oracle_attention(b, t["q"], t["k_pages"], t["v_pages"])
    K, V = _contiguous(b, t)
    o_ref, l_ref = _sdpa(t["q"].astype(np.float64), K, V, b.sm_scale, gqa=True)
    np.testing.assert_allclose(out, o_ref, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, l_ref, rtol=0, atol=1e-12)


def test_mixed_mask_equals_sdpa_explicit_mask_permuted_pages():
    segs = [(0, 20, 0, 0), (20, 33, 2, 8), (53, 30, 1, 0), (83, 7, 0, 0)]
    b = _one_request(60, 90, segs, window=41, identity=False, hq=4, hkv=2)
    t = W.make_tensors_numpy(b)
    out, lse = oracle_attention(b, t["q"], t["k_pages"], t["v_pages"])
    # explicit mask written straight from the segment wording
    ids = []
    for s0, ln, kind, blk in segs:
        base = (max(ids) + 1) if ids else 0
        ids += [base + (j if kind == 0 else 0 if kind == 1 else j // blk) for j in range(ln)]
    mask = np.array([[ids[tk] <= ids[p] and p - tk < 41 for tk in range(90)] for p in range(30, 90)])
    K, V = _contiguous(b, t)
    o_ref, l_ref = _sdpa(t["q"].astype(np.float64), K, V, b.sm_scale, mask=mask, gqa=True)
    np.testing.assert_allclose(out, o_ref, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, l_ref, rtol=0, atol=1e-12)


def test_one_visible_key_returns_its_value_row():
    # window 1: every row sees only itself
    b = _one_request(37, 37, [(0, 37, 0, 0)], window=1, identity=False)
    t = W.make_tensors_numpy(b)
    out, lse = oracle_attention(b, t["q"], t["k_pages"], t["v_pages"])
    K, V = _contiguous(b, t)
    for p in range(37):
        for h in range(2):
            assert np.array_equal(out[p, h], V[h, p])
            s = b.sm_scale * math.fsum(float(x) * float(y) for x, y in zip(t["q"][p, h], K[h, p]))
            assert abs(lse[p, h] - s) < 1e-12


def test_equal_scores_give_mean_of_visible_values():
    b = W.reduced("mixed")
    t = W.make_tensors_numpy(b)
    q0 = np.zeros_like(t["q"])
    out, lse = oracle_attention(b, q0, t["k_pages"], t["v_pages"])
    g = b.num_qo_heads // b.num_kv_heads
    for r in range(b.num_seqs):
        q_len, L, qs = (int(x) for x in b.seqs[r])
        vis = visible_matrix(q_len, L, block_ids(b.seq_segments(r), L), int(b.masks[r, 2]))
        K, V = _contiguous(b, t, r)
        for i in range(0, q_len, 7):
            n = int(vis[i].sum())
            for h in range(b.num_qo_heads):
                ref = np.mean(V[h // g][vis[i]], axis=0)
                np.testing.assert_allclose(out[qs + i, h], ref, rtol=0, atol=1e-12)
                assert abs(lse[qs + i, h] - math.log(n)) < 1e-12


def test_page_permutation_is_bitwise_invariant():
    b = W.reduced("mixed")
    t = W.make_tensors_numpy(b)
    o1, l1 = oracle_attention(b, t["q"], t["k_pages"], t["v_pages"])
    b2, t2 = W.permute_pages(b, t, seed=5)
    assert not np.array_equal(b2.block_table, b.block_table)
    o2, l2 = oracle_attention(b2, t2["q"], t2["k_pages"], t2["v_pages"])
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)


def test_singleton_blocks_equal_causal_and_wide_window_equals_none():
    bc = _one_request(50, 50, [(0, 50, 0, 0)], identity=False, seed=3)
    bb = _one_request(50, 50, [(0, 50, 2, 1)], identity=False, seed=3)
    bw = _one_request(50, 50, [(0, 50, 0, 0)], window=50, identity=False, seed=3)
    t = W.make_tensors_numpy(bc)
    ref = oracle_attention(bc, t["q"], t["k_pages"], t["v_pages"])
    for other in (bb, bw):
        got = oracle_attention(other, t["q"], t["k_pages"], t["v_pages"])
        assert np.array_equal(ref[0], got[0]) and np.array_equal(ref[1], got[1])


def test_gqa_equals_mha_with_repeated_kv_heads():
    b = W.reduced("stream_window_bf16")
    b = W._finish("t", 4, 2, 32, "f32", list(b.seqs[:, 0]), list(b.seqs[:, 1]),
                  [[tuple(s) for s in b.seq_segments(r)] for r in range(b.num_seqs)],
                  list(b.masks[:, 2]), b.block_table, b.num_pages, 0)
    t = W.make_tensors_numpy(b)
    o1, l1 = oracle_attention(b, t["q"], t["k_pages"], t["v_pages"])
    bm = W._finish("t", 4, 4, 32, "f32", list(b.seqs[:, 0]), list(b.seqs[:, 1]),
                   [[tuple(s) for s in b.seq_segments(r)] for r in range(b.num_seqs)],
                   list(b.masks[:, 2]), b.block_table, b.num_pages, 0)
    kr = np.repeat(t["k_pages"], 2, axis=2)
    vr = np.repeat(t["v_pages"], 2, axis=2)
    o2, l2 = oracle_attention(bm, t["q"], kr, vr)
    np.testing.assert_allclose(o1, o2, rtol=0, atol=1e-13)
    np.testing.assert_allclose(l1, l2, rtol=0, atol=1e-13)


def test_request_order_does_not_matter():
    b = W.reduced("decode_bf16")
    t = W.make_tensors_numpy(b)
    o1, l1 = oracle_attention(b, t["q"], t["k_pages"], t["v_pages"])
    order = np.random.default_rng(1).permutation(b.num_seqs)
    seqs = b.seqs[order].copy()
    seqs[:, 2] = np.concatenate([[0], np.cumsum(seqs[:-1, 0])])
    b2 = W.Batch(b.name, b.num_qo_heads, b.num_kv_heads, b.head_dim, b.dtype, seqs,
                 b.masks[order].copy(), b.segments, b.block_table[order].copy(), b.num_pages)
    q2 = np.concatenate([t["q"][b.seqs[r, 2]:b.seqs[r, 2] + b.seqs[r, 0]] for r in order])
    o2, l2 = oracle_attention(b2, q2, t["k_pages"], t["v_pages"])
    for new, r in enumerate(order):
        a, n = int(b.seqs[r, 2]), int(b.seqs[r, 0])
        c = int(seqs[new, 2])
        assert np.array_equal(o1[a:a + n], o2[c:c + n])
        assert np.array_equal(l1[a:a + n], l2[c:c + n])


def test_no_visible_key_gives_zero_and_minus_inf():
    q = np.ones((3, 4))
    K = np.ones((5, 4))
    V = np.arange(20.0).reshape(5, 4)
    vis = np.zeros((3, 5), dtype=bool)
    vis[1, 2] = True
    out, lse = attend(q, K, V, vis, 0.5)
    assert np.all(out[[0, 2]] == 0) and np.all(np.isneginf(lse[[0, 2]]))
    assert np.array_equal(out[1], V[2]) and lse[1] == 0.5 * 4


def test_large_scores_do_not_overflow():
    q = np.full((1, 2), 300.0)
    K = np.array([[1.0, 1.0], [1.0, 0.0]])
    V = np.array([[1.0, 0.0], [0.0, 1.0]])
    out, lse = attend(q, K, V, np.ones((1, 2), dtype=bool), 1.0)
    # scores 600 and 300: weight of the second is exp(-300)
    assert np.allclose(out[0], [1.0, math.exp(-300)], rtol=0, atol=1e-300)
    assert abs(lse[0] - (600 + math.log1p(math.exp(-300)))) < 1e-12


def test_golden_hand_derived_cases():
    with open(os.path.join(GOLDEN, "hand_cases.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        out, lse = attend(np.array(c["q"]), np.array(c["K"]), np.array(c["V"]),
                          np.array(c["visible"], dtype=bool), c["sm_scale"])
        np.testing.assert_allclose(out, np.array(c["out"]), rtol=0, atol=1e-12, err_msg=c["name"])
        exp_lse = [float("-inf") if x is None else x for x in c["lse_natural"]]
        np.testing.assert_allclose(lse, np.array(exp_lse), rtol=0, atol=1e-12, err_msg=c["name"])


@pytest.mark.parametrize("seed", range(4))
def test_scalar_oracle_agrees_on_tiny_batches(seed):
    rng = np.random.default_rng(seed)
    q_lens, kv_lens, segl, wins = [], [], [], []
    for _ in range(3):
        L = int(rng.integers(1, 41))
        # random segment tiling
        segs, pos = [], 0
        while pos < L:
            ln = int(rng.integers(1, L - pos + 1))
            kind = int(rng.integers(0, 3))
            segs.append((pos, ln, kind, int(rng.integers(1, 6)) if kind == 2 else 0))
            pos += ln
        q_lens.append(int(rng.integers(1, L + 1))); kv_lens.append(L)
        segl.append(segs); wins.append(int(rng.integers(0, 3)) * int(rng.integers(1, 12)))
    pages = sum((L + 15) // 16 for L in kv_lens) + 2
    perm = rng.permutation(pages).astype(np.int32)
    bt = np.full((3, 3), -1, dtype=np.int32)
    cur = 0
    for r, L in enumerate(kv_lens):
        n = (L + 15) // 16
        bt[r, :n] = perm[cur:cur + n]; cur += n
    b = W._finish("tiny", 4, 2, 8, "f32", q_lens, kv_lens, segl, wins, bt, pages, seed)
    t = W.make_tensors_numpy(b)
    out, lse = oracle_attention(b, t["q"], t["k_pages"], t["v_pages"])
    so, sl = scalar_attention(b, t["q"].tolist(), t["k_pages"].tolist(), t["v_pages"].tolist())
    np.testing.assert_allclose(out, np.array(so), rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, np.array(sl), rtol=0, atol=1e-12)


@pytest.mark.parametrize("seed", range(3))
def test_split_and_merge_equals_unsplit(seed):
    rng = np.random.default_rng(seed)
    M, N, d = 9, 130, 16
    q, K, V = rng.standard_normal((M, d)), rng.standard_normal((N, d)), rng.standard_normal((N, d))
    vis = rng.random((M, N)) < 0.6
    vis[:, :3] = False  # leading chunk empty for every row
    vis[4] = False
    vis[4, 100] = True  # a row with one key in one chunk only
    ref_o, ref_l = attend(q, K, V, vis, 0.3)
    cuts = np.sort(rng.choice(np.arange(1, N), size=5, replace=False))
    edges = [0, 3, *cuts.tolist(), N]
    outs, lses = [], []
    for a, e in zip(edges[:-1], edges[1:]):
        o, s = attend(q, K[a:e], V[a:e], vis[:, a:e], 0.3)
        outs.append(o); lses.append(s)
    mo, ml = merge_partials(outs, lses)
    np.testing.assert_allclose(mo, ref_o, rtol=0, atol=1e-12)
    np.testing.assert_allclose(ml, ref_l, rtol=0, atol=1e-12)
    # all chunks empty for a row -> zero / -inf
    mo2, ml2 = merge_partials([np.ones((1, 2))] * 2, [np.array([-np.inf])] * 2)
    assert np.all(mo2 == 0) and np.isneginf(ml2[0])


def test_sampled_rows_agree_with_scalar_oracle():
    b = W.reduced("tiny_causal_f32")
    segs = [[(0, 9, 0, 0), (9, 20, 2, 6), (29, 6, 1, 0)], [(0, 12, 0, 0)]]
    bt = np.array([[3, 0, 4], [1, 2, -1]], dtype=np.int32)
    b = W._finish("t", 4, 2, 8, "f32", [30, 5], [35, 12], segs, [0, 4], bt, 5, 0)
    t = W.make_tensors_numpy(b)
    so, sl = scalar_attention(b, t["q"].tolist(), t["k_pages"].tolist(), t["v_pages"].tolist())
    picks = [(0, 0, 0), (0, 11, 3), (0, 29, 1), (1, 0, 2), (1, 4, 0)]
    ro, rl = oracle_rows(b, t["q"], t["k_pages"], t["v_pages"], picks)
    for n, (r, i, h) in enumerate(picks):
        row = int(b.seqs[r, 2]) + i
        np.testing.assert_allclose(ro[n], so[row][h], rtol=0, atol=1e-12)
        assert abs(rl[n] - sl[row][h]) < 1e-12


def test_cfg_label_reading_aliased_pages_equals_a_private_copy():
    """The image-dropped CFG label reads the conditional label's text pages in
    place; giving it private copies of those pages changes nothing (bitwise),
    and each label equals unmasked SDPA over its concatenated context."""
    import dataclasses

    b = W.reduced("cfg_labels_bf16")
    t = W.make_tensors_numpy(b)
    o1, l1 = oracle_attention(b, t["q"], t["k_pages"], t["v_pages"])
    tp = 32 // 16
    bt = b.block_table.copy()
    k, v = t["k_pages"], t["v_pages"]
    extra_k, extra_v = [], []
    for r in range(2, b.num_seqs, 3):
        for j in range(tp):
            src = int(bt[r, j])
            extra_k.append(k[src]); extra_v.append(v[src])
            bt[r, j] = b.num_pages + len(extra_k) - 1
    b2 = dataclasses.replace(b, block_table=bt, num_pages=b.num_pages + len(extra_k))
    k2 = np.concatenate([k, np.stack(extra_k)]); v2 = np.concatenate([v, np.stack(extra_v)])
    o2, l2 = oracle_attention(b2, t["q"], k2, v2)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)
    for r in range(b.num_seqs):
        q_len, L, qs = (int(x) for x in b.seqs[r])
        K, V = _contiguous(b, t, r)
        q = t["q"][qs:qs + q_len].astype(np.float64)
        ro, rl = _sdpa(q, K, V, b.sm_scale, gqa=True)
        np.testing.assert_allclose(o1[qs:qs + q_len], ro, rtol=0, atol=1e-12)
        np.testing.assert_allclose(l1[qs:qs + q_len], rl, rtol=0, atol=1e-12)
