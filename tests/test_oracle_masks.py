"""Pins of the oracle's mask model (visibility) against predicates written
directly from each workload's wording, by brute force over every (row, key)
pair, and against closed-form visible-pair counts at full size."""
import numpy as np
import pytest

import workloads as W
from oracle import block_ids, useful_work, visible_matrix


def _vis(batch, r):
    q_len, kv_len, _ = batch.seqs[r]
    _, _, window = batch.masks[r]
    return visible_matrix(int(q_len), int(kv_len), block_ids(batch.seq_segments(r), int(kv_len)), int(window))


def _brute(q_len, kv_len, pred):
    out = np.zeros((q_len, kv_len), dtype=bool)
    for i in range(q_len):
        p = kv_len - q_len + i
        for t in range(kv_len):
            out[i, t] = pred(p, t)
    return out


def test_causal_prefill_matches_lower_triangle():
    b = W.tiny_causal_f32()
    for r in range(b.num_seqs):
        L = int(b.seqs[r, 1])
        assert np.array_equal(_vis(b, r), _brute(L, L, lambda p, t: t <= p))


def test_decode_row_sees_whole_context():
    b = W.reduced("decode_bf16")
    for r in range(b.num_seqs):
        L = int(b.seqs[r, 1])
        assert np.array_equal(_vis(b, r), _brute(1, L, lambda p, t: t <= p))
        assert _vis(b, r).sum() == L


def test_text_prefix_then_full_latent_block():
    b = W.reduced("text_latent_bf16")
    text = 37
    for r in range(b.num_seqs):
        L = int(b.seqs[r, 1])
        # text rows: causal, and they never see the latents;
        # latent rows: the whole prefix and the whole latent block.
        pred = lambda p, t: (t <= p) if p < text else True  # noqa: E731
        assert np.array_equal(_vis(b, r), _brute(L, L, pred))


def test_window_chunks_see_exactly_window_keys():
    b = W.reduced("stream_window_bf16")
    Wn = 100
    for r in range(b.num_seqs):
        q_len, L = int(b.seqs[r, 0]), int(b.seqs[r, 1])
        vis = _vis(b, r)
        assert np.array_equal(vis, _brute(q_len, L, lambda p, t: t <= p and p - t < Wn))
        for i in range(q_len):
            p = L - q_len + i
            assert vis[i].sum() == min(Wn, p + 1)
            # both boundary keys: the oldest visible and the first hidden one
            if p - Wn + 1 >= 0:
                assert vis[i, p - Wn + 1]
            if p - Wn >= 0:
                assert not vis[i, p - Wn]


def test_rollout_frames_over_shared_prefix():
    prefix, frame = 64, 40
    b = W.reduced("rollout_bf16")
    for r in range(b.num_seqs):
        q_len, L = int(b.seqs[r, 0]), int(b.seqs[r, 1])

        def pred(p, t):
            f = (p - prefix) // frame  # frame of the query
            return t < prefix or (t - prefix) // frame <= f

        assert np.array_equal(_vis(b, r), _brute(q_len, L, pred))
    # every block table starts with the same prefix pages
    assert (b.block_table[:, : prefix // 16] == b.block_table[0, : prefix // 16]).all()


def test_ragged_blocks_and_mixed_segments():
    segs = [(0, 5, W.SEG_CAUSAL, 0), (5, 11, W.SEG_BLOCKS, 4), (16, 3, W.SEG_FULL, 0), (19, 2, W.SEG_CAUSAL, 0)]
    blk = block_ids(segs, 21)
    # causal 0..4 -> 0..4; blocks of 4 over 11 tokens -> 5,5,5,5,6,6,6,6,7,7,7; full -> 8; causal -> 9,10
    expect = [0, 1, 2, 3, 4, 5, 5, 5, 5, 6, 6, 6, 6, 7, 7, 7, 8, 8, 8, 9, 10]
    assert blk.tolist() == expect
    vis = visible_matrix(21, 21, blk, 3)
    for p in range(21):
        for t in range(21):
            assert vis[p, t] == (expect[t] <= expect[p] and p - t < 3)


@pytest.mark.parametrize("bad", [
    [(0, 5, 0, 0), (6, 4, 0, 0)],       # gap
    [(0, 5, 0, 0)],                      # does not reach kv_len
    [(0, 10, 2, 0)],                     # BLOCKS without a block size
    [(0, 10, 7, 0)],                     # unknown kind
])
def test_segments_must_tile(bad):
    with pytest.raises(ValueError):
        block_ids(bad, 10)


def test_full_size_visible_pair_counts_closed_form():
    """Visible (row, key) pairs times query heads at full size, from each
    workload's wording."""
    c1 = W.tiny_causal_f32()
    assert useful_work(c1)["pairs"] == 2 * sum(L * (L + 1) // 2 for L in (17, 33, 64, 5))
    c3 = W.text_latent_bf16()
    assert useful_work(c3)["pairs"] == 8 * 28 * (256 * 257 // 2 + 4096 * 4352)
    c4 = W.stream_window_bf16()
    # every context is at least the window long, so each row sees exactly 1024 keys
    assert useful_work(c4)["pairs"] == 256 * 16 * 1024 * 16
    c5 = W.rollout_bf16()
    assert useful_work(c5)["pairs"] == 300 * 16 * sum(256 * (2048 + 256 * (f + 1)) for f in range(4))
    c2 = W.decode_bf16()
    assert useful_work(c2)["pairs"] == 28 * int(c2.seqs[:, 1].sum())


def test_kv_bytes_count_shared_pages_once():
    c5 = W.rollout_bf16()
    # 2048 shared prefix keys once + 300 x 1024 own keys; K and V; 16 heads x 64 x 2 bytes
    assert useful_work(c5)["kv_bytes"] == 2 * (2048 + 300 * 1024) * 16 * 64 * 2
    c4 = W.stream_window_bf16()
    # 16 rows with windows of 1024 ending at consecutive positions: 1039 distinct keys
    assert useful_work(c4)["kv_bytes"] == 2 * 256 * 1039 * 8 * 128 * 2


def test_cfg_labels_see_whole_context_and_alias_text_pages():
    """Every latent query row of every CFG label sees the label's whole context
    and its own block; the image-dropped label's text pages are the
    conditional label's; the text-dropped label shares no page."""
    text = 32
    b = W.reduced("cfg_labels_bf16")
    for r in range(b.num_seqs):
        q_len, L = int(b.seqs[r, 0]), int(b.seqs[r, 1])
        assert np.array_equal(_vis(b, r), _brute(q_len, L, lambda p, t: True))
    tp = text // 16
    for img in range(b.num_seqs // 3):
        cond, no_text, no_img = (b.block_table[3 * img + k] for k in range(3))
        n = [(int(b.seqs[3 * img + k, 1]) + 15) // 16 for k in range(3)]
        assert np.array_equal(no_img[:tp], cond[:tp])
        assert not set(no_img[tp:n[2]]) & set(cond[:n[0]])
        others = set(cond[:n[0]]) | set(no_img[:n[2]])
        assert not set(no_text[:n[1]]) & others


def test_cfg_labels_full_size_counts_closed_form():
    b = W.cfg_labels_bf16()
    w = useful_work(b)
    # 2 images x 28 heads x 4096 latent rows over (256+4096+4096) + (4096+4096) + (256+4096) keys
    assert w["pairs"] == 2 * 28 * 4096 * (8448 + 8192 + 4352)
    # distinct keys: per image 8448 + 8192 + 4096 (the text keys of the image-dropped label are shared)
    assert w["kv_bytes"] == 2 * 2 * (8448 + 8192 + 4096) * 4 * 128 * 2


def test_serving_mix_each_request_kind_by_its_own_predicate():
    """The node batch across Walks: decode rows see their whole context; the
    image request's text rows are causal and blind to the latents, its latent
    rows see everything; chunk rows are causal under a 96-key window; rollout
    frames see the shared prefix and frames up to their own."""
    b = W.reduced("serving_mix_bf16")
    text, latent, Wn, prefix, frame = 37, 200, 96, 64, 40
    kinds = ["decode"] * 5 + ["image"] + ["chunk"] * 4 + ["rollout"] * 3
    assert len(kinds) == b.num_seqs
    for r, kind in enumerate(kinds):
        q_len, L = int(b.seqs[r, 0]), int(b.seqs[r, 1])
        if kind == "decode":
            pred = lambda p, t: t <= p  # noqa: E731
            assert q_len == 1
        elif kind == "image":
            pred = lambda p, t: (t <= p) if p < text else True  # noqa: E731
            assert q_len == L == text + latent
        elif kind == "chunk":
            pred = lambda p, t: t <= p and p - t < Wn  # noqa: E731
            assert q_len == 16
        else:
            def pred(p, t):
                return t < prefix or (t - prefix) // frame <= (p - prefix) // frame
            assert q_len == 2 * frame and L == prefix + 2 * frame
        assert np.array_equal(_vis(b, r), _brute(q_len, L, pred)), (r, kind)
    first_roll = kinds.index("rollout")
    shared = b.block_table[first_roll, :prefix // 16]
    for r in range(first_roll, b.num_seqs):
        assert np.array_equal(b.block_table[r, :prefix // 16], shared)
    assert b.prefix_groups == [(list(range(first_roll, b.num_seqs)), prefix)]
