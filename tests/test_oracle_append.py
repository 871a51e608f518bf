"""Pins of the paged KV append oracle: rows land where an independent walk of
the block table says, every other slot keeps its value, and appending then
attending equals attention over the contiguous context with the new rows in
its last positions."""
import dataclasses

import numpy as np
import pytest
import torch

import workloads as W
from oracle import append_targets, kv_append, oracle_attention


def _new_rows(b, seed=5):
    rng = np.random.default_rng(seed)
    shape = (b.total_q, b.num_kv_heads, b.head_dim)
    return rng.standard_normal(shape).astype(np.float32), rng.standard_normal(shape).astype(np.float32)


@pytest.mark.parametrize("name", ["decode_bf16", "stream_window_bf16", "rollout_bf16", "cfg_labels_bf16", "mixed"])
def test_rows_land_at_their_positions_and_nothing_else_changes(name):
    b = W.reduced(name)
    t = W.make_tensors_numpy(b)
    kn, vn = _new_rows(b)
    k2, v2 = kv_append(b, kn, vn, t["k_pages"], t["v_pages"])
    touched = np.zeros(t["k_pages"].shape[:2], dtype=bool)
    for r in range(b.num_seqs):  # independent walk: position -> logical page -> physical page
        q_len, kv_len, q_start = (int(x) for x in b.seqs[r])
        for i in range(q_len):
            pos = kv_len - q_len + i
            page, slot = int(b.block_table[r][pos >> 4]), pos & 15
            assert np.array_equal(k2[page, slot], kn[q_start + i])
            assert np.array_equal(v2[page, slot], vn[q_start + i])
            touched[page, slot] = True
    assert np.array_equal(k2[~touched], t["k_pages"][~touched])
    assert np.array_equal(v2[~touched], t["v_pages"][~touched])
    assert touched.sum() == int(b.seqs[:, 0].sum())


def test_append_then_attend_equals_sdpa_over_the_contiguous_context():
    b = W.reduced("stream_window_bf16")
    b = dataclasses.replace(b, masks=b.masks * np.array([1, 1, 0]))  # no window: plain causal
    t = W.make_tensors_numpy(b)
    kn, vn = _new_rows(b)
    k2, v2 = kv_append(b, kn, vn, t["k_pages"], t["v_pages"])
    out, lse = oracle_attention(b, t["q"], k2, v2)
    g = b.num_qo_heads // b.num_kv_heads
    for r in range(b.num_seqs):
        q_len, L, qs = (int(x) for x in b.seqs[r])
        K = np.stack([t["k_pages"][b.block_table[r][p >> 4], p & 15] for p in range(L)]).astype(np.float64)
        V = np.stack([t["v_pages"][b.block_table[r][p >> 4], p & 15] for p in range(L)]).astype(np.float64)
        K[L - q_len:] = kn[qs:qs + q_len]
        V[L - q_len:] = vn[qs:qs + q_len]
        q = torch.from_numpy(t["q"][qs:qs + q_len].astype(np.float64)).transpose(0, 1)[None]
        kk = torch.from_numpy(K).transpose(0, 1).repeat_interleave(g, dim=0)[None]
        vv = torch.from_numpy(V).transpose(0, 1).repeat_interleave(g, dim=0)[None]
        mask = torch.ones(q_len, L, dtype=torch.bool).tril(diagonal=L - q_len)
        ref = torch.nn.functional.scaled_dot_product_attention(q, kk, vv, attn_mask=mask, scale=b.sm_scale)
        np.testing.assert_allclose(out[qs:qs + q_len], ref[0].transpose(0, 1).numpy(), rtol=0, atol=1e-12)


def test_two_rows_on_one_slot_are_rejected():
    b = W.reduced("decode_bf16")
    bt = b.block_table.copy()
    # request 1's last page becomes request 0's last page, and both new tokens sit in the same slot
    L0, L1 = int(b.seqs[0, 1]), int(b.seqs[1, 1])
    seqs = b.seqs.copy()
    seqs[1, 1] = L1 - (L1 % 16) + (L0 - 1) % 16 + 1 if L1 >= 16 else (L0 - 1) % 16 + 1
    bt[1, (int(seqs[1, 1]) - 1) >> 4] = bt[0, (L0 - 1) >> 4]
    b2 = dataclasses.replace(b, block_table=bt, seqs=seqs)
    with pytest.raises(ValueError):
        append_targets(b2)


def test_out_of_pool_page_is_rejected():
    b = W.reduced("decode_bf16")
    bt = b.block_table.copy()
    bt[0, (int(b.seqs[0, 1]) - 1) >> 4] = b.num_pages
    with pytest.raises(ValueError):
        append_targets(dataclasses.replace(b, block_table=bt))
