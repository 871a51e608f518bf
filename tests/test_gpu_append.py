"""GPU tests of the paged KV append (``mstar_kv_append``) through the C-ABI:
pages bitwise equal to the CPU oracle's, attention over the appended cache
against the oracle, the out-of-pool error bit, and a full-size property."""
import numpy as np
import pytest

import workloads as W
from oracle import append_targets, kv_append, oracle_attention
from paper_2606_12688_amd import attn
from tests.helpers import plan_for

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _new_rows(b, seed=9):
    import torch

    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    dt = torch.float32 if b.dtype == "f32" else torch.bfloat16
    shape = (b.total_q, b.num_kv_heads, b.head_dim)
    return (torch.randn(shape, generator=g, device=DEV).to(dt), torch.randn(shape, generator=g, device=DEV).to(dt))


def _host(t):
    return t.float().cpu().numpy()


@pytest.mark.parametrize("name", ["tiny_causal_f32", "decode_bf16", "stream_window_bf16", "rollout_bf16",
                                  "cfg_labels_bf16", "mixed"])
def test_append_matches_oracle_bitwise_then_attention_parity(name):
    import torch

    b = W.reduced(name)
    t = W.make_tensors_torch(b, DEV, poison_unused=True)
    kn, vn = _new_rows(b)
    ref_k, ref_v = kv_append(b, _host(kn), _host(vn), _host(t["k_pages"]), _host(t["v_pages"]))
    pl = plan_for(b)
    bt = torch.from_numpy(np.ascontiguousarray(b.block_table)).to(DEV)
    attn.kv_append(pl, kn, vn, bt, t["k_pages"], t["v_pages"])
    assert attn.check(pl) == 0
    # bitwise (NaN-poisoned untouched slots compare equal as bit patterns)
    assert np.array_equal(_host(t["k_pages"]).view(np.uint32), ref_k.view(np.uint32))
    assert np.array_equal(_host(t["v_pages"]).view(np.uint32), ref_v.view(np.uint32))
    out = torch.empty_like(t["q"])
    lse = torch.empty(t["q"].shape[:2], dtype=torch.float32, device=DEV)
    attn.fwd(pl, t["q"], t["k_pages"], t["v_pages"], bt, out, lse, attn.workspace(pl, DEV))
    assert attn.check(pl) == 0
    pl.destroy()
    ro, rl = oracle_attention(b, _host(t["q"]).astype(np.float64), ref_k.astype(np.float64), ref_v.astype(np.float64))
    tol_o = 1e-5 if b.dtype == "f32" else 1.5e-2
    eo = float(np.abs(_host(out).astype(np.float64) - ro).max())
    el = float(np.abs(lse.cpu().numpy().astype(np.float64) - rl).max())
    print(f"{name}: append bitwise, then max|dout|={eo:.3e} max|dlse|={el:.3e}", flush=True)
    assert eo <= tol_o and el <= 1e-3


def test_out_of_pool_target_sets_error_bit_and_other_rows_land():
    import torch

    b = W.reduced("decode_bf16")
    t = W.make_tensors_torch(b, DEV)
    kn, vn = _new_rows(b)
    bt_h = b.block_table.copy()
    L0 = int(b.seqs[0, 1])
    bt_h[0, (L0 - 1) >> 4] = b.num_pages + 3
    pl = plan_for(b)
    before = _host(t["k_pages"])
    attn.kv_append(pl, kn, vn, torch.from_numpy(bt_h).to(DEV), t["k_pages"], t["v_pages"])
    assert attn.check(pl) == attn.DEVERR_PAGE_RANGE
    pl.destroy()
    after = _host(t["k_pages"])
    kh = _host(kn)
    for r in range(1, b.num_seqs):
        L, qs = int(b.seqs[r, 1]), int(b.seqs[r, 2])
        page, slot = int(bt_h[r, (L - 1) >> 4]), (L - 1) & 15
        assert np.array_equal(after[page, slot], kh[qs])
    touched = np.zeros(before.shape[:2], dtype=bool)
    for r in range(1, b.num_seqs):
        L = int(b.seqs[r, 1])
        touched[bt_h[r, (L - 1) >> 4], (L - 1) & 15] = True
    assert np.array_equal(after[~touched].view(np.uint32), before[~touched].view(np.uint32))


@pytest.mark.parametrize("name", ["decode_bf16", "rollout_bf16"])
def test_full_size_append_property(name):
    """Every new row lands bitwise where the block table says; the untouched
    slots keep their bytes (compared on the device)."""
    import torch

    b = W.FULL_SIZE[name]()
    t = W.make_tensors_torch(b, DEV)
    kn, vn = _new_rows(b)
    targets = np.array(append_targets(b), dtype=np.int64)  # (row, page, slot)
    flat = torch.from_numpy(targets[:, 1] * 16 + targets[:, 2]).to(DEV)
    rows = torch.from_numpy(targets[:, 0]).to(DEV)
    kp_before = t["k_pages"].clone()
    pl = plan_for(b)
    bt = torch.from_numpy(np.ascontiguousarray(b.block_table)).to(DEV)
    attn.kv_append(pl, kn, vn, bt, t["k_pages"], t["v_pages"])
    assert attn.check(pl) == 0
    pl.destroy()
    kflat = t["k_pages"].view(-1, b.num_kv_heads, b.head_dim)
    vflat = t["v_pages"].view(-1, b.num_kv_heads, b.head_dim)
    assert torch.equal(kflat[flat].view(torch.int16), kn[rows].view(torch.int16))
    assert torch.equal(vflat[flat].view(torch.int16), vn[rows].view(torch.int16))
    keep = torch.ones(kflat.shape[0], dtype=torch.bool, device=DEV)
    keep[flat] = False
    assert torch.equal(kflat[keep].view(torch.int16), kp_before.view(-1, b.num_kv_heads, b.head_dim)[keep].view(torch.int16))
    print(f"{name}: {len(targets)} rows appended", flush=True)


@pytest.mark.parametrize("seed", range(20))
def test_append_on_random_batches_bitwise(seed):
    """The seeded random batches of the attention parity test (head layouts,
    bf16 and fp32, request shapes with and without rows, tails of any
    length inside or across pages): the pool after the append equals the
    oracle's bit for bit, unused slots (NaN-poisoned) included."""
    import torch

    from tests.test_gpu_random_batches import random_batch

    b, _ = random_batch(seed)
    t = W.make_tensors_torch(b, DEV, poison_unused=True)
    kn, vn = _new_rows(b, seed=100 + seed)
    ref_k, ref_v = kv_append(b, _host(kn), _host(vn), _host(t["k_pages"]), _host(t["v_pages"]))
    pl = plan_for(b)
    bt = torch.from_numpy(np.ascontiguousarray(b.block_table)).to(DEV)
    attn.kv_append(pl, kn, vn, bt, t["k_pages"], t["v_pages"])
    assert attn.check(pl) == 0
    pl.destroy()
    assert np.array_equal(_host(t["k_pages"]).view(np.uint32), ref_k.view(np.uint32)), f"seed {seed}: K pages"
    assert np.array_equal(_host(t["v_pages"]).view(np.uint32), ref_v.view(np.uint32)), f"seed {seed}: V pages"
