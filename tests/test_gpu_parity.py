"""GPU parity: the HIP path through the C-ABI against the CPU fp64 oracle.

Tolerances (max-abs over every compared element, unit-variance inputs):
out 1e-5 (fp32) / 1.5e-2 (bf16), lse 1e-3 (natural log)."""
import numpy as np
import pytest

import workloads as W
from oracle import oracle_rows
from paper_2606_12688_amd import attn
from tests.helpers import TOL, compare, host64, oracle_of, plan_for, run_gpu

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
_host = host64
_compare = compare
_oracle = oracle_of


REDUCED = ["tiny_causal_f32", "decode_bf16", "text_latent_bf16", "stream_window_bf16", "rollout_bf16",
           "cfg_labels_bf16", "shared_prefix_decode_bf16", "serving_mix_bf16", "mixed", "window_edges_bf16",
           "queried_prefix_bf16"]
CASCADE = ["rollout_bf16", "cfg_labels_bf16", "shared_prefix_decode_bf16", "serving_mix_bf16", "mixed",
           "queried_prefix_bf16"]
FLAGS = {"auto": 0, "force_split": attn.FLAG_FORCE_SPLIT, "no_split": attn.FLAG_NO_SPLIT}


@pytest.mark.parametrize("flag", list(FLAGS))
@pytest.mark.parametrize("name", REDUCED)
def test_reduced_parity(name, flag):
    b = W.reduced(name)
    t = W.make_tensors_torch(b, DEV)
    out, lse = run_gpu(b, t, FLAGS[flag])
    ro, rl = _oracle(b, t)
    _compare(b, out, lse, ro, rl, f"{name}/{flag}")


@pytest.mark.parametrize("flag", list(FLAGS))
@pytest.mark.parametrize("name", CASCADE)
def test_cascade_parity(name, flag):
    """Shared-prefix cascade plans (prefix attended once for all members'
    rows, own keys separately, merged by log-sum-exp) against the oracle,
    every member in the cascade and (default) only the decode-like ones."""
    b = W.reduced(name)
    t = W.make_tensors_torch(b, DEV, poison_unused=True)
    ro, rl = _oracle(b, t)
    for extra, tag in ((attn.FLAG_CASCADE_ALL, "all"), (0, "default")):
        out, lse = run_gpu(b, t, FLAGS[flag] | extra, cascade=True)
        _compare(b, out, lse, ro, rl, f"{name}/cascade-{tag}/{flag}")


@pytest.mark.parametrize("name,cascade", [("serving_mix_bf16", False), ("serving_mix_bf16", True),
                                          ("mixed", False), ("shared_prefix_decode_bf16", True)])
def test_side_stream_fork_equals_serial_bitwise(name, cascade):
    """A plan with tile and few-row work runs the few-row kernel on a side
    stream; with MSTAR_FLAG_SERIAL everything runs on the caller's stream.  The
    kernels do the same arithmetic either way: bitwise equal outputs."""
    import torch

    b = W.reduced(name)
    t = W.make_tensors_torch(b, DEV)
    pl = plan_for(b, 0, cascade=cascade)
    st = pl.stats()
    assert st["decode_items"] > 0 and (st["prefill_items"] > 0 or len(pl.items(4)) > 0)  # forks or not
    pl.destroy()
    o1, l1 = run_gpu(b, t, 0, cascade=cascade)
    o2, l2 = run_gpu(b, t, attn.FLAG_SERIAL, cascade=cascade)
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(l1.view(torch.int32), l2.view(torch.int32))
    _compare(b, o1, l1, *_oracle(b, t), f"{name} fork")


@pytest.mark.parametrize("seed", [1, 2])
@pytest.mark.parametrize("name", ["tiny_causal_f32", "decode_bf16"])
def test_more_seeds(name, seed):
    b = W.reduced(name, seed)
    t = W.make_tensors_torch(b, DEV)
    out, lse = run_gpu(b, t)
    _compare(b, out, lse, *_oracle(b, t), f"{name}/seed{seed}")


@pytest.mark.parametrize("d,hq,hkv,dtype", [(64, 8, 2, "bf16"), (64, 4, 4, "bf16"), (128, 6, 6, "bf16"),
                                            (128, 12, 2, "bf16"), (64, 4, 2, "f32"), (128, 2, 1, "f32")])
def test_mixed_launch_head_layouts(d, hq, hkv, dtype):
    b = W.mixed(seed=3, hq=hq, hkv=hkv, d=d, dtype=dtype)
    t = W.make_tensors_torch(b, DEV)
    for flag in (0, attn.FLAG_FORCE_SPLIT):
        out, lse = run_gpu(b, t, flag)
        _compare(b, out, lse, *_oracle(b, t), f"mixed d{d} {hq}/{hkv} {dtype} flags{flag}")


def test_determinism_and_page_permutation_bitwise():
    import torch

    b = W.reduced("mixed")
    t = W.make_tensors_torch(b, DEV)
    o1, l1 = run_gpu(b, t)
    o2, l2 = run_gpu(b, t)
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(l1.view(torch.int32), l2.view(torch.int32))
    b2, t2 = W.permute_pages(b, t, seed=11)
    o3, l3 = run_gpu(b2, t2)
    assert torch.equal(o1.view(torch.int16), o3.view(torch.int16))
    assert torch.equal(l1.view(torch.int32), l3.view(torch.int32))


@pytest.mark.parametrize("flag", ["auto", "force_split"])
@pytest.mark.parametrize("name", ["mixed", "serving_mix_bf16", "decode_bf16"])
def test_repeated_launches_of_one_plan_write_every_output(name, flag):
    """Launches of one plan back to back (the mixed batches run the few-row
    kernel beside the tile kernel on the side stream), with the outputs
    NaN-filled before each: every launch writes every output, and all agree
    bitwise."""
    import torch

    b = W.reduced(name)
    t = W.make_tensors_torch(b, DEV)
    pl = plan_for(b, FLAGS[flag])
    assert pl.stats()["decode_items"] > 0
    q = t["q"]
    bt = torch.from_numpy(np.ascontiguousarray(b.block_table)).to(DEV)
    ws = attn.workspace(pl, DEV)
    outs = []
    for _ in range(6):
        out = torch.full_like(q, float("nan"))
        lse = torch.full((q.shape[0], b.num_qo_heads), float("nan"), dtype=torch.float32, device=DEV)
        attn.fwd(pl, q, t["k_pages"], t["v_pages"], bt, out, lse, ws)
        outs.append((out, lse))
    torch.cuda.synchronize()
    assert attn.check(pl) == 0
    pl.destroy()
    _compare(b, outs[0][0], outs[0][1], *_oracle(b, t), f"{name}/{flag} first launch")
    for i, (o, l) in enumerate(outs[1:], 1):
        assert torch.equal(o.view(torch.int16), outs[0][0].view(torch.int16)), f"launch {i}"
        assert torch.equal(l.view(torch.int32), outs[0][1].view(torch.int32)), f"launch {i}"


@pytest.mark.parametrize("name,cascade", [("mixed", False), ("serving_mix_bf16", False), ("mixed", True),
                                          ("decode_bf16", False)])
def test_pool_beyond_2gb_takes_per_page_resources(name, cascade):
    """A K/V pool larger than 2 GB takes the kernels' per-page buffer-resource
    path (one resource per page instead of one per pool).  The batch's pages
    are moved to the top of a pool of just over 2 GB (byte offsets past 2^31)
    and the results must equal the compact batch's bitwise."""
    import dataclasses

    import torch

    b = W.reduced(name)
    t = W.make_tensors_torch(b, DEV)
    o_ref, l_ref = run_gpu(b, t, attn.FLAG_FORCE_SPLIT, cascade=cascade)
    page_bytes = 16 * b.num_kv_heads * b.head_dim * 2
    big = (1 << 31) // page_bytes + b.num_pages + 64
    assert (big - b.num_pages) * page_bytes > (1 << 31)
    # page p -> big - 1 - p: every page sits past the 2 GB mark
    bt = b.block_table.copy()
    valid = bt >= 0
    bt[valid] = big - 1 - bt[valid]
    nb = dataclasses.replace(b, block_table=bt, num_pages=big)
    nt = dict(t)
    idx = torch.arange(big - 1, big - 1 - b.num_pages, -1, device=DEV)
    for k in ("k_pages", "v_pages"):
        x = torch.zeros((big,) + tuple(t[k].shape[1:]), dtype=t[k].dtype, device=DEV)
        x[idx] = t[k]
        nt[k] = x
    o, l = run_gpu(nb, nt, attn.FLAG_FORCE_SPLIT, cascade=cascade)
    assert torch.equal(o.view(torch.int16), o_ref.view(torch.int16))
    assert torch.equal(l.view(torch.int32), l_ref.view(torch.int32))
    del nt
    torch.cuda.empty_cache()


def test_unused_slots_poisoned_with_nan():
    for name in ("mixed", "decode_bf16", "rollout_bf16", "tiny_causal_f32"):
        b = W.reduced(name)
        t = W.make_tensors_torch(b, DEV, poison_unused=True)
        for flag in (0, attn.FLAG_FORCE_SPLIT):
            out, lse = run_gpu(b, t, flag)
            _compare(b, out, lse, *_oracle(b, t), f"{name} NaN-poisoned flags{flag}")


@pytest.mark.parametrize("name", ["decode_bf16", "mixed", "rollout_bf16", "text_latent_bf16"])
def test_out_of_range_page_sets_error_bit_without_reading(name):
    """Block-table entries past the pool or negative, on the few-row path
    (decode), the tile path at d = 64 (rollouts) and d = 128 (text+latent)
    and both in one launch (mixed): the device error bit is set, read and
    cleared, and every output stays finite (the bad pages read as zeros)."""
    import torch

    b = W.reduced(name)
    t = W.make_tensors_torch(b, DEV)
    bt = b.block_table.copy()
    for r in range(b.num_seqs):
        if b.seqs[r, 1] > 0:
            bt[r, 0] = b.num_pages + 5 if r % 2 == 0 else -3
    pl = plan_for(b)
    out = torch.zeros_like(t["q"])
    lse = torch.zeros(t["q"].shape[:2], dtype=torch.float32, device=DEV)
    attn.fwd(pl, t["q"], t["k_pages"], t["v_pages"], torch.from_numpy(bt).to(DEV), out, lse, attn.workspace(pl, DEV))
    assert attn.check(pl) == attn.DEVERR_PAGE_RANGE
    assert attn.check(pl) == 0  # the word was cleared
    assert torch.isfinite(out.float()).all()
    pl.destroy()


def test_fwd_rejects_wrong_shapes_and_small_workspace():
    import torch

    b = W.reduced("decode_bf16")
    t = W.make_tensors_torch(b, DEV)
    pl = plan_for(b, attn.FLAG_FORCE_SPLIT)
    bt = torch.from_numpy(b.block_table).to(DEV)
    out = torch.empty_like(t["q"])
    lse = torch.empty(t["q"].shape[:2], dtype=torch.float32, device=DEV)
    with pytest.raises(ValueError):
        attn.fwd(pl, t["q"][:-1], t["k_pages"], t["v_pages"], bt, out, lse, attn.workspace(pl, DEV))
    with pytest.raises(attn.MStarError) as ei:
        attn.fwd(pl, t["q"], t["k_pages"], t["v_pages"], bt, out, lse, None)
    assert ei.value.code == attn.ERR_WORKSPACE
    small = torch.empty(16, dtype=torch.uint8, device=DEV)
    rc = attn.lib().mstar_attn_fwd(pl.handle, t["q"].data_ptr(), t["k_pages"].data_ptr(), t["v_pages"].data_ptr(),
                                   bt.data_ptr(), out.data_ptr(), lse.data_ptr(), small.data_ptr(), 16, None)
    assert rc == attn.ERR_WORKSPACE
    pl.destroy()


# ---------------------------------------------------------------------------
# Full sizes: sampled outputs against the oracle, and a property of every row.
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("name,cascade", [("tiny_causal_f32", False), ("decode_bf16", False),
                                          ("text_latent_bf16", False), ("stream_window_bf16", False),
                                          ("rollout_bf16", False), ("cfg_labels_bf16", False),
                                          ("shared_prefix_decode_bf16", False), ("shared_prefix_decode_bf16", True),
                                          ("rollout_bf16", True), ("cfg_labels_bf16", True),
                                          ("serving_mix_bf16", False), ("serving_mix_bf16", True)])
def test_full_size_sampled(name, cascade):
    import torch

    b = W.FULL_SIZE[name]()
    print(f"{name}: generating", flush=True)
    t = W.make_tensors_torch(b, DEV)
    out, lse = run_gpu(b, t, attn.FLAG_CASCADE_ALL if cascade else 0, cascade=cascade)
    torch.cuda.synchronize()
    print(f"{name}: fwd done", flush=True)
    # every output is a convex combination of value rows
    vmax = float(t["v_pages"].float().abs().max())
    assert torch.isfinite(out.float()).all() and torch.isfinite(lse).all()
    assert float(out.float().abs().max()) <= vmax * (1 + 2 ** -7)
    rng = np.random.default_rng(7)
    n = b.num_seqs
    reqs = sorted({0, n - 1, *rng.choice(n, size=min(n, 4), replace=False).tolist()})
    sb, q, kp, vp, rows = W.extract_requests(b, t, reqs, _host)
    picks = []
    for j in range(sb.num_seqs):
        ql = int(sb.seqs[j, 0])
        for i in sorted({0, ql - 1, *rng.integers(0, ql, size=3).tolist()}):
            for h in sorted({0, b.num_qo_heads - 1, int(rng.integers(b.num_qo_heads))}):
                picks.append((j, i, h))
    ro, rl = oracle_rows(sb, q, kp, vp, picks)
    got_o = np.stack([_host(out[rows[sb.seqs[j, 2] + i], h]) for j, i, h in picks])
    got_l = np.array([float(lse[rows[sb.seqs[j, 2] + i], h]) for j, i, h in picks])
    tol_o, tol_l = TOL[b.dtype]
    eo, el = float(np.abs(got_o - ro).max()), float(np.abs(got_l - rl).max())
    print(f"{name} full size{' (cascade)' if cascade else ''}, {len(picks)} sampled rows: "
          f"max|dout|={eo:.3e} max|dlse|={el:.3e}", flush=True)
    assert eo <= tol_o and el <= tol_l


@pytest.mark.parametrize("flag", ["auto", "force_split"])
@pytest.mark.parametrize("name,rate,cascade", [("decode_bf16", 0.03, False), ("text_latent_bf16", 0.03, False),
                                               ("stream_window_bf16", 0.03, False), ("rollout_bf16", 0.05, False),
                                               ("decode_bf16", -0.0006, False),
                                               ("rollout_bf16", 0.5, False), ("text_latent_bf16", 0.5, False),
                                               ("shared_prefix_decode_bf16", 0.03, True),
                                               ("rollout_bf16", 0.05, True)])
def test_growing_scores_move_the_lazy_reference(name, rate, cascade, flag):
    """Keys scaled by 1 + rate * position: with rate > 0 a row's maximum keeps
    growing from tile to tile, by about the lazy threshold of 2^8 per 64-key
    tile, so the kernels both keep a stale reference (probabilities up to 2^8)
    and move it (rescaling O); split pieces then carry very different LSEs
    into the merge.  With rate < 0 the maximum sits in the first keys.  With
    rate 0.5 the scores of later tiles overflow fp32 against the reference of
    a row's first tile (2^100 and beyond), so the tile kernel's fixed-reference
    tiles must be redone in exact mode.

    Peaked rows return single V values of magnitude up to ~4.5, where storing
    the output in bf16 alone can be off by half a unit in the last place,
    2^-8 of the value (0.0156 at 4): the output bar is 1.5e-2 plus 2^-8 of
    the reference.  The lse bar is unchanged."""
    import torch

    b = W.reduced(name)
    t = W.make_tensors_torch(b, DEV)
    scale = np.ones((b.num_pages, 16), dtype=np.float32)
    bt = np.asarray(b.block_table)
    for r in range(bt.shape[0]):
        for j in range(bt.shape[1]):
            p = int(bt[r, j])
            if p >= 0:
                scale[p] = 1.0 + rate * (16 * j + np.arange(16))
    s = torch.from_numpy(scale).to(DEV)[:, :, None, None]
    t["k_pages"] = (t["k_pages"].float() * s).to(t["k_pages"].dtype)
    extra = attn.FLAG_CASCADE_ALL if cascade else 0
    out, lse = run_gpu(b, t, FLAGS[flag] | extra, cascade=cascade)
    ro, rl = _oracle(b, t)
    _compare(b, out, lse, ro, rl, f"{name}/rate {rate}/cascade {cascade}/{flag}", rel_o=2.0**-8)
