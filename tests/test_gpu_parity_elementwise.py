"""Element-wise GPU parity where sampled rows are not enough.

Every output (all rows, all heads, out and lse) is compared with the CPU fp64
oracle for:

* long work items: tile items over 2048 keys, where the tile kernel refills
  the third window of its page-index ring, and few-row items over 4096 keys,
  where a wave's page indices span more than one register window (planned
  without key splitting so that each request stays one item, and also with
  the default and forced splitting);
* sliding windows at their small edges (1 key, fewer keys than a page, one
  page, one more) on the few-row and the tile path, for several head layouts;
* the whole full-size launches of the tiny fp32, decode and streaming-chunk
  workloads (the oracle reads only the pages holding visible keys);
* whole requests (every row and head) of the full-size text+latent, rollout
  and CFG-label launches: the requests of the first and the last workgroup
  in launch order.

Bars as in the other parity tests: out 1e-5 (fp32) / 1.5e-2 (bf16), lse 1e-3.
"""
import numpy as np
import pytest

import workloads as W
from oracle import oracle_attention
from paper_2606_12688_amd import attn
from tests.helpers import compare, host64, oracle_of, plan_for, run_gpu

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
FLAGS = {"no_split": attn.FLAG_NO_SPLIT, "auto": 0, "force_split": attn.FLAG_FORCE_SPLIT}


def _longest(b, flags, kind):
    pl = plan_for(b, flags | attn.FLAG_HOST_ONLY)
    it = pl.items(kind)
    pl.destroy()
    return int((it[:, 5] - it[:, 4]).max()) if len(it) else 0


@pytest.mark.parametrize("flag", list(FLAGS))
@pytest.mark.parametrize("name", W.LONG_ITEMS)
def test_long_items_every_output(name, flag):
    b = W.long_items(name)
    if flag == "no_split":  # the long-item paths are reached
        if name in ("text_latent_long", "rollout_long"):
            assert _longest(b, FLAGS[flag], 0) > 2048
        else:
            assert _longest(b, FLAGS[flag], 1) > 4096
    print(f"{name}/{flag}: {b.num_seqs} requests, kv_len up to {int(b.seqs[:, 1].max())}", flush=True)
    t = W.make_tensors_torch(b, DEV)
    out, lse = run_gpu(b, t, FLAGS[flag])
    compare(b, out, lse, *oracle_of(b, t), f"{name}/{flag}")


@pytest.mark.parametrize("flag", list(FLAGS))
@pytest.mark.parametrize("d,hq,hkv", [(128, 16, 8), (64, 8, 8), (128, 28, 4), (64, 16, 2)])
def test_window_edges_every_output(d, hq, hkv, flag):
    b = W.window_edges_bf16(seed=1, d=d, hq=hq, hkv=hkv)
    pl = plan_for(b, FLAGS[flag] | attn.FLAG_HOST_ONLY)
    st = pl.stats()
    pl.destroy()
    assert st["prefill_items"] > 0 and st["decode_items"] > 0  # both paths see the windows
    print(f"window edges d{d} {hq}/{hkv} {flag}: {st['prefill_items']} tile, {st['decode_items']} few-row items",
          flush=True)
    t = W.make_tensors_torch(b, DEV)
    out, lse = run_gpu(b, t, FLAGS[flag])
    compare(b, out, lse, *oracle_of(b, t), f"window edges d{d} {hq}/{hkv} {flag}")


def _compare_requests(b, t, out, lse, reqs, key_ranges, label):
    sb, q, kp, vp, rows = W.extract_requests(b, t, reqs, host64, key_ranges=key_ranges)
    ro, rl = oracle_attention(sb, q, kp, vp)
    import torch

    idx = torch.from_numpy(rows).to(out.device)
    return compare(b, out.index_select(0, idx), lse.index_select(0, idx), ro, rl, label)


# configurations 1 and 2 also at seeds 1 and 2 (new values and page permutation; new lengths for decode)
@pytest.mark.parametrize("name,seed", [("tiny_causal_f32", 0), ("tiny_causal_f32", 1), ("tiny_causal_f32", 2),
                                       ("decode_bf16", 0), ("decode_bf16", 1), ("decode_bf16", 2),
                                       ("stream_window_bf16", 0)])
def test_full_size_launch_every_output(name, seed):
    import torch

    b = W.FULL_SIZE[name](seed)
    print(f"{name} seed {seed}: generating", flush=True)
    t = W.make_tensors_torch(b, DEV)
    out, lse = run_gpu(b, t)
    torch.cuda.synchronize()
    pl = plan_for(b, attn.FLAG_HOST_ONLY)
    kr = pl.key_ranges()
    pl.destroy()
    worst = [0.0, 0.0]
    for chunk in np.array_split(np.arange(b.num_seqs), max(1, b.num_seqs // 32)):
        eo, el = _compare_requests(b, t, out, lse, chunk, kr[chunk], f"{name} requests {chunk[0]}..{chunk[-1]}")
        worst = [max(worst[0], eo), max(worst[1], el)]
    print(f"{name} seed {seed} full launch, every output: max|dout|={worst[0]:.3e} max|dlse|={worst[1]:.3e}",
          flush=True)


@pytest.mark.parametrize("name,which", [("text_latent_bf16", "first"), ("text_latent_bf16", "last"),
                                        ("rollout_bf16", "first"), ("rollout_bf16", "last"),
                                        ("cfg_labels_bf16", "first")])
def test_full_size_first_and_last_requests_every_output(name, which):
    """One whole request (every row and head) of a full-size launch: the one
    the first or the last workgroup in launch order works on.  One request
    per test keeps each oracle run within tens of seconds."""
    import torch

    b = W.FULL_SIZE[name]()
    print(f"{name}: generating", flush=True)
    t = W.make_tensors_torch(b, DEV)
    out, lse = run_gpu(b, t)
    torch.cuda.synchronize()
    pl = plan_for(b, attn.FLAG_HOST_ONLY)
    order, items = pl.tile_order(), pl.items(0)
    pl.destroy()
    live = order[order[:, 0] >= 0]
    r = int(items[live[0 if which == "first" else -1, 0], 0])
    print(f"{name}: oracle of request {r} ({int(b.seqs[r, 0])} rows x {b.num_qo_heads} heads)", flush=True)
    _compare_requests(b, t, out, lse, [r], None, f"{name} request {r} ({which} in launch order), every row and head")
