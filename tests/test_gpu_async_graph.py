"""GPU tests of asynchronous planning and graph capture: a serving loop that
builds each step's plan on the planner's thread and stream while the previous
step runs (results against the oracle; plain and shared-prefix cascade plans),
and kv_append + fwd captured in a HIP graph, replayed with eager work in
between, every replay bitwise equal to the eager call."""
import numpy as np
import pytest

import workloads as W
from oracle import oracle_attention
from paper_2606_12688_amd import attn
from tests.helpers import plan_for

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _host(t):
    return t.float().cpu().numpy().astype(np.float64)


def _args(b, flags=0):
    return (b.num_qo_heads, b.num_kv_heads, b.head_dim, b.dtype, b.seqs, b.masks, b.segments,
            b.block_table.shape[1], b.num_pages, b.sm_scale, flags)


def test_async_planner_serving_loop_against_oracle():
    import torch

    steps = [W.reduced(n, seed=s) for s, n in enumerate(
        ["decode_bf16", "mixed", "rollout_bf16", "stream_window_bf16", "cfg_labels_bf16", "text_latent_bf16",
         "shared_prefix_decode_bf16", "rollout_bf16"])]
    # the last two steps are planned as shared-prefix cascades (the second with every member in)
    cascade = {6: 0, 7: attn.FLAG_CASCADE_ALL}

    def submit(i):
        b = steps[i]
        if i in cascade:
            ap.submit(*_args(b, cascade[i]), prefix_groups=b.prefix_groups)
        else:
            ap.submit(*_args(b))

    stream = torch.cuda.current_stream()
    ap = attn.AsyncPlanner(depth=2)
    submit(0)
    for i, b in enumerate(steps):
        t = W.make_tensors_torch(b, DEV)
        if i + 1 < len(steps):
            submit(i + 1)  # planned on the worker while this step runs
        pl = ap.take(stream)                 # the stream waits for the upload on the device
        out = torch.empty_like(t["q"])
        lse = torch.empty(t["q"].shape[:2], dtype=torch.float32, device=DEV)
        bt = torch.from_numpy(np.ascontiguousarray(b.block_table)).to(DEV)
        attn.fwd(pl, t["q"], t["k_pages"], t["v_pages"], bt, out, lse, attn.workspace(pl, DEV), stream)
        assert attn.check(pl, stream) == 0
        pl.destroy()
        h = {k: _host(v) for k, v in t.items()}
        ro, rl = oracle_attention(b, h["q"], h["k_pages"], h["v_pages"])
        eo, el = float(np.abs(_host(out) - ro).max()), float(np.abs(lse.cpu().numpy() - rl).max())
        print(f"step {i} {b.name}: max|dout|={eo:.3e} max|dlse|={el:.3e}", flush=True)
        assert eo <= 1.5e-2 and el <= 1e-3
    ap.close()


@pytest.mark.parametrize("name,flags,cascade", [("mixed", 0, False), ("decode_bf16", attn.FLAG_FORCE_SPLIT, False),
                                                ("rollout_bf16", 0, False), ("shared_prefix_decode_bf16", 0, True),
                                                ("rollout_bf16", attn.FLAG_CASCADE_ALL, True)])
def test_append_and_fwd_captured_in_a_graph_replay_bitwise(name, flags, cascade):
    import torch

    b = W.reduced(name)
    t = W.make_tensors_torch(b, DEV)
    g0 = torch.Generator(device=DEV)
    g0.manual_seed(5)
    kn = torch.randn((b.total_q, b.num_kv_heads, b.head_dim), generator=g0, device=DEV).to(torch.bfloat16)
    vn = torch.randn((b.total_q, b.num_kv_heads, b.head_dim), generator=g0, device=DEV).to(torch.bfloat16)
    pl = plan_for(b, flags, cascade=cascade)
    bt = torch.from_numpy(np.ascontiguousarray(b.block_table)).to(DEV)
    ws = attn.workspace(pl, DEV)
    out = torch.empty_like(t["q"])
    lse = torch.empty(t["q"].shape[:2], dtype=torch.float32, device=DEV)

    def step(stream=None):
        attn.kv_append(pl, kn, vn, bt, t["k_pages"], t["v_pages"], stream)
        attn.fwd(pl, t["q"], t["k_pages"], t["v_pages"], bt, out, lse, ws, stream)

    step()
    torch.cuda.synchronize()
    ref_o, ref_l = out.clone(), lse.clone()
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        with torch.cuda.graph(graph, stream=side):
            step(side)
    torch.cuda.current_stream().wait_stream(side)
    for rep in range(4):
        out.zero_()  # eager work between replays, on the same tensors
        lse.fill_(float("nan"))
        scratch = torch.randn(1 << 16, device=DEV).sum()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), ref_o.view(torch.int16)), f"replay {rep}"
        assert torch.equal(lse.view(torch.int32), ref_l.view(torch.int32)), f"replay {rep}"
        assert torch.isfinite(scratch)
    assert attn.check(pl) == 0
    del graph
    pl.destroy()
