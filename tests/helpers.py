"""Shared test helpers: build plans from workload descriptors and run the HIP
path through the C-ABI binding."""
import numpy as np

from paper_2606_12688_amd import attn


def plan_for(b, flags=0, stream=None, cascade=False):
    """Plan for a workload batch; with ``cascade`` its shared-prefix groups go to
    mstar_attn_plan_cascade."""
    return attn.plan(b.num_qo_heads, b.num_kv_heads, b.head_dim, b.dtype, b.seqs, b.masks, b.segments,
                     b.block_table.shape[1], b.num_pages, b.sm_scale, flags, stream,
                     prefix_groups=b.prefix_groups if cascade else None)


def run_gpu(b, tensors, flags=0, device="cuda:0", out_fill=None, cascade=False):
    """Plan + fwd on the GPU; returns (out, lse) as torch tensors on the device."""
    import torch

    pl = plan_for(b, flags, cascade=cascade)
    q = tensors["q"]
    out = torch.empty_like(q) if out_fill is None else torch.full_like(q, out_fill)
    lse = torch.full((q.shape[0], b.num_qo_heads), float("nan"), dtype=torch.float32, device=device)
    bt = torch.from_numpy(np.ascontiguousarray(b.block_table)).to(device)
    ws = attn.workspace(pl, device)
    attn.fwd(pl, q, tensors["k_pages"], tensors["v_pages"], bt, out, lse, ws)
    bits = attn.check(pl)
    assert bits == 0, f"device error bits {bits}"
    pl.destroy()
    return out, lse
