"""Shared test helpers: build plans from workload descriptors, run the HIP
path through the C-ABI binding, and compare with the CPU oracle.

Tolerances (max-abs over every compared element, unit-variance inputs):
out 1e-5 (fp32) / 1.5e-2 (bf16), lse 1e-3 (natural log)."""
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


TOL = {"f32": (1e-5, 1e-3), "bf16": (1.5e-2, 1e-3)}


def host64(t):
    """A torch tensor as a float64 numpy array on the host."""
    return t.float().cpu().numpy().astype(np.float64)


def compare(b, out, lse, ref_o, ref_l, label="", rel_o=0.0):
    """Max-abs errors of (out, lse) against the oracle's, within the bars
    above; rel_o widens the output bar by rel_o * |reference|."""
    tol_o, tol_l = TOL[b.dtype]
    o = out if isinstance(out, np.ndarray) else host64(out)
    l = lse if isinstance(lse, np.ndarray) else lse.cpu().numpy().astype(np.float64)
    assert np.isfinite(o).all(), f"{label}: non-finite output"
    assert np.isfinite(l).all(), f"{label}: non-finite lse"
    eo = float((np.abs(o - ref_o) - rel_o * np.abs(ref_o)).max()) if o.size else 0.0
    el = float(np.abs(l - ref_l).max()) if l.size else 0.0
    print(f"{label}: max|dout|={eo:.3e} max|dlse|={el:.3e} over {o.size} outputs", flush=True)
    assert eo <= tol_o, f"{label}: out error {eo} > {tol_o}"
    assert el <= tol_l, f"{label}: lse error {el} > {tol_l}"
    return eo, el


def oracle_of(b, t):
    """The oracle over a whole batch whose tensors live on the GPU."""
    from oracle import oracle_attention

    h = {k: host64(v) for k, v in t.items()}
    return oracle_attention(b, h["q"], h["k_pages"], h["v_pages"])
