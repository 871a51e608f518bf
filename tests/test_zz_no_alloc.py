"""The allocation-free entry point (mstar_attn_fwd_noalloc) against the
workspace entry point (mstar_attn_fwd), through the C-ABI.

Two calls in a row share the library's static device scratch: a split plan
first, then a smaller one, each bitwise equal to mstar_attn_fwd with a caller
workspace on the same plan (the kernels are the same; only where the partials
live differs) and within the oracle bars.  A plan needing more scratch than the
array holds is refused before anything is enqueued."""
import numpy as np
import pytest

import workloads as W
from paper_2606_12688_amd import attn
from tests.helpers import compare, oracle_of, plan_for

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _call(fn, b, t, pl, stream, ws=None):
    import torch

    out = torch.full_like(t["q"], float("nan"))
    lse = torch.full((t["q"].shape[0], b.num_qo_heads), float("nan"), dtype=torch.float32, device=DEV)
    bt = torch.from_numpy(np.ascontiguousarray(b.block_table)).to(DEV)
    L = attn.lib()
    ptrs = (pl.handle, t["q"].data_ptr(), t["k_pages"].data_ptr(), t["v_pages"].data_ptr(), bt.data_ptr(),
            out.data_ptr(), lse.data_ptr())
    if fn == "noalloc":
        rc = L.mstar_attn_fwd_noalloc(*ptrs, stream.cuda_stream)
    else:
        rc = L.mstar_attn_fwd(*ptrs, ws.data_ptr() if ws is not None else None,
                              ws.numel() if ws is not None else 0, stream.cuda_stream)
    assert rc == 0, attn.last_error()
    assert attn.check(pl, stream) == 0
    return out, lse


def test_noalloc_equals_workspace_entry_point_on_two_calls():
    import torch

    stream = torch.cuda.current_stream()
    # first a plan with many split partials, then a smaller one: the second
    # call finds the first call's partials in the scratch and must not read them
    cases = [(W.reduced("serving_mix_bf16"), attn.FLAG_FORCE_SPLIT, True),
             (W.reduced("decode_bf16"), attn.FLAG_FORCE_SPLIT, False)]
    sizes = []
    for b, flags, cascade in cases:
        t = W.make_tensors_torch(b, DEV)
        pl = plan_for(b, flags, stream, cascade=cascade)
        need = pl.workspace_bytes
        assert 0 < need <= 32 << 20
        sizes.append(need)
        ws = attn.workspace(pl, DEV)
        o_ref, l_ref = _call("fwd", b, t, pl, stream, ws)
        o, l = _call("noalloc", b, t, pl, stream)
        assert torch.equal(o.view(torch.int16), o_ref.view(torch.int16))
        assert torch.equal(l.view(torch.int32), l_ref.view(torch.int32))
        compare(b, o, l, *oracle_of(b, t), f"noalloc {b.name} flags {flags}")
        pl.destroy()
    assert sizes[1] < sizes[0]


def test_noalloc_refuses_a_plan_beyond_the_scratch():
    import torch

    stream = torch.cuda.current_stream()
    b = W.FULL_SIZE["decode_bf16"]()
    pl = plan_for(b, attn.FLAG_FORCE_SPLIT, stream)
    assert pl.workspace_bytes > 32 << 20
    t = W.make_tensors_torch(b, DEV)  # tensors of the planned shapes: the refusal is the only thing tested
    bt = torch.from_numpy(np.ascontiguousarray(b.block_table)).to(DEV)
    out = torch.empty_like(t["q"])
    lse = torch.empty((b.total_q, b.num_qo_heads), dtype=torch.float32, device=DEV)
    rc = attn.lib().mstar_attn_fwd_noalloc(pl.handle, t["q"].data_ptr(), t["k_pages"].data_ptr(),
                                           t["v_pages"].data_ptr(), bt.data_ptr(), out.data_ptr(), lse.data_ptr(),
                                           stream.cuda_stream)
    assert rc == attn.ERR_WORKSPACE
    assert "scratch" in attn.last_error()
    torch.cuda.synchronize()
    pl.destroy()
