"""Plans reuse pooled device buffers: a plan destroyed right after its fwd was
enqueued (no synchronization) hands its buffers to the next plan, whose upload
must wait on the device for that fwd before overwriting the work list.  Both
calls must give the results they give alone (bitwise), through the
synchronous planner and the asynchronous one."""
import numpy as np
import pytest

import workloads as W
from paper_2606_12688_amd import attn
from tests.helpers import compare, oracle_of, plan_for, run_gpu

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _block_class(nbytes):
    """Capacity of the pooled block a work list of `nbytes` takes: a power of two, at least 64 KiB."""
    cap = 64 << 10
    while cap < nbytes:
        cap <<= 1
    return cap


def _alloc(b, t):
    import torch

    out = torch.empty_like(t["q"])
    lse = torch.empty((t["q"].shape[0], b.num_qo_heads), dtype=torch.float32, device=DEV)
    bt = torch.from_numpy(np.ascontiguousarray(b.block_table)).to(DEV)
    return out, lse, bt


@pytest.mark.parametrize("first,second", [
    # full size: the first fwd (~2 ms) is still running when the second plan's upload is enqueued
    (("text_latent_bf16", {}), ("text_latent_bf16", {"latent": 4000})),
    (("rollout_bf16", {"n": 5, "prefix": 64, "frames": 4, "frame": 40}), ("mixed", {})),
])
def test_destroy_while_running_then_reuse(first, second):
    """Plan A's fwd is enqueued and A destroyed at once; plan B, whose work
    list takes a pooled block of the same capacity as A's, is uploaded on another
    stream and takes A's block (the most recently released among equally
    small ones), so only the wait on A's use event keeps B's upload from
    overwriting A's work list under the running kernel."""
    import torch

    stream = torch.cuda.current_stream()
    upload = torch.cuda.Stream()
    build = {"text_latent_bf16": W.text_latent_bf16, "rollout_bf16": W.rollout_bf16, "mixed": W.mixed}
    a, b = build[first[0]](**first[1]), build[second[0]](**second[1])
    ta, tb = W.make_tensors_torch(a, DEV), W.make_tensors_torch(b, DEV)
    ref_a = run_gpu(a, ta)
    ref_b = run_gpu(b, tb)
    for rep in range(3):
        pa = plan_for(a, 0, stream)
        oa, la, bta = _alloc(a, ta)
        attn.fwd(pa, ta["q"], ta["k_pages"], ta["v_pages"], bta, oa, la, attn.workspace(pa, DEV), stream)
        bytes_a = pa.stats()["device_bytes"]
        pa.destroy()  # no synchronization: the fwd may still be running
        pb = plan_for(b, 0, upload)  # its upload goes on another stream
        assert _block_class(bytes_a) == _block_class(pb.stats()["device_bytes"])
        stream.wait_stream(upload)
        ob, lb, btb = _alloc(b, tb)
        attn.fwd(pb, tb["q"], tb["k_pages"], tb["v_pages"], btb, ob, lb, attn.workspace(pb, DEV), stream)
        torch.cuda.synchronize()
        assert attn.check(pb) == 0
        pb.destroy()
        assert torch.equal(oa.view(torch.int16), ref_a[0].view(torch.int16)), f"rep {rep}: first call"
        assert torch.equal(la.view(torch.int32), ref_a[1].view(torch.int32))
        assert torch.equal(ob.view(torch.int16), ref_b[0].view(torch.int16)), f"rep {rep}: second call"
        assert torch.equal(lb.view(torch.int32), ref_b[1].view(torch.int32))
    compare(b, ob, lb, *oracle_of(b, tb), f"{second[0]} after {first[0]}")


def test_async_planner_reuses_buffers_of_plans_destroyed_in_flight():
    import torch

    stream = torch.cuda.current_stream()
    names = ["mixed", "decode_bf16", "rollout_bf16", "mixed", "stream_window_bf16", "decode_bf16"]
    batches = [W.reduced(n, seed=i) for i, n in enumerate(names)]
    tens = [W.make_tensors_torch(bb, DEV) for bb in batches]
    refs = [run_gpu(bb, tt) for bb, tt in zip(batches, tens)]

    def args(bb):
        return (bb.num_qo_heads, bb.num_kv_heads, bb.head_dim, bb.dtype, bb.seqs, bb.masks, bb.segments,
                bb.block_table.shape[1], bb.num_pages, bb.sm_scale, 0)

    ap = attn.AsyncPlanner(depth=2)
    ap.submit(*args(batches[0]))
    outs = []
    for i, bb in enumerate(batches):
        if i + 1 < len(batches):
            ap.submit(*args(batches[i + 1]))
        pl = ap.take(stream)
        o, l, bt = _alloc(bb, tens[i])
        attn.fwd(pl, tens[i]["q"], tens[i]["k_pages"], tens[i]["v_pages"], bt, o, l, attn.workspace(pl, DEV), stream)
        pl.destroy()  # in flight; the worker may hand its buffers to the next plan
        outs.append((o, l))
    torch.cuda.synchronize()
    ap.close()
    for i, ((o, l), (ro, rl)) in enumerate(zip(outs, refs)):
        assert torch.equal(o.view(torch.int16), ro.view(torch.int16)), f"step {i} {names[i]}"
        assert torch.equal(l.view(torch.int32), rl.view(torch.int32)), f"step {i} {names[i]}"
