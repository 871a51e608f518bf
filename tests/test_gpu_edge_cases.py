"""GPU edge cases of the batch descriptors: an empty batch, requests without
query rows (with and without cached keys) between ordinary ones, single-key
requests, and a request whose rows each see one key, on the bf16 tile and
few-row paths and the fp32 path, under every split policy.  Outputs are
pre-filled with NaN, so a row the kernels skip fails the comparison."""
import numpy as np
import pytest

import workloads as W
from paper_2606_12688_amd import attn
from tests.helpers import compare, oracle_of, plan_for, run_gpu

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
FLAGS = {"auto": 0, "force_split": attn.FLAG_FORCE_SPLIT, "no_split": attn.FLAG_NO_SPLIT}
C = W.SEG_CAUSAL


def _zero_query_batch(d, hq, hkv, dtype):
    """Requests with q_len = 0 (kv_len 0, 40 and 700) around a decode token, a
    16-token chunk, a 200-row prefill and a one-token first step."""
    q_lens = [0, 1, 0, 16, 0, 200, 1]
    kv_lens = [0, 33, 40, 90, 700, 200, 1]
    segs = [[] if L == 0 else [(0, L, C, 0)] for L in kv_lens]
    return W.custom(f"zero_query_{dtype}_d{d}", hq, hkv, d, q_lens, kv_lens, segs, [0] * len(q_lens), seed=3,
                    dtype=dtype)


def _one_key_batch(d, hq, hkv, dtype):
    """Every row sees exactly one key: single-token requests over one cached
    key, and a 150-row prefill with a window of one."""
    q_lens = [1, 1, 150, 1]
    kv_lens = [1, 1, 150, 1]
    segs = [[(0, L, C, 0)] for L in kv_lens]
    return W.custom(f"one_key_{dtype}_d{d}", hq, hkv, d, q_lens, kv_lens, segs, [0, 0, 1, 0], seed=5, dtype=dtype)


SHAPES = [(64, 8, 2, "bf16"), (128, 4, 4, "bf16"), (128, 28, 4, "bf16"), (64, 2, 1, "f32")]


@pytest.mark.parametrize("flag", list(FLAGS))
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"d{s[0]}-{s[1]}x{s[2]}-{s[3]}")
@pytest.mark.parametrize("build", [_zero_query_batch, _one_key_batch], ids=["zero_query", "one_key"])
def test_degenerate_requests(build, shape, flag):
    b = build(*shape)
    t = W.make_tensors_torch(b, DEV)
    out, lse = run_gpu(b, t, FLAGS[flag], out_fill=float("nan"))
    compare(b, out, lse, *oracle_of(b, t), f"{b.name}/{flag}")
    if build is _one_key_batch:
        # one visible key: out is that key's V row exactly (up to the output
        # rounding), whatever the scores
        ro, _ = oracle_of(b, t)
        assert np.abs(out.float().cpu().numpy() - ro).max() <= (1e-6 if shape[3] == "f32" else 2 ** -8)


@pytest.mark.parametrize("d", [64, 128])
def test_empty_batch_runs_nothing(d):
    import torch

    p = dict(num_qo_heads=4, num_kv_heads=2, head_dim=d, dtype="bf16", seqs=np.zeros((0, 3), np.int32),
             masks=np.zeros((0, 3), np.int32), segments=np.zeros((0, 4), np.int32), max_blocks_per_seq=1,
             num_pages=1, sm_scale=d ** -0.5, flags=0)
    pl = attn.plan(**p)
    assert pl.stats()["total_q"] == 0 and pl.workspace_bytes == 0
    q = torch.zeros((0, 4, d), dtype=torch.bfloat16, device=DEV)
    kv = torch.zeros((1, 16, 2, d), dtype=torch.bfloat16, device=DEV)
    out = torch.zeros_like(q)
    lse = torch.zeros((0, 4), dtype=torch.float32, device=DEV)
    bt = torch.zeros((0, 1), dtype=torch.int32, device=DEV)
    attn.fwd(pl, q, kv, kv, bt, out, lse, None)
    torch.cuda.synchronize()
    assert attn.check(pl) == 0
    pl.destroy()


def test_zero_query_requests_leave_their_neighbours_rows_alone():
    """Requests without rows sit between others in the packed row space: every
    written row belongs to a request with rows (the rows of the others are
    all written, and nothing is written past total_q)."""
    import torch

    b = _zero_query_batch(128, 28, 4, "bf16")
    t = W.make_tensors_torch(b, DEV)
    pl = plan_for(b, 0)
    total_q = int(pl.stats()["total_q"])
    assert total_q == int(b.seqs[:, 0].sum())
    q = t["q"]
    pad = 8
    out = torch.full((total_q + pad,) + tuple(q.shape[1:]), float("nan"), dtype=q.dtype, device=DEV)
    lse = torch.full((total_q + pad, b.num_qo_heads), float("nan"), dtype=torch.float32, device=DEV)
    bt = torch.from_numpy(np.ascontiguousarray(b.block_table)).to(DEV)
    attn.fwd(pl, q, t["k_pages"], t["v_pages"], bt, out[:total_q], lse[:total_q], attn.workspace(pl, DEV))
    torch.cuda.synchronize()
    assert attn.check(pl) == 0
    pl.destroy()
    assert torch.isnan(out[total_q:].float()).all() and torch.isnan(lse[total_q:]).all()
    compare(b, out[:total_q], lse[:total_q], *oracle_of(b, t), "zero_query neighbours")


@pytest.mark.parametrize("cascade", [False, True], ids=["plain", "cascade"])
@pytest.mark.parametrize("flag", list(FLAGS))
def test_request_rows_in_any_order_with_gaps(flag, cascade):
    """Requests may place their packed rows anywhere in q / out / lse: here in
    reverse request order with gaps of one to three rows between them and
    before the first.  Every row of a request matches the oracle and every
    row of no request keeps its NaN fill (plain plans, and cascades with
    every group member joined)."""
    import dataclasses

    import torch

    base = W.mixed(seed=4)
    seqs = base.seqs.copy()
    pos = 5
    for r in reversed(range(base.num_seqs)):
        seqs[r, 2] = pos
        pos += int(seqs[r, 0]) + 1 + r % 3
    b = dataclasses.replace(base, seqs=seqs, name="mixed_scattered_rows")
    t = W.make_tensors_torch(b, DEV)
    # as a cascade every member of the shared-prefix group joins it
    flags = FLAGS[flag] | (attn.FLAG_CASCADE_ALL if cascade else 0)
    out, lse = run_gpu(b, t, flags, out_fill=float("nan"), cascade=cascade)
    rows = np.concatenate([np.arange(qs, qs + ql) for ql, _, qs in seqs.tolist()])
    gaps = np.setdiff1d(np.arange(b.total_q), rows)
    assert len(gaps) > 0
    g = torch.from_numpy(gaps).to(DEV)
    assert torch.isnan(out.index_select(0, g).float()).all() and torch.isnan(lse.index_select(0, g)).all()
    ro, rl = oracle_of(b, t)
    idx = torch.from_numpy(rows).to(DEV)
    compare(b, out.index_select(0, idx), lse.index_select(0, idx), ro[rows], rl[rows], f"{b.name}/{flag}/cascade={cascade}")
