"""Host-side tests of the asynchronous, double-buffered planner (no GPU
needed: host-only plans make no HIP call): plans come back in submission order
and equal synchronous plans, submit blocks at the depth, errors surface at
take, and submit/take work from different threads."""
import threading
import time

import numpy as np
import pytest

import workloads as W
from paper_2606_12688_amd import attn
from tests.helpers import plan_for

NAMES = ["decode_bf16", "text_latent_bf16", "stream_window_bf16", "rollout_bf16", "cfg_labels_bf16", "mixed",
         "tiny_causal_f32"]


def _args(b, flags=attn.FLAG_HOST_ONLY):
    return (b.num_qo_heads, b.num_kv_heads, b.head_dim, b.dtype, b.seqs, b.masks, b.segments,
            b.block_table.shape[1], b.num_pages, b.sm_scale, flags)


def _same(p1, p2):
    for kind in range(4):
        assert np.array_equal(p1.items(kind), p2.items(kind))
    assert np.array_equal(p1.tile_order(), p2.tile_order())
    s1, s2 = p1.stats(), p2.stats()
    for k in ("visible_pairs", "prefill_items", "decode_items", "f32_items", "merge_rows", "partial_slots"):
        assert s1[k] == s2[k]


def test_plans_come_back_in_order_and_equal_synchronous_plans():
    batches = [W.reduced(n) for n in NAMES]
    ap = attn.AsyncPlanner(depth=2)
    ap.submit(*_args(batches[0]))
    for i, b in enumerate(batches):
        if i + 1 < len(batches):
            ap.submit(*_args(batches[i + 1]))  # the next batch is planned while this one "runs"
        got = ap.take()
        ref = plan_for(b, attn.FLAG_HOST_ONLY)
        _same(got, ref)
        got.destroy()
        ref.destroy()
    ap.close()


def test_submit_blocks_at_depth_until_a_take():
    b = W.reduced("mixed")
    ap = attn.AsyncPlanner(depth=2)
    ap.submit(*_args(b))
    ap.submit(*_args(b))
    done = threading.Event()

    def third():
        ap.submit(*_args(b))
        done.set()

    th = threading.Thread(target=third)
    th.start()
    time.sleep(0.3)
    assert not done.is_set()  # two outstanding: the third waits
    ap.take().destroy()
    th.join(timeout=10)
    assert done.is_set()
    ap.take().destroy()
    ap.take().destroy()
    ap.close()


def test_planning_error_surfaces_at_take_and_the_planner_goes_on():
    good = W.reduced("decode_bf16")
    bad = W.reduced("decode_bf16")
    seqs = bad.seqs.copy()
    seqs[0, 0] = seqs[0, 1] + 1  # q_len > kv_len
    ap = attn.AsyncPlanner(depth=2)
    ap.submit(*((good.num_qo_heads, good.num_kv_heads, good.head_dim, good.dtype, seqs) + _args(good)[5:]))
    ap.submit(*_args(good))
    with pytest.raises(attn.MStarError) as ei:
        ap.take()
    assert ei.value.code == attn.ERR_INVALID_ARG and "q_len" in str(ei.value)
    p = ap.take()
    ref = plan_for(good, attn.FLAG_HOST_ONLY)
    _same(p, ref)
    p.destroy()
    ref.destroy()
    with pytest.raises(attn.MStarError):
        ap.take()  # nothing outstanding
    ap.close()


def test_submit_and_take_from_different_threads():
    batches = [W.reduced(n, seed=s) for s in range(3) for n in ("decode_bf16", "mixed")]
    ap = attn.AsyncPlanner(depth=2)
    errors = []

    def producer():
        try:
            for b in batches:
                ap.submit(*_args(b))
        except Exception as e:  # pragma: no cover
            errors.append(e)

    th = threading.Thread(target=producer)
    th.start()
    for b in batches:
        while not ap._pending:  # the Python side records a submit after the C call returns
            time.sleep(0.001)
        got = ap.take()
        ref = plan_for(b, attn.FLAG_HOST_ONLY)
        _same(got, ref)
        got.destroy()
        ref.destroy()
    th.join(timeout=10)
    assert not errors
    ap.close()


def test_close_with_untaken_plans_releases_them():
    ap = attn.AsyncPlanner(depth=3)
    for n in ("decode_bf16", "mixed", "rollout_bf16"):
        ap.submit(*_args(W.reduced(n)))
    ap.close()  # joins the worker and destroys the three plans


@pytest.mark.parametrize("name", ["shared_prefix_decode_bf16", "rollout_bf16", "mixed"])
def test_cascade_plans_through_the_planner_equal_synchronous_ones(name):
    """mstar_planner_submit_cascade builds the same plan as mstar_attn_plan_cascade."""
    b = W.reduced(name)
    ap = attn.AsyncPlanner(depth=2)
    for flags in (attn.FLAG_HOST_ONLY, attn.FLAG_HOST_ONLY | attn.FLAG_CASCADE_ALL):
        ap.submit(*_args(b, flags), prefix_groups=b.prefix_groups)
        got = ap.take()
        ref = plan_for(b, flags, cascade=True)
        _same(got, ref)
        for kind in (4, 5):
            assert np.array_equal(got.items(kind), ref.items(kind))
        assert np.array_equal(got.tile_order(cascade=True), ref.tile_order(cascade=True))
        got.destroy()
        ref.destroy()
    with pytest.raises(attn.MStarError):  # a bad group surfaces at take
        ap.submit(*_args(b), prefix_groups=[([0, 0], 64)])
        ap.take()
    ap.close()
