#!/usr/bin/env python
"""Benchmark of batched paged-KV attention with per-request masks on one MI355X.

    python bench.py [--gpus 1] [--steps 50] [--warmup 10] [--workload decode_bf16]

A step is one ``mstar_attn_fwd`` over one synthetic batch (every kernel of the
path: page-table gather, masked tile or few-row attention, split-K merge).
The plan (mask descriptors -> row intervals -> work list -> upload) is built
once before the timed region, as the serving runtime builds it off the
critical path; its host time is reported separately as ``plan_host_us``.

Inputs are resident in HBM before timing starts.  Several copies of Q/K/V
are rotated from step to step so that the 256 MB Infinity Cache cannot serve
one step's K/V reads from the previous step.

Prints ONE JSON line.  ``value`` is the whole-job rate in the metric's unit
for the workload's bound: KV-read GB/s for HBM-bound workloads (decode,
streaming chunks), useful TFLOP/s for MFMA-bound ones (prefill, rollouts, CFG
labels).
Useful FLOPs are 4 * head_dim per visible (row, key) pair per query head;
KV bytes count every distinct visible key of a request and KV head once for
K and once for V, pages shared between requests once.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "attention useful TFLOP/s and KV-read HBM GB/s, as fraction of MI355X peak"
PEAK_HBM_GBS = 8000.0
PEAK_BF16_TFLOPS = 2516.6   # dense MFMA: 256 CU x 2.4 GHz x 4096 FLOP/clk
PEAK_FP32_TFLOPS = 157.3
BOUND = {"tiny_causal_f32": "alu", "decode_bf16": "hbm", "text_latent_bf16": "mfma",
         "stream_window_bf16": "hbm", "rollout_bf16": "mfma", "cfg_labels_bf16": "mfma",
         "shared_prefix_decode_bf16": "hbm", "serving_mix_bf16": "mfma"}
# kernel classes of mstar_attn_fwd_timed: 0 multi-row tiles, 1 few-row items, 2 fp32, 3 merge, 4 cascade
KERNEL_NAMES = ["tile_kernel", "few_kernel", "f32_kernel", "merge_kernel", "cascade_kernel"]
DOMINANT = {"tiny_causal_f32": 2, "decode_bf16": 1, "text_latent_bf16": 0, "stream_window_bf16": 1,
            "rollout_bf16": 0, "cfg_labels_bf16": 0, "shared_prefix_decode_bf16": 1, "serving_mix_bf16": 0}
KERNEL_SRC = os.path.join(ROOT, "paper_2606_12688_amd", "csrc", "kernels.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def kernel_source_sha() -> str:
    with open(KERNEL_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def kv_bytes(b, key_ranges) -> int:
    """Distinct visible K and V rows (shared pages once) times their size."""
    slots = []
    for r in range(b.num_seqs):
        lo, hi = int(key_ranges[r, 0]), int(key_ranges[r, 1])
        if hi <= lo:
            continue
        t = np.arange(lo, hi, dtype=np.int64)
        slots.append(b.block_table[r, t // b.page_size].astype(np.int64) * b.page_size + t % b.page_size)
    n = len(np.unique(np.concatenate(slots))) if slots else 0
    esize = 4 if b.dtype == "f32" else 2
    return 2 * n * b.num_kv_heads * b.head_dim * esize


def describe(b) -> dict:
    q, kv = b.seqs[:, 0], b.seqs[:, 1]
    return {"workload": b.name, "requests": b.num_seqs, "num_qo_heads": b.num_qo_heads,
            "num_kv_heads": b.num_kv_heads, "head_dim": b.head_dim, "page_size": b.page_size,
            "q_len": [int(q.min()), int(q.max())], "kv_len": [int(kv.min()), int(kv.max())],
            "windows": sorted({int(w) for w in b.masks[:, 2]}), "total_q": b.total_q, "num_pages": b.num_pages}


def cpu_baseline(b, tensors, unit, budget_s=15.0):
    """The oracle, as it stands, timed on this host on a bounded sample of the
    workload (about ``budget_s`` seconds of wall time), scaled to the metric's
    unit.  The sample is whole requests (every query head) when one request
    fits the budget several times over, else the first query heads of one
    request (a full-size text+latent request alone takes tens of seconds)."""
    import workloads as W
    from oracle import oracle_attention
    from paper_2606_12688_amd import attn

    def measure(reqs, heads):
        sb, q, kp, vp, _ = W.extract_requests(b, tensors, reqs)
        pl = attn.plan(sb.num_qo_heads, sb.num_kv_heads, sb.head_dim, sb.dtype, sb.seqs, sb.masks,
                       sb.segments, sb.block_table.shape[1], sb.num_pages, sb.sm_scale, attn.FLAG_HOST_ONLY)
        pairs, kr = pl.stats()["visible_pairs"], pl.key_ranges()
        pl.destroy()
        frac = len(heads) / b.num_qo_heads
        kv_heads = len({h // (b.num_qo_heads // b.num_kv_heads) for h in heads})
        c0, t0 = time.process_time(), time.perf_counter()
        oracle_attention(sb, q, kp, vp, heads=heads)
        wall = time.perf_counter() - t0
        return wall, time.process_time() - c0, pairs * frac, kv_bytes(sb, kr) * kv_heads / b.num_kv_heads

    order = np.random.default_rng(123).permutation(b.num_seqs)
    all_heads = list(range(b.num_qo_heads))
    w1, _, _, _ = measure(order[:1], [0])  # one request, one head
    if w1 * b.num_qo_heads * 3 <= budget_s:
        heads = all_heads
        n = int(max(1, min(b.num_seqs, budget_s / max(w1 * b.num_qo_heads, 1e-3))))
    else:
        n = 1
        heads = all_heads[:int(max(1, min(b.num_qo_heads, budget_s / max(w1, 1e-3))))]
    wall, cpu, pairs, nbytes = measure(order[:n], heads)
    reps = 1
    while wall < budget_s * 0.66 and reps < 100:  # a small sample: repeat it (wall, cpu are totals)
        w2, c2, _, _ = measure(order[:n], heads)
        wall, cpu, reps = wall + w2, cpu + c2, reps + 1
    wall, cpu = wall / reps, cpu / reps
    flop = 4.0 * b.head_dim * pairs
    value = nbytes / wall / 1e9 if unit == "GB/s" else flop / wall / 1e12
    return {"value": value, "unit": unit, "cores": max(1, int(round(cpu / wall))), "kind": "oracle",
            "sample": f"{n} of {b.num_seqs} requests x {len(heads)} of {b.num_qo_heads} query heads, fp64 NumPy "
                      f"oracle, mean of {reps} run(s) of {wall:.2f} s wall, {flop / wall / 1e9:.2f} GFLOP/s, "
                      f"{nbytes / wall / 1e9:.3f} GB/s KV"}


def bench_append(args, b, dev):
    """Time ``mstar_kv_append`` alone: every new K and V row of the workload is
    read once and written once (HBM-bound); one JSON line."""
    import torch

    import workloads as W
    from paper_2606_12688_amd import attn

    stream = torch.cuda.current_stream()
    pl = attn.plan(b.num_qo_heads, b.num_kv_heads, b.head_dim, b.dtype, b.seqs, b.masks, b.segments,
                   b.block_table.shape[1], b.num_pages, b.sm_scale, 0, stream)
    t = W.make_tensors_torch(b, dev, seed=args.seed)
    g = torch.Generator(device=dev)
    g.manual_seed(args.seed + 77)
    shape = (b.total_q, b.num_kv_heads, b.head_dim)
    dt = t["q"].dtype
    kn = torch.randn(shape, generator=g, device=dev).to(dt)
    vn = torch.randn(shape, generator=g, device=dev).to(dt)
    bt = torch.from_numpy(np.ascontiguousarray(b.block_table)).to(dev)
    attn.kv_append(pl, kn, vn, bt, t["k_pages"], t["v_pages"], stream)
    assert attn.check(pl, stream) == 0
    L = attn.lib()
    call = (pl.handle, kn.data_ptr(), vn.data_ptr(), bt.data_ptr(), t["k_pages"].data_ptr(),
            t["v_pages"].data_ptr(), stream.cuda_stream)
    for _ in range(args.warmup):
        L.mstar_kv_append(*call)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        rc = L.mstar_kv_append(*call)
        if rc != 0:
            raise attn.MStarError(rc, attn.last_error())
    e1.record(stream)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / args.steps
    kernel_ms = e0.elapsed_time(e1) / args.steps
    assert attn.check(pl, stream) == 0
    esize = 4 if b.dtype == "f32" else 2
    nbytes = 2 * 2 * b.total_q * b.num_kv_heads * b.head_dim * esize  # K and V, read and written
    gbs = nbytes / (ms * 1e-3) / 1e9
    achieved = nbytes / (kernel_ms * 1e-3) / 1e9
    print(json.dumps({
        "metric": "paged KV append HBM GB/s (new K/V rows read and written)", "value": round(gbs, 3),
        "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": b.dtype, "data": "synthetic",
        "config": dict(describe(b), op="kv_append", new_rows=b.total_q),
        "roofline": {"bound": "hbm", "achieved": round(achieved, 3), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": None},
        "bytes_per_step": nbytes}), flush=True)
    pl.destroy()


def bench_serve(args, b, dev):
    """A serving loop over one workload: every step plans the batch again (the
    batch changes from step to step in a server), runs the attention and waits
    for it (standing in for reading back the step's tokens).  Inline: plan,
    then attention, on the critical path.  Async: the plan of step i+1 is built
    on the planner's thread and stream while step i runs (Sec. 3.3, Runtime).
    One JSON line with the per-step wall time of both."""
    import torch

    import workloads as W
    from paper_2606_12688_amd import attn

    stream = torch.cuda.current_stream()
    t = W.make_tensors_torch(b, dev, seed=args.seed)
    out = torch.empty_like(t["q"])
    lse = torch.empty(t["q"].shape[:2], dtype=torch.float32, device=dev)
    bt = torch.from_numpy(np.ascontiguousarray(b.block_table)).to(dev)
    flags = attn.FLAG_SERIAL if args.serial else 0
    args_plan = (b.num_qo_heads, b.num_kv_heads, b.head_dim, b.dtype, b.seqs, b.masks, b.segments,
                 b.block_table.shape[1], b.num_pages, b.sm_scale, flags)
    groups = b.prefix_groups if args.cascade else None
    pl0 = attn.plan(*args_plan, stream, prefix_groups=groups)
    ws = attn.workspace(pl0, dev)  # the same shapes every step: one workspace
    pl0.destroy()

    def inline(n):
        for _ in range(n):
            pl = attn.plan(*args_plan, stream, prefix_groups=groups)
            attn.fwd(pl, t["q"], t["k_pages"], t["v_pages"], bt, out, lse, ws, stream)
            torch.cuda.synchronize()
            pl.destroy()

    ap = attn.AsyncPlanner(depth=2)

    def overlapped(n):
        ap.submit(*args_plan, prefix_groups=groups)
        for i in range(n):
            if i + 1 < n:
                ap.submit(*args_plan, prefix_groups=groups)
            pl = ap.take(stream)
            attn.fwd(pl, t["q"], t["k_pages"], t["v_pages"], bt, out, lse, ws, stream)
            torch.cuda.synchronize()
            pl.destroy()

    res = {}
    for name, fn in (("inline", inline), ("async", overlapped)):
        fn(args.warmup)
        t0 = time.perf_counter()
        fn(args.steps)
        res[name] = (time.perf_counter() - t0) * 1e3 / args.steps
    ap.close()
    st = attn.plan(*args_plan[:-1], flags | attn.FLAG_HOST_ONLY, prefix_groups=groups)
    plan_us = st.stats()["plan_host_us"]
    st.destroy()
    print(json.dumps({
        "metric": "serving-loop step time, plan + attention + wait (ms)", "value": round(res["async"], 5),
        "unit": "ms", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(res["async"], 5),
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": b.dtype, "data": "synthetic",
        "config": dict(describe(b), op="serve", cascade=bool(args.cascade)),
        "inline_ms_per_step": round(res["inline"], 5),
        "async_ms_per_step": round(res["async"], 5), "plan_host_us": round(plan_us, 1)}), flush=True)


CONFIGS = ["tiny_causal_f32", "decode_bf16", "text_latent_bf16", "stream_window_bf16", "rollout_bf16"]
HEADLINE = "rollout_bf16"  # the largest configuration (3.38 TFLOP, 2.54 GB per step)


def host_cpu():
    """CPU model and the logical CPUs this process may use."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return model, len(os.sched_getaffinity(0))


def bench_attention(args, name, dev, cpu_budget_s):
    """One workload: build the plan, rotate input copies, time K steps of
    ``mstar_attn_fwd`` with nothing else on the stream (the step time), then a
    separate sampled loop with HIP events around each kernel (per-kernel
    durations for the roofline).  Returns the per-configuration record."""
    import torch

    import workloads as W
    from paper_2606_12688_amd import attn

    b = W.FULL_SIZE[name](args.seed)
    if args.cascade and not b.prefix_groups:
        raise SystemExit(f"{name} declares no shared-prefix group")
    bound = BOUND[name]
    stream = torch.cuda.current_stream()

    def make_plan():
        return attn.plan(b.num_qo_heads, b.num_kv_heads, b.head_dim, b.dtype, b.seqs, b.masks, b.segments,
                         b.block_table.shape[1], b.num_pages, b.sm_scale, attn.FLAG_SERIAL if args.serial else 0,
                         stream, prefix_groups=b.prefix_groups if args.cascade else None)
    # the first plan of a process includes one-time set-up (pools, HIP context
    # work); the reported planning time is that of a later plan
    pl_first = make_plan()
    plan_first_us = pl_first.stats()["plan_host_us"]
    pl_first.destroy()
    plan_us = []
    for _ in range(5):
        p2 = make_plan()
        plan_us.append(p2.stats()["plan_host_us"])
        p2.destroy()
    pl = make_plan()
    st = pl.stats()
    flop = 4.0 * b.head_dim * st["visible_pairs"]
    nbytes = kv_bytes(b, pl.key_ranges())

    # rotate enough copies that one step's K/V is out of the 256 MB MALL by the next use
    n_rot = min(8, max(2, int(np.ceil(1.0e9 / max(nbytes, 1)))))
    copies = []
    for i in range(n_rot):
        t = W.make_tensors_torch(b, dev, seed=args.seed + 1000 * i)
        t["out"] = torch.empty_like(t["q"])
        t["lse"] = torch.empty(t["q"].shape[:2], dtype=torch.float32, device=dev)
        copies.append(t)
    bt = torch.from_numpy(np.ascontiguousarray(b.block_table)).to(dev)
    ws = attn.workspace(pl, dev)
    # validate every copy once through the checked binding, then call the C entry point directly
    for t in copies:
        attn.fwd(pl, t["q"], t["k_pages"], t["v_pages"], bt, t["out"], t["lse"], ws, stream)
    assert attn.check(pl, stream) == 0
    L = attn.lib()
    sh = stream.cuda_stream
    ws_ptr, ws_n = (ws.data_ptr(), ws.numel()) if ws is not None else (None, 0)
    calls = [(pl.handle, t["q"].data_ptr(), t["k_pages"].data_ptr(), t["v_pages"].data_ptr(), bt.data_ptr(),
              t["out"].data_ptr(), t["lse"].data_ptr(), ws_ptr, ws_n, sh) for t in copies]

    def run(i):
        rc = L.mstar_attn_fwd(*calls[i % n_rot])
        if rc != 0:
            raise attn.MStarError(rc, attn.last_error())

    # ---- the step time: K calls back to back, nothing else on the stream
    K = args.steps
    for i in range(args.warmup):
        run(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(K):
        run(i)
    torch.cuda.synchronize()
    ms_per_step = (time.perf_counter() - t0) * 1e3 / K

    # ---- per-kernel durations: a separate loop with the library's HIP events
    # recorded right before / after each kernel on the stream it runs on, and
    # a pair around the whole call on the caller's stream
    launched = [k for k, n in enumerate(("prefill_items", "decode_items", "f32_items", "merge_rows")) if st[n] > 0]
    if len(pl.items(4)):
        launched.append(4)
    n_ev = max(8, min(32, K))
    evs = [[[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(2)] for _ in range(n_ev)]
    span = [[torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)] for _ in range(n_ev)]
    arrays = []
    for i in range(n_ev):
        arr = [(ctypes.c_void_p * 5)(), (ctypes.c_void_p * 5)()]
        for side in range(2):
            for k in launched:
                evs[i][side][k].record(stream)  # creates the event
                arr[side][k] = evs[i][side][k].cuda_event
        arrays.append(arr)
    torch.cuda.synchronize()
    for i in range(n_ev):
        span[i][0].record(stream)
        rc = L.mstar_attn_fwd_timed(*calls[i % n_rot], arrays[i][0], arrays[i][1])
        span[i][1].record(stream)
        if rc != 0:
            raise attn.MStarError(rc, attn.last_error())
    torch.cuda.synchronize()
    per_kernel = {KERNEL_NAMES[k]: np.array([evs[i][0][k].elapsed_time(evs[i][1][k]) for i in range(n_ev)])
                  for k in launched}
    span_ms = np.array([span[i][0].elapsed_time(span[i][1]) for i in range(n_ev)])
    if len([k for k in launched if k in (0, 1, 4)]) > 1:
        # the step's work is spread over several kernels, some side by side: the call's span
        kernel_ms, dominant = span_ms, "call(" + "+".join(KERNEL_NAMES[k] for k in launched) + ")"
    else:
        dominant = KERNEL_NAMES[DOMINANT[name]]
        kernel_ms = per_kernel[dominant]
    assert attn.check(pl, stream) == 0

    tflops = flop / (ms_per_step * 1e-3) / 1e12
    gbps = nbytes / (ms_per_step * 1e-3) / 1e9
    k_mean = float(kernel_ms.mean())
    if bound == "hbm":
        value, unit = gbps, "GB/s"
        achieved, peak, runit = nbytes / (k_mean * 1e-3) / 1e9, PEAK_HBM_GBS, "GB/s"
    elif bound == "mfma":
        value, unit = tflops, "TFLOP/s"
        achieved, peak, runit = flop / (k_mean * 1e-3) / 1e12, PEAK_BF16_TFLOPS, "TFLOP/s"
    else:
        value, unit = tflops, "TFLOP/s"
        achieved, peak, runit = flop / (k_mean * 1e-3) / 1e12, PEAK_FP32_TFLOPS, "TFLOP/s"

    traffic = None
    traffic_note = "no counter run recorded for this kernel source"
    if os.path.exists(TRAFFIC_FILE):
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f).get(name + ("+cascade" if args.cascade else ""))
        if rec and rec.get("kernel_src_sha") == kernel_source_sha():
            traffic = rec["hbm_bytes_per_launch"]
            traffic_note = rec.get("note", "")
        elif rec:
            traffic_note = "kernels changed since the counters were taken"

    def stats(v):
        return {"mean": round(float(v.mean()), 5), "median": round(float(np.median(v)), 5),
                "p95": round(float(np.percentile(v, 95)), 5)}

    res = {
        "workload": name, "value": round(value, 3), "unit": unit, "ms_per_step": round(ms_per_step, 5),
        "dtype": b.dtype, "config": describe(b),
        "roofline": {"bound": bound, "achieved": round(achieved, 3), "peak": peak, "unit": runit,
                     "frac": round(achieved / peak, 4), "traffic": traffic},
        "tflops": round(tflops, 3), "kv_gbps": round(gbps, 3),
        "tflops_frac_bf16_peak": round(tflops / PEAK_BF16_TFLOPS, 4),
        "kv_gbps_frac_hbm_peak": round(gbps / PEAK_HBM_GBS, 4),
        "dominant_kernel": dominant, "kernel_ms": {k: stats(v) for k, v in per_kernel.items()},
        "call_ms": stats(span_ms), "event_sampled_calls": n_ev,
        "useful_flop": flop, "kv_bytes": nbytes, "plan_host_us": round(float(np.median(plan_us)), 1),
        "plan_host_us_first_call": round(plan_first_us, 1),
        "plan": {k: st[k] for k in ("prefill_items", "decode_items", "f32_items", "merge_rows", "partial_slots")},
        "rotated_input_copies": n_rot, "traffic_note": traffic_note,
    }
    if cpu_budget_s > 0:
        res["cpu_baseline"] = cpu_baseline(b, copies[0], unit, cpu_budget_s)
    pl.destroy()
    del copies, ws
    torch.cuda.empty_cache()
    return res


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=None, choices=sorted(BOUND),
                    help="time this workload only (default: the five configurations, rollouts as the headline)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=15.0,
                    help="seconds of oracle time for the headline's cpu_baseline (a third of it for each other "
                         "configuration)")
    ap.add_argument("--serial", action="store_true",
                    help="plan with MSTAR_FLAG_SERIAL: every kernel on the caller's stream, none beside another")
    ap.add_argument("--cascade", action="store_true",
                    help="plan with the workload's shared-prefix groups (mstar_attn_plan_cascade); the roofline "
                         "then divides by the span of the whole call")
    ap.add_argument("--op", default="attention", choices=["attention", "append", "serve"],
                    help="append: time mstar_kv_append (the step's new K/V rows into their pages); serve: a "
                         "serving loop that re-plans every step, planning inline vs on the async planner")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="run only a plain 1 GiB device copy (for HBM counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path (the attention would "
              "shard by request or by KV head, each GPU running its share with no exchange).", file=sys.stderr)
        sys.exit(2)

    import torch

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")

    if args.calibrate_copy:
        n = 1 << 30
        src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        for _ in range(args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": n, "launches": args.steps}))
        return

    import workloads as W

    if args.op in ("append", "serve"):
        b = W.FULL_SIZE[args.workload or "decode_bf16"](args.seed)
        if args.cascade and not b.prefix_groups:
            print(f"{b.name} declares no shared-prefix group", file=sys.stderr)
            sys.exit(2)
        (bench_append if args.op == "append" else bench_serve)(args, b, dev)
        return

    budget = 0.0 if args.no_cpu_baseline else args.cpu_budget
    model, nproc = host_cpu()
    if args.workload:
        names, head = [args.workload], args.workload
    else:
        names, head = CONFIGS, HEADLINE
    configs = {}
    for name in names:
        print(f"[bench] {name}", file=sys.stderr, flush=True)
        configs[name] = bench_attention(args, name, dev, budget if name == head else budget / 3)
        if "cpu_baseline" in configs[name]:
            configs[name]["cpu_baseline"].update(cpu_model=model, host_logical_cpus=nproc)
    h = configs[head]
    res = {
        "metric": METRIC, "value": h["value"], "unit": h["unit"], "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": h["ms_per_step"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": h["dtype"], "data": "synthetic",
        "config": h["config"], "roofline": h["roofline"],
    }
    if "cpu_baseline" in h:
        res["cpu_baseline"] = h["cpu_baseline"]
    res.update({k: v for k, v in h.items() if k not in res and k not in ("workload",)})
    res["cascade"], res["serial"] = bool(args.cascade), bool(args.serial)
    if len(names) > 1:
        res["configs"] = {f"c{CONFIGS.index(n) + 1}_{n}": {
            k: configs[n][k] for k in ("value", "unit", "ms_per_step", "roofline", "cpu_baseline", "tflops",
                                       "kv_gbps", "useful_flop", "kv_bytes", "dominant_kernel", "kernel_ms",
                                       "call_ms", "plan_host_us", "config") if k in configs[n]} for n in names}
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
