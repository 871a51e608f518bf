"""GPU parity on seeded random batches.  Each seed draws a head layout (G = 1,
2, 4 or 7 query heads per KV head), a head dimension, a dtype, and up to six
requests of random shape (single tokens, chunks, prefills, requests without
query rows) whose key range is cut into one to three segments of random kind
(causal, one full block, blocks of a random length), with or without a
sliding window; pages are a seeded permutation of the pool and the split
policy is drawn too.  Every output is compared with the oracle."""
import numpy as np
import pytest

import workloads as W
from paper_2606_12688_amd import attn
from tests.helpers import compare, oracle_of, run_gpu

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
FLAGS = [0, attn.FLAG_FORCE_SPLIT, attn.FLAG_NO_SPLIT]


def random_batch(seed):
    rng = np.random.default_rng(1000 + seed)
    d = int(rng.choice([64, 128]))
    dtype = "f32" if rng.random() < 0.15 else "bf16"
    hkv = int(rng.choice([1, 2, 4]))
    hq = hkv * int(rng.choice([1, 2, 4, 7]))
    q_lens, kv_lens, seg_lists, windows = [], [], [], []
    for _ in range(int(rng.integers(1, 7))):
        kind = rng.choice(["decode", "chunk", "prefill", "empty"], p=[0.3, 0.25, 0.35, 0.1])
        kv = int(rng.integers(1, 900))
        if kind == "decode":
            q = 1
        elif kind == "chunk":
            q = int(rng.integers(2, 33))
        elif kind == "prefill":
            q = int(rng.integers(1, min(kv, 300) + 1))
        else:
            q = 0
        q = min(q, kv)
        # one to three segments tiling [0, kv)
        cuts = sorted(set(int(c) for c in rng.integers(1, kv, size=int(rng.integers(0, 3))))) if kv > 1 else []
        bounds = [0] + cuts + [kv]
        segs = []
        for a, b in zip(bounds[:-1], bounds[1:]):
            k = int(rng.choice([W.SEG_CAUSAL, W.SEG_FULL, W.SEG_BLOCKS]))
            segs.append((a, b - a, k, int(rng.integers(1, 70)) if k == W.SEG_BLOCKS else 0))
        q_lens.append(q)
        kv_lens.append(kv)
        seg_lists.append(segs)
        windows.append(0 if rng.random() < 0.6 else int(rng.integers(1, 300)))
    b = W.custom(f"random_{seed}", hq, hkv, d, q_lens, kv_lens, seg_lists, windows, seed=seed, dtype=dtype,
                 pool_pages=int(sum((x + 15) // 16 for x in kv_lens)) + int(rng.integers(0, 40)))
    return b, FLAGS[int(rng.integers(0, 3))]


@pytest.mark.parametrize("seed", range(40))
def test_random_batch(seed):
    b, flag = random_batch(seed)
    t = W.make_tensors_torch(b, DEV)
    out, lse = run_gpu(b, t, flag, out_fill=float("nan"))
    compare(b, out, lse, *oracle_of(b, t), f"random batch {seed} (d{b.head_dim} {b.dtype} "
            f"{b.num_qo_heads}/{b.num_kv_heads}, {b.num_seqs} requests, flags {flag})")
