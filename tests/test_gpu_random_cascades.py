"""GPU parity on seeded random shared-prefix cascades.  Each seed draws a head
layout, a head dimension, a page-aligned prefix of 16 to 1024 keys whose
pages every block table shares, and two to eight requests.  Members of the
prefix group are decode tokens, 16-token chunks, prefills past the prefix,
rows that start inside the prefix's block and requests without rows; the
others read the same pages but stay outside the group.  Every member row sees
the whole prefix: the prefix is one full block, followed by the member's own
keys, causal or in blocks.  Every output is compared with the oracle under
both member policies (decode-like members only, every member) and the three
split policies."""
import numpy as np
import pytest

import workloads as W
from paper_2606_12688_amd import attn
from tests.helpers import compare, oracle_of, run_gpu

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
FLAGS = [0, attn.FLAG_FORCE_SPLIT, attn.FLAG_NO_SPLIT]


def random_cascade(seed):
    rng = np.random.default_rng(5000 + seed)
    d = int(rng.choice([64, 128]))
    hkv = int(rng.choice([1, 2, 4]))
    hq = hkv * int(rng.choice([1, 2, 4, 7]))
    prefix = 16 * int(rng.integers(1, 65))
    n = int(rng.integers(2, 9))
    q_lens, kv_lens, seg_lists, windows, members = [], [], [], [], []
    for r in range(n):
        own = int(rng.integers(0, 400))
        L = prefix + own
        member = r == 0 or rng.random() < 0.75
        if member:
            kind = rng.choice(["decode", "chunk", "prefill", "inside", "empty"], p=[0.35, 0.2, 0.2, 0.15, 0.1])
            if kind == "decode":
                q = 1
            elif kind == "chunk":
                q = min(16, L)
            elif kind == "prefill":
                q = min(int(rng.integers(17, 300)), L)
            elif kind == "inside":  # the first rows lie inside the prefix's block
                q = own + int(rng.integers(1, min(prefix, 200) + 1))
            else:
                q = 0
            segs = [(0, prefix, W.SEG_FULL, 0)]
            if own:
                own_kind = int(rng.choice([W.SEG_CAUSAL, W.SEG_BLOCKS]))
                segs.append((prefix, own, own_kind, int(rng.integers(1, 70)) if own_kind == W.SEG_BLOCKS else 0))
            window = 0
            members.append(r)
        else:  # same pages, outside the group: any mask
            q = min(int(rng.choice([1, 16, 150])), L)
            segs = [(0, L, W.SEG_CAUSAL, 0)]
            window = 0 if rng.random() < 0.5 else int(rng.integers(1, 500))
        q_lens.append(q)
        kv_lens.append(L)
        seg_lists.append(segs)
        windows.append(window)
    b = W.custom(f"random_cascade_{seed}", hq, hkv, d, q_lens, kv_lens, seg_lists, windows, seed=seed,
                 shared_prefix_pages=prefix // W.PAGE)
    b.prefix_groups = [(members, prefix)]
    return b


@pytest.mark.parametrize("seed", range(24))
def test_random_cascade(seed):
    b = random_cascade(seed)
    t = W.make_tensors_torch(b, DEV)
    ro, rl = oracle_of(b, t)
    for policy, tag in ((0, "decode-like members"), (attn.FLAG_CASCADE_ALL, "every member")):
        for flag in FLAGS:
            out, lse = run_gpu(b, t, flag | policy, out_fill=float("nan"), cascade=True)
            compare(b, out, lse, ro, rl, f"random cascade {seed} (d{b.head_dim} {b.num_qo_heads}/{b.num_kv_heads}, "
                    f"{b.num_seqs} requests, prefix {b.prefix_groups[0][1]}, {tag}, flags {flag})")
