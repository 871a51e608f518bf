"""Second, scalar oracle in plain Python for tiny inputs.

TEST INFRASTRUCTURE ONLY: it exists to catch implementation slips in the NumPy
oracle (``attention.py``).  It restates the same definition with explicit
loops and exactly rounded sums (``math.fsum``), walking the segments token by
token instead of vectorising them, and it reads every key through the block
table one element at a time.
"""
from __future__ import annotations

import math


def _block_of_each_token(segments):
    ids = []
    counter = 0
    for start, length, kind, blk in segments:
        assert start == len(ids)
        for j in range(length):
            if kind == 0:      # causal: every token starts a new block
                ids.append(counter + j)
            elif kind == 1:    # full: one block for the whole segment
                ids.append(counter)
            else:              # fixed-size blocks
                ids.append(counter + j // blk)
        if kind == 0:
            counter += length
        elif kind == 1:
            counter += 1
        else:
            counter += (length + blk - 1) // blk
    return ids


def scalar_attention(batch, q, k_pages, v_pages):
    """Same contract as ``oracle_attention`` but returns nested lists:
    ``out[row][head][dim]`` and ``lse[row][head]`` for every packed row."""
    hq, hkv = batch.num_qo_heads, batch.num_kv_heads
    group = hq // hkv
    d = len(q[0][0])
    ps = batch.page_size
    total_q = len(q)
    out = [[[0.0] * d for _ in range(hq)] for _ in range(total_q)]
    lse = [[-math.inf] * hq for _ in range(total_q)]
    for r in range(batch.num_seqs):
        q_len, kv_len, q_start = (int(x) for x in batch.seqs[r])
        seg_b, seg_c, window = (int(x) for x in batch.masks[r])
        segs = [tuple(int(v) for v in batch.segments[s]) for s in range(seg_b, seg_b + seg_c)]
        ids = _block_of_each_token(segs)
        for i in range(q_len):
            p = kv_len - q_len + i
            keys = [t for t in range(kv_len)
                    if ids[t] <= ids[p] and (window == 0 or p - t < window)]
            for h in range(hq):
                kvh = h // group
                qv = [float(x) for x in q[q_start + i][h]]
                scores = []
                rows = []
                for t in keys:
                    page = int(batch.block_table[r][t // ps])
                    krow = [float(x) for x in k_pages[page][t % ps][kvh]]
                    vrow = [float(x) for x in v_pages[page][t % ps][kvh]]
                    scores.append(batch.sm_scale * math.fsum(a * b for a, b in zip(qv, krow)))
                    rows.append(vrow)
                if not keys:
                    continue
                mx = max(scores)
                w = [math.exp(s - mx) for s in scores]
                den = math.fsum(w)
                out[q_start + i][h] = [math.fsum(w[n] * rows[n][c] for n in range(len(keys))) / den
                                       for c in range(d)]
                lse[q_start + i][h] = mx + math.log(den)
    return out, lse
