"""Paged KV append: the step's new key/value rows written into their pages.

TEST INFRASTRUCTURE ONLY (see the package docstring): never imported by the
product path.

Each node execution of the paper's transformer engine first stores the K/V of
the tokens it processes in the paged cache and then attends over the cache:
decode steps, flow steps over latents, and rollout frames reuse the cache
instead of re-prefilling (Sec. 3.3, Runtime; Sec. 4.4).  Reading (the paper
gives no data layout): request ``r``'s ``q_len`` new tokens are its positions
``kv_len - q_len .. kv_len - 1`` (the same placement as its queries); the new
row ``q_start + i`` of ``k_new`` / ``v_new`` (``[total_q, Hkv, d]``) goes to
``pages[block_table[r][pos // page_size], pos % page_size]`` with
``pos = kv_len - q_len + i``.  Every other slot keeps its value.  Two new rows
must not target one slot (requests that share pages share only their cached
prefix, never the slots of new tokens).
"""
from __future__ import annotations

import numpy as np


def append_targets(batch):
    """(packed row, physical page, slot) of every new token, in request order.

    Raises ``ValueError`` if a target page is outside the pool or two new rows
    target the same slot."""
    out = []
    seen = set()
    for r in range(batch.num_seqs):
        q_len, kv_len, q_start = (int(x) for x in batch.seqs[r])
        for i in range(q_len):
            pos = kv_len - q_len + i
            page = int(batch.block_table[r, pos // batch.page_size])
            slot = pos % batch.page_size
            if not 0 <= page < batch.num_pages:
                raise ValueError(f"request {r}: page {page} of position {pos} is outside the pool")
            if (page, slot) in seen:
                raise ValueError(f"request {r}: slot ({page}, {slot}) is the target of two new rows")
            seen.add((page, slot))
            out.append((q_start + i, page, slot))
    return out


def kv_append(batch, k_new, v_new, k_pages, v_pages):
    """New page arrays with the step's rows written in; the inputs are left as
    they are.  Values are copied exactly (no arithmetic)."""
    k_out = np.array(k_pages, copy=True)
    v_out = np.array(v_pages, copy=True)
    for row, page, slot in append_targets(batch):
        k_out[page, slot] = k_new[row]
        v_out[page, slot] = v_new[row]
    return k_out, v_out
