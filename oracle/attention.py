"""fp64 dense masked-softmax attention read through paged block tables.

TEST INFRASTRUCTURE ONLY (see the package docstring): never imported by the
product path.

Readings of the paper (it fixes none of these; each is the documented reading
the library boundary also states):

* Mask model.  A request's keys ``[0, kv_len)`` are tiled in order by segments.
  Walking them with a counter ``c`` assigns every position a block id:
  CAUSAL gives token ``j`` of the segment id ``c + j`` (each token its own
  block); FULL gives every token id ``c`` (one block); BLOCKS(b) gives token
  ``j`` id ``c + floor(j / b)`` (consecutive full blocks of ``b`` tokens, the
  last possibly short).  Key ``t`` is visible to the query at position ``p``
  iff ``blk[t] <= blk[p]`` and, with a window ``W > 0``, ``p - t < W`` (the
  row sees exactly ``W`` keys ending at itself, plus any later keys of its
  own block).  These cover the paper's causal text decoding, full-attention
  image/latent blocks inside flow loops (Sec. 3.1, image-generation Walk),
  streamed chunks (Sec. 3.1, chunk policies) and frame-by-frame rollouts
  over a cached context (Sec. 4.4).
* Query placement.  A request's ``q_len`` queries are its last ``q_len``
  positions, ``kv_len - q_len .. kv_len - 1``: new tokens are appended to the
  paged cache before attention reads it (Sec. 4.4: rollouts reuse the paged KV
  cache instead of re-prefilling).
* Paging.  Key ``t`` of request ``r`` lives at
  ``pages[block_table[r][t // page_size], t % page_size, kv_head, :]``; one
  pool serves every request and pages may be shared (Sec. 4.1: several
  contexts as labels over one paged pool, read in place; App. A: K candidates
  in one batched forward over a shared context).
* GQA.  Query head ``h`` reads KV head ``h // (Hq / Hkv)``.
* Output.  ``out = sum_t softmax(s)_t V[t]`` with ``s_t = sm_scale * q.K[t]``
  over visible ``t``; ``lse = log(sum_t exp(s_t))`` in natural log.  A row with
  no visible key gets ``out = 0`` and ``lse = -inf``.
"""
from __future__ import annotations

import numpy as np

SEG_CAUSAL = 0
SEG_FULL = 1
SEG_BLOCKS = 2


def block_ids(segments, kv_len: int) -> np.ndarray:
    """Block id of every key position of one request (mask model above).

    ``segments``: rows ``(start, len, kind, block)`` tiling ``[0, kv_len)`` in
    order.  Raises ``ValueError`` if they do not.
    """
    ids = np.empty(kv_len, dtype=np.int64)
    c = 0
    pos = 0
    for start, length, kind, blk in np.asarray(segments, dtype=np.int64).reshape(-1, 4):
        if start != pos or length < 0:
            raise ValueError("segments must tile [0, kv_len) in order")
        j = np.arange(length, dtype=np.int64)
        if kind == SEG_CAUSAL:
            ids[pos:pos + length] = c + j
            c += length
        elif kind == SEG_FULL:
            ids[pos:pos + length] = c
            c += 1
        elif kind == SEG_BLOCKS:
            if blk <= 0:
                raise ValueError("BLOCKS segment needs a positive block size")
            ids[pos:pos + length] = c + j // blk
            c += -(-length // blk)
        else:
            raise ValueError("unknown segment kind")
        pos += length
    if pos != kv_len:
        raise ValueError("segments must tile [0, kv_len) in order")
    return ids


def visible_matrix(q_len: int, kv_len: int, blk: np.ndarray, window: int) -> np.ndarray:
    """bool ``[q_len, kv_len]``: may query row ``i`` (position
    ``kv_len - q_len + i``) see key ``t``?"""
    p = np.arange(kv_len - q_len, kv_len, dtype=np.int64)[:, None]
    t = np.arange(kv_len, dtype=np.int64)[None, :]
    vis = blk[t] <= blk[p]
    if window > 0:
        vis &= (p - t) < window
    return vis


def gather_kv(pages: np.ndarray, bt_row: np.ndarray, kv_len: int, kvh: int,
              positions=None) -> np.ndarray:
    """Rows of one KV head of one request, read through its block table, as
    fp64 ``[len(positions), d]`` (default: every position ``0..kv_len-1``)."""
    page_size = pages.shape[1]
    t = np.arange(kv_len) if positions is None else np.asarray(positions, dtype=np.int64)
    phys = np.asarray(bt_row, dtype=np.int64)[t // page_size]
    return np.asarray(pages[phys, t % page_size, kvh, :], dtype=np.float64)


def attend(q: np.ndarray, K: np.ndarray, V: np.ndarray, vis: np.ndarray, sm_scale: float):
    """Masked softmax attention of query rows ``q [M, d]`` over ``K, V [N, d]``
    with visibility ``vis [M, N]``; returns ``out [M, d]``, ``lse [M]`` (fp64)."""
    q = np.asarray(q, dtype=np.float64)
    s = (q @ np.asarray(K, dtype=np.float64).T) * float(sm_scale)
    s = np.where(vis, s, -np.inf)
    m = s.max(axis=1, initial=-np.inf)
    empty = ~np.isfinite(m)
    m_safe = np.where(empty, 0.0, m)
    e = np.exp(s - m_safe[:, None])  # exp(-inf) = 0 for hidden keys
    l = e.sum(axis=1)
    out = (e @ np.asarray(V, dtype=np.float64)) / np.where(empty, 1.0, l)[:, None]
    lse = m_safe + np.log(np.where(empty, 1.0, l))
    out[empty] = 0.0
    lse[empty] = -np.inf
    return out, lse


def _request_rows(batch, r):
    q_len, kv_len, q_start = (int(x) for x in batch.seqs[r])
    seg_b, seg_c, window = (int(x) for x in batch.masks[r])
    blk = block_ids(batch.segments[seg_b:seg_b + seg_c], kv_len)
    return q_len, kv_len, q_start, window, blk


def oracle_attention(batch, q, k_pages, v_pages, heads=None):
    """Whole-batch oracle.  ``q [total_q, Hq, d]``, pages ``[P, page, Hkv, d]``
    (any real dtype; read as fp64).  Returns ``out [total_q, Hq, d]`` and
    ``lse [total_q, Hq]`` in fp64; rows that belong to no request stay 0 / -inf.

    Only keys visible to some row of a request are gathered (the rest would get
    weight zero), which bounds memory for windowed requests."""
    hq, hkv = batch.num_qo_heads, batch.num_kv_heads
    g = hq // hkv
    total_q = q.shape[0]
    d = q.shape[2]
    out = np.zeros((total_q, hq, d), dtype=np.float64)
    lse = np.full((total_q, hq), -np.inf, dtype=np.float64)
    heads = range(hq) if heads is None else heads
    for r in range(batch.num_seqs):
        q_len, kv_len, q_start, window, blk = _request_rows(batch, r)
        if q_len == 0:
            continue
        vis = visible_matrix(q_len, kv_len, blk, window)
        cols = np.nonzero(vis.any(axis=0))[0]
        vis = vis[:, cols]
        kv_cache = {}
        for h in heads:
            kvh = h // g
            if kvh not in kv_cache:
                kv_cache = {kvh: (gather_kv(k_pages, batch.block_table[r], kv_len, kvh, cols),
                                  gather_kv(v_pages, batch.block_table[r], kv_len, kvh, cols))}
            K, V = kv_cache[kvh]
            o, s = attend(q[q_start:q_start + q_len, h, :], K, V, vis, batch.sm_scale)
            out[q_start:q_start + q_len, h, :] = o
            lse[q_start:q_start + q_len, h] = s
    return out, lse


def oracle_rows(batch, q, k_pages, v_pages, picks):
    """Oracle for selected outputs only: ``picks`` is a list of
    ``(request, query_row, head)``.  Returns ``out [n, d]``, ``lse [n]`` fp64.
    Each pick gathers just the keys its row may see."""
    g = batch.num_qo_heads // batch.num_kv_heads
    d = q.shape[2]
    outs = np.zeros((len(picks), d), dtype=np.float64)
    lses = np.zeros(len(picks), dtype=np.float64)
    for n, (r, i, h) in enumerate(picks):
        q_len, kv_len, q_start, window, blk = _request_rows(batch, r)
        vis = visible_matrix(q_len, kv_len, blk, window)[i]
        cols = np.nonzero(vis)[0]
        K = gather_kv(k_pages, batch.block_table[r], kv_len, h // g, cols)
        V = gather_kv(v_pages, batch.block_table[r], kv_len, h // g, cols)
        o, s = attend(q[q_start + i:q_start + i + 1, h, :], K, V,
                      np.ones((1, len(cols)), dtype=bool), batch.sm_scale)
        outs[n] = o[0]
        lses[n] = s[0]
    return outs, lses


def merge_partials(outs, lses):
    """Combine attention results over disjoint key subsets of the same rows.

    ``outs [S, M, d]`` are each subset's normalised outputs and ``lses [S, M]``
    its natural-log log-sum-exps.  Since ``exp(lse_s)`` is subset ``s``'s
    softmax denominator, the union's denominator is ``sum_s exp(lse_s)`` and
    its output is the denominator-weighted mean of the subset outputs.  Subsets
    with no visible key (``lse = -inf``) carry weight zero."""
    outs = np.asarray(outs, dtype=np.float64)
    lses = np.asarray(lses, dtype=np.float64)
    m = lses.max(axis=0)
    empty = ~np.isfinite(m)
    m_safe = np.where(empty, 0.0, m)
    w = np.exp(lses - m_safe[None, :])
    tot = w.sum(axis=0)
    out = (w[:, :, None] * outs).sum(axis=0) / np.where(empty, 1.0, tot)[:, None]
    lse = m_safe + np.log(np.where(empty, 1.0, tot))
    out[empty] = 0.0
    lse[empty] = -np.inf
    return out, lse


def useful_work(batch):
    """Visible (row, key) pairs summed over query heads, useful FLOPs
    (``4 d`` per pair and head: ``2 d`` for the score, ``2 d`` for the weighted
    value sum) and algorithmic KV bytes (each distinct visible key of a request
    and KV head read once for K and once for V; pages shared between requests
    counted once).  Returns a dict."""
    hq, hkv, d = batch.num_qo_heads, batch.num_kv_heads, batch.head_dim
    esize = 4 if batch.dtype == "f32" else 2
    pairs = 0
    phys_slots = set()
    for r in range(batch.num_seqs):
        q_len, kv_len, q_start, window, blk = _request_rows(batch, r)
        if q_len == 0:
            continue
        lo, hi = _row_intervals(q_len, kv_len, blk, window)
        pairs += int((hi - lo).sum())
        t0, t1 = int(lo.min()), int(hi.max())
        t = np.arange(t0, t1, dtype=np.int64)
        ps = batch.page_size
        phys = np.asarray(batch.block_table[r], dtype=np.int64)[t // ps] * ps + t % ps
        phys_slots.update(phys.tolist())
    kv_bytes = 2 * len(phys_slots) * hkv * d * esize
    return {"pairs": pairs * hq, "flop": 4.0 * d * pairs * hq, "kv_bytes": float(kv_bytes)}


def _row_intervals(q_len, kv_len, blk, window):
    """Visible keys of each row as ``[lo, hi)``: block ids never decrease along
    the sequence, so a row sees every key up to the end of its own block, and a
    window only cuts keys off from below."""
    p = np.arange(kv_len - q_len, kv_len, dtype=np.int64)
    # end of p's block: first index whose block id exceeds blk[p]
    hi = np.searchsorted(blk, blk[p], side="right")
    lo = np.maximum(0, p - window + 1) if window > 0 else np.zeros_like(p)
    return lo, hi
