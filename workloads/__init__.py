"""Seeded synthetic inputs for batched paged-KV attention with per-request masks.

This module is shared by the tests, the benchmark and the smoke check.  It
holds no attention arithmetic: it only draws request lengths, lays requests
out in a paged KV pool, writes mask descriptors and draws Q/K/V values.  Both
the CPU oracle and the HIP path consume what it returns; neither is imported
here.

Workload shapes stand in for the serving scenarios the paper runs (it gives no
per-layer attention shapes and its datasets are not used):

* ``tiny_causal_f32``   - a tiny causal prefill in fp32 (parity case).
* ``decode_bf16``       - one new token per request over a long context, GQA 7:1
                          (autoregressive decode inside a ``DynamicLoop``,
                          Sec. 3.1 "Loop optimizations"; Sec. 4.2 / 4.3).
* ``text_latent_bf16``  - causal text prefix followed by a full-attention latent
                          block (BAGEL's flow loop over latents, Sec. 3.1
                          listing of the image-generation Walk; Sec. 4.1).
* ``stream_window_bf16``- 16-token streamed chunks over a long context under a
                          sliding window (streaming edges, Sec. 3.1 "Flexible
                          chunk policies").
* ``rollout_bf16``      - K candidate rollouts appending frame blocks over one
                          shared context whose pages every block table points
                          to (V-JEPA 2 rollout and MPC, Sec. 4.4 and App. A).
* ``cfg_labels_bf16``   - an image-editing flow step under classifier-free
                          guidance: the three CFG contexts (conditional,
                          text dropped, image dropped) as three labels over
                          one paged pool, the image-dropped label reading the
                          conditional label's text pages in place (Sec. 4.1;
                          App. F, CFG Walk).
* ``shared_prefix_decode_bf16`` - one new token for each of many requests over
                          one shared context plus their own tokens (candidates
                          continued from one context, App. A).
* ``queried_prefix_bf16`` - requests over a shared full-attention prefix whose
                          first query rows lie inside that prefix (a shared-
                          prefix group where some rows see only the prefix).
* ``mixed``             - requests of all the kinds above in one launch (one
                          ``LLM`` replica serving every Walk, Sec. 3.2).

Descriptor layout (mirrors the C structs of the library boundary):

* ``seqs``      int32 ``[n, 3]``: ``q_len, kv_len, q_start``.  Queries sit at the
                last ``q_len`` positions of the request's ``kv_len`` keys.
* ``masks``     int32 ``[n, 3]``: ``seg_begin, seg_count, window``.
* ``segments``  int32 ``[S, 4]``: ``start, len, kind, block``; kinds are
                ``CAUSAL`` (0), ``FULL`` (1) and ``BLOCKS`` (2).
* ``block_table`` int32 ``[n, max_blocks]``: physical page of each logical page.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

SEG_CAUSAL = 0
SEG_FULL = 1
SEG_BLOCKS = 2
PAGE = 16

# Sub-seed offsets: every random field has its own stream.
_SUB_LENGTHS = 1
_SUB_PERM = 2
_SUB_Q = 3
_SUB_K = 4
_SUB_V = 5


@dataclasses.dataclass
class Batch:
    """Descriptors of one attention launch (no tensor data)."""

    name: str
    num_qo_heads: int
    num_kv_heads: int
    head_dim: int
    dtype: str  # "f32" or "bf16"
    seqs: np.ndarray
    masks: np.ndarray
    segments: np.ndarray
    block_table: np.ndarray
    num_pages: int
    page_size: int = PAGE
    sm_scale: float = 0.0
    seed: int = 0
    # shared-prefix groups: [(member request indices, prefix_len), ...]; the
    # members' block tables agree on the first prefix_len / 16 pages and all
    # their query rows see those keys (for a cascade plan)
    prefix_groups: Optional[list] = None

    def __post_init__(self):
        if self.sm_scale == 0.0:
            self.sm_scale = float(1.0 / np.sqrt(self.head_dim))

    @property
    def num_seqs(self) -> int:
        return int(self.seqs.shape[0])

    @property
    def total_q(self) -> int:
        if self.num_seqs == 0:
            return 0
        return int((self.seqs[:, 0] + self.seqs[:, 2]).max())

    def seq_segments(self, r: int) -> np.ndarray:
        b, c, _ = self.masks[r]
        return self.segments[b:b + c]


def _rng(seed: int, sub: int) -> np.random.Generator:
    return np.random.default_rng([int(seed), int(sub)])


def _layout_pages(kv_lens, pool_pages: Optional[int], rng, shared_prefix_pages: int = 0):
    """Assign physical pages to requests from a seeded permutation of the pool.

    Pages are handed out in permutation order; the first ``shared_prefix_pages``
    of the permutation are referenced by every request's first logical pages.
    """
    need = [(int(L) + PAGE - 1) // PAGE for L in kv_lens]
    own = [n - shared_prefix_pages for n in need]
    total = shared_prefix_pages + sum(own)
    pool = total if pool_pages is None else int(pool_pages)
    if pool < total:
        raise ValueError("page pool too small")
    perm = rng.permutation(pool).astype(np.int32)
    max_blocks = max(need) if need else 1
    bt = np.full((len(kv_lens), max(max_blocks, 1)), -1, dtype=np.int32)
    shared = perm[:shared_prefix_pages]
    cur = shared_prefix_pages
    for r, n in enumerate(own):
        bt[r, :shared_prefix_pages] = shared
        bt[r, shared_prefix_pages:shared_prefix_pages + n] = perm[cur:cur + n]
        cur += n
    return bt, pool


def _finish(name, hq, hkv, d, dtype, q_lens, kv_lens, seg_lists, windows, bt, pool, seed):
    n = len(q_lens)
    seqs = np.zeros((n, 3), dtype=np.int32)
    masks = np.zeros((n, 3), dtype=np.int32)
    segs = []
    qs = 0
    for r in range(n):
        seqs[r] = (q_lens[r], kv_lens[r], qs)
        qs += q_lens[r]
        masks[r] = (len(segs), len(seg_lists[r]), windows[r])
        segs.extend(seg_lists[r])
    segments = np.array(segs, dtype=np.int32).reshape(-1, 4)
    return Batch(name=name, num_qo_heads=hq, num_kv_heads=hkv, head_dim=d, dtype=dtype,
                 seqs=seqs, masks=masks, segments=segments, block_table=bt,
                 num_pages=pool, seed=seed)


# --------------------------------------------------------------------------
# The five workloads at full size, plus scaled-down variants for tests.
# --------------------------------------------------------------------------

def tiny_causal_f32(seed: int = 0) -> Batch:
    """4 causal prefills of lengths 17, 33, 64, 5; 2 query heads over 1 KV head;
    head_dim 64; fp32; pages permuted by seed."""
    lens = [17, 33, 64, 5]
    bt, pool = _layout_pages(lens, None, _rng(seed, _SUB_PERM))
    segs = [[(0, L, SEG_CAUSAL, 0)] for L in lens]
    return _finish("tiny_causal_f32", 2, 1, 64, "f32", lens, lens, segs, [0] * 4, bt, pool, seed)


def decode_bf16(seed: int = 0, n: int = 64, lmin: int = 512, lmax: int = 8192,
                hq: int = 28, hkv: int = 4, d: int = 128, pool_pages: Optional[int] = 40000) -> Batch:
    """n requests, each one new query token over a context of length
    L ~ U{lmin..lmax} (the new token's K/V is already cached: kv_len = L)."""
    L = _rng(seed, _SUB_LENGTHS).integers(lmin, lmax + 1, size=n)
    kv = [int(x) for x in L]
    bt, pool = _layout_pages(kv, pool_pages, _rng(seed, _SUB_PERM))
    segs = [[(0, x, SEG_CAUSAL, 0)] for x in kv]
    return _finish("decode_bf16", hq, hkv, d, "bf16", [1] * n, kv, segs, [0] * n, bt, pool, seed)


def text_latent_bf16(seed: int = 0, n: int = 8, text: int = 256, latent: int = 4096,
                     hq: int = 28, hkv: int = 4, d: int = 128) -> Batch:
    """n prefills of a causal text prefix followed by a latent block with full
    attention inside the block and full view of the prefix."""
    L = text + latent
    kv = [L] * n
    bt, pool = _layout_pages(kv, None, _rng(seed, _SUB_PERM))
    segs = [[(0, text, SEG_CAUSAL, 0), (text, latent, SEG_FULL, 0)] for _ in range(n)]
    return _finish("text_latent_bf16", hq, hkv, d, "bf16", kv, kv, segs, [0] * n, bt, pool, seed)


def stream_window_bf16(seed: int = 0, n: int = 256, chunk: int = 16, cmin: int = 1024,
                       cmax: int = 16384, window: int = 1024, hq: int = 16, hkv: int = 8,
                       d: int = 128) -> Batch:
    """n requests each appending a causal chunk over an existing context of
    length C ~ U{cmin..cmax}, under a sliding window of ``window`` keys."""
    C = _rng(seed, _SUB_LENGTHS).integers(cmin, cmax + 1, size=n)
    kv = [int(c) + chunk for c in C]
    bt, pool = _layout_pages(kv, None, _rng(seed, _SUB_PERM))
    segs = [[(0, x, SEG_CAUSAL, 0)] for x in kv]
    return _finish("stream_window_bf16", hq, hkv, d, "bf16", [chunk] * n, kv, segs,
                   [window] * n, bt, pool, seed)


def rollout_bf16(seed: int = 0, n: int = 300, prefix: int = 2048, frames: int = 4,
                 frame: int = 256, hq: int = 16, hkv: int = 16, d: int = 64) -> Batch:
    """n candidate rollouts sharing one context of ``prefix`` tokens (its pages
    are referenced by every block table) and each appending ``frames`` frames of
    ``frame`` tokens: full attention inside a frame, causal across frames, full
    view of the prefix.  Only the appended frames are queried."""
    if prefix % PAGE:
        raise ValueError("shared prefix must be page aligned")
    q = frames * frame
    L = prefix + q
    kv = [L] * n
    bt, pool = _layout_pages(kv, None, _rng(seed, _SUB_PERM), shared_prefix_pages=prefix // PAGE)
    segs = [[(0, prefix, SEG_FULL, 0), (prefix, q, SEG_BLOCKS, frame)] for _ in range(n)]
    b = _finish("rollout_bf16", hq, hkv, d, "bf16", [q] * n, kv, segs, [0] * n, bt, pool, seed)
    b.prefix_groups = [(list(range(n)), prefix)]
    return b


def shared_prefix_decode_bf16(seed: int = 0, n: int = 128, prefix: int = 4096, own_min: int = 256,
                              own_max: int = 1024, hq: int = 28, hkv: int = 4, d: int = 128) -> Batch:
    """n requests decoding one token each over one shared ``prefix``-token
    context (its pages are referenced by every block table) followed by their
    own ``own ~ U{own_min..own_max}`` tokens: K candidates or samples continued
    from one context in one batched step (App. A, V-JEPA 2 MPC Walk; Sec. 4.1,
    contexts as labels over one pool).  One prefix group holds every request."""
    if prefix % PAGE:
        raise ValueError("shared prefix must be page aligned")
    own = _rng(seed, _SUB_LENGTHS).integers(own_min, own_max + 1, size=n)
    kv = [prefix + int(x) for x in own]
    bt, pool = _layout_pages(kv, None, _rng(seed, _SUB_PERM), shared_prefix_pages=prefix // PAGE)
    segs = [[(0, L, SEG_CAUSAL, 0)] for L in kv]
    b = _finish("shared_prefix_decode_bf16", hq, hkv, d, "bf16", [1] * n, kv, segs, [0] * n, bt, pool, seed)
    b.prefix_groups = [(list(range(n)), prefix)]
    return b


def cfg_labels_bf16(seed: int = 0, n: int = 2, text: int = 256, image: int = 4096, latent: int = 4096,
                    hq: int = 28, hkv: int = 4, d: int = 128) -> Batch:
    """n image-editing requests at one flow step, each as three CFG labels over
    one page pool; in every label the ``latent`` tokens are the queries and form
    one full-attention block that sees the label's whole context:

    * conditional:   causal text (``text``), full condition image (``image``), latents;
    * text dropped:  full condition image (its own pages), latents;
    * image dropped: causal text, latents.  Its text pages are the conditional
      label's text pages (the same causal prefix, read in place).

    Requests are ordered image by image: conditional, text dropped, image dropped.
    """
    if text % PAGE:
        raise ValueError("the shared text prefix must be page aligned")
    rng = _rng(seed, _SUB_PERM)
    q_lens, kv_lens, seg_lists = [], [], []
    for _ in range(n):
        q_lens += [latent] * 3
        kv_lens += [text + image + latent, image + latent, text + latent]
        seg_lists += [
            [(0, text, SEG_CAUSAL, 0), (text, image, SEG_FULL, 0), (text + image, latent, SEG_FULL, 0)],
            [(0, image, SEG_FULL, 0), (image, latent, SEG_FULL, 0)],
            [(0, text, SEG_CAUSAL, 0), (text, latent, SEG_FULL, 0)],
        ]
    need = [(x + PAGE - 1) // PAGE for x in kv_lens]
    tp = text // PAGE
    own = [need[r] - (tp if r % 3 == 2 else 0) for r in range(len(need))]
    pool = sum(own)
    perm = rng.permutation(pool).astype(np.int32)
    bt = np.full((len(kv_lens), max(need)), -1, dtype=np.int32)
    cur = 0
    for r in range(len(kv_lens)):
        if r % 3 == 2:  # image dropped: the conditional label's text pages, then its own
            bt[r, :tp] = bt[r - 2, :tp]
            bt[r, tp:tp + own[r]] = perm[cur:cur + own[r]]
        else:
            bt[r, :own[r]] = perm[cur:cur + own[r]]
        cur += own[r]
    b = _finish("cfg_labels_bf16", hq, hkv, d, "bf16", q_lens, kv_lens, seg_lists, [0] * len(q_lens),
                bt, pool, seed)
    b.prefix_groups = [([3 * i, 3 * i + 2], text) for i in range(n)]  # conditional + image dropped
    return b


def queried_prefix_bf16(seed: int = 0, n: int = 4, prefix: int = 2048, tail: int = 256, q: int = 400,
                        hq: int = 8, hkv: int = 2, d: int = 128) -> Batch:
    """n requests over one shared ``prefix`` (one full-attention block whose
    pages every block table points to) followed by ``tail`` causal tokens of
    their own; the last ``q`` positions are queried, so the first query rows lie
    inside the prefix's block (they see exactly the prefix) and the rest see the
    prefix plus their causal tail.  One prefix group holds every request."""
    if prefix % PAGE:
        raise ValueError("shared prefix must be page aligned")
    L = prefix + tail
    if not tail < q <= L:
        raise ValueError("the queried rows must start inside the prefix")
    kv = [L] * n
    bt, pool = _layout_pages(kv, None, _rng(seed, _SUB_PERM), shared_prefix_pages=prefix // PAGE)
    segs = [[(0, prefix, SEG_FULL, 0), (prefix, tail, SEG_CAUSAL, 0)] for _ in range(n)]
    b = _finish("queried_prefix_bf16", hq, hkv, d, "bf16", [q] * n, kv, segs, [0] * n, bt, pool, seed)
    b.prefix_groups = [(list(range(n)), prefix)]
    return b


def mixed(seed: int = 0, hq: int = 8, hkv: int = 2, d: int = 128, dtype: str = "bf16",
          scale: int = 1) -> Batch:
    """Requests of every kind in one launch: decode, text+latent prefill,
    windowed chunks, frame-block rollouts over shared prefix pages, and a
    block-causal request with a ragged final block."""
    rng = _rng(seed, _SUB_LENGTHS)
    q_lens, kv_lens, seg_lists, windows = [], [], [], []
    # decode requests
    for L in rng.integers(40, 700 * scale, size=3):
        L = int(L)
        q_lens.append(1); kv_lens.append(L); seg_lists.append([(0, L, SEG_CAUSAL, 0)]); windows.append(0)
    # text + latent prefill
    t, lat = 37, 160 * scale + 3
    q_lens.append(t + lat); kv_lens.append(t + lat)
    seg_lists.append([(0, t, SEG_CAUSAL, 0), (t, lat, SEG_FULL, 0)]); windows.append(0)
    # windowed chunks
    for C in rng.integers(100, 600 * scale, size=2):
        C = int(C)
        q_lens.append(16); kv_lens.append(C + 16); seg_lists.append([(0, C + 16, SEG_CAUSAL, 0)])
        windows.append(96)
    # block-causal with a ragged last block, queried partly
    L = 211 * scale
    q_lens.append(150 * scale); kv_lens.append(L)
    seg_lists.append([(0, 19, SEG_CAUSAL, 0), (19, L - 19, SEG_BLOCKS, 48)]); windows.append(0)
    kv_rollout_start = len(kv_lens)
    # rollouts over one shared prefix (added last so the prefix pages are shared)
    prefix, fr, nf = 64, 32, 3
    n_roll = 3
    for _ in range(n_roll):
        q_lens.append(nf * fr); kv_lens.append(prefix + nf * fr)
        seg_lists.append([(0, prefix, SEG_FULL, 0), (prefix, nf * fr, SEG_BLOCKS, fr)]); windows.append(0)
    # page layout: non-rollout requests get private pages, rollouts share a prefix
    prng = _rng(seed, _SUB_PERM)
    need = [(x + PAGE - 1) // PAGE for x in kv_lens]
    shared_pages = prefix // PAGE
    own = [need[r] - (shared_pages if r >= kv_rollout_start else 0) for r in range(len(need))]
    pool = sum(own) + shared_pages + 7  # a few unreferenced pages
    perm = prng.permutation(pool).astype(np.int32)
    bt = np.full((len(kv_lens), max(need)), -1, dtype=np.int32)
    shared = perm[:shared_pages]
    cur = shared_pages
    for r in range(len(kv_lens)):
        off = 0
        if r >= kv_rollout_start:
            bt[r, :shared_pages] = shared
            off = shared_pages
        bt[r, off:off + own[r]] = perm[cur:cur + own[r]]
        cur += own[r]
    b = _finish("mixed", hq, hkv, d, dtype, q_lens, kv_lens, seg_lists, windows, bt, pool, seed)
    b.prefix_groups = [(list(range(kv_rollout_start, kv_rollout_start + n_roll)), prefix)]
    return b


def serving_mix_bf16(seed: int = 0, n_decode: int = 48, lmin: int = 512, lmax: int = 8192, text: int = 256,
                     latent: int = 4096, n_chunk: int = 64, cmin: int = 1024, cmax: int = 16384,
                     window: int = 1024, n_roll: int = 16, prefix: int = 2048, frames: int = 2, frame: int = 256,
                     hq: int = 28, hkv: int = 4, d: int = 128) -> Batch:
    """One node's batch across Walks (Sec. 3.2: one LLM replica serves requests
    at different graph positions in one launch): decode steps, one image
    request's text + latent prefill, streaming speech chunks under a sliding
    window, and world-model rollout frames over a shared context, with one
    head layout.  The rollouts form a shared-prefix group."""
    rng = _rng(seed, _SUB_LENGTHS)
    q_lens, kv_lens, seg_lists, windows = [], [], [], []
    for L in rng.integers(lmin, lmax + 1, size=n_decode):
        L = int(L)
        q_lens.append(1); kv_lens.append(L); seg_lists.append([(0, L, SEG_CAUSAL, 0)]); windows.append(0)
    q_lens.append(text + latent); kv_lens.append(text + latent)
    seg_lists.append([(0, text, SEG_CAUSAL, 0), (text, latent, SEG_FULL, 0)]); windows.append(0)
    for C in rng.integers(cmin, cmax + 1, size=n_chunk):
        C = int(C)
        q_lens.append(16); kv_lens.append(C + 16); seg_lists.append([(0, C + 16, SEG_CAUSAL, 0)])
        windows.append(window)
    first_roll = len(kv_lens)
    if prefix % PAGE:
        raise ValueError("shared prefix must be page aligned")
    for _ in range(n_roll):
        q_lens.append(frames * frame); kv_lens.append(prefix + frames * frame)
        seg_lists.append([(0, prefix, SEG_FULL, 0), (prefix, frames * frame, SEG_BLOCKS, frame)])
        windows.append(0)
    # private pages for every request; the rollouts' first prefix / 16 pages are shared
    prng = _rng(seed, _SUB_PERM)
    shared_pages = prefix // PAGE
    need = [(x + PAGE - 1) // PAGE for x in kv_lens]
    own = [need[r] - (shared_pages if r >= first_roll else 0) for r in range(len(need))]
    pool = sum(own) + (shared_pages if n_roll else 0)
    perm = prng.permutation(pool).astype(np.int32)
    bt = np.full((len(kv_lens), max(need)), -1, dtype=np.int32)
    cur = shared_pages if n_roll else 0
    for r in range(len(kv_lens)):
        off = 0
        if r >= first_roll:
            bt[r, :shared_pages] = perm[:shared_pages]
            off = shared_pages
        bt[r, off:off + own[r]] = perm[cur:cur + own[r]]
        cur += own[r]
    b = _finish("serving_mix_bf16", hq, hkv, d, "bf16", q_lens, kv_lens, seg_lists, windows, bt, pool, seed)
    b.prefix_groups = [(list(range(first_roll, first_roll + n_roll)), prefix)] if n_roll else None
    return b


def custom(name: str, hq: int, hkv: int, d: int, q_lens, kv_lens, seg_lists, windows, seed: int = 0,
           dtype: str = "bf16", pool_pages: Optional[int] = None, shared_prefix_pages: int = 0) -> Batch:
    """A batch from explicit per-request lengths, segment lists and windows,
    laid out in a seeded permutation of the pool (the first
    ``shared_prefix_pages`` pages shared by every request)."""
    bt, pool = _layout_pages(kv_lens, pool_pages, _rng(seed, _SUB_PERM), shared_prefix_pages)
    return _finish(name, hq, hkv, d, dtype, list(q_lens), list(kv_lens), seg_lists, list(windows), bt, pool, seed)


def window_edges_bf16(seed: int = 0, d: int = 128, hq: int = 16, hkv: int = 8) -> Batch:
    """Sliding windows at their small edges (1 key, fewer keys than a page,
    exactly a page, one more) on every query shape: single-token decode and
    16-token chunks (few-row path) and 300-row prefills (tile path) under
    causal, full-block and block-causal segments, next to windows wider than
    the context."""
    q_lens, kv_lens, seg_lists, windows = [], [], [], []
    rng = _rng(seed, _SUB_LENGTHS)
    for w in (1, 5, 16, 17):
        for q, ctx in ((1, int(rng.integers(40, 900))), (16, int(rng.integers(0, 700)))):
            L = ctx + q
            q_lens.append(q); kv_lens.append(L); seg_lists.append([(0, L, SEG_CAUSAL, 0)]); windows.append(w)
        L = 300 + int(rng.integers(0, 400))
        q_lens.append(300); kv_lens.append(L); seg_lists.append([(0, L, SEG_CAUSAL, 0)]); windows.append(w)
        # full block after a causal head: rows in the block see later keys of it
        q_lens.append(300); kv_lens.append(340)
        seg_lists.append([(0, 40, SEG_CAUSAL, 0), (40, 300, SEG_FULL, 0)]); windows.append(w)
        # frame blocks of 48 with a ragged last one
        q_lens.append(250); kv_lens.append(307)
        seg_lists.append([(0, 19, SEG_CAUSAL, 0), (19, 288, SEG_BLOCKS, 48)]); windows.append(w)
    # windows wider than the whole context
    q_lens.append(16); kv_lens.append(116); seg_lists.append([(0, 116, SEG_CAUSAL, 0)]); windows.append(5000)
    q_lens.append(300); kv_lens.append(300); seg_lists.append([(0, 300, SEG_CAUSAL, 0)]); windows.append(300)
    return custom("window_edges_bf16", hq, hkv, d, q_lens, kv_lens, seg_lists, windows, seed)


def long_items(name: str, seed: int = 0) -> Batch:
    """Small batches whose single work items are long: tile items over 2048
    keys (the tile kernel's page-index ring refills its third window) and
    few-row items over 4096 keys (a wave's page indices span more than one
    register window).  Planned without key splitting, each request's range
    stays one item."""
    if name == "text_latent_long":
        return text_latent_bf16(seed, n=2, text=64, latent=2500, hq=4, hkv=1)
    if name == "rollout_long":
        return rollout_bf16(seed, n=2, prefix=2048, frames=2, frame=128, hq=4, hkv=4, d=64)
    if name == "decode_long":
        return decode_bf16(seed, n=8, lmin=6000, lmax=9000, hq=8, hkv=2, pool_pages=None)
    if name == "chunk_long":
        return stream_window_bf16(seed, n=4, cmin=6000, cmax=9000, window=5000, hq=8, hkv=4)
    raise KeyError(name)


LONG_ITEMS = ["text_latent_long", "rollout_long", "decode_long", "chunk_long"]


FULL_SIZE = {
    "tiny_causal_f32": tiny_causal_f32,
    "decode_bf16": decode_bf16,
    "text_latent_bf16": text_latent_bf16,
    "stream_window_bf16": stream_window_bf16,
    "rollout_bf16": rollout_bf16,
    "cfg_labels_bf16": cfg_labels_bf16,
    "shared_prefix_decode_bf16": shared_prefix_decode_bf16,
    "serving_mix_bf16": serving_mix_bf16,
}


def reduced(name: str, seed: int = 0) -> Batch:
    """Scaled-down variant of a workload: same mask structure and head layout,
    sizes small enough for the CPU oracle to finish in seconds while still
    spanning several tiles and ragged tails."""
    if name == "tiny_causal_f32":
        return tiny_causal_f32(seed)
    if name == "decode_bf16":
        return decode_bf16(seed, n=9, lmin=1, lmax=1500, pool_pages=None)
    if name == "text_latent_bf16":
        return text_latent_bf16(seed, n=2, text=37, latent=300)
    if name == "stream_window_bf16":
        return stream_window_bf16(seed, n=7, cmin=1, cmax=700, window=100)
    if name == "rollout_bf16":
        return rollout_bf16(seed, n=5, prefix=64, frames=4, frame=40)
    if name == "cfg_labels_bf16":
        return cfg_labels_bf16(seed, n=2, text=32, image=101, latent=70, hq=7, hkv=1)
    if name == "shared_prefix_decode_bf16":
        return shared_prefix_decode_bf16(seed, n=37, prefix=320, own_min=1, own_max=150, hq=8, hkv=2)
    if name == "serving_mix_bf16":
        return serving_mix_bf16(seed, n_decode=5, lmin=1, lmax=900, text=37, latent=200, n_chunk=4, cmin=1,
                                cmax=600, window=96, n_roll=3, prefix=64, frames=2, frame=40, hq=7, hkv=1)
    if name == "mixed":
        return mixed(seed)
    if name == "window_edges_bf16":
        return window_edges_bf16(seed)
    if name == "queried_prefix_bf16":
        return queried_prefix_bf16(seed, n=3, prefix=192, tail=64, q=200, hq=4, hkv=1, d=64)
    raise KeyError(name)


# --------------------------------------------------------------------------
# Tensor values.
# --------------------------------------------------------------------------

def tensor_shapes(b: Batch):
    return {
        "q": (b.total_q, b.num_qo_heads, b.head_dim),
        "k_pages": (b.num_pages, b.page_size, b.num_kv_heads, b.head_dim),
        "v_pages": (b.num_pages, b.page_size, b.num_kv_heads, b.head_dim),
    }


def make_tensors_numpy(b: Batch, seed: Optional[int] = None):
    """Q/K/V iid N(0,1) drawn in float32 on the host (small batches only).
    For bf16 batches the values are rounded to bf16 (nearest even) and returned
    as float32 arrays holding exactly the bf16 values."""
    seed = b.seed if seed is None else seed
    out = {}
    for name, sub in (("q", _SUB_Q), ("k_pages", _SUB_K), ("v_pages", _SUB_V)):
        x = _rng(seed, sub).standard_normal(tensor_shapes(b)[name], dtype=np.float32)
        if b.dtype == "bf16":
            x = round_to_bf16(x)
        out[name] = x
    return out


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even); float32 result."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16
    return r.astype(np.uint32).view(np.float32).reshape(x.shape)


def make_tensors_torch(b: Batch, device, seed: Optional[int] = None, poison_unused: bool = False):
    """Q/K/V iid N(0,1) drawn with torch's generator on ``device`` (float32, then
    rounded to the batch dtype).  With ``poison_unused`` every page slot that no
    request references (unreferenced pages and the tail slots of each request's
    last page) is set to NaN."""
    import torch

    seed = b.seed if seed is None else seed
    dt = torch.float32 if b.dtype == "f32" else torch.bfloat16
    g = torch.Generator(device=device)
    out = {}
    for name, sub in (("q", _SUB_Q), ("k_pages", _SUB_K), ("v_pages", _SUB_V)):
        g.manual_seed(int(seed) * 1000003 + sub)
        x = torch.randn(tensor_shapes(b)[name], generator=g, device=device, dtype=torch.float32)
        out[name] = x.to(dt)
        del x
    if poison_unused:
        used = used_slots(b)
        mask = torch.from_numpy(~used).to(device)
        for name in ("k_pages", "v_pages"):
            out[name][mask] = float("nan")
    return out


def used_slots(b: Batch) -> np.ndarray:
    """bool ``[num_pages, page_size]``: slots that hold a key of some request."""
    used = np.zeros((b.num_pages, b.page_size), dtype=bool)
    for r in range(b.num_seqs):
        L = int(b.seqs[r, 1])
        for t0 in range(0, L, b.page_size):
            p = int(b.block_table[r, t0 // b.page_size])
            used[p, :min(b.page_size, L - t0)] = True
    return used


def permute_pages(b: Batch, tensors: dict, seed: int):
    """The same logical batch stored under a different physical page order:
    page ``p`` moves to ``perm[p]`` and block tables are rewritten to match."""
    perm = np.random.default_rng([seed, 99]).permutation(b.num_pages).astype(np.int32)
    bt = b.block_table.copy()
    valid = bt >= 0
    bt[valid] = perm[bt[valid]]
    nb = dataclasses.replace(b, block_table=bt)
    inv = np.empty_like(perm)
    inv[perm] = np.arange(b.num_pages, dtype=np.int32)
    nt = dict(tensors)
    for name in ("k_pages", "v_pages"):
        x = tensors[name]
        nt[name] = x[inv] if isinstance(x, np.ndarray) else x[_as_index(x, inv)]
    return nb, nt


def _as_index(x, idx):
    import torch

    return torch.from_numpy(idx.astype(np.int64)).to(x.device)


def extract_requests(b: Batch, tensors: dict, reqs, to_host=None, key_ranges=None):
    """The requests ``reqs`` of ``b`` as a batch of their own, with only their
    pages (renumbered) and their query rows.  ``tensors`` may live on any
    device; ``to_host`` converts a tensor to a float64 numpy array (default:
    ``.float().cpu().numpy()``).  With ``key_ranges`` (one ``(lo, hi)`` per
    selected request, covering every key its rows may see) only the pages
    holding those keys are copied and the other block-table entries become
    -1.  Returns ``(sub_batch, q, k_pages, v_pages, rows)`` where ``rows`` are
    the packed query rows of the originals."""
    reqs = [int(r) for r in reqs]
    if to_host is None:
        def to_host(t):
            return np.asarray(t.float().cpu().numpy(), dtype=np.float64) if not isinstance(t, np.ndarray) \
                else np.asarray(t, dtype=np.float64)
    bt = b.block_table[reqs].copy()
    if key_ranges is not None:
        for j, (lo, hi) in enumerate(key_ranges):
            keep = np.zeros(bt.shape[1], dtype=bool)
            keep[int(lo) // b.page_size:(int(hi) + b.page_size - 1) // b.page_size] = True
            bt[j, ~keep] = -1
    pages = np.unique(bt[bt >= 0])
    nbt = np.where(bt >= 0, np.searchsorted(pages, bt), -1).astype(np.int32)
    seqs = b.seqs[reqs].copy()
    rows = np.concatenate([np.arange(s[2], s[2] + s[0]) for s in b.seqs[reqs]]).astype(np.int64)
    segl = [[tuple(int(v) for v in x) for x in b.seq_segments(r)] for r in reqs]
    sb = _finish(b.name + "/sub", b.num_qo_heads, b.num_kv_heads, b.head_dim, b.dtype, [int(x) for x in seqs[:, 0]],
                 [int(x) for x in seqs[:, 1]], segl, [int(x) for x in b.masks[reqs, 2]], nbt, len(pages), b.seed)
    kp, vp, q = tensors["k_pages"], tensors["v_pages"], tensors["q"]
    if isinstance(kp, np.ndarray):
        return sb, to_host(q[rows]), to_host(kp[pages]), to_host(vp[pages]), rows
    import torch

    pidx = torch.from_numpy(pages.astype(np.int64)).to(kp.device)
    ridx = torch.from_numpy(rows).to(q.device)
    return sb, to_host(q.index_select(0, ridx)), to_host(kp.index_select(0, pidx)), \
        to_host(vp.index_select(0, pidx)), rows
