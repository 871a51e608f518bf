"""Python binding of the attention library's C-ABI (``include/mstar_attn.h``).

Argument marshalling only: every step of the computation runs in the HIP
library.  PyTorch supplies device memory and streams.  The names follow the C
entry points: :func:`plan` (``mstar_attn_plan``), :meth:`Plan.workspace_bytes`,
:func:`fwd` (``mstar_attn_fwd``), :func:`fwd_noalloc` (``mstar_attn_fwd_noalloc``),
:func:`kv_append` (``mstar_kv_append``),
:func:`check` (``mstar_attn_check``),
:class:`AsyncPlanner` (``mstar_planner_*``), :meth:`Plan.stats`, :meth:`Plan.key_ranges`, :meth:`Plan.items`,
:meth:`Plan.destroy` and :func:`last_error`.

If ``libmstar_attn.so`` has not been built, loading fails loudly; there is no
fallback implementation.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

# MSTAR_ATTN_LIB names another build of the same library (the host-only
# sanitizer build the CPU tests load); by default the in-tree HIP build.
LIB_PATH = os.environ.get("MSTAR_ATTN_LIB") or os.path.join(os.path.dirname(os.path.abspath(__file__)),
                                                            "libmstar_attn.so")

OK = 0
ERR_INVALID_ARG = -1
ERR_UNSUPPORTED = -2
ERR_WORKSPACE = -3
ERR_HIP = -4
ERR_NOMEM = -5

SEG_CAUSAL, SEG_FULL, SEG_BLOCKS = 0, 1, 2
DTYPE_F32, DTYPE_BF16 = 0, 1
FLAG_FORCE_SPLIT, FLAG_NO_SPLIT, FLAG_HOST_ONLY, FLAG_CASCADE_ALL, FLAG_SERIAL = 1, 2, 4, 8, 16
DEVERR_PAGE_RANGE = 1

EXPORTS = [
    "mstar_attn_plan",
    "mstar_attn_plan_cascade",
    "mstar_attn_workspace_bytes",
    "mstar_attn_fwd",
    "mstar_attn_fwd_timed",
    "mstar_attn_fwd_noalloc",
    "mstar_attn_check",
    "mstar_attn_plan_stats",
    "mstar_attn_plan_key_ranges",
    "mstar_attn_plan_items",
    "mstar_attn_plan_tile_order",
    "mstar_attn_plan_cascade_order",
    "mstar_kv_append",
    "mstar_planner_create",
    "mstar_planner_submit",
    "mstar_planner_submit_cascade",
    "mstar_planner_take",
    "mstar_attn_plan_wait",
    "mstar_planner_destroy",
    "mstar_attn_plan_destroy",
    "mstar_last_error",
]


class Segment(ctypes.Structure):
    _fields_ = [("start", ctypes.c_int32), ("len", ctypes.c_int32), ("kind", ctypes.c_int32),
                ("block", ctypes.c_int32)]


class MaskSpec(ctypes.Structure):
    _fields_ = [("seg_begin", ctypes.c_int32), ("seg_count", ctypes.c_int32), ("window", ctypes.c_int32)]


class PrefixGroup(ctypes.Structure):
    _fields_ = [("member_begin", ctypes.c_int32), ("member_count", ctypes.c_int32), ("prefix_len", ctypes.c_int32)]


class SeqDesc(ctypes.Structure):
    _fields_ = [("q_len", ctypes.c_int32), ("kv_len", ctypes.c_int32), ("q_start", ctypes.c_int32)]


class Params(ctypes.Structure):
    _fields_ = [("num_qo_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("page_size", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("max_blocks_per_seq", ctypes.c_int32), ("num_pages", ctypes.c_int32),
                ("flags", ctypes.c_uint32), ("sm_scale", ctypes.c_float)]


class PlanStats(ctypes.Structure):
    _fields_ = [("visible_pairs", ctypes.c_int64), ("prefill_items", ctypes.c_int64),
                ("decode_items", ctypes.c_int64), ("f32_items", ctypes.c_int64),
                ("merge_rows", ctypes.c_int64), ("partial_slots", ctypes.c_int64),
                ("total_q", ctypes.c_int64), ("plan_host_us", ctypes.c_double),
                ("device_bytes", ctypes.c_int64)]


class MStarError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"mstar error {code}: {msg}")
        self.code = code


_lib = None


def lib() -> ctypes.CDLL:
    """Load the built library (raises if it is missing)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2606_12688_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    L.mstar_attn_plan.argtypes = [ctypes.POINTER(Params), ctypes.POINTER(SeqDesc), ctypes.POINTER(MaskSpec), i32,
                                  ctypes.POINTER(Segment), i32, vp, ctypes.POINTER(vp)]
    L.mstar_attn_plan.restype = ctypes.c_int
    L.mstar_attn_plan_cascade.argtypes = [ctypes.POINTER(Params), ctypes.POINTER(SeqDesc), ctypes.POINTER(MaskSpec),
                                          i32, ctypes.POINTER(Segment), i32, ctypes.POINTER(PrefixGroup), i32,
                                          ctypes.POINTER(i32), i32, vp, ctypes.POINTER(vp)]
    L.mstar_attn_plan_cascade.restype = ctypes.c_int
    L.mstar_attn_workspace_bytes.argtypes = [vp]
    L.mstar_attn_workspace_bytes.restype = sz
    L.mstar_attn_fwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    L.mstar_attn_fwd.restype = ctypes.c_int
    L.mstar_attn_fwd_timed.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, sz, vp, vp, vp]
    L.mstar_attn_fwd_timed.restype = ctypes.c_int
    L.mstar_attn_fwd_noalloc.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp]
    L.mstar_attn_fwd_noalloc.restype = ctypes.c_int
    L.mstar_attn_check.argtypes = [vp, vp, ctypes.POINTER(i32)]
    L.mstar_attn_check.restype = ctypes.c_int
    L.mstar_attn_plan_stats.argtypes = [vp, ctypes.POINTER(PlanStats)]
    L.mstar_attn_plan_stats.restype = ctypes.c_int
    L.mstar_attn_plan_key_ranges.argtypes = [vp, vp, i32]
    L.mstar_attn_plan_key_ranges.restype = ctypes.c_int
    L.mstar_attn_plan_items.argtypes = [vp, i32, vp, i64, ctypes.POINTER(i64)]
    L.mstar_attn_plan_items.restype = ctypes.c_int
    L.mstar_attn_plan_tile_order.argtypes = [vp, vp, i64, ctypes.POINTER(i64)]
    L.mstar_attn_plan_tile_order.restype = ctypes.c_int
    L.mstar_attn_plan_cascade_order.argtypes = [vp, vp, i64, ctypes.POINTER(i64)]
    L.mstar_attn_plan_cascade_order.restype = ctypes.c_int
    L.mstar_kv_append.argtypes = [vp, vp, vp, vp, vp, vp, vp]
    L.mstar_kv_append.restype = ctypes.c_int
    L.mstar_planner_create.argtypes = [i32, ctypes.POINTER(vp)]
    L.mstar_planner_create.restype = ctypes.c_int
    L.mstar_planner_submit.argtypes = [vp, ctypes.POINTER(Params), ctypes.POINTER(SeqDesc), ctypes.POINTER(MaskSpec),
                                       i32, ctypes.POINTER(Segment), i32]
    L.mstar_planner_submit.restype = ctypes.c_int
    L.mstar_planner_submit_cascade.argtypes = [vp, ctypes.POINTER(Params), ctypes.POINTER(SeqDesc),
                                               ctypes.POINTER(MaskSpec), i32, ctypes.POINTER(Segment), i32,
                                               ctypes.POINTER(PrefixGroup), i32, ctypes.POINTER(i32), i32]
    L.mstar_planner_submit_cascade.restype = ctypes.c_int
    L.mstar_planner_take.argtypes = [vp, vp, ctypes.POINTER(vp)]
    L.mstar_planner_take.restype = ctypes.c_int
    L.mstar_attn_plan_wait.argtypes = [vp, vp]
    L.mstar_attn_plan_wait.restype = ctypes.c_int
    L.mstar_planner_destroy.argtypes = [vp]
    L.mstar_planner_destroy.restype = None
    L.mstar_attn_plan_destroy.argtypes = [vp]
    L.mstar_attn_plan_destroy.restype = None
    L.mstar_last_error.argtypes = []
    L.mstar_last_error.restype = ctypes.c_char_p
    _lib = L
    return L


def last_error() -> str:
    return lib().mstar_last_error().decode()


def _check_rc(rc: int):
    if rc != OK:
        raise MStarError(rc, last_error())


def _array(ctype, rows, width):
    rows = np.ascontiguousarray(np.asarray(rows, dtype=np.int32).reshape(-1, width))
    n = rows.shape[0]
    arr = (ctype * max(n, 1))()
    if n:
        ctypes.memmove(arr, rows.ctypes.data, rows.nbytes)
    return arr, n


def _stream_handle(stream) -> Optional[int]:
    if stream is None:
        try:
            import torch

            if torch.cuda.is_available():
                return torch.cuda.current_stream().cuda_stream
        except Exception:
            pass
        return None
    return getattr(stream, "cuda_stream", stream)


class Plan:
    """Owns an ``mstar_plan_t``.  Build with :func:`plan`."""

    def __init__(self, handle: int, params: Params, num_seqs: int, total_q: int):
        self._h = ctypes.c_void_p(handle)
        self.params = params
        self.num_seqs = num_seqs
        self.total_q = total_q

    @property
    def handle(self):
        if not self._h:
            raise ValueError("plan destroyed")
        return self._h

    @property
    def workspace_bytes(self) -> int:
        return int(lib().mstar_attn_workspace_bytes(self.handle))

    def stats(self) -> dict:
        st = PlanStats()
        _check_rc(lib().mstar_attn_plan_stats(self.handle, ctypes.byref(st)))
        return {f: getattr(st, f) for f, _ in PlanStats._fields_}

    def key_ranges(self) -> np.ndarray:
        out = np.zeros((max(self.num_seqs, 1), 2), dtype=np.int32)
        _check_rc(lib().mstar_attn_plan_key_ranges(self.handle, out.ctypes.data, self.num_seqs))
        return out[: self.num_seqs]

    def items(self, kind: int) -> np.ndarray:
        cnt = ctypes.c_int64(0)
        _check_rc(lib().mstar_attn_plan_items(self.handle, kind, None, 0, ctypes.byref(cnt)))
        out = np.zeros((max(cnt.value, 1), 8), dtype=np.int32)
        _check_rc(lib().mstar_attn_plan_items(self.handle, kind, out.ctypes.data, cnt.value, ctypes.byref(cnt)))
        return out[: cnt.value]

    def tile_order(self, cascade: bool = False) -> np.ndarray:
        """(tile item, query head) of every multi-row workgroup in launch order, as an int32 [n, 2] array
        (``mstar_attn_plan_tile_order``, or ``mstar_attn_plan_cascade_order`` for the cascade kernel);
        (-1, -1) marks padding."""
        fn = lib().mstar_attn_plan_cascade_order if cascade else lib().mstar_attn_plan_tile_order
        cnt = ctypes.c_int64(0)
        _check_rc(fn(self.handle, None, 0, ctypes.byref(cnt)))
        out = np.zeros((cnt.value, 2), dtype=np.int32)
        _check_rc(fn(self.handle, out.ctypes.data, cnt.value, ctypes.byref(cnt)))
        return out

    def destroy(self):
        if self._h:
            lib().mstar_attn_plan_destroy(self._h)
            self._h = ctypes.c_void_p(None)

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass


def _descriptors(num_qo_heads, num_kv_heads, head_dim, dtype, seqs, masks, segments, max_blocks_per_seq,
                 num_pages, sm_scale, flags, page_size):
    p = Params()
    p.num_qo_heads, p.num_kv_heads, p.head_dim, p.page_size = num_qo_heads, num_kv_heads, head_dim, page_size
    p.dtype = {"f32": DTYPE_F32, "bf16": DTYPE_BF16}[dtype] if isinstance(dtype, str) else int(dtype)
    p.max_blocks_per_seq, p.num_pages, p.flags = max_blocks_per_seq, num_pages, flags
    p.sm_scale = float(sm_scale) if sm_scale is not None else float(1.0 / np.sqrt(head_dim))
    s_arr, n = _array(SeqDesc, seqs, 3)
    m_arr, nm = _array(MaskSpec, masks, 3)
    g_arr, ns = _array(Segment, segments, 4)
    if nm != n:
        raise ValueError("seqs and masks differ in length")
    sq = np.asarray(seqs, dtype=np.int64).reshape(-1, 3)
    total_q = int((sq[:, 0] + sq[:, 2]).max()) if n else 0
    return p, s_arr, n, m_arr, g_arr, ns, total_q


def _groups(prefix_groups):
    """``[(member request indices, prefix_len), ...]`` -> mstar_prefix_group array and member array."""
    members = [int(r) for mem, _ in prefix_groups for r in mem]
    gr = (PrefixGroup * len(prefix_groups))()
    k = 0
    for i, (mem, plen) in enumerate(prefix_groups):
        gr[i].member_begin, gr[i].member_count, gr[i].prefix_len = k, len(mem), int(plen)
        k += len(mem)
    mem_arr = (ctypes.c_int32 * max(len(members), 1))(*members)
    return gr, len(prefix_groups), mem_arr, len(members)


def plan(num_qo_heads: int, num_kv_heads: int, head_dim: int, dtype: str, seqs, masks, segments,
         max_blocks_per_seq: int, num_pages: int, sm_scale: Optional[float] = None, flags: int = 0,
         stream=None, page_size: int = 16, prefix_groups=None) -> Plan:
    """``mstar_attn_plan``: ``seqs [n,3]`` (q_len, kv_len, q_start), ``masks [n,3]``
    (seg_begin, seg_count, window), ``segments [S,4]`` (start, len, kind, block).
    With ``prefix_groups`` (``[(member request indices, prefix_len), ...]``),
    ``mstar_attn_plan_cascade``."""
    p, s_arr, n, m_arr, g_arr, ns, total_q = _descriptors(num_qo_heads, num_kv_heads, head_dim, dtype, seqs, masks,
                                                          segments, max_blocks_per_seq, num_pages, sm_scale,
                                                          flags, page_size)
    h = ctypes.c_void_p(None)
    stream_h = None if flags & FLAG_HOST_ONLY else _stream_handle(stream)
    if prefix_groups:
        gr, ng, mem_arr, nm = _groups(prefix_groups)
        _check_rc(lib().mstar_attn_plan_cascade(ctypes.byref(p), s_arr, m_arr, n, g_arr, ns, gr, ng, mem_arr, nm,
                                                stream_h, ctypes.byref(h)))
    else:
        _check_rc(lib().mstar_attn_plan(ctypes.byref(p), s_arr, m_arr, n, g_arr, ns, stream_h, ctypes.byref(h)))
    return Plan(h.value, p, n, total_q)


class AsyncPlanner:
    """``mstar_planner_*``: plans built in submission order on a native worker
    thread with its own HIP stream, at most ``depth`` outstanding (double
    buffering with the default 2).  :meth:`submit` takes the arguments of
    :func:`plan` (without ``stream``; with ``prefix_groups`` it is
    ``mstar_planner_submit_cascade``); :meth:`take` returns the oldest plan
    after making ``stream`` wait for its upload."""

    def __init__(self, depth: int = 2):
        h = ctypes.c_void_p(None)
        _check_rc(lib().mstar_planner_create(int(depth), ctypes.byref(h)))
        self._h = h
        self._pending = []

    def submit(self, num_qo_heads, num_kv_heads, head_dim, dtype, seqs, masks, segments, max_blocks_per_seq,
               num_pages, sm_scale=None, flags=0, page_size=16, prefix_groups=None):
        p, s_arr, n, m_arr, g_arr, ns, total_q = _descriptors(num_qo_heads, num_kv_heads, head_dim, dtype, seqs,
                                                              masks, segments, max_blocks_per_seq, num_pages,
                                                              sm_scale, flags, page_size)
        if prefix_groups:
            gr, ng, mem_arr, nm = _groups(prefix_groups)
            _check_rc(lib().mstar_planner_submit_cascade(self._h, ctypes.byref(p), s_arr, m_arr, n, g_arr, ns, gr, ng,
                                                         mem_arr, nm))
        else:
            _check_rc(lib().mstar_planner_submit(self._h, ctypes.byref(p), s_arr, m_arr, n, g_arr, ns))
        self._pending.append((p, n, total_q))

    def take(self, stream=None) -> Plan:
        if not self._pending:
            raise MStarError(ERR_INVALID_ARG, "no plan was submitted")
        p, n, total_q = self._pending.pop(0)
        h = ctypes.c_void_p(None)
        stream_h = None if p.flags & FLAG_HOST_ONLY else _stream_handle(stream)
        _check_rc(lib().mstar_planner_take(self._h, stream_h, ctypes.byref(h)))
        return Plan(h.value, p, n, total_q)

    def close(self):
        if self._h:
            lib().mstar_planner_destroy(self._h)
            self._h = ctypes.c_void_p(None)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _need(cond, msg):
    if not cond:
        raise ValueError(msg)


def _check_fwd_tensors(pl: Plan, q, k_pages, v_pages, block_table, out, lse):
    """Shapes, dtypes and devices, so that the kernels never read outside the
    tensors."""
    import torch

    p = pl.params
    dt = torch.float32 if p.dtype == DTYPE_F32 else torch.bfloat16
    D, hq, hkv = p.head_dim, p.num_qo_heads, p.num_kv_heads
    dev = q.device
    for name, t in (("q", q), ("k_pages", k_pages), ("v_pages", v_pages), ("block_table", block_table),
                    ("out", out), ("lse", lse)):
        _need(t.is_cuda and t.device == dev, f"{name} must be on {dev}")
        _need(t.is_contiguous(), f"{name} must be contiguous")
    _need(q.dtype == dt and out.dtype == dt and k_pages.dtype == dt and v_pages.dtype == dt, "dtype mismatch")
    _need(tuple(q.shape) == (pl.total_q, hq, D) and tuple(out.shape) == (pl.total_q, hq, D),
          f"q/out must be [{pl.total_q}, {hq}, {D}]")
    _need(tuple(lse.shape) == (pl.total_q, hq) and lse.dtype == torch.float32, "lse must be float32 [total_q, Hq]")
    kv_shape = (p.num_pages, p.page_size, hkv, D)
    _need(tuple(k_pages.shape) == kv_shape and tuple(v_pages.shape) == kv_shape, f"pages must be {kv_shape}")
    _need(block_table.dtype == torch.int32 and tuple(block_table.shape) == (pl.num_seqs, p.max_blocks_per_seq),
          f"block_table must be int32 [{pl.num_seqs}, {p.max_blocks_per_seq}]")
    return dev


def fwd(pl: Plan, q, k_pages, v_pages, block_table, out, lse, workspace=None, stream=None):
    """``mstar_attn_fwd`` on torch tensors."""
    dev = _check_fwd_tensors(pl, q, k_pages, v_pages, block_table, out, lse)
    need = pl.workspace_bytes
    ws_ptr, ws_bytes = None, 0
    if workspace is not None:
        _need(workspace.is_cuda and workspace.device == dev and workspace.is_contiguous(), "bad workspace")
        ws_ptr, ws_bytes = workspace.data_ptr(), workspace.numel() * workspace.element_size()
    if need > 0 and ws_bytes < need:
        raise MStarError(ERR_WORKSPACE, f"workspace of {need} bytes required")
    _check_rc(lib().mstar_attn_fwd(pl.handle, q.data_ptr(), k_pages.data_ptr(), v_pages.data_ptr(),
                                   block_table.data_ptr(), out.data_ptr(), lse.data_ptr(), ws_ptr, ws_bytes,
                                   _stream_handle(stream)))


def fwd_noalloc(pl: Plan, q, k_pages, v_pages, block_table, out, lse, stream=None):
    """``mstar_attn_fwd_noalloc`` on torch tensors: split-K partials in the
    library's static device scratch instead of a workspace."""
    _check_fwd_tensors(pl, q, k_pages, v_pages, block_table, out, lse)
    _check_rc(lib().mstar_attn_fwd_noalloc(pl.handle, q.data_ptr(), k_pages.data_ptr(), v_pages.data_ptr(),
                                           block_table.data_ptr(), out.data_ptr(), lse.data_ptr(),
                                           _stream_handle(stream)))


def kv_append(pl: Plan, k_new, v_new, block_table, k_pages, v_pages, stream=None):
    """``mstar_kv_append`` on torch tensors: write the plan's new K/V rows
    (``[total_q, Hkv, d]``, the same row numbering as q) into their pages."""
    import torch

    p = pl.params
    dt = torch.float32 if p.dtype == DTYPE_F32 else torch.bfloat16
    dev = k_new.device
    for name, t in (("k_new", k_new), ("v_new", v_new), ("block_table", block_table), ("k_pages", k_pages),
                    ("v_pages", v_pages)):
        _need(t.is_cuda and t.device == dev, f"{name} must be on {dev}")
        _need(t.is_contiguous(), f"{name} must be contiguous")
    _need(k_new.dtype == dt and v_new.dtype == dt and k_pages.dtype == dt and v_pages.dtype == dt, "dtype mismatch")
    row = (pl.total_q, p.num_kv_heads, p.head_dim)
    _need(tuple(k_new.shape) == row and tuple(v_new.shape) == row, f"k_new/v_new must be {list(row)}")
    kv_shape = (p.num_pages, p.page_size, p.num_kv_heads, p.head_dim)
    _need(tuple(k_pages.shape) == kv_shape and tuple(v_pages.shape) == kv_shape, f"pages must be {kv_shape}")
    _need(block_table.dtype == torch.int32 and tuple(block_table.shape) == (pl.num_seqs, p.max_blocks_per_seq),
          f"block_table must be int32 [{pl.num_seqs}, {p.max_blocks_per_seq}]")
    _check_rc(lib().mstar_kv_append(pl.handle, k_new.data_ptr(), v_new.data_ptr(), block_table.data_ptr(),
                                    k_pages.data_ptr(), v_pages.data_ptr(), _stream_handle(stream)))


def check(pl: Plan, stream=None) -> int:
    """``mstar_attn_check``: synchronize and return (and clear) the device error bits."""
    bits = ctypes.c_int32(0)
    rc = lib().mstar_attn_check(pl.handle, _stream_handle(stream), ctypes.byref(bits))
    if rc not in (OK, ERR_INVALID_ARG):
        _check_rc(rc)
    return int(bits.value)


def workspace(pl: Plan, device):
    """A device buffer of the plan's workspace size (or None if none is needed)."""
    import torch

    n = pl.workspace_bytes
    return torch.empty(n, dtype=torch.uint8, device=device) if n else None
