"""PaDoc tree attention on MI355X: thin Python binding of ``libpadoc_attn``.

Every step of the computation runs in the HIP library; this module only
marshals arguments.  PyTorch provides device memory and the current stream.

    segs = segments_from_pages(pages, block_size=0)        # tree -> segments
    plan = TreePlan(segs, Hq, Hkv, d, "bf16", block_size=0,
                    num_kv_rows=T, num_q_rows=n_q)
    o, lse = tree_attn_fwd(q, k, v, plan)                    # packed forward
    o, lse = branch_decode(q, k_cache, v_cache, bt, plan)    # paged decode step
"""
from __future__ import annotations

import ctypes as C
import math
from typing import Optional, Sequence

import numpy as np

from . import _lib
from ._lib import PadocError, SEGMENT_DTYPE, WORK_DTYPE, RANGE_DTYPE, BWD_DTYPE

__all__ = ["TreePlan", "segments_from_pages", "segments_layout", "tree_attn_fwd", "tree_attn_bwd", "branch_decode",
           "DecodeSession", "tree_depths", "tree_remaining", "cache_from_rows", "PadocError", "SEGMENT_DTYPE", "version", "set_kernel_events", "make_workspace"]

_DTYPES = {"f32": _lib.F32, "fp32": _lib.F32, "float32": _lib.F32, "bf16": _lib.BF16, "bfloat16": _lib.BF16}


def version() -> str:
    return _lib.lib().padoc_version().decode()


def _page_struct(pg, keep):
    get = (lambda k: pg[k]) if isinstance(pg, dict) else (lambda k: getattr(pg, k))
    br = list(get("branches"))
    bget = lambda b, k: b[k] if isinstance(b, dict) else getattr(b, k)
    f = np.ascontiguousarray([bget(b, "fork") for b in br], dtype=np.int32)
    ln = np.ascontiguousarray([bget(b, "length") for b in br], dtype=np.int32)
    ql = np.ascontiguousarray([bget(b, "q_len") for b in br], dtype=np.int32)
    keep.extend([f, ln, ql])
    P = C.POINTER(C.c_int32)
    return _lib.Page(int(get("prefix_len")), int(get("prefix_q")), int(get("stream_len")), int(get("stream_q")),
                     len(br), f.ctypes.data_as(P), ln.ctypes.data_as(P), ql.ctypes.data_as(P))


def segments_from_pages(pages: Sequence, block_size: int = 0) -> np.ndarray:
    """Pages ``[prefix | stream | Y_1..Y_N]`` -> segment records in packed
    order (``padoc_tree_from_pages``)."""
    L = _lib.lib()
    keep: list = []
    arr = (_lib.Page * max(1, len(pages)))(*[_page_struct(p, keep) for p in pages])
    n = C.c_int32(0)
    L.padoc_tree_from_pages(arr, len(pages), block_size, None, 0, C.byref(n))
    out = np.zeros(n.value, dtype=SEGMENT_DTYPE)
    _lib.check(L.padoc_tree_from_pages(arr, len(pages), block_size, out.ctypes.data_as(C.c_void_p),
                                       n.value, C.byref(n)))
    return out


def segments_layout(nodes, block_size: int = 0) -> np.ndarray:
    """Generic nodes ``(parent, fork, len, q_len)`` -> segment records with the
    canonical packed offsets (``padoc_tree_layout``)."""
    out = np.zeros(len(nodes), dtype=SEGMENT_DTYPE)
    for i, n in enumerate(nodes):
        if isinstance(n, tuple):
            out[i] = (n[0], n[1], n[2], n[3], 0, 0)
        else:
            out[i] = (n.parent, n.fork, n.length, n.q_len, 0, 0)
    _lib.check(_lib.lib().padoc_tree_layout(out.ctypes.data_as(C.c_void_p), len(out), block_size))
    return out


def tree_depths(segments: np.ndarray):
    """Per page root of a segment tree: ``(root index, D_seq, D_crit)``
    arrays (``padoc_tree_depths``: sequential decoding depth and concurrent
    critical path, Sec. 3.1 / App. D); ``R_step = 1 - D_crit / D_seq``."""
    segs = np.ascontiguousarray(segments, dtype=SEGMENT_DTYPE)
    n = len(segs)
    d_seq = np.zeros(n, np.int64)
    d_crit = np.zeros(n, np.int64)
    _lib.check(_lib.lib().padoc_tree_depths(segs.ctypes.data if n else None, n, d_seq.ctypes.data,
                                            d_crit.ctypes.data))
    roots = np.nonzero(segs["parent"] < 0)[0]
    return roots, d_seq[roots], d_crit[roots]


def tree_remaining(segments: np.ndarray, progress=None) -> np.ndarray:
    """Remaining critical path of every segment (``padoc_tree_remaining``,
    Sec. 3.1) when segment s has produced ``progress[s]`` tokens (None: 0);
    int64, one entry per segment."""
    segs = np.ascontiguousarray(segments, dtype=SEGMENT_DTYPE)
    n = len(segs)
    prog = None
    if progress is not None:
        prog = np.ascontiguousarray(progress, dtype=np.int32)
        if prog.shape != (n,):
            raise ValueError(f"progress needs one entry per segment ({n}), got shape {prog.shape}")
    out = np.zeros(n, np.int64)
    _lib.check(_lib.lib().padoc_tree_remaining(segs.ctypes.data if n else None, n,
                                               prog.ctypes.data if prog is not None and n else None,
                                               out.ctypes.data if n else None))
    return out


def cache_from_rows(k_rows, v_rows, k_cache=None, v_cache=None, stream=None):
    """Paged K/V blocks in row layout ``[num_blocks, Hkv, 16, d]`` rewritten
    into the library's paged layouts (``padoc_cache_from_rows``): K
    ``[num_blocks, Hkv, d/8, 16, 8]``, V ``[num_blocks, Hkv, d, 16]``, block
    for block.  Returns ``(k_cache, v_cache)`` (allocated when not given)."""
    import torch
    if k_rows.dim() != 4 or k_rows.shape[2] != 16 or tuple(v_rows.shape) != tuple(k_rows.shape):
        raise ValueError("k_rows / v_rows must both be [num_blocks, Hkv, 16, d]")
    nb, hkv, _, d = k_rows.shape
    dt = k_rows.dtype
    if dt not in (torch.bfloat16, torch.float32) or v_rows.dtype != dt:
        raise ValueError("k_rows / v_rows must share dtype bfloat16 or float32")
    dev = k_rows.device
    for name, t in (("k_rows", k_rows), ("v_rows", v_rows)):
        _check_tensor(name, t, dt, dev)
    if k_cache is None:
        k_cache = torch.empty((nb, hkv, d // 8, 16, 8), dtype=dt, device=dev)
    if v_cache is None:
        v_cache = torch.empty((nb, hkv, d, 16), dtype=dt, device=dev)
    for name, t, shape in (("k_cache", k_cache, (nb, hkv, d // 8, 16, 8)), ("v_cache", v_cache, (nb, hkv, d, 16))):
        _check_tensor(name, t, dt, dev)
        if tuple(t.shape) != shape:
            raise ValueError(f"{name} must be {shape}")
    s = torch.cuda.current_stream(dev) if stream is None else stream
    _lib.check(_lib.lib().padoc_cache_from_rows(_ptr(k_rows), _ptr(v_rows), _ptr(k_cache), _ptr(v_cache), int(nb),
                                                int(hkv), int(d), _lib.BF16 if dt == torch.bfloat16 else _lib.F32,
                                                C.c_void_p(s.cuda_stream)))
    return k_cache, v_cache


class TreePlan:
    """A validated tree and its schedule (``padoc_plan``)."""

    def __init__(self, segments: np.ndarray, num_heads_q: int, num_heads_kv: int, head_dim: int,
                 dtype: str = "bf16", block_size: int = 0, num_kv_rows: int = 0, num_q_rows: Optional[int] = None,
                 softmax_scale: Optional[float] = None, block_table_host: Optional[np.ndarray] = None,
                 block_table_len: Optional[int] = None, max_chunk_keys: int = 0, target_workgroups: int = 0):
        segs = np.ascontiguousarray(segments, dtype=SEGMENT_DTYPE)
        self.segments = segs
        self.num_heads_q, self.num_heads_kv, self.head_dim = num_heads_q, num_heads_kv, head_dim
        self.dtype = dtype
        self.block_size = block_size
        if num_q_rows is None:
            num_q_rows = int((segs["q_off"] + segs["q_len"]).max()) if len(segs) else 0
        self.num_q_rows = num_q_rows
        self.softmax_scale = 1.0 / math.sqrt(head_dim) if softmax_scale is None else softmax_scale
        bt = None
        if block_table_host is not None:
            bt = np.ascontiguousarray(block_table_host, dtype=np.int32)
            if block_table_len is None:
                block_table_len = bt.size
        if block_table_len is None:
            block_table_len = 0
        self.block_table_len = block_table_len
        desc = _lib.TreeDesc(len(segs), segs.ctypes.data if len(segs) else None, num_heads_q, num_heads_kv,
                             head_dim, float(self.softmax_scale), _DTYPES[dtype], block_size, int(num_kv_rows),
                             int(num_q_rows), bt.ctypes.data if bt is not None else None, int(block_table_len),
                             int(max_chunk_keys), int(target_workgroups))
        h = C.c_void_p()
        L = _lib.lib()
        _lib.check(L.padoc_plan_create(C.byref(desc), C.byref(h)))
        self._h = h
        sz = C.c_size_t(0)
        _lib.check(L.padoc_plan_workspace_bytes(h, C.byref(sz)))
        self.workspace_bytes = sz.value
        self._ws = None

    @property
    def handle(self):
        if self._h is None:
            raise ValueError("plan is closed")
        return self._h

    def close(self):
        if getattr(self, "_h", None) is not None:
            _lib.lib().padoc_plan_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def export(self) -> dict:
        """Schedule as numpy arrays (copies)."""
        return _export_schedule(self.handle)

    def backward_workspace_bytes(self) -> int:
        n = C.c_size_t(0)
        _lib.check(_lib.lib().padoc_plan_backward_workspace_bytes(self.handle, C.byref(n)))
        return int(n.value)

    def backward_workspace(self, device):
        """A cached device workspace for the backward (256-byte aligned)."""
        import torch
        if getattr(self, "_bws", None) is None or self._bws[0] != torch.device(device):
            nb = self.backward_workspace_bytes()
            raw = torch.empty(nb + 256, dtype=torch.uint8, device=device)
            off = (-raw.data_ptr()) % 256
            self._bws = (torch.device(device), raw, raw[off: off + nb])
        return self._bws[2]

    def workspace(self, device):
        """A cached device workspace of the plan's size (256-byte aligned)."""
        import torch
        if self._ws is None or self._ws[0] != torch.device(device):
            raw = torch.empty(self.workspace_bytes + 256, dtype=torch.uint8, device=device)
            off = (-raw.data_ptr()) % 256
            self._ws = (torch.device(device), raw, raw[off: off + self.workspace_bytes])
        return self._ws[2]


def _carray(ptr, n, dt):
    if n == 0 or not ptr:
        return np.zeros(0, dtype=dt)
    buf = (C.c_char * (int(n) * np.dtype(dt).itemsize)).from_address(ptr)
    return np.frombuffer(buf, dtype=dt).copy()


def _export_schedule(handle) -> dict:
    v = _lib.ScheduleView()
    _lib.check(_lib.lib().padoc_plan_export(handle, C.byref(v)))
    arr = _carray
    return {
        "kind": v.kind, "tile_cols": v.tile_cols, "tile_keys": v.tile_keys, "n_work_shared": v.n_work_shared,
        "work": arr(v.work, v.n_work, WORK_DTYPE), "ranges": arr(v.ranges, v.n_range, RANGE_DTYPE),
        "lims": arr(v.lims, v.n_lim, np.int32), "toks": arr(v.toks, v.n_tok, np.int32),
        "tile_class": arr(v.tile_class, v.n_tile_class, np.int8),
        "tile_class_off": arr(v.tile_class_off, v.n_range, np.int64),
        "comb_ptr": arr(v.comb_ptr, v.n_comb_ptr, np.int32), "comb_slot": arr(v.comb_slot, v.n_comb, np.int32),
        "comb_rows": arr(v.comb_rows, v.n_comb_rows, np.int32),
        "bwd": arr(v.bwd, v.n_bwd, BWD_DTYPE), "btoks": arr(v.btoks, v.n_btok, np.int32),
        "blims": arr(v.blims, v.n_blim, np.int32),
        "n_slots": v.n_slots, "workspace_bytes": v.workspace_bytes,
    }


def make_workspace(plan: TreePlan, device):
    return plan.workspace(device)


def _ptr(t):
    return C.c_void_p(t.data_ptr())


def _check_tensor(name, t, dtype, device):
    import torch
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if t.dtype != dtype:
        raise TypeError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _torch_dtype(plan):
    import torch
    return torch.bfloat16 if _DTYPES[plan.dtype] == _lib.BF16 else torch.float32


def _outputs(plan, q, out, lse):
    import torch
    if out is None:
        out = torch.empty(plan.num_q_rows, plan.num_heads_q, plan.head_dim, dtype=q.dtype, device=q.device)
    if lse is None:
        lse = torch.empty(plan.num_q_rows, plan.num_heads_q, dtype=torch.float32, device=q.device)
    return out, lse


def tree_attn_fwd(q, k, v, plan: TreePlan, out=None, lse=None, workspace=None, stream=None):
    """Packed forward (``padoc_tree_attn_fwd``).  q ``[n_q, Hq, d]``; k, v
    ``[T, Hkv, d]``; returns ``(O [n_q, Hq, d], LSE [n_q, Hq] float32)``."""
    import torch
    dt = _torch_dtype(plan)
    dev = q.device
    for name, t in (("q", q), ("k", k), ("v", v)):
        _check_tensor(name, t, dt, dev)
    out, lse = _outputs(plan, q, out, lse)
    ws = plan.workspace(dev) if workspace is None else workspace
    s = torch.cuda.current_stream(dev) if stream is None else stream
    _lib.check(_lib.lib().padoc_tree_attn_fwd(plan.handle, _ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse),
                                              _ptr(ws), ws.numel(), C.c_void_p(s.cuda_stream)))
    return out, lse


def _repeat_call(plan, key):
    """The C arguments of the plan's previous call when this call passes the
    same tensors (same objects at the same addresses) on the same stream,
    else None.  A decode loop calls with the same buffers every step; this
    skips the per-call checks and argument marshalling."""
    last = getattr(plan, "_last_call", None)
    return last[1] if last is not None and last[0] == key else None


def branch_decode(q, k_cache, v_cache, block_table, plan: TreePlan, out=None, lse=None, workspace=None,
                  stream=None):
    """Decode step over a paged cache (``padoc_branch_decode``).  q ``[n_q,
    Hq, d]``; K cache chunk-major ``[blocks, Hkv, d/8, 16, 8]``, V cache
    d-major ``[blocks, Hkv, d, 16]`` (layouts in ``padoc_attn.h``);
    block_table int32 on the device; returns ``(O, LSE)``."""
    import torch
    if out is not None and lse is not None and workspace is not None:
        s = torch.cuda.current_stream(q.device) if stream is None else stream
        key = ("decode", plan.handle, s.cuda_stream) + tuple(
            (id(t), t.data_ptr(), t.shape, t.stride(), t.dtype) for t in (q, k_cache, v_cache, block_table, out, lse, workspace))
        args = _repeat_call(plan, key)
        if args is not None:
            _lib.check(_lib.lib().padoc_branch_decode(*args))
            return out, lse
    dt = _torch_dtype(plan)
    dev = q.device
    for name, t in (("q", q), ("k_cache", k_cache), ("v_cache", v_cache)):
        _check_tensor(name, t, dt, dev)
    _check_tensor("block_table", block_table, torch.int32, dev)
    out, lse = _outputs(plan, q, out, lse)
    ws = plan.workspace(dev) if workspace is None else workspace
    s = torch.cuda.current_stream(dev) if stream is None else stream
    args = (plan.handle, _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(block_table), _ptr(out), _ptr(lse), _ptr(ws),
            ws.numel(), C.c_void_p(s.cuda_stream))
    _lib.check(_lib.lib().padoc_branch_decode(*args))
    if workspace is not None:
        plan._last_call = (("decode", plan.handle, s.cuda_stream) + tuple(
            (id(t), t.data_ptr(), t.shape, t.stride(), t.dtype) for t in (q, k_cache, v_cache, block_table, out, lse, workspace)),
            args)
    return out, lse


NO_ALLOC_WORKSPACE_BYTES = 64 << 20   # PADOC_NO_ALLOC_WORKSPACE_BYTES


def plan_upload(plan: TreePlan, workspace, stream=None):
    """Copy a decode plan's schedule into ``workspace`` (``padoc_plan_upload``)
    for ``branch_decode_resident`` calls: every layer of a decode step runs
    over the same tree, so one upload serves all of them."""
    import torch
    _check_tensor("workspace", workspace, torch.uint8, workspace.device)
    s = torch.cuda.current_stream(workspace.device) if stream is None else stream
    _lib.check(_lib.lib().padoc_plan_upload(plan.handle, _ptr(workspace), workspace.numel(),
                                            C.c_void_p(s.cuda_stream)))
    return workspace


def branch_decode_resident(q, k_cache, v_cache, block_table, plan: TreePlan, out, lse, workspace, stream=None):
    """Decode step on a workspace that holds the plan's schedule
    (``padoc_branch_decode_resident``, after ``plan_upload``): the kernels of
    ``branch_decode`` without the schedule copy."""
    import torch
    s = torch.cuda.current_stream(q.device) if stream is None else stream
    key = ("resident", plan.handle, s.cuda_stream) + tuple(
        (id(t), t.data_ptr(), t.shape, t.stride(), t.dtype) for t in (q, k_cache, v_cache, block_table, out, lse, workspace))
    args = _repeat_call(plan, key)
    if args is None:
        dt = _torch_dtype(plan)
        dev = q.device
        for name, t in (("q", q), ("k_cache", k_cache), ("v_cache", v_cache), ("out", out)):
            _check_tensor(name, t, dt, dev)
        _check_tensor("block_table", block_table, torch.int32, dev)
        _check_tensor("lse", lse, torch.float32, dev)
        _check_tensor("workspace", workspace, torch.uint8, dev)
        args = (plan.handle, _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(block_table), _ptr(out), _ptr(lse),
                _ptr(workspace), workspace.numel(), C.c_void_p(s.cuda_stream))
    _lib.check(_lib.lib().padoc_branch_decode_resident(*args))
    plan._last_call = (key, args)
    return out, lse


def branch_decode_no_alloc(q, k_cache, v_cache, block_table, plan: TreePlan, out, lse, stream=None):
    """Decode step with the library's fixed per-GPU workspace
    (``padoc_branch_decode_no_alloc``): the caller passes every input and
    both outputs; nothing is allocated.  Calls that overlap on one GPU race
    on that workspace."""
    import torch
    dt = _torch_dtype(plan)
    dev = q.device
    for name, t in (("q", q), ("k_cache", k_cache), ("v_cache", v_cache), ("out", out)):
        _check_tensor(name, t, dt, dev)
    _check_tensor("block_table", block_table, torch.int32, dev)
    _check_tensor("lse", lse, torch.float32, dev)
    s = torch.cuda.current_stream(dev) if stream is None else stream
    _lib.check(_lib.lib().padoc_branch_decode_no_alloc(plan.handle, _ptr(q), _ptr(k_cache), _ptr(v_cache),
                                                       _ptr(block_table), _ptr(out), _ptr(lse),
                                                       C.c_void_p(s.cuda_stream)))
    return out, lse


def tree_attn_bwd(q, k, v, o, lse, dout, plan: TreePlan, dq=None, dk=None, dv=None, workspace=None, stream=None):
    """Backward of the packed forward (``padoc_tree_attn_bwd``, bf16 plans).
    q, o, dout ``[n_q, Hq, d]``; k, v ``[T, Hkv, d]``; lse float32 ``[n_q,
    Hq]`` (the forward's outputs); returns ``(dQ, dK, dV)``."""
    import torch
    dt = _torch_dtype(plan)
    dev = q.device
    for name, t in (("q", q), ("k", k), ("v", v), ("o", o), ("dout", dout)):
        _check_tensor(name, t, dt, dev)
    _check_tensor("lse", lse, torch.float32, dev)
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(k) if dk is None else dk
    dv = torch.empty_like(v) if dv is None else dv
    for name, t, ref in (("dq", dq, q), ("dk", dk, k), ("dv", dv, v)):
        _check_tensor(name, t, dt, dev)
        if t.shape != ref.shape:
            raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(ref.shape)}")
    ws = plan.backward_workspace(dev) if workspace is None else workspace
    s = torch.cuda.current_stream(dev) if stream is None else stream
    _lib.check(_lib.lib().padoc_tree_attn_bwd(plan.handle, _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), _ptr(dout),
                                              _ptr(dq), _ptr(dk), _ptr(dv), _ptr(ws), ws.numel(),
                                              C.c_void_p(s.cuda_stream)))
    return dq, dk, dv


class DecodeSession:
    """Decode session (``padoc_session_*``): the step loop of masked parallel
    decoding (App. E) over caller-owned paged caches.

    ``open(parent, fork)`` starts a stream (``parent=-1``: a page root) that
    sees the first ``fork`` tokens of ``parent``; ``close(id)`` retires one.
    A step is ``prepare(n_new, n_query)`` (host: grow every open stream by
    ``n_new[i]`` tokens, plan the attention of the last ``n_query[i]``) then
    ``launch(q, k_new, v_new)`` (device: append the K/V rows, patch the block
    table, attention); rows follow ascending open stream id.  Without caches
    (``k_cache=None``) the session is host-only: steps are completed with
    ``commit()`` and inspected with ``view()``."""

    def __init__(self, num_heads_q: int, num_heads_kv: int, head_dim: int, num_blocks: int, dtype: str = "bf16",
                 k_cache=None, v_cache=None, block_table=None, block_table_capacity: Optional[int] = None,
                 softmax_scale: Optional[float] = None, max_chunk_keys: int = 0, target_workgroups: int = 0):
        self.num_heads_q, self.num_heads_kv, self.head_dim = num_heads_q, num_heads_kv, head_dim
        self.dtype = dtype
        self.num_blocks = int(num_blocks)
        self.softmax_scale = 1.0 / math.sqrt(head_dim) if softmax_scale is None else softmax_scale
        dev = (k_cache, v_cache, block_table)
        if any(t is not None for t in dev) and any(t is None for t in dev):
            raise ValueError("pass k_cache, v_cache and block_table together (or none of them)")
        self.k_cache, self.v_cache, self.block_table = k_cache, v_cache, block_table
        if block_table is not None:
            import torch
            dt = torch.bfloat16 if _DTYPES[dtype] == _lib.BF16 else torch.float32
            dv = k_cache.device
            _check_tensor("k_cache", k_cache, dt, dv)
            _check_tensor("v_cache", v_cache, dt, dv)
            _check_tensor("block_table", block_table, torch.int32, dv)
            want_k = (self.num_blocks, num_heads_kv, head_dim // 8, 16, 8)
            want_v = (self.num_blocks, num_heads_kv, head_dim, 16)
            if tuple(k_cache.shape) != want_k or tuple(v_cache.shape) != want_v:
                raise ValueError(f"caches must be K {want_k} and V {want_v}")
            if block_table_capacity is None:
                block_table_capacity = block_table.numel()
            if block_table_capacity > block_table.numel():
                raise ValueError("block_table_capacity exceeds the block table")
            self.device = dv
        else:
            self.device = None
        if block_table_capacity is None:
            block_table_capacity = 2 * self.num_blocks + 1024
        self.block_table_capacity = int(block_table_capacity)
        desc = _lib.SessionDesc(num_heads_q, num_heads_kv, head_dim, float(self.softmax_scale), _DTYPES[dtype],
                                self.num_blocks, self.block_table_capacity,
                                k_cache.data_ptr() if k_cache is not None else None,
                                v_cache.data_ptr() if v_cache is not None else None,
                                block_table.data_ptr() if block_table is not None else None,
                                int(max_chunk_keys), int(target_workgroups))
        h = C.c_void_p()
        _lib.check(_lib.lib().padoc_session_create(C.byref(desc), C.byref(h)))
        self._h = h
        self.n_open = 0
        self.n_kv_rows = self.n_q_rows = 0
        self.workspace_bytes = 0
        self._ws = None

    @property
    def handle(self):
        if self._h is None:
            raise ValueError("session is closed")
        return self._h

    def destroy(self):
        if getattr(self, "_h", None) is not None:
            _lib.lib().padoc_session_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass

    def open(self, parent: int = -1, fork: int = 0) -> int:
        i = C.c_int32(0)
        _lib.check(_lib.lib().padoc_session_open(self.handle, int(parent), int(fork), C.byref(i)))
        self.n_open += 1
        return int(i.value)

    def close(self, stream_id: int) -> None:
        _lib.check(_lib.lib().padoc_session_close(self.handle, int(stream_id)))
        self.n_open -= 1

    def select(self, max_rows: int, priority=None):
        """``(n_new, n_query)`` for a step that takes at most ``max_rows``
        rows (``padoc_session_select``): the open streams with the largest
        ``priority`` (one entry per open stream, ascending id), or the oldest
        when ``priority`` is None."""
        n_new = np.zeros(self.n_open, np.int32)
        n_query = np.zeros(self.n_open, np.int32)
        pr = None
        if priority is not None:
            pr = np.ascontiguousarray(priority, dtype=np.int64)
            if pr.shape != (self.n_open,):
                raise ValueError(f"need one priority per open stream ({self.n_open}), got shape {pr.shape}")
        _lib.check(_lib.lib().padoc_session_select(self.handle, int(max_rows),
                                                   pr.ctypes.data if pr is not None and self.n_open else None,
                                                   n_new.ctypes.data, n_query.ctypes.data))
        return n_new, n_query

    def prepare(self, n_new=None, n_query=None):
        """Returns ``(n_kv_rows, n_q_rows, workspace_bytes)`` of the step."""
        arrs = []
        for a in (n_new, n_query):
            if a is None:
                arrs.append(None)
                continue
            a = np.ascontiguousarray(a, dtype=np.int32)
            if a.shape != (self.n_open,):
                raise ValueError(f"need one entry per open stream ({self.n_open}), got shape {a.shape}")
            arrs.append(a)
        if (arrs[0] is None) != (arrs[1] is None):
            raise ValueError("pass n_new and n_query together (or neither: one token and one query each)")
        nk, nq, ws = C.c_int32(0), C.c_int32(0), C.c_size_t(0)
        ptr = [a.ctypes.data if a is not None else None for a in arrs]
        _lib.check(_lib.lib().padoc_session_prepare(self.handle, ptr[0], ptr[1], C.byref(nk), C.byref(nq),
                                                    C.byref(ws)))
        self.n_kv_rows, self.n_q_rows, self.workspace_bytes = int(nk.value), int(nq.value), int(ws.value)
        return self.n_kv_rows, self.n_q_rows, self.workspace_bytes

    def workspace(self):
        """A cached device workspace of at least the prepared step's size."""
        import torch
        need = max(256, self.workspace_bytes)
        if self._ws is None or self._ws[2].numel() < need:
            cap = need + need // 4
            raw = torch.empty(cap + 256, dtype=torch.uint8, device=self.device)
            off = (-raw.data_ptr()) % 256
            self._ws = (self.device, raw, raw[off: off + cap])
        return self._ws[2]

    def launch(self, q, k_new, v_new, out=None, lse=None, workspace=None, stream=None):
        """Run the prepared step; q ``[n_q_rows, Hq, d]``, k_new / v_new
        ``[n_kv_rows, Hkv, d]``.  Returns ``(O, LSE)``."""
        import torch
        if self.device is None:
            raise RuntimeError("host-only session: use commit()")
        dt = self.k_cache.dtype
        dev = self.device
        if self.n_kv_rows:
            for name, t in (("k_new", k_new), ("v_new", v_new)):
                _check_tensor(name, t, dt, dev)
                if tuple(t.shape) != (self.n_kv_rows, self.num_heads_kv, self.head_dim):
                    raise ValueError(f"{name} must be [{self.n_kv_rows}, {self.num_heads_kv}, {self.head_dim}]")
        if out is None:
            out = torch.empty(self.n_q_rows, self.num_heads_q, self.head_dim, dtype=dt, device=dev)
        if lse is None:
            lse = torch.empty(self.n_q_rows, self.num_heads_q, dtype=torch.float32, device=dev)
        if self.n_q_rows:
            _check_tensor("q", q, dt, dev)
            if tuple(q.shape) != (self.n_q_rows, self.num_heads_q, self.head_dim):
                raise ValueError(f"q must be [{self.n_q_rows}, {self.num_heads_q}, {self.head_dim}]")
            _check_tensor("out", out, dt, dev)
            _check_tensor("lse", lse, torch.float32, dev)
            if tuple(out.shape) != tuple(q.shape) or tuple(lse.shape) != tuple(q.shape[:2]):
                raise ValueError("out / lse shape does not match q")
        ws = self.workspace() if workspace is None else workspace
        s = torch.cuda.current_stream(dev) if stream is None else stream

        def p(t, n):
            return _ptr(t) if n else None
        _lib.check(_lib.lib().padoc_session_launch(self.handle, p(q, self.n_q_rows), p(k_new, self.n_kv_rows),
                                                   p(v_new, self.n_kv_rows), p(out, self.n_q_rows),
                                                   p(lse, self.n_q_rows), _ptr(ws), ws.numel(),
                                                   C.c_void_p(s.cuda_stream)))
        return out, lse

    def step(self, q, k_new, v_new, n_new=None, n_query=None, **kw):
        """``prepare`` then ``launch``."""
        self.prepare(n_new, n_query)
        return self.launch(q, k_new, v_new, **kw)

    def commit(self) -> None:
        _lib.check(_lib.lib().padoc_session_commit(self.handle))

    def view(self, schedule: bool = False, block_table: bool = True) -> dict:
        """The prepared step (or the tree as it stands) as numpy copies
        (``block_table=False`` skips copying the host block table)."""
        v = _lib.SessionView()
        _lib.check(_lib.lib().padoc_session_view_get(self.handle, C.byref(v)))
        arr = _carray
        n = v.n_rows
        prepared = bool(v.plan)
        out = {
            "seg": arr(v.seg, v.n_seg, SEGMENT_DTYPE), "seg_id": arr(v.seg_id, v.n_seg, np.int32),
            "row_id": arr(v.row_id, n, np.int32),
            "block_table": arr(v.block_table, self.block_table_capacity if block_table else 0, np.int32),
            "free_blocks": int(v.free_blocks), "prepared": prepared,
        }
        if prepared:
            new_off = arr(v.new_off, n + 1, np.int32)
            out.update({
                "new_off": new_off, "q_off": arr(v.q_off, n + 1, np.int32),
                "new_slot": arr(v.new_slot, 2 * int(new_off[-1]), np.int32).reshape(-1, 2),
                "patch": arr(v.patch, 2 * v.n_patch, np.int32).reshape(-1, 2),
                "workspace_bytes": int(v.workspace_bytes), "plan": int(v.plan),
            })
            if schedule:
                out["schedule"] = _export_schedule(C.c_void_p(v.plan))
        return out


def set_kernel_events(before=None, after=None):
    """Record torch CUDA events around all kernels of later calls on this
    thread (``padoc_set_kernel_events``); call with no arguments to stop."""
    b = C.c_void_p(before.cuda_event) if before is not None else None
    a = C.c_void_p(after.cuda_event) if after is not None else None
    _lib.check(_lib.lib().padoc_set_kernel_events(b, a))
