"""ctypes binding of ``libpadoc_attn.so`` (argument marshalling only).

The shared library must have been built (``python -m
paper_2608_06146_amd.build``); there is no fallback: loading fails loudly when
it is missing.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libpadoc_attn.so")

OK, ERR_ARG, ERR_TREE, ERR_SHAPE, ERR_DTYPE, ERR_BOUNDS, ERR_WORKSPACE, ERR_HIP, ERR_MODE = 0, -1, -2, -3, -4, -5, -6, -7, -8
STATUS_NAMES = {0: "PADOC_OK", -1: "PADOC_ERR_ARG", -2: "PADOC_ERR_TREE", -3: "PADOC_ERR_SHAPE",
                -4: "PADOC_ERR_DTYPE", -5: "PADOC_ERR_BOUNDS", -6: "PADOC_ERR_WORKSPACE",
                -7: "PADOC_ERR_HIP", -8: "PADOC_ERR_MODE"}
F32, BF16 = 0, 1

SEGMENT_DTYPE = np.dtype([("parent", "<i4"), ("fork", "<i4"), ("len", "<i4"), ("q_len", "<i4"),
                          ("kv_off", "<i8"), ("q_off", "<i8")])
WORK_DTYPE = np.dtype([("tok_begin", "<i4"), ("ntok", "<i4"), ("rng_begin", "<i4"), ("rng_count", "<i4"),
                       ("kvh", "<i4"), ("out_base", "<i4"), ("cost", "<i4"), ("col0", "<i4"),
                       ("ncol", "<i4"), ("direct", "<i4", (3,))])
BWD_DTYPE = np.dtype([("key_row0", "<i8"), ("n_keys", "<i4"), ("tok_begin", "<i4"), ("ntok", "<i4"),
                      ("lim_begin", "<i4"), ("col0", "<i4"), ("ncol", "<i4"), ("kvh", "<i4"), ("cost", "<i4")])
RANGE_DTYPE = np.dtype([("kv_start", "<i8"), ("n_keys", "<i4"), ("min_lim", "<i4"), ("lim_off", "<i4"),
                        ("seg", "<i4"), ("key_begin", "<i4"), ("reserved", "<i4")])


class Segment(C.Structure):
    _fields_ = [("parent", C.c_int32), ("fork", C.c_int32), ("len", C.c_int32), ("q_len", C.c_int32),
                ("kv_off", C.c_int64), ("q_off", C.c_int64)]


class Page(C.Structure):
    _fields_ = [("prefix_len", C.c_int32), ("prefix_q_len", C.c_int32), ("stream_len", C.c_int32),
                ("stream_q_len", C.c_int32), ("n_branches", C.c_int32),
                ("branch_fork", C.POINTER(C.c_int32)), ("branch_len", C.POINTER(C.c_int32)),
                ("branch_q_len", C.POINTER(C.c_int32))]


class TreeDesc(C.Structure):
    _fields_ = [("n_seg", C.c_int32), ("seg", C.c_void_p), ("num_heads_q", C.c_int32),
                ("num_heads_kv", C.c_int32), ("head_dim", C.c_int32), ("softmax_scale", C.c_float),
                ("dtype", C.c_int32), ("block_size", C.c_int32), ("num_kv_rows", C.c_int64),
                ("num_q_rows", C.c_int64), ("block_table_host", C.c_void_p), ("block_table_len", C.c_int64),
                ("max_chunk_keys", C.c_int32), ("target_workgroups", C.c_int32)]


class ScheduleView(C.Structure):
    _fields_ = [("kind", C.c_int32), ("tile_cols", C.c_int32), ("tile_keys", C.c_int32),
                ("n_work", C.c_int32), ("work", C.c_void_p), ("n_work_shared", C.c_int32),
                ("n_range", C.c_int32), ("ranges", C.c_void_p),
                ("n_lim", C.c_int32), ("lims", C.c_void_p),
                ("n_tok", C.c_int32), ("toks", C.c_void_p),
                ("n_tile_class", C.c_int64), ("tile_class", C.c_void_p), ("tile_class_off", C.c_void_p),
                ("n_comb_ptr", C.c_int64), ("comb_ptr", C.c_void_p),
                ("n_comb", C.c_int64), ("comb_slot", C.c_void_p),
                ("n_comb_rows", C.c_int64), ("comb_rows", C.c_void_p),
                ("n_bwd", C.c_int32), ("bwd", C.c_void_p),
                ("n_btok", C.c_int64), ("btoks", C.c_void_p),
                ("n_blim", C.c_int64), ("blims", C.c_void_p),
                ("n_slots", C.c_int64), ("workspace_bytes", C.c_size_t)]


class SessionDesc(C.Structure):
    _fields_ = [("num_heads_q", C.c_int32), ("num_heads_kv", C.c_int32), ("head_dim", C.c_int32),
                ("softmax_scale", C.c_float), ("dtype", C.c_int32), ("num_blocks", C.c_int64),
                ("block_table_capacity", C.c_int64), ("k_cache", C.c_void_p), ("v_cache", C.c_void_p),
                ("block_table", C.c_void_p), ("max_chunk_keys", C.c_int32), ("target_workgroups", C.c_int32)]


class SessionView(C.Structure):
    _fields_ = [("n_seg", C.c_int32), ("seg", C.c_void_p), ("seg_id", C.c_void_p),
                ("n_rows", C.c_int32), ("row_id", C.c_void_p), ("new_off", C.c_void_p), ("q_off", C.c_void_p),
                ("new_slot", C.c_void_p), ("n_patch", C.c_int32), ("patch", C.c_void_p),
                ("block_table", C.c_void_p), ("plan", C.c_void_p), ("free_blocks", C.c_int64),
                ("workspace_bytes", C.c_size_t)]


EXPORTED = [
    "padoc_tree_from_pages", "padoc_tree_layout", "padoc_plan_create", "padoc_plan_workspace_bytes",
    "padoc_plan_export", "padoc_plan_destroy", "padoc_tree_attn_fwd", "padoc_branch_decode",
    "padoc_branch_decode_no_alloc", "padoc_plan_upload", "padoc_branch_decode_resident", "padoc_last_error",
    "padoc_set_kernel_events", "padoc_version",
    "padoc_plan_backward_workspace_bytes", "padoc_tree_attn_bwd",
    "padoc_session_create", "padoc_session_destroy", "padoc_session_open", "padoc_session_close",
    "padoc_session_prepare", "padoc_session_launch", "padoc_session_commit", "padoc_session_view_get",
    "padoc_tree_depths", "padoc_tree_remaining", "padoc_session_select", "padoc_cache_from_rows",
]

_lib = None


def lib():
    """Load the library once; raise if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2608_06146_amd.build` "
                           "(the HIP library is required; there is no fallback path)")
    L = C.CDLL(LIB_PATH)
    vp, i32, i64, sz = C.c_void_p, C.c_int32, C.c_int64, C.c_size_t
    L.padoc_tree_from_pages.argtypes = [C.POINTER(Page), i32, i32, vp, i32, C.POINTER(i32)]
    L.padoc_tree_layout.argtypes = [vp, i32, i32]
    L.padoc_plan_create.argtypes = [C.POINTER(TreeDesc), C.POINTER(vp)]
    L.padoc_plan_workspace_bytes.argtypes = [vp, C.POINTER(sz)]
    L.padoc_plan_export.argtypes = [vp, C.POINTER(ScheduleView)]
    L.padoc_plan_destroy.argtypes = [vp]
    L.padoc_plan_destroy.restype = None
    L.padoc_tree_attn_fwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, sz, vp]
    L.padoc_branch_decode.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    L.padoc_branch_decode_no_alloc.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp]
    L.padoc_plan_upload.argtypes = [vp, vp, sz, vp]
    L.padoc_branch_decode_resident.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    L.padoc_plan_backward_workspace_bytes.argtypes = [vp, C.POINTER(sz)]
    L.padoc_tree_attn_bwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    L.padoc_session_create.argtypes = [C.POINTER(SessionDesc), C.POINTER(vp)]
    L.padoc_session_destroy.argtypes = [vp]
    L.padoc_session_destroy.restype = None
    L.padoc_session_open.argtypes = [vp, i32, i32, C.POINTER(i32)]
    L.padoc_session_close.argtypes = [vp, i32]
    L.padoc_session_prepare.argtypes = [vp, vp, vp, C.POINTER(i32), C.POINTER(i32), C.POINTER(sz)]
    L.padoc_session_launch.argtypes = [vp, vp, vp, vp, vp, vp, vp, sz, vp]
    L.padoc_session_commit.argtypes = [vp]
    L.padoc_session_view_get.argtypes = [vp, C.POINTER(SessionView)]
    L.padoc_tree_depths.argtypes = [vp, i32, vp, vp]
    L.padoc_tree_remaining.argtypes = [vp, i32, vp, vp]
    L.padoc_session_select.argtypes = [vp, i32, vp, vp, vp]
    L.padoc_cache_from_rows.argtypes = [vp, vp, vp, vp, C.c_int64, i32, i32, C.c_int, vp]
    L.padoc_last_error.argtypes = []
    L.padoc_last_error.restype = C.c_char_p
    L.padoc_set_kernel_events.argtypes = [vp, vp]
    L.padoc_version.argtypes = []
    L.padoc_version.restype = C.c_char_p
    for name in ("padoc_tree_from_pages", "padoc_tree_layout", "padoc_plan_create", "padoc_plan_workspace_bytes",
                 "padoc_plan_export", "padoc_tree_attn_fwd", "padoc_branch_decode", "padoc_branch_decode_no_alloc",
                 "padoc_plan_upload", "padoc_branch_decode_resident", "padoc_set_kernel_events",
                 "padoc_plan_backward_workspace_bytes", "padoc_tree_attn_bwd", "padoc_session_create",
                 "padoc_session_open", "padoc_session_close", "padoc_session_prepare", "padoc_session_launch",
                 "padoc_session_commit", "padoc_session_view_get", "padoc_tree_depths",
                 "padoc_tree_remaining", "padoc_session_select", "padoc_cache_from_rows"):
        getattr(L, name).restype = C.c_int
    _lib = L
    return L


class PadocError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


def check(status: int) -> None:
    if status != OK:
        raise PadocError(status, lib().padoc_last_error().decode(errors="replace"))
