"""ctypes declarations of libmosaic (include/mosaic.h).  Marshalling only."""
from __future__ import annotations

import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmosaic.so")

MOSAIC_OK = 0
STATUS_NAMES = {0: "OK", -1: "INVALID", -2: "UNSUPPORTED", -3: "CAPACITY", -4: "STATE", -5: "HIP"}
OP_COMPRESS, OP_APPEND, OP_DECODE, OP_WINDOW_ROTATIONS = 0, 1, 2, 3

EXPORTED = [
    "mosaic_params_default", "mosaic_cache_create", "mosaic_cache_arena_bytes", "mosaic_cache_bind",
    "mosaic_cache_destroy", "mosaic_cache_layout", "mosaic_workspace_bytes", "mosaic_decode_ws_layout",
    "mosaic_compress", "mosaic_append", "mosaic_decode_attention", "mosaic_dense_workspace_bytes",
    "mosaic_dense_decode_attention", "mosaic_cache_stats", "mosaic_seq_tokens", "mosaic_last_error",
    "mosaic_set_timing", "mosaic_decode_timing", "mosaic_rotation_workspace_bytes", "mosaic_compute_rotations",
    "mosaic_reorder_workspace_bytes", "mosaic_reorder_rotations", "mosaic_decode_attention_noalloc",
    "mosaic_window_poll", "mosaic_window_close", "mosaic_cache_create_ragged", "mosaic_cache_pair_regions",
    "mosaic_window_rotations",
]


class MosaicParams(C.Structure):
    _fields_ = [
        ("head_dim", C.c_int32), ("num_kv_heads", C.c_int32), ("group_size", C.c_int32), ("dtype", C.c_int32),
        ("seg_len", C.c_int32), ("rot_window", C.c_int32), ("update_buf", C.c_int32),
        ("keep_cand", C.c_int32 * 3), ("group_cand", C.c_int32 * 3), ("block_cand", C.c_int32 * 3),
        ("default_keep", C.c_int32), ("default_group", C.c_int32), ("default_block", C.c_int32),
        ("tau_channel", C.c_float), ("tau_block", C.c_float),
        ("select_num", C.c_int32), ("select_den", C.c_int32), ("force_default_strategy", C.c_int32),
        ("trunc_channels", C.c_int32), ("value_fp8", C.c_int32),
        ("dyn_windows", C.c_int32), ("tau_window", C.c_float), ("min_window", C.c_int32),
    ]


class MosaicLayout(C.Structure):
    _fields_ = [(n, C.c_uint64) for n in (
        "meta_off", "meta_stride", "desc_off", "desc_stride", "score_off", "score_stride", "token_off",
        "token_stride", "buf_off", "buf_stride", "stage_off", "stage_stride", "rot_off", "rot_stride", "total")] + [
        ("num_pairs", C.c_int32), ("max_desc", C.c_int32), ("num_windows", C.c_int32), ("reserved", C.c_int32),
        ("cov_off", C.c_uint64), ("cov_stride", C.c_uint64), ("pairs_off", C.c_uint64)]


class MosaicWsLayout(C.Structure):
    _fields_ = [(n, C.c_uint64) for n in (
        "qrot_off", "qrot_stride", "score_off", "score_stride", "sel_off", "sel_stride", "wsel_off", "wsel_stride",
        "part_off", "part_stride", "tag_off", "tag_stride", "binfo_off", "binfo_stride", "bsize_off", "bsize_stride", "selinfo_off",
        "selinfo_stride", "wres_off", "wres_stride", "total")] + [
        ("max_blocks", C.c_int32), ("max_splits", C.c_int32), ("gp", C.c_int32), ("reserved", C.c_int32),
        ("tkx_off", C.c_uint64), ("tkx_stride", C.c_uint64)]


class MosaicStats(C.Structure):
    _fields_ = [("tokens", C.c_int64), ("dense_bytes", C.c_int64), ("used_bytes", C.c_int64),
                ("rotation_bytes", C.c_int64), ("segments", C.c_int64), ("strategy_hist", C.c_int64 * 27)]


_lib = None


class MosaicError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"mosaic {STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


def load() -> C.CDLL:
    """Load the in-tree HIP library; raise if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with paper_2607_00760_amd.build.build() "
                              "(there is no fallback path)")
        _lib = bind_signatures(C.CDLL(LIB_PATH))
    return _lib


def bind_signatures(L: C.CDLL) -> C.CDLL:
    """Set the argument and result types of every exported entry point of L."""
    vp, sz = C.c_void_p, C.c_size_t
    L.mosaic_params_default.argtypes = [C.POINTER(MosaicParams)]
    L.mosaic_params_default.restype = None
    L.mosaic_cache_create.argtypes = [C.POINTER(MosaicParams), C.c_int32, C.c_int32, C.c_int32, C.POINTER(vp)]
    L.mosaic_cache_create_ragged.argtypes = [C.POINTER(MosaicParams), C.c_int32, C.POINTER(C.c_int32), C.c_int32,
                                             C.POINTER(vp)]
    L.mosaic_cache_pair_regions.argtypes = [vp, C.POINTER(C.c_uint64)]
    L.mosaic_cache_arena_bytes.argtypes = [vp, C.POINTER(sz)]
    L.mosaic_cache_bind.argtypes = [vp, vp, sz]
    L.mosaic_cache_destroy.argtypes = [vp]
    L.mosaic_cache_layout.argtypes = [vp, C.POINTER(MosaicLayout)]
    L.mosaic_workspace_bytes.argtypes = [vp, C.c_int32, C.POINTER(sz)]
    L.mosaic_decode_ws_layout.argtypes = [vp, C.POINTER(MosaicWsLayout)]
    L.mosaic_compress.argtypes = [vp, vp, vp, C.c_int64, C.POINTER(C.c_int32), vp, vp, vp, sz, vp]
    L.mosaic_append.argtypes = [vp, vp, vp, vp]
    L.mosaic_decode_attention.argtypes = [vp, vp, vp, C.c_float, vp, sz, vp]
    L.mosaic_decode_attention_noalloc.argtypes = [vp, vp, vp, C.c_float, vp]
    L.mosaic_dense_workspace_bytes.argtypes = [C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.POINTER(sz)]
    L.mosaic_dense_decode_attention.argtypes = [vp, vp, vp, vp, C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                                                C.c_int32, C.c_int64, C.c_int32, vp, C.c_float, vp, sz, vp]
    L.mosaic_cache_stats.argtypes = [vp, C.POINTER(MosaicStats), vp]
    L.mosaic_rotation_workspace_bytes.argtypes = [C.POINTER(MosaicParams), C.c_int32, C.c_int32, C.POINTER(sz)]
    L.mosaic_compute_rotations.argtypes = [C.POINTER(MosaicParams), C.c_int32, C.c_int32, vp, vp, C.c_int64,
                                           C.POINTER(C.c_int32), vp, vp, vp, vp, vp, sz, vp]
    L.mosaic_reorder_workspace_bytes.argtypes = [C.POINTER(MosaicParams), C.c_int32, C.c_int32, C.POINTER(sz)]
    L.mosaic_reorder_rotations.argtypes = [C.POINTER(MosaicParams), C.c_int32, C.c_int32, vp, vp, C.c_int64,
                                           C.POINTER(C.c_int32), vp, vp, vp, sz, vp]
    L.mosaic_window_poll.argtypes = [vp, C.POINTER(C.c_int32), C.POINTER(C.c_int32), vp]
    L.mosaic_window_close.argtypes = [vp, vp, vp, vp, vp, C.c_int64, vp]
    L.mosaic_window_rotations.argtypes = [vp, vp, vp, vp, sz, vp]
    L.mosaic_set_timing.argtypes = [vp, C.c_int32]
    L.mosaic_decode_timing.argtypes = [vp, C.POINTER(C.c_float)]
    L.mosaic_seq_tokens.argtypes = [vp, C.c_int32]
    L.mosaic_seq_tokens.restype = C.c_int32
    L.mosaic_last_error.argtypes = []
    L.mosaic_last_error.restype = C.c_char_p
    for n in EXPORTED:
        f = getattr(L, n)
        if f.restype is C.c_int:   # default restype -> mosaic_status
            f.restype = C.c_int32
    return L


def check(status: int):
    if status != MOSAIC_OK:
        raise MosaicError(status, load().mosaic_last_error().decode())
    return status
