"""MI355X (gfx950) MosaicKV hot path: compressed KV cache + decode attention.

Thin Python layer over libmosaic (include/mosaic.h).  PyTorch provides device
memory and the current HIP stream; every step of the method runs in the HIP
kernels.  There is no CPU or PyTorch fallback: if the library is not built,
using the cache raises.
"""
from __future__ import annotations

import ctypes as C
from dataclasses import dataclass

from ._lib import (OP_APPEND, OP_COMPRESS, OP_DECODE, OP_WINDOW_ROTATIONS, MosaicError, MosaicLayout, MosaicParams, MosaicStats,
                   MosaicWsLayout, check, load)

__all__ = ["Params", "MosaicCache", "dense_decode", "MosaicError", "load"]

D = 128


@dataclass
class Params:
    """Method parameters (the strategy set of Sec. 4.3, candidates of Sec. 5.5,
    defaults of Sec. 6.1)."""
    num_kv_heads: int = 8
    group_size: int = 4
    dtype: str = "fp16"
    rot_window: int = 65536
    keep_cand: tuple = (16, 32, 48)
    group_cand: tuple = (4, 2, 1)
    block_cand: tuple = (16, 8, 4)
    default: tuple = (32, 1, 8)
    tau_channel: float = 0.30
    tau_block: float = 0.90
    select: tuple = (1, 10)
    force_default: bool = False
    trunc: int = 128                 # channels represented in the bitmaps (Sec. 5.2 channel truncation)
    fp8: bool = False                # K/V token values as E4M3 codes (Sec. 7, combining with quantization)
    dyn_windows: bool = False        # decode windows closed by their compression loss (Sec. 4.3, Sec. 5.5)
    tau_window: float = 8.0
    min_window: int = 1024

    def to_c(self) -> MosaicParams:
        p = MosaicParams()
        load().mosaic_params_default(C.byref(p))
        p.num_kv_heads, p.group_size = self.num_kv_heads, self.group_size
        p.dtype = 1 if self.dtype == "bf16" else 0
        p.rot_window = self.rot_window
        for i in range(3):
            p.keep_cand[i], p.group_cand[i], p.block_cand[i] = self.keep_cand[i], self.group_cand[i], self.block_cand[i]
        p.default_keep, p.default_group, p.default_block = self.default
        p.tau_channel, p.tau_block = self.tau_channel, self.tau_block
        p.select_num, p.select_den = self.select
        p.force_default_strategy = 1 if self.force_default else 0
        p.trunc_channels = self.trunc
        p.value_fp8 = 1 if self.fp8 else 0
        p.dyn_windows = 1 if self.dyn_windows else 0
        p.tau_window, p.min_window = self.tau_window, self.min_window
        return p


def _stream(device=None):
    import torch
    return C.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _ptr(t):
    return C.c_void_p(t.data_ptr()) if t is not None else None


def _check_tensor(t, name, dtype, device):
    import torch
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on a GPU")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, cache on {device}")


class MosaicCache:
    """One layer's compressed KV cache for `num_seqs` sequences."""

    def __init__(self, params: Params, num_seqs: int, max_tokens, rotated: bool = True, device="cuda"):
        """max_tokens: one capacity for every sequence, or a list of per-sequence
        capacities (each pair's regions then sized for its own sequence)."""
        import torch
        self.lib = load()
        self.params = params
        ragged = not isinstance(max_tokens, int)
        caps = [int(x) for x in max_tokens] if ragged else None
        if ragged and len(caps) != num_seqs:
            raise ValueError(f"{len(caps)} capacities for {num_seqs} sequences")
        self.num_seqs, self.max_tokens, self.rotated = num_seqs, (max(caps) if ragged else max_tokens), bool(rotated)
        self.device = torch.device(device)
        if self.device.index is None:
            self.device = torch.device("cuda", torch.cuda.current_device())
        self.elem = torch.bfloat16 if params.dtype == "bf16" else torch.float16
        self._p = params.to_c()
        h = C.c_void_p()
        if ragged:
            check(self.lib.mosaic_cache_create_ragged(C.byref(self._p), num_seqs, (C.c_int32 * num_seqs)(*caps),
                                                      int(self.rotated), C.byref(h)))
        else:
            check(self.lib.mosaic_cache_create(C.byref(self._p), num_seqs, max_tokens, int(self.rotated), C.byref(h)))
        self._h = h
        n = C.c_size_t()
        check(self.lib.mosaic_cache_arena_bytes(self._h, C.byref(n)))
        self.arena = torch.empty(n.value, dtype=torch.uint8, device=self.device)
        check(self.lib.mosaic_cache_bind(self._h, _ptr(self.arena), n.value))
        check(self.lib.mosaic_workspace_bytes(self._h, OP_DECODE, C.byref(n)))
        self.workspace = torch.empty(max(n.value, 256), dtype=torch.uint8, device=self.device)
        self.layout = MosaicLayout()
        check(self.lib.mosaic_cache_layout(self._h, C.byref(self.layout)))
        self.ws_layout = MosaicWsLayout()
        check(self.lib.mosaic_decode_ws_layout(self._h, C.byref(self.ws_layout)))
        tab = (C.c_uint64 * (4 * self.num_pairs))()
        check(self.lib.mosaic_cache_pair_regions(self._h, tab))
        self.pair_regions = [tuple(tab[4 * p: 4 * p + 4]) for p in range(self.num_pairs)]

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            try:
                self.lib.mosaic_cache_destroy(h)
            except Exception:
                pass
            self._h = None

    @property
    def num_pairs(self):
        return self.num_seqs * self.params.num_kv_heads

    def seq_tokens(self, s):
        return int(self.lib.mosaic_seq_tokens(self._h, s))

    def compress(self, k, v, ctx_lens, rot_k=None, rot_v=None, single_pass: bool = True):
        """k, v: [num_seqs][Hkv][seq_stride][128] (cache dtype); ctx_lens: host ints;
        rot_k/rot_v: [num_seqs][Hkv][ceil(max_tokens / rot_window)][128][128] fp32 or None.
        single_pass: rotate each token once, packing through a transient
        workspace (the library's worst-case segment slots); False: two passes,
        no extra memory.  Both write the same bytes."""
        import torch
        _check_tensor(k, "k", self.elem, self.device)
        _check_tensor(v, "v", self.elem, self.device)
        if k.shape != v.shape or k.dim() != 4 or k.shape[0] != self.num_seqs or k.shape[1] != self.params.num_kv_heads \
                or k.shape[3] != D:
            raise ValueError(f"k/v shape {tuple(k.shape)} does not match the cache")
        if rot_k is not None:
            _check_tensor(rot_k, "rot_k", torch.float32, self.device)
            _check_tensor(rot_v, "rot_v", torch.float32, self.device)
            nw = -(-self.max_tokens // self.params.rot_window)       # fixed windows of the prefill
            want = (self.num_seqs, self.params.num_kv_heads, nw, D, D)
            if tuple(rot_k.shape) != want or tuple(rot_v.shape) != want:
                raise ValueError(f"rotation shape {tuple(rot_k.shape)} != {want}")
        lens = (C.c_int32 * self.num_seqs)(*[int(x) for x in ctx_lens])
        ws = None
        if single_pass:
            n = C.c_size_t()
            check(self.lib.mosaic_workspace_bytes(self._h, OP_COMPRESS, C.byref(n)))
            ws = torch.empty(max(n.value, 16), dtype=torch.uint8, device=self.device)
        with torch.cuda.device(self.device):
            check(self.lib.mosaic_compress(self._h, _ptr(k), _ptr(v), k.shape[2], lens, _ptr(rot_k), _ptr(rot_v),
                                           _ptr(ws), 0 if ws is None else ws.numel(), _stream(self.device)))
        self._keep = (k, v, rot_k, rot_v, ws)  # alive until the enqueued work completes

    def append(self, k_new, v_new):
        """k_new, v_new: [num_seqs][Hkv][128]."""
        _check_tensor(k_new, "k_new", self.elem, self.device)
        _check_tensor(v_new, "v_new", self.elem, self.device)
        if tuple(k_new.shape) != (self.num_seqs, self.params.num_kv_heads, D) or k_new.shape != v_new.shape:
            raise ValueError(f"k_new shape {tuple(k_new.shape)}")
        import torch
        with torch.cuda.device(self.device):
            check(self.lib.mosaic_append(self._h, _ptr(k_new), _ptr(v_new), _stream(self.device)))
        self._keep_app = (k_new, v_new)

    def decode(self, q, sm_scale: float, out=None):
        """q: [num_seqs][Hkv * G][128] -> fp32 [num_seqs][Hq][128]."""
        import torch
        _check_tensor(q, "q", self.elem, self.device)
        hq = self.params.num_kv_heads * self.params.group_size
        if tuple(q.shape) != (self.num_seqs, hq, D):
            raise ValueError(f"q shape {tuple(q.shape)} != {(self.num_seqs, hq, D)}")
        if out is None:
            out = torch.empty((self.num_seqs, hq, D), dtype=torch.float32, device=self.device)
        _check_tensor(out, "out", torch.float32, self.device)
        with torch.cuda.device(self.device):
            check(self.lib.mosaic_decode_attention(self._h, _ptr(q), _ptr(out), float(sm_scale), _ptr(self.workspace),
                                                   self.workspace.numel(), _stream(self.device)))
        return out

    def window_poll(self):
        """Windows closed by their loss and awaiting their rotation (synchronizes):
        {pair: (window, first token, tokens)}."""
        import torch
        out = (C.c_int32 * (3 * self.num_pairs))()
        n = C.c_int32()
        with torch.cuda.device(self.device):
            check(self.lib.mosaic_window_poll(self._h, out, C.byref(n), _stream(self.device)))
        return {p: (out[3 * p], out[3 * p + 1], out[3 * p + 2]) for p in range(self.num_pairs) if out[3 * p] >= 0}

    def window_rotations(self):
        """Rotations of the polled windows from their incremental covariances,
        on the GPU: (rot_k, rot_v) [num_seqs][Hkv][128][128] fp32 (identity for
        pairs with nothing to close)."""
        import torch
        n = C.c_size_t()
        check(self.lib.mosaic_workspace_bytes(self._h, OP_WINDOW_ROTATIONS, C.byref(n)))
        ws = torch.empty(max(n.value, 256), dtype=torch.uint8, device=self.device)
        rk = torch.empty((self.num_seqs, self.params.num_kv_heads, D, D), dtype=torch.float32, device=self.device)
        rv = torch.empty_like(rk)
        with torch.cuda.device(self.device):
            check(self.lib.mosaic_window_rotations(self._h, _ptr(rk), _ptr(rv), _ptr(ws), ws.numel(),
                                                   _stream(self.device)))
        self._keep_wrot = ws
        return rk, rv

    def window_close(self, rot_k, rot_v, k, v):
        """rot_k, rot_v: [num_seqs][Hkv][128][128] fp32, each polled pair's new
        rotation; k, v: [num_seqs][Hkv][stride][128] each closed window's raw
        tokens from its first one."""
        import torch
        for t, nm in ((rot_k, "rot_k"), (rot_v, "rot_v")):
            _check_tensor(t, nm, torch.float32, self.device)
            if tuple(t.shape) != (self.num_seqs, self.params.num_kv_heads, D, D):
                raise ValueError(f"{nm} shape {tuple(t.shape)}")
        for t, nm in ((k, "k"), (v, "v")):
            _check_tensor(t, nm, self.elem, self.device)
            if t.dim() != 4 or tuple(t.shape[:2]) != (self.num_seqs, self.params.num_kv_heads) or t.shape[3] != D:
                raise ValueError(f"{nm} shape {tuple(t.shape)}")
        if k.shape != v.shape:
            raise ValueError("k and v shapes differ")
        with torch.cuda.device(self.device):
            check(self.lib.mosaic_window_close(self._h, _ptr(rot_k), _ptr(rot_v), _ptr(k), _ptr(v), k.shape[2],
                                               _stream(self.device)))
        self._keep_close = (rot_k, rot_v, k, v)

    def window_cov(self, pair: int, window: int):
        """(K, V) incremental covariances [128][128] fp64 of a window of a pair
        (dynamic windows; valid for the open window and the one before it)."""
        import torch
        base = self.layout.cov_off + pair * self.layout.cov_stride + (window & 1) * 2 * D * D * 8
        raw = self.arena[base: base + 2 * D * D * 8].view(torch.float64).reshape(2, D, D)
        return raw[0], raw[1]

    KERNELS = ("qrot", "score", "topk", "attn", "reduce")

    def set_timing(self, enable: bool = True):
        check(self.lib.mosaic_set_timing(self._h, int(enable)))

    def decode_timing(self) -> dict:
        """Per-kernel ms of the last decode (after set_timing(True))."""
        ms = (C.c_float * 5)()
        check(self.lib.mosaic_decode_timing(self._h, ms))
        return dict(zip(self.KERNELS, list(ms)))

    def stats(self) -> dict:
        st = MosaicStats()
        import torch
        with torch.cuda.device(self.device):
            check(self.lib.mosaic_cache_stats(self._h, C.byref(st), _stream(self.device)))
        hist = {}
        p = self.params
        for ri in range(3):
            for gi in range(3):
                for bi in range(3):
                    n = st.strategy_hist[ri * 9 + gi * 3 + bi]
                    if n:
                        hist[(p.keep_cand[ri], p.group_cand[gi], p.block_cand[bi])] = n
        return dict(tokens=st.tokens, dense_bytes=st.dense_bytes, used_bytes=st.used_bytes,
                    rotation_bytes=st.rotation_bytes, segments=st.segments, strategies=hist,
                    ratio=(st.dense_bytes / st.used_bytes) if st.used_bytes else float("nan"))

    # ---- inspection (tests): raw bytes of a pair's regions -------------------
    def region(self, name: str, pair: int, nbytes: int | None = None):
        off = getattr(self.layout, name + "_off")
        stride = getattr(self.layout, name + "_stride")
        if name in ("desc", "score", "token"):            # located by the pair table
            pos = off + self.pair_regions[pair][("desc", "score", "token").index(name)]
            n = self.pair_regions[pair][3] if nbytes is None and name == "token" else nbytes
            if n is None:
                raise ValueError(f"give the bytes of the {name} region")
            return self.arena[pos: pos + n]
        n = stride if nbytes is None else nbytes
        return self.arena[off + pair * stride: off + pair * stride + n]

    def ws_region(self, name: str, pair: int, nbytes: int | None = None):
        off = getattr(self.ws_layout, name + "_off")
        stride = getattr(self.ws_layout, name + "_stride")
        n = stride if nbytes is None else nbytes
        return self.workspace[off + pair * stride: off + pair * stride + n]


def dense_decode(q, k, v, ctx_lens_dev, sm_scale: float, max_ctx: int, group_size: int, out=None, ws=None):
    """Uncompressed split-K decode attention (baseline).  q [S][Hq][128];
    k, v [S][Hkv][seq_stride][128]; ctx_lens_dev int32 [S] on the GPU."""
    import torch
    lib = load()
    S, Hkv, stride, _ = k.shape
    _check_tensor(k, "k", None, None)
    _check_tensor(v, "v", k.dtype, k.device)
    _check_tensor(q, "q", k.dtype, k.device)
    _check_tensor(ctx_lens_dev, "ctx_lens", torch.int32, k.device)
    n = C.c_size_t()
    check(lib.mosaic_dense_workspace_bytes(S, Hkv, group_size, max_ctx, C.byref(n)))
    if ws is None or ws.numel() < n.value:
        ws = torch.empty(max(n.value, 256), dtype=torch.uint8, device=k.device)
    if out is None:
        out = torch.empty((S, Hkv * group_size, D), dtype=torch.float32, device=k.device)
    dt = 1 if k.dtype == torch.bfloat16 else 0
    with torch.cuda.device(k.device):
        check(lib.mosaic_dense_decode_attention(_ptr(q), _ptr(k), _ptr(v), _ptr(out), S, Hkv, group_size, D, dt, stride,
                                                max_ctx, _ptr(ctx_lens_dev), float(sm_scale), _ptr(ws), ws.numel(),
                                                _stream(k.device)))
    return out


def compute_rotations(params: Params, k, v, ctx_lens, max_tokens: int, evals: bool = False, ws=None):
    """Rotation matrices of every window from the cache itself (GPU covariance
    and Jacobi eigensolver): k, v [S][Hkv][seq_stride][128] on the GPU,
    ctx_lens a list of ints.  Returns (rot_k, rot_v) [S][Hkv][nw][128][128]
    fp32, plus (evals_k, evals_v) [S][Hkv][nw][128] when evals is set."""
    import torch
    lib = load()
    S, Hkv, stride, _ = k.shape
    _check_tensor(k, "k", None, None)
    _check_tensor(v, "v", k.dtype, k.device)
    p = params.to_c()
    p.num_kv_heads = Hkv
    p.dtype = 1 if k.dtype == torch.bfloat16 else 0
    n = C.c_size_t()
    check(lib.mosaic_rotation_workspace_bytes(C.byref(p), S, max_tokens, C.byref(n)))
    if ws is None or ws.numel() < n.value:
        ws = torch.empty(n.value, dtype=torch.uint8, device=k.device)
    nw = -(-max_tokens // params.rot_window)
    rk = torch.empty((S, Hkv, nw, D, D), dtype=torch.float32, device=k.device)
    rv = torch.empty_like(rk)
    ek = ev = None
    if evals:
        ek = torch.empty((S, Hkv, nw, D), dtype=torch.float32, device=k.device)
        ev = torch.empty_like(ek)
    lens = (C.c_int32 * S)(*[int(x) for x in ctx_lens])
    with torch.cuda.device(k.device):
        check(lib.mosaic_compute_rotations(C.byref(p), S, max_tokens, _ptr(k), _ptr(v), stride, lens, _ptr(rk),
                                           _ptr(rv), _ptr(ek) if evals else None, _ptr(ev) if evals else None,
                                           _ptr(ws), ws.numel(), _stream(k.device)))
    return (rk, rv, ek, ev) if evals else (rk, rv)


def reorder_rotations(params: Params, k, v, ctx_lens, max_tokens: int, rot_k, rot_v, ws=None):
    """Selection-pattern reorder of the rows of rot_k / rot_v in place (the
    layout compute_rotations returns), counted over the tokens of k, v
    [S][Hkv][seq_stride][128] on the GPU with params.default[0] kept channels."""
    import torch
    lib = load()
    S, Hkv, stride, _ = k.shape
    _check_tensor(k, "k", None, None)
    _check_tensor(v, "v", k.dtype, k.device)
    nw = -(-max_tokens // params.rot_window)
    for t, name in ((rot_k, "rot_k"), (rot_v, "rot_v")):
        _check_tensor(t, name, torch.float32, k.device)
        if tuple(t.shape) != (S, Hkv, nw, D, D):
            raise ValueError(f"{name}: shape {tuple(t.shape)}, expected {(S, Hkv, nw, D, D)}")
    p = params.to_c()
    p.num_kv_heads = Hkv
    p.dtype = 1 if k.dtype == torch.bfloat16 else 0
    n = C.c_size_t()
    check(lib.mosaic_reorder_workspace_bytes(C.byref(p), S, max_tokens, C.byref(n)))
    if ws is None or ws.numel() < n.value:
        ws = torch.empty(n.value, dtype=torch.uint8, device=k.device)
    lens = (C.c_int32 * S)(*[int(x) for x in ctx_lens])
    with torch.cuda.device(k.device):
        check(lib.mosaic_reorder_rotations(C.byref(p), S, max_tokens, _ptr(k), _ptr(v), stride, lens, _ptr(rot_k),
                                           _ptr(rot_v), _ptr(ws), ws.numel(), _stream(k.device)))
    return rot_k, rot_v
