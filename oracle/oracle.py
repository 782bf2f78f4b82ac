"""ctypes binding of the plain C oracle (mosaic_oracle.c).

TEST INFRASTRUCTURE ONLY: imported by tests/, __graft_entry__.smoke() and the
cpu_baseline leg of bench.py, never by the product package.  The oracle is
independent of the HIP library: it shares no code with it, only the dense
inputs (K, V, q) and the rotation matrices, which are inputs of the method.

Every function follows a passage of the paper (arXiv 2607.00760); see the
header comment of mosaic_oracle.c for the section map and the readings.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mosaic_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
# a separately built copy of the same source to load instead (the sanitizer
# test builds one with AddressSanitizer and UndefinedBehaviorSanitizer)
_LIB_OVERRIDE = os.environ.get("MOSAIC_ORACLE_LIB")
D = 128

CFLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared"]


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (no SIMD intrinsics, no FMA contraction)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", *CFLAGS, "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


class OrcParams(C.Structure):
    _fields_ = [
        ("group", C.c_int32), ("dtype", C.c_int32), ("seg_len", C.c_int32),
        ("rot_window", C.c_int32), ("update_buf", C.c_int32),
        ("keep_cand", C.c_int32 * 3), ("group_cand", C.c_int32 * 3), ("block_cand", C.c_int32 * 3),
        ("def_keep", C.c_int32), ("def_group", C.c_int32), ("def_block", C.c_int32),
        ("tau_channel", C.c_float), ("tau_block", C.c_float),
        ("select_num", C.c_int32), ("select_den", C.c_int32), ("force_default", C.c_int32),
        ("trunc", C.c_int32), ("fp8", C.c_int32),
        ("dyn", C.c_int32), ("tau_window", C.c_float), ("min_window", C.c_int32),
    ]


class OrcDesc(C.Structure):
    _fields_ = [("tok_off", C.c_uint32), ("sc_off", C.c_uint32), ("first_block", C.c_uint32),
                ("r", C.c_uint8), ("log2g", C.c_uint8), ("log2b", C.c_uint8), ("flags", C.c_uint8)]


class OrcInfo(C.Structure):
    _fields_ = [("L", C.c_int32), ("n_final", C.c_int32), ("prov", C.c_int32), ("n_buf", C.c_int32),
                ("n_desc", C.c_int32), ("nblk_final", C.c_int32), ("nblk", C.c_int32),
                ("tok_tail", C.c_uint32), ("sc_tail", C.c_uint32), ("used_bytes", C.c_uint64)]


@dataclass
class Params:
    """Method parameters (Sec. 4.3 strategy set; Sec. 6.1 defaults)."""
    group: int = 4
    dtype: str = "fp16"             # "fp16" | "bf16"
    seg_len: int = 64
    rot_window: int = 65536
    update_buf: int = 32
    keep_cand: tuple = (16, 32, 48)
    group_cand: tuple = (4, 2, 1)
    block_cand: tuple = (16, 8, 4)
    default: tuple = (32, 1, 8)
    tau_channel: float = 0.30
    tau_block: float = 0.90
    select: tuple = (1, 10)
    force_default: bool = False
    trunc: int = 128                # channels represented in the bitmap (Sec. 5.2 channel truncation)
    fp8: bool = False               # K/V token values as E4M3 (Sec. 7, combining with quantization)
    dyn: bool = False               # decode windows closed by their accumulated loss (Sec. 4.3, R-23)
    tau_window: float = 8.0
    min_window: int = 1024

    def to_c(self) -> OrcParams:
        p = OrcParams()
        p.group = self.group
        p.dtype = 1 if self.dtype == "bf16" else 0
        p.seg_len, p.rot_window, p.update_buf = self.seg_len, self.rot_window, self.update_buf
        for i in range(3):
            p.keep_cand[i] = self.keep_cand[i]
            p.group_cand[i] = self.group_cand[i]
            p.block_cand[i] = self.block_cand[i]
        p.def_keep, p.def_group, p.def_block = self.default
        p.tau_channel, p.tau_block = self.tau_channel, self.tau_block
        p.select_num, p.select_den = self.select
        p.force_default = 1 if self.force_default else 0
        p.trunc = self.trunc
        p.fp8 = 1 if self.fp8 else 0
        p.dyn = 1 if self.dyn else 0
        p.tau_window, p.min_window = self.tau_window, self.min_window
        return p


_lib = None


def lib():
    global _lib
    if _lib is None:
        if _LIB_OVERRIDE:
            L = C.CDLL(_LIB_OVERRIDE)
        else:
            if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
                build(force=True)
            L = C.CDLL(_LIB)
        fp, u16p, u8p, i32p, f64p = (C.POINTER(C.c_float), C.POINTER(C.c_uint16), C.POINTER(C.c_uint8),
                                     C.POINTER(C.c_int32), C.POINTER(C.c_double))
        L.orc_f16_to_f32.argtypes = [C.c_uint16]; L.orc_f16_to_f32.restype = C.c_float
        L.orc_f32_to_f16.argtypes = [C.c_float]; L.orc_f32_to_f16.restype = C.c_uint16
        L.orc_bf16_to_f32.argtypes = [C.c_uint16]; L.orc_bf16_to_f32.restype = C.c_float
        L.orc_e4m3_to_f32.argtypes = [C.c_uint8]; L.orc_e4m3_to_f32.restype = C.c_float
        L.orc_f32_to_e4m3.argtypes = [C.c_float]; L.orc_f32_to_e4m3.restype = C.c_uint8
        L.orc_f32_to_bf16.argtypes = [C.c_float]; L.orc_f32_to_bf16.restype = C.c_uint16
        L.orc_tree_sum.argtypes = [fp, C.c_int]; L.orc_tree_sum.restype = C.c_float
        L.orc_rotate.argtypes = [fp, fp, fp]; L.orc_rotate.restype = None
        L.orc_group_scores.argtypes = [fp, C.c_int, fp]; L.orc_group_scores.restype = None
        L.orc_topk_mask.argtypes = [fp, C.c_int, C.c_int, u8p]; L.orc_topk_mask.restype = C.c_int
        L.orc_pack_vector.argtypes = [fp, C.c_int, C.c_int, C.c_int, u8p]; L.orc_pack_vector.restype = None
        L.orc_bitmap_bytes.argtypes = [C.c_int]; L.orc_bitmap_bytes.restype = C.c_int
        L.orc_vec_bytes.argtypes = [C.c_int, C.c_int, C.c_int]; L.orc_vec_bytes.restype = C.c_int
        L.orc_vec_bytes_t.argtypes = [C.c_int, C.c_int, C.c_int, C.c_int]; L.orc_vec_bytes_t.restype = C.c_int
        L.orc_choose_strategy.argtypes = [C.POINTER(OrcParams), fp, fp, C.c_int, i32p, i32p, i32p]
        L.orc_choose_strategy.restype = None
        L.orc_pair_new.argtypes = [C.POINTER(OrcParams), C.c_int, fp, fp, C.c_int]
        L.orc_pair_new.restype = C.c_void_p
        L.orc_pair_free.argtypes = [C.c_void_p]; L.orc_pair_free.restype = None
        L.orc_pair_compress.argtypes = [C.c_void_p, u16p, u16p, C.c_int]; L.orc_pair_compress.restype = C.c_int
        L.orc_pair_append.argtypes = [C.c_void_p, u16p, u16p]; L.orc_pair_append.restype = C.c_int
        L.orc_pair_info.argtypes = [C.c_void_p, C.POINTER(OrcInfo)]; L.orc_pair_info.restype = None
        for nm, rt in (("orc_pair_tok", u8p), ("orc_pair_sc", u8p), ("orc_pair_desc", C.POINTER(OrcDesc)),
                       ("orc_pair_bufk", u16p), ("orc_pair_bufv", u16p),
                       ("orc_pair_stgk", u16p), ("orc_pair_stgv", u16p)):
            getattr(L, nm).argtypes = [C.c_void_p]; getattr(L, nm).restype = rt
        L.orc_pair_scores.argtypes = [C.c_void_p, u16p, fp, C.c_int]; L.orc_pair_scores.restype = C.c_int
        L.orc_segment_loss.argtypes = [C.POINTER(OrcParams), fp, fp, C.c_int, C.c_int, C.c_int]
        L.orc_segment_loss.restype = C.c_float
        L.orc_max_windows.argtypes = [C.POINTER(OrcParams), C.c_int]; L.orc_max_windows.restype = C.c_int
        L.orc_pair_close.argtypes = [C.c_void_p, fp, fp, u16p, u16p]; L.orc_pair_close.restype = C.c_int
        L.orc_pair_windows.argtypes = [C.c_void_p, i32p, i32p, fp, i32p]; L.orc_pair_windows.restype = None
        L.orc_pair_cov.argtypes = [C.c_void_p, C.c_int, C.c_int, f64p]; L.orc_pair_cov.restype = None
        L.orc_select_count.argtypes = [C.c_int, C.c_int, C.c_int]; L.orc_select_count.restype = C.c_int
        L.orc_select_budget.argtypes = [C.c_int, C.c_int, C.c_int]; L.orc_select_budget.restype = C.c_int
        L.orc_select_blocks.argtypes = [fp, i32p, C.c_int, C.c_int, u8p]; L.orc_select_blocks.restype = C.c_int
        L.orc_pair_decode.argtypes = [C.c_void_p, u16p, C.c_float, f64p, i32p, C.c_int]
        L.orc_pair_decode.restype = C.c_int
        L.orc_dense_attention.argtypes = [u16p, u16p, u16p, C.c_int, C.c_int, C.c_int, C.c_float, f64p]
        L.orc_dense_attention.restype = None
        L.orc_bytes_per_token.argtypes = [C.c_int, C.c_int, C.c_int, C.c_int]
        L.orc_bytes_per_token.restype = C.c_double
        L.orc_bytes_per_token_t.argtypes = [C.c_int, C.c_int, C.c_int, C.c_int, C.c_int]
        L.orc_bytes_per_token_t.restype = C.c_double
        _lib = L
    return _lib


def _p(a, t):
    return a.ctypes.data_as(C.POINTER(t))


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _u16(a):
    return np.ascontiguousarray(a, dtype=np.uint16)


# ---- scalar conversions ----------------------------------------------------
def f32_to_f16_bits(x):
    L = lib()
    return np.array([L.orc_f32_to_f16(float(v)) for v in np.asarray(x, np.float32).ravel()], np.uint16)


def f32_to_bf16_bits(x):
    L = lib()
    return np.array([L.orc_f32_to_bf16(float(v)) for v in np.asarray(x, np.float32).ravel()], np.uint16)


def f16_bits_to_f32(b):
    L = lib()
    return np.array([L.orc_f16_to_f32(int(v)) for v in np.asarray(b, np.uint16).ravel()], np.float32)


def bf16_bits_to_f32(b):
    L = lib()
    return np.array([L.orc_bf16_to_f32(int(v)) for v in np.asarray(b, np.uint16).ravel()], np.float32)


def f32_to_e4m3(x):
    L = lib()
    return np.array([L.orc_f32_to_e4m3(float(v)) for v in np.asarray(x, np.float32).ravel()], np.uint8)


def e4m3_to_f32(b):
    L = lib()
    return np.array([L.orc_e4m3_to_f32(int(v)) for v in np.asarray(b, np.uint8).ravel()], np.float32)


# ---- vector primitives -----------------------------------------------------
def tree_sum(a) -> np.float32:
    a = _f32(a)
    return np.float32(lib().orc_tree_sum(_p(a, C.c_float), a.size))


def rotate(x, R=None):
    """Sec. 2.3: y = x . R^T (fp32 fused chain per output channel)."""
    x = _f32(x).reshape(-1, D)
    y = np.empty_like(x)
    Rk = _f32(R) if R is not None else None
    for t in range(x.shape[0]):
        lib().orc_rotate(_p(x[t], C.c_float), _p(Rk, C.c_float) if Rk is not None else None, _p(y[t], C.c_float))
    return y


def group_scores(y, g):
    y = _f32(y)
    s = np.empty(D // g, np.float32)
    lib().orc_group_scores(_p(y, C.c_float), g, _p(s, C.c_float))
    return s


def topk_mask(s, k):
    s = _f32(s)
    keep = np.zeros(s.size, np.uint8)
    rc = lib().orc_topk_mask(_p(s, C.c_float), s.size, k, _p(keep, C.c_uint8))
    if rc != 0:
        raise ValueError("non-finite input")
    return keep.astype(bool)


def vec_bytes(r, g, elem_bytes=2, trunc=D):
    return lib().orc_vec_bytes_t(r, g, elem_bytes, trunc)


def bitmap_bytes(g):
    return lib().orc_bitmap_bytes(g)


def pack_vector(y, r, g, dtype="fp16"):
    y = _f32(y)
    out = np.zeros(vec_bytes(r, g), np.uint8)
    lib().orc_pack_vector(_p(y, C.c_float), r, g, 1 if dtype == "bf16" else 0, _p(out, C.c_uint8))
    return out


def choose_strategy(params: Params, yk, yv):
    yk, yv = _f32(yk).reshape(-1, D), _f32(yv).reshape(-1, D)
    r, g, b = C.c_int32(), C.c_int32(), C.c_int32()
    P = params.to_c()
    lib().orc_choose_strategy(C.byref(P), _p(yk, C.c_float), _p(yv, C.c_float), yk.shape[0],
                              C.byref(r), C.byref(g), C.byref(b))
    return r.value, g.value, b.value


def segment_loss(params: Params, yk, yv, r, g):
    """Compression loss of a 64-token segment under (r, g) (R-23): the larger
    of K's and V's relative dropped energy."""
    yk, yv = _f32(yk).reshape(-1, D), _f32(yv).reshape(-1, D)
    P = params.to_c()
    return float(np.float32(lib().orc_segment_loss(C.byref(P), _p(yk, C.c_float), _p(yv, C.c_float), yk.shape[0], r, g)))


def max_windows(params: Params, cap: int) -> int:
    P = params.to_c()
    return lib().orc_max_windows(C.byref(P), cap)


def select_count(nblk, num, den):
    return lib().orc_select_count(nblk, num, den)


def select_budget(ntok, num, den):
    """Tokens to select: ceil(rho * ntok) in integers, at least 1 (R-7)."""
    return lib().orc_select_budget(ntok, num, den)


def select_blocks(scores, sizes, budget):
    """Blocks taken in (score desc, index asc) order while fewer than budget
    tokens are taken (R-7) -> boolean mask."""
    s = _f32(scores)
    z = np.ascontiguousarray(sizes, dtype=np.int32)
    keep = np.zeros(s.size, np.uint8)
    rc = lib().orc_select_blocks(_p(s, C.c_float), _p(z, C.c_int32), s.size, budget, _p(keep, C.c_uint8))
    if rc < 0:
        raise ValueError("non-finite input")
    return keep.astype(bool)


def bytes_per_token(r, g, B, elem_bytes=2, trunc=D):
    """Bytes per token of a full segment: two packed vectors (K, V) and 1/B of
    a block key; the bitmap represents the first trunc channels."""
    return lib().orc_bytes_per_token_t(r, g, B, elem_bytes, trunc)


def dense_attention(q, k, v, scale, dtype="fp16"):
    """Textbook dense attention of one GQA group: q [G][D], k/v [L][D] raw bits."""
    q, k, v = _u16(q), _u16(k), _u16(v)
    G, L = q.shape[0], k.shape[0]
    out = np.zeros((G, D), np.float64)
    lib().orc_dense_attention(_p(q, C.c_uint16), _p(k, C.c_uint16), _p(v, C.c_uint16), L, G,
                              1 if dtype == "bf16" else 0, scale, _p(out, C.c_double))
    return out


# ---- per-(sequence, kv head) cache -------------------------------------------
class Pair:
    """Oracle cache of one (sequence, kv head): compress, append, decode."""

    def __init__(self, params: Params, cap: int, rot_k=None, rot_v=None):
        self.params = params
        self._P = params.to_c()
        self.cap = cap
        if rot_k is not None:
            rk, rv = _f32(rot_k).reshape(-1, D, D), _f32(rot_v).reshape(-1, D, D)
            nw = rk.shape[0]
            self._h = lib().orc_pair_new(C.byref(self._P), cap, _p(rk, C.c_float), _p(rv, C.c_float), nw)
        else:
            self._h = lib().orc_pair_new(C.byref(self._P), cap, None, None, 0)
        if not self._h:
            raise MemoryError("orc_pair_new")

    def __del__(self):
        h = getattr(self, "_h", None)
        if h and _lib is not None:
            try:
                _lib.orc_pair_free(h)
            except Exception:
                pass
            self._h = None

    @property
    def elem_bytes(self):
        """Bytes per kept value in the K and V token records."""
        return 1 if self.params.fp8 else 2

    def compress(self, k, v):
        k, v = _u16(k).reshape(-1, D), _u16(v).reshape(-1, D)
        rc = lib().orc_pair_compress(self._h, _p(k, C.c_uint16), _p(v, C.c_uint16), k.shape[0])
        if rc:
            raise ValueError("compress: capacity")

    def append(self, k, v):
        k, v = _u16(k).reshape(D), _u16(v).reshape(D)
        rc = lib().orc_pair_append(self._h, _p(k, C.c_uint16), _p(v, C.c_uint16))
        if rc:
            raise ValueError("append: capacity")

    def append_status(self, k, v) -> int:
        """Append returning the oracle's status (0, -3 capacity, -4 a closed
        window awaits its rotation) instead of raising."""
        k, v = _u16(k).reshape(D), _u16(v).reshape(D)
        return lib().orc_pair_append(self._h, _p(k, C.c_uint16), _p(v, C.c_uint16))

    def windows(self):
        """-> dict(nwin, pend, wloss, wseg list): the window table (R-23)."""
        nwin, pend, wl = C.c_int32(), C.c_int32(), C.c_float()
        lib().orc_pair_windows(self._h, C.byref(nwin), C.byref(pend), C.byref(wl), None)
        ws = np.zeros(max(nwin.value, 1), np.int32)
        lib().orc_pair_windows(self._h, C.byref(nwin), C.byref(pend), C.byref(wl), _p(ws, C.c_int32))
        return dict(nwin=nwin.value, pend=pend.value, wloss=float(np.float32(wl.value)), wseg=ws[:nwin.value].tolist())

    def cov(self, w):
        """(K, V) incremental covariances [D][D] fp64 of window w (R-23)."""
        out = []
        for which in (0, 1):
            a = np.zeros((D, D), np.float64)
            lib().orc_pair_cov(self._h, w, which, _p(a, C.c_double))
            out.append(a)
        return tuple(out)

    def close(self, rot_k, rot_v, k, v):
        """Close of the window awaiting its rotation: new R (rows = channels)
        and the window's raw tokens."""
        rk, rv = _f32(rot_k).reshape(D, D), _f32(rot_v).reshape(D, D)
        k, v = _u16(k).reshape(-1, D), _u16(v).reshape(-1, D)
        rc = lib().orc_pair_close(self._h, _p(rk, C.c_float), _p(rv, C.c_float), _p(k, C.c_uint16), _p(v, C.c_uint16))
        if rc:
            raise ValueError("close: no window awaits a rotation")

    def info(self) -> OrcInfo:
        o = OrcInfo()
        lib().orc_pair_info(self._h, C.byref(o))
        return o

    def _bytes(self, fn, n):
        ptr = getattr(lib(), fn)(self._h)
        return np.ctypeslib.as_array(ptr, shape=(n,)).copy() if n > 0 else np.zeros(0, np.uint8)

    def token_arena(self):
        i = self.info()
        n = i.tok_tail
        if i.prov:
            d = self.descriptors()[-1]
            n = d["tok_off"] + self.params.update_buf * 2 * vec_bytes(d["r"], 1 << d["log2g"], self.elem_bytes,
                                                                     self.params.trunc)
        return self._bytes("orc_pair_tok", n)

    def score_arena(self):
        i = self.info()
        n = i.sc_tail
        if i.prov:
            d = self.descriptors()[-1]
            n = d["sc_off"] + (self.params.update_buf >> d["log2b"]) * vec_bytes(d["r"], 1 << d["log2g"], 2,
                                                                                self.params.trunc)
        return self._bytes("orc_pair_sc", n)

    def descriptors(self):
        i = self.info()
        ptr = lib().orc_pair_desc(self._h)
        out = []
        for j in range(i.n_desc):
            d = ptr[j]
            out.append(dict(tok_off=d.tok_off, sc_off=d.sc_off, first_block=d.first_block, r=d.r,
                            log2g=d.log2g, log2b=d.log2b, flags=d.flags))
        return out

    def descriptor_bytes(self):
        """Descriptors as the 16-byte little-endian records they are stored as."""
        ds = self.descriptors()
        a = np.zeros((len(ds), 16), np.uint8)
        for j, d in enumerate(ds):
            a[j, 0:4] = np.frombuffer(np.uint32(d["tok_off"]).tobytes(), np.uint8)
            a[j, 4:8] = np.frombuffer(np.uint32(d["sc_off"]).tobytes(), np.uint8)
            a[j, 8:12] = np.frombuffer(np.uint32(d["first_block"]).tobytes(), np.uint8)
            a[j, 12:16] = [d["r"], d["log2g"], d["log2b"], d["flags"]]
        return a.reshape(-1)

    def buffer(self):
        """(k, v) raw bits of the live update-buffer tokens."""
        n = self.info().n_buf
        bk = np.ctypeslib.as_array(lib().orc_pair_bufk(self._h), shape=(32 * D,)).reshape(32, D)[:n].copy()
        bv = np.ctypeslib.as_array(lib().orc_pair_bufv(self._h), shape=(32 * D,)).reshape(32, D)[:n].copy()
        return bk, bv

    def staging(self):
        """(k, v) raw bits of the trailing segment's tokens held for finalize."""
        m = self.info().L % self.params.seg_len
        sk = np.ctypeslib.as_array(lib().orc_pair_stgk(self._h), shape=(64 * D,)).reshape(64, D)[:m].copy()
        sv = np.ctypeslib.as_array(lib().orc_pair_stgv(self._h), shape=(64 * D,)).reshape(64, D)[:m].copy()
        return sk, sv

    def scores(self, q):
        q = _u16(q).reshape(-1, D)
        nb = self.info().nblk
        s = np.zeros(max(nb, 1), np.float32)
        n = lib().orc_pair_scores(self._h, _p(q, C.c_uint16), _p(s, C.c_float), nb)
        return s[:n]

    def decode(self, q, scale):
        """-> (out [G][D] fp64, selected block indices ascending)."""
        q = _u16(q).reshape(-1, D)
        G = q.shape[0]
        out = np.zeros((G, D), np.float64)
        nb = max(self.info().nblk, 1)
        sel = np.zeros(nb, np.int32)
        ns = lib().orc_pair_decode(self._h, _p(q, C.c_uint16), scale, _p(out, C.c_double),
                                   _p(sel, C.c_int32), nb)
        if ns < 0:
            raise ValueError("decode: non-finite block score")
        return out, sel[:ns].copy()
