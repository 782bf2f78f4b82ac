"""C ABI of libmosaic on the CPU: the library loads, exports every symbol the
header declares, and validates arguments before touching the GPU."""
import ctypes as C
import os
import re
import subprocess

import pytest

import paper_2607_00760_amd as M
from paper_2607_00760_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mosaic.h")


def declared_functions():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(mosaic_[a-z_]+)\s*\(", txt)))


def test_header_and_exports_agree():
    names = declared_functions()
    assert "mosaic_compress" in names and "mosaic_append" in names and "mosaic_decode_attention" in names
    out = subprocess.run(["nm", "-D", "--defined-only", _lib.LIB_PATH], capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\bT (mosaic_\w+)", out))
    assert set(names) <= exported, set(names) - exported
    assert set(names) == set(_lib.EXPORTED)
    L = _lib.load()
    for n in names:
        assert getattr(L, n) is not None


def _create(**kw):
    L = _lib.load()
    raw = {"head_dim", "seg_len", "update_buf", "group_size", "num_kv_heads", "dtype", "rot_window"}
    p = M.Params(**{k: v for k, v in kw.items() if k in M.Params.__dataclass_fields__ and k not in raw}).to_c()
    for k, v in kw.items():
        if k in raw:
            setattr(p, k, v)
    h = C.c_void_p()
    st = L.mosaic_cache_create(C.byref(p), kw.get("num_seqs", 2), kw.get("max_tokens", 1000), kw.get("rotated", 1),
                               C.byref(h))
    return st, h


def test_defaults_match_paper():
    p = _lib.MosaicParams()
    _lib.load().mosaic_params_default(C.byref(p))
    assert (p.head_dim, p.seg_len, p.update_buf, p.rot_window) == (128, 64, 32, 65536)
    assert list(p.keep_cand) == [16, 32, 48] and list(p.group_cand) == [4, 2, 1] and list(p.block_cand) == [16, 8, 4]
    assert (p.default_keep, p.default_group, p.default_block) == (32, 1, 8)
    assert (p.select_num, p.select_den) == (1, 10)
    assert (p.trunc_channels, p.value_fp8) == (128, 0)


@pytest.mark.parametrize("kw,status", [
    (dict(head_dim=64), -2), (dict(seg_len=32), -2), (dict(update_buf=16), -2),
    (dict(group_size=9), -1), (dict(group_size=0), -1), (dict(num_kv_heads=0), -1), (dict(dtype=3), -1),
    (dict(rot_window=100), -1), (dict(keep_cand=(16, 30, 48)), -1), (dict(group_cand=(3, 2, 1)), -1),
    (dict(block_cand=(16, 8, 2)), -1), (dict(default=(33, 1, 8)), -1), (dict(tau_channel=float("nan")), -1),
    (dict(select=(0, 10)), -1), (dict(max_tokens=0), -1), (dict(num_seqs=0), -1),
    (dict(max_tokens=40_000_000), -3), (dict(trunc=100), -1), (dict(trunc=96, default=(128, 1, 8)), -1),
    # one-byte values keep records 4-byte aligned only with kept counts that are multiples of 4
    (dict(fp8=True, keep_cand=(18, 32, 48), group_cand=(2, 2, 1)), -1),
    (dict(fp8=True, default=(18, 2, 8), group_cand=(2, 2, 1)), -1),
])
def test_create_rejects(kw, status):
    st, h = _create(**kw)
    assert st == status
    assert _lib.load().mosaic_last_error().decode() != ""


def test_layout_and_workspace():
    L = _lib.load()
    st, h = _create(num_seqs=3, max_tokens=70000, num_kv_heads=2, group_size=7)
    assert st == 0
    n = C.c_size_t()
    assert L.mosaic_cache_arena_bytes(h, C.byref(n)) == 0
    lay = _lib.MosaicLayout()
    assert L.mosaic_cache_layout(h, C.byref(lay)) == 0
    assert lay.num_pairs == 6 and lay.num_windows == 2 and lay.total == n.value
    offs = [lay.meta_off, lay.desc_off, lay.score_off, lay.token_off, lay.buf_off, lay.stage_off, lay.rot_off]
    strides = [lay.meta_stride, lay.desc_stride, lay.score_stride, lay.token_stride, lay.buf_stride,
               lay.stage_stride, lay.rot_stride]
    for a, b, s in zip(offs, offs[1:], strides):
        assert a % 256 == 0 and s % 256 == 0 and a + 6 * s <= b
    assert lay.rot_stride >= 2 * 3 * 128 * 128 * 4
    assert lay.token_stride >= (70000 // 64 + 1) * 64 * 2 * (2 * 48 + 16)
    for op, pos in ((0, True), (1, False), (2, True)):
        assert L.mosaic_workspace_bytes(h, op, C.byref(n)) == 0
        assert (n.value > 0) == pos
    # the optional single-pass compression workspace: a worst-case slot per (pair, segment)
    assert L.mosaic_workspace_bytes(h, 0, C.byref(n)) == 0
    assert n.value >= 6 * (70000 // 64 + 1) * 64 * 2 * (2 * 48 + 16)
    assert L.mosaic_workspace_bytes(h, 7, C.byref(n)) == -1
    wl = _lib.MosaicWsLayout()
    assert L.mosaic_decode_ws_layout(h, C.byref(wl)) == 0 and wl.gp == 8 and wl.max_splits > 0
    L.mosaic_cache_destroy(h)


def test_calls_out_of_order_or_bad_pointers_fail_before_launch():
    L = _lib.load()
    st, h = _create(num_seqs=1, max_tokens=128, rotated=0)
    assert st == 0
    lens = (C.c_int32 * 1)(64)
    fake = C.c_void_p(0x100000)
    # not bound
    assert L.mosaic_compress(h, fake, fake, 128, lens, None, None, None, 0, None) == -4
    assert L.mosaic_append(h, fake, fake, None) == -4
    assert L.mosaic_decode_attention(h, fake, fake, 0.1, fake, 1 << 20, None) == -4
    # misaligned arena, too small arena
    assert L.mosaic_cache_bind(h, C.c_void_p(0x100010), 1 << 30) == -1
    assert L.mosaic_cache_bind(h, C.c_void_p(0x100000), 16) == -1
    assert L.mosaic_cache_bind(h, C.c_void_p(0x100000), 1 << 30) == 0
    # bound but not compressed
    assert L.mosaic_append(h, fake, fake, None) == -4
    assert L.mosaic_decode_attention(h, fake, fake, 0.1, fake, 1 << 20, None) == -4
    # compress argument checks (all before any HIP call)
    assert L.mosaic_compress(h, None, fake, 128, lens, None, None, None, 0, None) == -1
    assert L.mosaic_compress(h, C.c_void_p(0x100002), fake, 128, lens, None, None, None, 0, None) == -1
    assert L.mosaic_compress(h, fake, fake, 128, lens, fake, fake, None, 0, None) == -1      # not a rotated cache
    big = (C.c_int32 * 1)(129)
    assert L.mosaic_compress(h, fake, fake, 256, big, None, None, None, 0, None) == -3
    neg = (C.c_int32 * 1)(-1)
    assert L.mosaic_compress(h, fake, fake, 128, neg, None, None, None, 0, None) == -1
    assert L.mosaic_compress(h, fake, fake, 32, lens, None, None, None, 0, None) == -1       # stride < length
    assert "seq_stride" in L.mosaic_last_error().decode()
    L.mosaic_cache_destroy(h)


def test_dense_argument_checks():
    L = _lib.load()
    n = C.c_size_t()
    assert L.mosaic_dense_workspace_bytes(2, 8, 4, 4096, C.byref(n)) == 0 and n.value > 0
    fake = C.c_void_p(0x100000)
    assert L.mosaic_dense_decode_attention(fake, fake, fake, fake, 1, 8, 4, 64, 0, 128, 128, fake, 0.1, fake,
                                           n.value, None) == -2
    assert L.mosaic_dense_decode_attention(fake, fake, fake, fake, 1, 8, 4, 128, 0, 64, 128, fake, 0.1, fake,
                                           n.value, None) == -1
    assert L.mosaic_dense_decode_attention(fake, fake, fake, fake, 1, 8, 4, 128, 0, 128, 128, fake, 0.1, fake,
                                           16, None) == -1


def test_package_has_no_fallback(monkeypatch, tmp_path):
    monkeypatch.setattr(_lib, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(_lib, "_lib", None)
    with pytest.raises(ImportError):
        _lib.load()


def test_rotation_and_reorder_argument_checks():
    """The rotation and reorder entry points validate everything before any
    HIP call (workspace sizes, NULL and misaligned pointers, lengths)."""
    L = _lib.load()
    p = M.Params(num_kv_heads=2, rot_window=1024).to_c()
    n_rot, n_reo = C.c_size_t(), C.c_size_t()
    assert L.mosaic_rotation_workspace_bytes(C.byref(p), 3, 2500, C.byref(n_rot)) == 0
    assert L.mosaic_reorder_workspace_bytes(C.byref(p), 3, 2500, C.byref(n_reo)) == 0
    nw = 3                                                    # ceil(2500 / 1024)
    assert n_reo.value >= 3 * 2 * 2 * nw * 128 * 4 + 3 * 2 * 2 * nw * 128 * 128 * 4
    assert L.mosaic_reorder_workspace_bytes(C.byref(p), 0, 2500, C.byref(n_reo)) == -1
    lens = (C.c_int32 * 3)(2500, 10, 0)
    fake, ws = C.c_void_p(0x100000), C.c_void_p(0x200000)
    big_ws = 1 << 40
    args = lambda **kw: [C.byref(p), 3, 2500, kw.get("k", fake), fake, kw.get("stride", 2500), kw.get("lens", lens),
                         kw.get("rk", fake), fake, kw.get("ws", ws), kw.get("ws_bytes", big_ws), None]
    assert L.mosaic_reorder_rotations(*args(k=None)) == -1
    assert L.mosaic_reorder_rotations(*args(rk=C.c_void_p(0x100004))) == -1                 # misaligned R
    assert L.mosaic_reorder_rotations(*args(ws=C.c_void_p(0x200010))) == -1                 # ws not 256-aligned
    assert L.mosaic_reorder_rotations(*args(ws_bytes=16)) == -1                              # small workspace
    assert L.mosaic_reorder_rotations(*args(stride=100)) == -1                               # stride < length
    assert L.mosaic_reorder_rotations(*args(lens=(C.c_int32 * 3)(2501, 0, 0))) == -3         # past max_tokens
    assert L.mosaic_reorder_rotations(*args(lens=(C.c_int32 * 3)(-1, 0, 0))) == -1
    p.default_keep = 0
    assert L.mosaic_reorder_rotations(*args()) == -1
    assert "default_keep" in L.mosaic_last_error().decode()


def test_ragged_capacities_layout():
    """Per-sequence capacities: each pair's desc, score and token regions are
    sized for its own sequence, 256-byte aligned, in pair order, disjoint and
    inside the arena, located only by the pair table (strides 0); the arena is
    smaller than with the longest capacity everywhere; uniform caches report
    p * stride in the same table."""
    L = _lib.load()
    p = M.Params(num_kv_heads=2, group_size=4).to_c()
    caps = (C.c_int32 * 3)(100, 5000, 70000)
    h = C.c_void_p()
    assert L.mosaic_cache_create_ragged(C.byref(p), 3, caps, 1, C.byref(h)) == 0
    lay = _lib.MosaicLayout()
    assert L.mosaic_cache_layout(h, C.byref(lay)) == 0
    assert lay.desc_stride == lay.score_stride == lay.token_stride == 0 and lay.num_windows == 2
    tab = (C.c_uint64 * 24)()
    assert L.mosaic_cache_pair_regions(h, tab) == 0
    rows = [tuple(tab[4 * q: 4 * q + 4]) for q in range(6)]
    starts = (lay.desc_off, lay.score_off, lay.token_off)
    for r, nxt in ((0, lay.score_off), (1, lay.token_off), (2, lay.buf_off)):
        offs = [starts[r] + row[r] for row in rows]
        assert all(o % 256 == 0 for o in offs) and offs == sorted(offs) and offs[0] == starts[r]
        assert offs[-1] < nxt
    tok = [rows[q][3] for q in range(6)]
    assert tok[0] == tok[1] < tok[2] == tok[3] < tok[4] == tok[5]
    assert tok[4] >= (70000 // 64 + 1) * 64 * 2 * (2 * 48 + 16) and tok[0] < (100 // 64 + 3) * 64 * 2 * (2 * 48 + 16) + 512
    for q in range(5):
        assert rows[q][2] + tok[q] <= rows[q + 1][2]
    n_r, n_u = C.c_size_t(), C.c_size_t()
    assert L.mosaic_cache_arena_bytes(h, C.byref(n_r)) == 0
    st, hu = _create(num_seqs=3, max_tokens=70000, num_kv_heads=2, group_size=4)
    assert st == 0 and L.mosaic_cache_arena_bytes(hu, C.byref(n_u)) == 0
    assert n_r.value < 0.4 * n_u.value
    lu = _lib.MosaicLayout()
    assert L.mosaic_cache_layout(hu, C.byref(lu)) == 0 and L.mosaic_cache_pair_regions(hu, tab) == 0
    assert [tuple(tab[4 * q: 4 * q + 4]) for q in range(6)] == \
        [(q * lu.desc_stride, q * lu.score_stride, q * lu.token_stride, lu.token_stride) for q in range(6)]
    L.mosaic_cache_destroy(h)
    L.mosaic_cache_destroy(hu)
    for bad in ((100, 0, 5), (100, -3, 5)):
        assert L.mosaic_cache_create_ragged(C.byref(p), 3, (C.c_int32 * 3)(*bad), 1, C.byref(h)) == -1
    assert L.mosaic_cache_create_ragged(C.byref(p), 3, None, 1, C.byref(h)) == -1
    assert L.mosaic_cache_create_ragged(C.byref(p), 0, caps, 1, C.byref(h)) == -1
