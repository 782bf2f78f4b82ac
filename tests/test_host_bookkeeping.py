"""Host bookkeeping of the C ABI, on the CPU: the real host layer (csrc/api.hip)
linked with a launch layer that records what it is asked to launch
(tests/hostsim/fake_launch.hip) instead of running kernels.

Checked: the append schedule (a flush exactly when a sequence's update buffer
reaches U = 32 tokens, a finalize exactly when its segment reaches S = 64
tokens, ragged lengths OR-ed into one launch), the launch plan of compress and
decode, capacity exhaustion, and the validation errors of every entry point,
each of which must return its status, launch nothing and leave the handle
unchanged.  The same checks run again with the host code built with
AddressSanitizer and UndefinedBehaviorSanitizer, in a child process that
preloads the sanitizer runtime.
"""
from __future__ import annotations

import ctypes as C
import math
import os
import subprocess
import sys


HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "hostsim"))
sys.path.insert(0, os.path.dirname(HERE))

import build as hostsim_build  # noqa: E402  (tests/hostsim/build.py)
from paper_2607_00760_amd import _lib  # noqa: E402

U, S = 32, 64
OK, INVALID, UNSUPPORTED, CAPACITY, STATE = 0, -1, -2, -3, -4


class Sim:
    def __init__(self, path):
        self.L = _lib.bind_signatures(C.CDLL(path))
        self.L.fake_log_count.restype = C.c_int
        self.L.fake_log_entry.restype = C.c_char_p
        self.L.fake_log_entry.argtypes = [C.c_int]
        self.keep = []

    def log(self):
        out = [self.L.fake_log_entry(i).decode() for i in range(self.L.fake_log_count())]
        self.L.fake_log_clear()
        return out

    def params(self, **kw):
        p = _lib.MosaicParams()
        self.L.mosaic_params_default(C.byref(p))
        for k, v in kw.items():
            setattr(p, k, v)
        return p

    def buf(self, n, align=256, offset=0):
        """A host buffer standing in for device memory (the recording layer never reads it)."""
        raw = C.create_string_buffer(n + align + offset)
        self.keep.append(raw)
        return C.c_void_p(((C.addressof(raw) + align - 1) // align) * align + offset)

    def cache(self, num_seqs, max_tokens, rotated=0, **kw):
        p = self.params(**kw)
        h = C.c_void_p()
        assert self.L.mosaic_cache_create(C.byref(p), num_seqs, max_tokens, rotated, C.byref(h)) == OK
        n = C.c_size_t()
        assert self.L.mosaic_cache_arena_bytes(h, C.byref(n)) == OK
        return h, p, n.value

    def tokens(self, h, num_seqs):
        return [self.L.mosaic_seq_tokens(h, q) for q in range(num_seqs)]


def expected_maintain(lengths):
    """What the append that brings each sequence to lengths + 1 must launch:
    a finalize if some sequence completes a segment, a flush if some sequence
    fills its buffer without completing a segment."""
    fin = any((L + 1) % S == 0 for L in lengths)
    flush = any((L + 1) % U == 0 and (L + 1) % S != 0 for L in lengths)
    return fin, flush


def run_checks(path):
    sim = Sim(path)
    L = sim.L
    sim.log()
    # ---- compress plan
    ns, hkv, cap = 3, 2, 400
    h, p, arena = sim.cache(ns, cap, num_kv_heads=hkv)
    kv = sim.buf(4 * 128 * 2 * ns * hkv * 128, 16)
    ctx = (C.c_int32 * ns)(0, 31, 100)
    assert L.mosaic_compress(h, kv, kv, 100, ctx, None, None, None, 0, None) == STATE     # not bound yet
    assert sim.log() == []
    assert L.mosaic_cache_bind(h, sim.buf(arena), arena) == OK
    assert L.mosaic_append(h, kv, kv, None) == STATE                                       # before compress
    q = sim.buf(ns * hkv * 4 * 128 * 2, 16)
    out = sim.buf(ns * hkv * 4 * 128 * 4, 16)
    wsz = C.c_size_t()
    assert L.mosaic_workspace_bytes(h, 2, C.byref(wsz)) == OK
    ws = sim.buf(wsz.value)
    assert L.mosaic_decode_attention(h, q, out, C.c_float(0.1), ws, wsz.value, None) == STATE
    assert sim.log() == []
    # compress errors: nothing launched, nothing changed
    bad = [
        (dict(k=None), INVALID), (dict(k=C.c_void_p(kv.value + 2)), INVALID), (dict(stride=99), INVALID),
        (dict(ctx=(C.c_int32 * ns)(0, cap + 1, 5)), CAPACITY), (dict(ctx=(C.c_int32 * ns)(0, -1, 5)), INVALID),
        (dict(rot=sim.buf(64, 16)), INVALID),                                 # cache created without rotation
    ]
    for kw, st in bad:
        r = L.mosaic_compress(h, kw.get("k", kv), kv, kw.get("stride", 100), kw.get("ctx", ctx),
                              kw.get("rot"), kw.get("rot"), None, 0, None)
        assert r == st, (kw, r)
        assert L.mosaic_last_error()
    assert sim.log() == []
    assert L.mosaic_compress(h, kv, kv, 100, ctx, None, None, None, 0, None) == OK
    log = sim.log()
    assert log[0] == "ctx_copy 0 31 100" and log[1].startswith(f"pairs_copy npairs={ns * hkv} tok 0 ")
    assert log[2:] == [f"compress npairs={ns * hkv} stride=100 segs=1 tail=1"]
    lengths = [0, 31, 100]
    assert sim.tokens(h, ns) == lengths
    # ---- the append schedule over 320 appends (ragged lengths cross U and S at different steps)
    for t in range(cap - 100):
        fin, flush = expected_maintain(lengths)
        assert L.mosaic_append(h, kv, kv, None) == OK, t
        want = [f"append npairs={ns * hkv}"]
        if fin or flush:
            want.append(f"maintain mode=0 flush={int(flush)} finalize={int(fin)}")
        assert sim.log() == want, (t, lengths)
        lengths = [x + 1 for x in lengths]
        assert sim.tokens(h, ns) == lengths
    # the longest sequence is full: the next append fails and changes nothing
    assert max(lengths) == cap
    assert L.mosaic_append(h, kv, kv, None) == CAPACITY
    assert sim.log() == [] and sim.tokens(h, ns) == lengths
    # append errors
    assert L.mosaic_append(h, None, kv, None) == INVALID
    assert L.mosaic_append(h, C.c_void_p(kv.value + 2), kv, None) == INVALID
    assert sim.log() == [] and sim.tokens(h, ns) == lengths
    # ---- decode plan and errors
    desc = max(x // S + (1 if x % S >= U else 0) for x in lengths)
    wins = max(1, min(math.ceil(cap / p.rot_window), math.ceil(max(lengths) / p.rot_window)))
    for kw, st in [(dict(q=None), INVALID), (dict(wsz=wsz.value - 1), INVALID), (dict(ws=sim.buf(wsz.value, 256, 16)), INVALID),
                   (dict(scale=float("nan")), INVALID), (dict(q=C.c_void_p(q.value + 2)), INVALID)]:
        r = L.mosaic_decode_attention(h, kw.get("q", q), out, C.c_float(kw.get("scale", 0.1)), kw.get("ws", ws),
                                      kw.get("wsz", wsz.value), None)
        assert r == st, (kw, r)
    assert sim.log() == []
    assert L.mosaic_decode_attention(h, q, out, C.c_float(0.125), ws, wsz.value, None) == OK
    assert sim.log() == [f"decode npairs={ns * hkv} desc={desc} windows={wins} scale=0.125000"]
    assert L.mosaic_workspace_bytes(h, 7, C.byref(wsz)) == INVALID
    assert L.mosaic_cache_destroy(h) == OK
    # ---- creation errors
    h2 = C.c_void_p()
    for kw, st in [(dict(head_dim=64), UNSUPPORTED), (dict(seg_len=32), UNSUPPORTED), (dict(update_buf=16), UNSUPPORTED),
                   (dict(num_kv_heads=0), INVALID), (dict(group_size=9), INVALID), (dict(dtype=5), INVALID),
                   (dict(rot_window=100), INVALID), (dict(select_den=0), INVALID), (dict(tau_channel=float("nan")), INVALID),
                   (dict(trunc_channels=80), INVALID), (dict(default_keep=130), INVALID)]:
        pp = sim.params(**kw)
        assert L.mosaic_cache_create(C.byref(pp), 2, 100, 0, C.byref(h2)) == st, kw
    pp = sim.params()
    assert L.mosaic_cache_create(C.byref(pp), 0, 100, 0, C.byref(h2)) == INVALID
    assert L.mosaic_cache_create(C.byref(pp), 1, 0, 0, C.byref(h2)) == INVALID
    # a rotated cache needs its rotations; the rotation copy is planned before the compression
    h3, _, arena3 = sim.cache(1, 200, rotated=1, num_kv_heads=1, rot_window=128)
    assert L.mosaic_cache_bind(h3, sim.buf(arena3), arena3) == OK
    ctx1 = (C.c_int32 * 1)(130)
    assert L.mosaic_compress(h3, kv, kv, 130, ctx1, None, None, None, 0, None) == INVALID
    rot = sim.buf(2 * 128 * 128 * 4, 16)
    assert L.mosaic_compress(h3, kv, kv, 130, ctx1, rot, rot, None, 0, None) == OK
    assert sim.log() == ["ctx_copy 130", "pairs_copy npairs=1 tok 0", "copy_rot npairs=1 nw=2 src=2",
                         "compress npairs=1 stride=130 segs=2 tail=1"]
    assert L.mosaic_cache_destroy(h3) == OK
    # ---- dynamic windows: parameters, window slots, and the poll-before-compress rule
    for kw, st in [(dict(dyn_windows=2), INVALID), (dict(dyn_windows=1, min_window=100), INVALID),
                   (dict(dyn_windows=1, min_window=0), INVALID), (dict(dyn_windows=1, tau_window=float("nan")), INVALID),
                   (dict(dyn_windows=1, rot_window=256, min_window=512), INVALID)]:
        pp = sim.params(**kw)
        assert L.mosaic_cache_create(C.byref(pp), 1, 1000, 1, C.byref(h2)) == st, kw
    pp = sim.params(dyn_windows=1)
    assert L.mosaic_cache_create(C.byref(pp), 1, 1000, 0, C.byref(h2)) == INVALID         # needs rotations
    pp = sim.params(dyn_windows=1, min_window=64)
    assert L.mosaic_cache_create(C.byref(pp), 1, 70000, 1, C.byref(h2)) == UNSUPPORTED    # 1094 windows > 1024
    h4, p4, arena4 = sim.cache(2, 1000, rotated=1, num_kv_heads=1, rot_window=512, dyn_windows=1, min_window=128)
    lay = _lib.MosaicLayout()
    assert L.mosaic_cache_layout(h4, C.byref(lay)) == OK
    assert lay.num_windows == 1000 // 128 + 1 and lay.meta_stride >= 64 + 4 * (lay.num_windows + 1)
    assert L.mosaic_cache_bind(h4, sim.buf(arena4), arena4) == OK
    ctx4 = (C.c_int32 * 2)(62, 10)
    rot4 = sim.buf(2 * 2 * 128 * 128 * 4, 16)
    assert L.mosaic_compress(h4, kv, kv, 100, ctx4, rot4, rot4, None, 0, None) == OK
    assert sim.log()[2] == "copy_rot npairs=2 nw=8 src=2"
    closed = (C.c_int32 * 6)()
    nclosed = C.c_int32()
    h5, _, _ = sim.cache(1, 100)
    assert L.mosaic_window_poll(h5, closed, C.byref(nclosed), None) == INVALID               # a fixed-window cache
    assert L.mosaic_cache_destroy(h5) == OK
    assert L.mosaic_window_close(h4, rot4, rot4, kv, kv, 64, None) == OK                     # nothing to close
    assert sim.log() == []
    assert L.mosaic_append(h4, kv, kv, None) == OK                                           # sequence 0: 63 tokens
    assert L.mosaic_append(h4, kv, kv, None) == OK                                           # 64: finalize
    assert sim.log()[-1] == "maintain mode=0 flush=0 finalize=1"
    assert L.mosaic_window_close(h4, rot4, rot4, kv, kv, 64, None) == STATE                  # poll first
    wrb = C.c_size_t()
    assert L.mosaic_workspace_bytes(h4, 3, C.byref(wrb)) == OK and wrb.value >= 2 * 2 * 128 * 128 * 4
    wr = sim.buf(wrb.value)
    assert L.mosaic_window_rotations(h4, rot4, rot4, wr, wrb.value, None) == STATE           # poll first too
    assert L.mosaic_window_rotations(h4, rot4, rot4, wr, wrb.value - 1, None) == STATE
    for _ in range(19):                                                                      # no compression due
        assert L.mosaic_append(h4, kv, kv, None) == OK
    # sequence 1 would reach 32 tokens: its buffer would be compressed before a poll
    assert sim.tokens(h4, 2) == [83, 31]
    sim.log()
    assert L.mosaic_append(h4, kv, kv, None) == STATE
    assert sim.log() == [] and sim.tokens(h4, 2) == [83, 31]
    assert "poll" in L.mosaic_last_error().decode()
    assert L.mosaic_cache_destroy(h4) == OK
    # ---- per-sequence capacities: each sequence checked against its own
    pr = sim.params(num_kv_heads=1)
    h6 = C.c_void_p()
    assert L.mosaic_cache_create_ragged(C.byref(pr), 2, (C.c_int32 * 2)(40, 300), 0, C.byref(h6)) == OK
    n6 = C.c_size_t()
    assert L.mosaic_cache_arena_bytes(h6, C.byref(n6)) == OK
    assert L.mosaic_cache_bind(h6, sim.buf(n6.value), n6.value) == OK
    assert L.mosaic_compress(h6, kv, kv, 100, (C.c_int32 * 2)(41, 100), None, None, None, 0, None) == CAPACITY
    assert sim.log() == []
    assert L.mosaic_compress(h6, kv, kv, 100, (C.c_int32 * 2)(38, 100), None, None, None, 0, None) == OK
    log = sim.log()
    tok = [int(x) for x in log[1].split(" tok ")[1].split()]
    assert log[0] == "ctx_copy 38 100" and log[1].startswith("pairs_copy npairs=2 tok 0 ")
    assert 0 < tok[1] < 8 * 64 * 2 * 112        # the short sequence's token slot: (40 / 64 + 2) segments
    assert L.mosaic_append(h6, kv, kv, None) == OK and L.mosaic_append(h6, kv, kv, None) == OK
    assert L.mosaic_append(h6, kv, kv, None) == CAPACITY                                     # sequence 0 holds 40
    assert sim.tokens(h6, 2) == [40, 102]
    assert L.mosaic_cache_destroy(h6) == OK
    return True


def test_host_bookkeeping_with_recording_launcher():
    assert run_checks(hostsim_build.build())


def test_host_bookkeeping_under_address_and_ub_sanitizers():
    lib = hostsim_build.build(sanitize=True)
    env = dict(os.environ, LD_PRELOAD=hostsim_build.asan_runtime(), ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    code = f"import sys; sys.path.insert(0, {HERE!r}); import test_host_bookkeeping as T; T.run_checks({lib!r}); print('clean')"
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0 and "clean" in r.stdout, (r.returncode, r.stdout[-2000:], r.stderr[-4000:])
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr[-4000:]


def test_oracle_pins_under_address_and_ub_sanitizers(tmp_path):
    """The oracle built with gcc's AddressSanitizer and UndefinedBehaviorSanitizer
    runs its whole pin suite in a child process."""
    src = os.path.join(os.path.dirname(HERE), "oracle", "mosaic_oracle.c")
    lib = str(tmp_path / "liboracle_san.so")
    subprocess.run(["gcc", "-O1", "-g", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
                    "-o", lib, src, "-lm"], check=True)
    rt = [subprocess.run(["gcc", f"-print-file-name={n}"], capture_output=True, text=True).stdout.strip()
          for n in ("libasan.so", "libubsan.so")]
    env = dict(os.environ, LD_PRELOAD=" ".join(rt), MOSAIC_ORACLE_LIB=lib, ASAN_OPTIONS="detect_leaks=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(HERE, "test_oracle_pins.py")], env=env, capture_output=True, text=True,
                       timeout=600, cwd=os.path.dirname(HERE))
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-3000:])
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr[-3000:]
