#!/usr/bin/env python3
"""Benchmark of the MosaicKV decode step on one MI355X.

Workload (the metric's configuration, the default): decode attention over a
compressed KV cache, batch 8 x 131072-token contexts, 32 query / 8 kv heads,
head dim 128, bf16, ~3x compression, 5 % of segments planted to carry 80 % of
the softmax mass.  A step is one mosaic_decode_attention call (q rotation,
block scoring, top-k, split-K packed attention, combine with back-rotation)
over the resident cache.  A 1 GiB buffer is read before every step so that
the 256 MB MALL holds none of the step's data; only the step itself sits
between the step's events.

Other workloads (--config): c1 (one 4K sequence), c2 and c5 (a step is one
append of a token to every sequence plus one decode, as those workloads
define it), c4 (one decode step across the 32 layers of a 1M-token cache,
each layer its own cache; per-layer and total times).

Prints ONE JSON line: value = microseconds per step (lower is better), plus
the roofline of the dominant kernel against the nominal 8 TB/s and against the
streaming-read bandwidth measured in the same run, the dense attention of the
same shape (this library's kernel and PyTorch SDPA), the compression pass and
the CPU oracle timed on the host's cores on a bounded sample.
"""
from __future__ import annotations

import argparse
import ctypes as C
import concurrent.futures as cf
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "compressed decode-attn µs/step + effective HBM GB/s, 128K ctx ×8 seqs vs dense"
HBM_PEAK_GBPS = 8000.0
D = 128


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="c3")
    ap.add_argument("--trunc", type=int, default=128,
                    help="channels represented in the bitmaps (channel truncation; 128 = none)")
    ap.add_argument("--force-default", action="store_true",
                    help="every segment takes the default strategy (32, 1, 8) instead of the search")
    ap.add_argument("--fp8", action="store_true",
                    help="K and V token values stored as E4M3 codes (block keys stay 16-bit)")
    ap.add_argument("--mode", choices=("mosaic", "quest"), default="mosaic",
                    help="quest: every channel kept, 16-token blocks, no rotation (sequence-only "
                         "compression on the same kernels)")
    ap.add_argument("--ctx", type=int, default=0, help="override the context length (smoke runs)")
    ap.add_argument("--flush-mb", type=int, default=1024)
    ap.add_argument("--dense-steps", type=int, default=5)
    ap.add_argument("--cpu-sample-pairs", type=int, default=0,
                    help="pairs the CPU oracle decodes (0: one per host core, up to every pair)")
    ap.add_argument("--layers", type=int, default=None, help="layers of c4 (default: all 32)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--no-graph", action="store_true")
    ap.add_argument("--no-rotations", action="store_true", help="skip timing the GPU rotation computation")
    ap.add_argument("--no-extras", action="store_true", help="skip the append-path and encoding-overlap timings")
    ap.add_argument("--calib-copy", type=int, default=0, metavar="MIB",
                    help="only run 5 device-to-device copies of MIB MiB (the reference kernel that scales the "
                         "FETCH_SIZE / WRITE_SIZE counters to bytes) and exit")
    return ap.parse_args()


def algorithmic_bytes(cache, spec, nb_list, sel_list, desc_list):
    """Bytes the method must move per decode step, per kernel (score / attn /
    qrot / reduce) and in total: block keys and descriptors (score), the
    selected blocks' packed K and V and the update-buffer tokens (attn), R_k^T
    per window and q (qrot), R_v per window with selected blocks and the fp32
    output (reduce, which rotates each window's merged sum back)."""
    G = spec.group
    W = spec.rot_window
    tot = dict(score=0, attn=0, qrot=0, reduce=0)
    sel_tok = scoreable_tok = 0
    nwq = max(1, -(-max(spec.ctx) // W))
    for p, (nb, sel, descs) in enumerate(zip(nb_list, sel_list, desc_list)):
        L = spec.ctx[p // spec.hkv]
        n_desc = len(descs)
        bmb = [(cache.params.trunc >> d[4]) >> 3 for d in descs]          # exactly T / g bits
        srec = [2 * d[3] + b for d, b in zip(descs, bmb)]                  # block keys: 16-bit values
        rec = [(1 if cache.params.fp8 else 2) * d[3] + b for d, b in zip(descs, bmb)]   # K / V tokens
        blocks_per = [((32 if d[6] & 1 else 64) >> d[5]) for d in descs]
        tot["score"] += sum(r * n for r, n in zip(srec, blocks_per)) + 16 * n_desc
        # selected blocks -> descriptor (first_block ascending)
        fb = [d[2] for d in descs]
        import bisect
        wins = set()
        for b in sel:
            i = bisect.bisect_right(fb, b) - 1
            B = 1 << descs[i][5]
            tot["attn"] += B * 2 * rec[i]
            sel_tok += B
            wins.add((i * 64) // W)
        scoreable_tok += sum(32 if d[6] & 1 else 64 for d in descs)
        m = L % 64
        nbuf = m - (32 if m >= 32 else 0)
        tot["attn"] += nbuf * 2 * D * 2
        tot["qrot"] += (nwq if cache.rotated else 0) * D * D * 4 + G * D * 2
        tot["reduce"] += (len(wins) if cache.rotated else 0) * D * D * 4    # R_v of each window, in the combine
        tot["reduce"] += G * D * 4
    tot["total"] = sum(tot.values())
    return tot, dict(selected_tokens=sel_tok, scoreable_tokens=scoreable_tok,
                     fraction=round(sel_tok / max(scoreable_tok, 1), 5))


def source_hash():
    h = hashlib.sha256()
    for f in ("decode.hip", "mosaic_internal.h"):
        h.update(open(os.path.join(ROOT, "paper_2607_00760_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def log(msg):
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def update_path_us(M, gen, spec, params, dev):
    """Append calls of the c3 batch shape (every (sequence, kv head) pair at
    once) on a short cache: the calls whose 32nd token fills the update buffer
    (provisional flush, Sec. 5.4) and the calls that complete a 64-token
    segment (finalize with its own strategy), against plain appends; medians
    over 256 appends (4 of each kind)."""
    import torch
    n = 256
    small = gen.spec(spec.name, ctx=(4096,) * spec.num_seqs, appends=n)
    lay = gen.make_layer(small, 0, device=dev, capacity=small.capacity)
    cache = M.MosaicCache(params, small.num_seqs, small.capacity, rotated=small.rotate, device=dev)
    cache.compress(lay["k"], lay["v"], lay["ctx_lens"], lay["rot_k"], lay["rot_v"])
    apps = [tuple(x.to(dev) for x in gen.make_appends(small, t)) for t in range(n)]
    torch.cuda.synchronize()
    times = []
    for t in range(n):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        cache.append(*apps[t])
        b.record()
        torch.cuda.synchronize()
        times.append(1e3 * a.elapsed_time(b))
    med = lambda xs: round(float(sorted(xs)[len(xs) // 2]), 1)
    kind = lambda t: (t + 1) % 64 == 0 and 2 or ((t + 1) % 32 == 0 and 1) or 0   # 4096 + t + 1 tokens after call t
    return {"pairs": small.num_seqs * small.hkv, "append_us": med([x for t, x in enumerate(times) if kind(t) == 0]),
            "append_with_flush_us": med([x for t, x in enumerate(times) if kind(t) == 1]),
            "append_with_finalize_us": med([x for t, x in enumerate(times) if kind(t) == 2]), "samples": n}


def dyn_window_us(M, gen, spec, params, dev, reps=3):
    """Windows closed by their loss (Sec. 4.3 dynamic partitioning of output
    tokens, Sec. 5.5), c3 batch shape, 4096-token windows: a 4032-token
    prefill per pair, so that the 64th append completes the window's last
    segment and closes it (maximum length).  Times that append (finalize plus
    the loss update), mosaic_window_rotations (every pair's K and V rotation
    from the window's incremental covariance, Jacobi on the GPU) and
    mosaic_window_close (the new rotations and the re-encoding of each pair's
    4096 tokens, strategy and packing passes); medians over `reps` fresh
    caches."""
    import dataclasses
    import torch
    W = 4096
    small = gen.spec(spec.name, ctx=(W - 64,) * spec.num_seqs, appends=64, rot_window=W)
    lay = gen.make_layer(small, 0, device=dev, capacity=small.capacity)
    dp = dataclasses.replace(params, rot_window=W, dyn_windows=True, min_window=1024, tau_window=1e30)
    apps = [tuple(x.to(dev) for x in gen.make_appends(small, t)) for t in range(64)]
    kw = torch.cat([lay["k"][:, :, :W - 64], torch.stack([a[0] for a in apps], dim=2)], dim=2).contiguous()
    vw = torch.cat([lay["v"][:, :, :W - 64], torch.stack([a[1] for a in apps], dim=2)], dim=2).contiguous()
    fin, rot, close = [], [], []
    for _ in range(reps):
        cache = M.MosaicCache(dp, small.num_seqs, small.capacity, rotated=True, device=dev)
        cache.compress(lay["k"], lay["v"], lay["ctx_lens"], lay["rot_k"], lay["rot_v"])
        for t in range(63):
            cache.append(*apps[t])
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
        ev[0].record()
        cache.append(*apps[63])
        ev[1].record()
        closed = cache.window_poll()                 # synchronizes
        if len(closed) != cache.num_pairs or any(x[2] != W for x in closed.values()):
            raise RuntimeError(f"expected every window to close at {W} tokens: {closed}")
        ev[2].record()
        rk, rv = cache.window_rotations()
        ev[3].record()
        ev[4].record()
        cache.window_close(rk, rv, kw, vw)
        ev[5].record()
        torch.cuda.synchronize()
        fin.append(1e3 * ev[0].elapsed_time(ev[1]))
        rot.append(1e3 * ev[2].elapsed_time(ev[3]))
        close.append(1e3 * ev[4].elapsed_time(ev[5]))
        del cache
    med = lambda xs: float(sorted(xs)[len(xs) // 2])
    pairs = small.num_seqs * small.hkv
    return {"pairs": pairs, "window_tokens": W, "append_with_finalize_and_close_us": round(med(fin), 1),
            "window_rotations_us": round(med(rot), 1), "window_close_us": round(med(close), 1), "close_tokens_per_s": round(pairs * W / (med(close) * 1e-6)),
            "reps": reps}


def encoding_overlap(cache, lay, dev, compress_ms):
    """Compression of one layer on a second stream while a stand-in of the
    next layer's prefill compute runs on the first (Sec. 5.5 asynchronous
    encoding): bf16 GEMMs sized to take about as long as the compression."""
    import torch
    a = torch.randn(8192, 8192, device=dev, dtype=torch.bfloat16)
    b = torch.randn(8192, 8192, device=dev, dtype=torch.bfloat16)
    c = torch.empty(8192, 8192, device=dev, dtype=torch.bfloat16)

    def compute(n):
        for _ in range(n):
            torch.matmul(a, b, out=c)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    compute(2)
    torch.cuda.synchronize()
    e0.record()
    compute(10)
    e1.record()
    torch.cuda.synchronize()
    per = e0.elapsed_time(e1) / 10
    n = max(1, int(round(compress_ms / per)))

    def run(side):
        torch.cuda.synchronize()
        e0.record()
        if side is None:
            compute(n)
            cache.compress(lay["k"], lay["v"], lay["ctx_lens"], lay["rot_k"], lay["rot_v"])
        else:
            side.wait_event(e0)
            with torch.cuda.stream(side):
                cache.compress(lay["k"], lay["v"], lay["ctx_lens"], lay["rot_k"], lay["rot_v"])
            compute(n)
            done = torch.cuda.Event()
            done.record(side)
            torch.cuda.current_stream().wait_event(done)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1)
    side = torch.cuda.Stream(device=dev)                   # default priority
    serial = min(run(None) for _ in range(2))
    overlapped = min(run(side) for _ in range(2))
    compute_ms = n * per
    return {"compute_ms": round(compute_ms, 2), "compress_ms": round(compress_ms, 2),
            "serial_ms": round(serial, 2), "overlapped_ms": round(overlapped, 2),
            "hidden_fraction": round((serial - overlapped) / compress_ms, 3)}


def arena_one_capacity(M, params, spec, cap):
    """Arena bytes of the same cache with the longest capacity for every
    sequence (host bookkeeping only, nothing allocated)."""
    L = M.load()
    h = C.c_void_p()
    p = params.to_c()
    M._lib.check(L.mosaic_cache_create(C.byref(p), spec.num_seqs, cap, int(spec.rotate), C.byref(h)))
    n = C.c_size_t()
    L.mosaic_cache_arena_bytes(h, C.byref(n))
    L.mosaic_cache_destroy(h)
    return int(n.value)


def cpu_info():
    """(CPU model, cores this process may run on)."""
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:
        cores = os.cpu_count() or 1
    # a shared host grants this process a share of its cores: OMP_NUM_THREADS
    # states it where it is set
    share = os.environ.get("OMP_NUM_THREADS", "")
    if share.isdigit() and int(share) > 0:
        cores = min(cores, int(share))
    return model, cores


def read_bandwidth(buf, reps=5):
    """Attainable streaming-read bandwidth: a read of the whole buffer (larger
    than the MALL) timed with HIP events, best of `reps`, in GB/s."""
    import torch
    sink = torch.zeros((), dtype=torch.int64, device=buf.device)
    v = buf.view(torch.int64)
    best = None
    for _ in range(reps + 1):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        torch.sum(v, dim=0, out=sink)
        b.record()
        b.synchronize()
        ms = a.elapsed_time(b)
        best = ms if best is None else min(best, ms)
    return buf.numel() / (best * 1e-3) / 1e9


def sdpa_dense_us(q, k, v, ctx_len, scale, evict, reps):
    """PyTorch's scaled_dot_product_attention over the same dense K/V (fp16,
    grouped-query heads), same flush protocol; None if it cannot run here."""
    import torch
    import torch.nn.functional as F
    if len(set(ctx_len)) != 1:
        return None                                      # ragged contexts: no single SDPA call
    L = ctx_len[0]
    qd = q[:, :, None, :]                                # [S][Hq][1][D]
    kd, vd = k[:, :, :L], v[:, :, :L]                    # [S][Hkv][L][D] (views)
    try:
        F.scaled_dot_product_attention(qd, kd, vd, scale=scale, enable_gqa=True)
        ts = []
        for i in range(reps + 1):
            evict()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            F.scaled_dot_product_attention(qd, kd, vd, scale=scale, enable_gqa=True)
            b.record()
            b.synchronize()
            if i:
                ts.append(a.elapsed_time(b))
        return 1e3 * sum(ts) / len(ts)
    except (RuntimeError, TypeError) as exc:
        log(f"SDPA not run: {exc}")
        return None


def main():
    args = parse()
    if args.gpus != 1:
        sys.exit("bench.py measures one GPU: this build has no multi-GPU path (run with --gpus 1)")
    import numpy as np
    import torch

    import paper_2607_00760_amd as M
    from workloads import gen

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    if args.calib_copy:
        n = args.calib_copy << 20
        src = torch.ones(n, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calib_copy_bytes": n, "copies": 5}), flush=True)
        return
    spec = gen.spec(args.config)
    if args.ctx:
        spec = gen.spec(args.config, ctx=(args.ctx,) * spec.num_seqs)
    # method parameters beyond the workload's: the quest mode keeps all D
    # channels of every vector in 16-token blocks, unrotated (the sequence-only
    # baseline of the paper's evaluation, run on this library's own kernels)
    extra = {} if args.trunc == D else dict(trunc=args.trunc)
    if args.force_default:
        extra["force_default"] = True
    if args.mode == "quest":
        spec = gen.spec(args.config, ctx=spec.ctx, rotate=False)
        extra = dict(default=(D, 1, 16), force_default=True)
    if args.fp8:
        extra["fp8"] = True
    appends = spec.appends > 0                               # c2, c5: a step appends a token, then decodes
    nlayers = spec.layers if args.layers is None else args.layers
    cap = spec.max_ctx + (args.warmup + args.steps if appends else 0)
    # ragged contexts: a capacity per sequence, so each pair's regions are
    # sized for its own sequence (the rotations still cover the longest)
    n_app = args.warmup + args.steps if appends else 0
    caps = [L + n_app for L in spec.ctx] if len(set(spec.ctx)) > 1 else cap
    params = M.Params(num_kv_heads=spec.hkv, group_size=spec.group, dtype=spec.dtype, rot_window=spec.rot_window,
                      tau_channel=spec.tau_channel, tau_block=spec.tau_block, select=spec.select, **extra)
    flush = torch.empty(args.flush_mb << 20, dtype=torch.uint8, device=dev)
    flush.fill_(1)
    sink = torch.zeros((), dtype=torch.int64, device=dev)

    def evict():
        # read (not write) a buffer larger than the 256 MB MALL, so that the
        # next step finds neither its data nor dirty lines to write back
        torch.sum(flush.view(torch.int64), dim=0, out=sink)

    read_gbps = read_bandwidth(flush)
    log(f"attainable streaming read {read_gbps:.0f} GB/s ({args.flush_mb} MiB)")

    # ---- the caches (one per layer), built from the seeded workload
    log(f"generating {spec.name}: {nlayers} layer(s) x {spec.num_seqs} x {spec.max_ctx} tokens, {spec.hkv} kv heads")
    t0 = time.time()
    caches, queries, lay0, compress_ms, stats = [], [], None, None, None
    for layer in range(nlayers):
        lay = gen.make_layer(spec, layer, device=dev, capacity=cap)
        q = lay["queries"] if lay["queries"] is not None else gen.make_queries(spec, 0, layer, device=dev)
        cache = M.MosaicCache(params, spec.num_seqs, caps, rotated=spec.rotate, device=dev)
        cache.compress(lay["k"], lay["v"], lay["ctx_lens"], lay["rot_k"], lay["rot_v"])
        if layer == 0:
            # the compression pass, timed once after one untimed pass
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            cache.compress(lay["k"], lay["v"], lay["ctx_lens"], lay["rot_k"], lay["rot_v"])
            e1.record()
            torch.cuda.synchronize()
            compress_ms = e0.elapsed_time(e1)
            lay0 = lay                                       # kept: dense baselines, rotations, oracle
        else:
            torch.cuda.synchronize()
            del lay
        caches.append(cache)
        queries.append(q)
        if nlayers > 1:
            log(f"layer {layer + 1}/{nlayers} compressed ({time.time() - t0:.1f}s)")
    torch.cuda.synchronize()
    t_gen = time.time() - t0
    stats = [c.stats() for c in caches]
    ratio = sum(st["dense_bytes"] for st in stats) / sum(st["used_bytes"] for st in stats)
    log(f"data + compression {t_gen:.1f}s, compress (layer 0) {compress_ms:.2f} ms, ratio {ratio:.3f}")
    cache, lay, q = caches[0], lay0, queries[0]

    # the rotation matrices computed on the GPU from the same K/V (covariance
    # and Jacobi eigensolver; the caches above use the host's rotations)
    rotations_ms = None
    reorder = None
    if spec.rotate and not args.no_rotations and nlayers == 1:
        rk_g, rv_g = M.compute_rotations(params, lay["k"], lay["v"], lay["ctx_lens"], cap)
        n = C.c_size_t()
        M.load().mosaic_rotation_workspace_bytes(C.byref(params.to_c()), spec.num_seqs, cap, C.byref(n))
        rws = torch.empty(n.value, dtype=torch.uint8, device=dev)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        M.compute_rotations(params, lay["k"], lay["v"], lay["ctx_lens"], cap, ws=rws)
        e1.record()
        torch.cuda.synchronize()
        rotations_ms = e0.elapsed_time(e1)
        log(f"rotations on the GPU {rotations_ms:.2f} ms")

        def ratio_with(rk_, rv_):
            c2 = M.MosaicCache(params, spec.num_seqs, cap, rotated=True, device=dev)
            c2.compress(lay["k"], lay["v"], lay["ctx_lens"], rk_, rv_)
            r_ = c2.stats()["ratio"]
            del c2
            return r_
        ratio_gpu_rot = ratio_with(rk_g, rv_g)
        M.load().mosaic_reorder_workspace_bytes(C.byref(params.to_c()), spec.num_seqs, cap, C.byref(n))
        ows = torch.empty(n.value, dtype=torch.uint8, device=dev)
        M.reorder_rotations(params, lay["k"], lay["v"], lay["ctx_lens"], cap, rk_g, rv_g, ws=ows)
        torch.cuda.synchronize()
        e0.record()
        M.reorder_rotations(params, lay["k"], lay["v"], lay["ctx_lens"], cap, rk_g, rv_g, ws=ows)   # same work again
        e1.record()
        torch.cuda.synchronize()
        reorder = {"reorder_ms": round(e0.elapsed_time(e1), 3), "ratio_gpu_rotations": round(ratio_gpu_rot, 4),
                   "ratio_gpu_rotations_reordered": round(ratio_with(rk_g, rv_g), 4)}
        del rk_g, rv_g, rws, ows
        log(f"reorder {reorder}")

    update_path = None
    dyn_windows = None
    overlap = None
    if not args.no_extras and nlayers == 1 and not appends:
        update_path = update_path_us(M, gen, spec, params, dev)
        log(f"append {update_path}")
        if spec.rotate:
            dyn_windows = dyn_window_us(M, gen, spec, params, dev)
            log(f"windows closed by their loss {dyn_windows}")
        overlap = encoding_overlap(cache, lay, dev, compress_ms)
        log(f"encoding overlap {overlap}")

    scale = 1.0 / math.sqrt(D)
    outs = [torch.empty((spec.num_seqs, spec.hq, D), dtype=torch.float32, device=dev) for _ in range(nlayers)]
    app = []
    if appends:
        app = [tuple(x.to(dev) for x in gen.make_appends(spec, t)) for t in range(args.warmup + args.steps)]
        qs_app = [gen.make_queries(spec, t + 1, device=dev) for t in range(args.warmup + args.steps)]
    nstep = [0]

    def step(timed_layers=False):
        """One step: the MALL read, then (append,) decode of every layer."""
        evict()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        lev = []
        a.record()
        for li, c in enumerate(caches):
            qq = queries[li]
            if appends:
                c.append(*app[nstep[0]])
                qq = qs_app[nstep[0]]
            c.decode(qq, scale, out=outs[li])
            if timed_layers:
                ev = torch.cuda.Event(enable_timing=True)
                ev.record()
                lev.append(ev)
        b.record()
        nstep[0] += 1
        return a, b, lev

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # the timed steps: plain library calls (per-layer events only between layers)
    step_ms, layer_ms = [], []
    w0 = time.time()
    for _ in range(args.steps):
        a, b, lev = step(timed_layers=nlayers > 1)
        b.synchronize()
        step_ms.append(a.elapsed_time(b))
        if lev:
            prev = a
            per = []
            for ev in lev:
                per.append(prev.elapsed_time(ev))
                prev = ev
            layer_ms.append(per)
    torch.cuda.synchronize()
    wall = time.time() - w0
    ms = float(np.mean(step_ms))
    log(f"{'append + ' if appends else ''}decode {1e3 * ms:.1f} us/step over {args.steps} steps"
        + (f" ({nlayers} layers)" if nlayers > 1 else ""))
    ref_out = outs[0].clone()
    # per-kernel durations: more steps with events on the launch stream (the
    # append configs' caches have room for warmup + steps appends only, so
    # their kernel timings re-run the decode of the last step)
    for c in caches:
        c.set_timing(True)
    kern = {k: [] for k in M.MosaicCache.KERNELS}
    for _ in range(args.steps):
        evict()
        for li, c in enumerate(caches):
            c.decode(qs_app[nstep[0] - 1] if appends else queries[li], scale, out=outs[li])
            for k_, v_ in c.decode_timing().items():
                kern[k_].append(v_)
    torch.cuda.synchronize()
    for c in caches:
        c.set_timing(False)
    kern_us = {k: 1e3 * float(np.mean(v)) for k, v in kern.items()}        # per launch (per layer)

    graph_us = None
    if not args.no_graph and nlayers == 1 and not appends:
        def graph_replay():
            """Capture one call into a HIP graph and time its replays; every
            replay must reproduce the eager output bit for bit."""
            out = outs[0]
            gs = torch.cuda.Stream()
            gs.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(gs):
                cache.decode(q, scale, out=out)
            torch.cuda.current_stream().wait_stream(gs)
            torch.cuda.synchronize()
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                cache.decode(q, scale, out=out)
            torch.cuda.synchronize()
            gms, same = [], True
            for i in range(args.steps + 1):
                evict()
                out.zero_()
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record()
                graph.replay()
                b.record()
                b.synchronize()
                same &= bool(torch.equal(out, ref_out))
                if i:
                    gms.append(a.elapsed_time(b))
            del graph
            if not same:
                log("graph replay output differs from the eager call; not reported")
                return None
            return 1e3 * float(np.mean(gms))
        try:
            graph_us = graph_replay()
            if graph_us is not None:
                log(f"graph replay {graph_us:.1f} us/step")
        except RuntimeError as exc:          # capture not supported here: no graph figure
            log(f"graph capture failed: {exc}")
            torch.cuda.synchronize()
        outs[0].copy_(ref_out)

    # algorithmic bytes from every cache's own descriptors and selections
    ab_tot, sel_tot = None, dict(selected_tokens=0, scoreable_tokens=0)
    for c in caches:
        nb_list, sel_list, desc_list = [], [], []
        for p in range(c.num_pairs):
            L = c.seq_tokens(p // spec.hkv)
            nd = L // 64 + (1 if L % 64 >= 32 else 0)
            raw = c.region("desc", p, 16 * nd).cpu().numpy()
            dd = []
            for j in range(nd):
                r = raw[16 * j:16 * j + 16]
                u = r[:12].view(np.uint32)
                dd.append((int(u[0]), int(u[1]), int(u[2]), int(r[12]), int(r[13]), int(r[14]), int(r[15])))
            desc_list.append(dd)
            nw = c.layout.num_windows
            wsel = c.ws_region("wsel", p, 4 * (nw + 2)).cpu().numpy().view(np.int32)
            k = int(wsel[nw])
            sel_list.append(c.ws_region("sel", p, 4 * max(k, 1)).cpu().numpy().view(np.int32)[:k].tolist())
            nb_list.append(int(wsel[nw + 1]))
        spec_now = gen.spec(spec.name, ctx=tuple(c.seq_tokens(b) for b in range(spec.num_seqs)),
                            num_seqs=spec.num_seqs) if appends else spec
        ab, selected = algorithmic_bytes(c, spec_now, nb_list, sel_list, desc_list)
        ab_tot = ab if ab_tot is None else {k: ab_tot[k] + ab[k] for k in ab}
        sel_tot = {k: sel_tot[k] + selected[k] for k in ("selected_tokens", "scoreable_tokens")}
    sel_tot["fraction"] = round(sel_tot["selected_tokens"] / max(sel_tot["scoreable_tokens"], 1), 5)
    dom = max(("score", "attn"), key=lambda k: kern_us[k])
    per_launch = ab_tot[dom] / nlayers
    achieved = per_launch / (kern_us[dom] * 1e-6) / 1e9
    traffic = None
    tf = os.path.join(ROOT, "profiles", f"traffic_{args.config}.json")
    if os.path.exists(tf) and not args.ctx and args.mode == "mosaic" and args.trunc == D and not args.force_default \
            and not args.fp8:
        t = json.load(open(tf))
        if t.get("source_hash") == source_hash() and t.get("kernel") == dom:
            traffic = t.get("bytes_per_launch")

    # dense attention of the same shape (one layer, fp16): this library's
    # split-K kernel and PyTorch SDPA, same flush protocol
    dense_us = sdpa_us = None
    if not args.no_dense:
        kd = lay["k"].to(torch.float16)
        vd = lay["v"].to(torch.float16)
        qd = q.to(torch.float16)
        ctx_l = list(lay["ctx_lens"])
        ctx = torch.tensor(ctx_l, dtype=torch.int32, device=dev)
        dout = M.dense_decode(qd, kd, vd, ctx, scale, spec.max_ctx, spec.group)
        n = C.c_size_t()
        M.load().mosaic_dense_workspace_bytes(spec.num_seqs, spec.hkv, spec.group, spec.max_ctx, C.byref(n))
        ws = torch.empty(n.value, dtype=torch.uint8, device=dev)
        dts = []
        for i in range(args.dense_steps + 1):
            evict()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            M.dense_decode(qd, kd, vd, ctx, scale, spec.max_ctx, spec.group, out=dout, ws=ws)
            b.record()
            torch.cuda.synchronize()
            if i:
                dts.append(a.elapsed_time(b))
        dense_us = 1e3 * float(np.mean(dts)) * nlayers
        sdpa_us = sdpa_dense_us(qd, kd, vd, ctx_l, scale, evict, args.dense_steps)
        if sdpa_us is not None:
            sdpa_us *= nlayers
        log(f"dense fp16: own kernel {dense_us:.1f} us/step, SDPA {sdpa_us} us/step"
            + (f" (one layer timed, x{nlayers})" if nlayers > 1 else ""))
        del kd, vd
    dense_bytes = nlayers * sum(2 * L * spec.hkv * D * 2 for L in lay["ctx_lens"])    # fp16 K and V read once
    dense_roofline_us = dense_bytes / (HBM_PEAK_GBPS * 1e9) * 1e6

    # CPU oracle on a bounded sample: one (sequence, kv head) pair per host
    # thread, compressed, then decoded; the decode is scaled to the whole step
    cpu = None
    parity = None
    if not args.no_cpu_baseline:
        from oracle import oracle as O
        model, cores = cpu_info()
        npairs = cache.num_pairs
        ns = min(npairs, cores, args.cpu_sample_pairs) if args.cpu_sample_pairs else min(npairs, cores)
        pairs_s = sorted(int(x) for x in np.random.default_rng(1).choice(npairs, size=ns, replace=False))
        op = O.Params(group=spec.group, dtype=spec.dtype, rot_window=spec.rot_window, tau_channel=spec.tau_channel,
                      tau_block=spec.tau_block, select=spec.select, **extra)
        qb = gen.bits(qs_app[nstep[0] - 1] if appends else q)
        # one layer; c4's 1M-token pairs are sampled on a prefix of 1/8 of their tokens
        frac = 8 if spec.max_ctx > (1 << 19) else 1
        kb_, vb_ = lay["k"], lay["v"]

        def comp(p):
            b, h = divmod(p, spec.hkv)
            L = lay["ctx_lens"][b] // frac
            pr = O.Pair(op, cap, lay["rot_k"][b, h].cpu().numpy() if spec.rotate else None,
                        lay["rot_v"][b, h].cpu().numpy() if spec.rotate else None)
            t = time.time()
            pr.compress(gen.bits(kb_[b, h, :L]), gen.bits(vb_[b, h, :L]))
            if appends:
                for t_ in range(nstep[0]):
                    pr.append(gen.bits(app[t_][0])[b, h], gen.bits(app[t_][1])[b, h])
            return pr, time.time() - t

        log(f"oracle: compressing {ns} pairs on {ns} threads ({cores} cores: {model})")
        with cf.ThreadPoolExecutor(ns) as ex:
            res = list(ex.map(comp, pairs_s))
        opairs = [r[0] for r in res]

        def dec(i):
            p = pairs_s[i]
            b, h = divmod(p, spec.hkv)
            t = time.time()
            o = opairs[i].decode(qb[b, h * spec.group:(h + 1) * spec.group], scale)
            return o, time.time() - t

        t = time.time()
        with cf.ThreadPoolExecutor(ns) as ex:
            outs_o = list(ex.map(dec, range(ns)))
        t_dec = time.time() - t
        per_pair = float(np.mean([r[1] for r in outs_o]))
        rounds = -(-npairs // cores) * nlayers * frac      # rounds of `cores` pairs a whole step needs
        cpu = dict(value=round(per_pair * rounds * 1e6, 1), unit="us/step", cores=ns, kind="oracle",
                   host_cores=cores, cpu_model=model, single_thread_us_per_pair=round(per_pair * 1e6, 1),
                   sample=(f"oracle decode of {ns} of {npairs} (sequence, kv head) pairs, one per thread on {ns} "
                           f"threads ({t_dec:.2f} s wall); a step of {npairs} pairs x {nlayers} layer(s) is "
                           f"{rounds} rounds of {min(npairs, cores)} pairs at the mean per-pair time"
                           + (f"; pairs compressed on the first 1/{frac} of their tokens, x{frac}" if frac > 1 else "")
                           + f"; oracle compress of the sample took {sum(r[1] for r in res):.1f} thread-s"))
        if frac == 1:
            got = outs[0].cpu().numpy() if not appends else outs[0].cpu().numpy()
            err, rel, sel_ok = 0.0, 0.0, True
            for i, p in enumerate(pairs_s):
                b, h = divmod(p, spec.hkv)
                o, s_o = outs_o[i][0]
                g_ = got[b, h * spec.group:(h + 1) * spec.group]
                err = max(err, float(np.abs(g_ - o).max()))
                rel = max(rel, float(np.linalg.norm(g_ - o) / max(np.linalg.norm(o), 1e-30)))
                nwl = cache.layout.num_windows
                wsel = cache.ws_region("wsel", p, 4 * (nwl + 2)).cpu().numpy().view(np.int32)
                kk = int(wsel[nwl])
                gsel = cache.ws_region("sel", p, 4 * max(kk, 1)).cpu().numpy().view(np.int32)[:kk].tolist()
                sel_ok &= list(s_o) == gsel
            parity = dict(pairs=ns, max_abs=err, rel_l2=rel, selected_blocks_identical=bool(sel_ok))

    value = ms * 1e3
    cfg_desc = {
        "c1": "decode attention over a compressed KV cache, batch 1 x 4096 tokens",
        "c2": "one appended token per sequence + decode attention over a compressed KV cache, batch 4 x 32768 tokens",
        "c3": "decode attention over a compressed KV cache, batch 8 x 131072 tokens",
        "c4": f"decode attention across {nlayers} layers of a compressed 1 x 1048576-token KV cache",
        "c5": "one appended token per sequence + decode attention over a compressed KV cache, batch 16 ragged "
              "16K..96K tokens",
    }[spec.name]
    res = {
        "metric": METRIC, "value": round(value, 3), "unit": "us/step", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 5), "higher_is_better": False, "scaling": "weak",
        "vs_baseline": None, "dtype": spec.dtype, "data": "synthetic",
        "config": {"workload": f"{spec.name}: {cfg_desc}, {spec.hq} q / {spec.hkv} kv heads, d=128, {spec.dtype}, "
                               f"select 1/10 of tokens"
                               + (", planted 5% of segments" if spec.kind == "planted" else "")
                               + ("; quest mode: all channels kept, 16-token blocks, no rotation"
                                  if args.mode == "quest" else "")
                               + (f"; bitmaps of the first {args.trunc} channels" if args.trunc != D else "")
                               + ("; default strategy forced" if args.force_default else "")
                               + ("; E4M3 token values" if args.fp8 else ""),
                   "mode": args.mode,
                   "num_seqs": spec.num_seqs, "ctx": spec.max_ctx, "q_heads": spec.hq, "kv_heads": spec.hkv,
                   "head_dim": D, "layers": nlayers, "select": f"{spec.select[0]}/{spec.select[1]}",
                   "mall_flush_mb": args.flush_mb},
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": traffic,
                     "algorithmic_bytes_per_launch": int(per_launch), "mean_launch_us": round(kern_us[dom], 3),
                     "attainable_read_gbps": round(read_gbps, 1),
                     "frac_of_attainable": round(achieved / read_gbps, 4)},
        "effective_gbps": round(ab_tot["total"] / (ms * 1e-3) / 1e9, 1),
        "algorithmic_bytes_per_step": ab_tot,
        "selected": sel_tot,
        "kernels_us": {k: round(v, 3) for k, v in kern_us.items()},
        "layer_us": ([round(1e3 * float(x), 2) for x in np.mean(np.array(layer_ms), axis=0)] if layer_ms else None),
        "graph_replay_us_per_step": None if graph_us is None else round(graph_us, 3),
        "dense_us_per_step": None if dense_us is None else round(dense_us, 2),
        "sdpa_us_per_step": None if sdpa_us is None else round(sdpa_us, 2),
        "speedup_vs_dense": None if dense_us is None else round(dense_us / value, 2),
        "speedup_vs_sdpa": None if sdpa_us is None else round(sdpa_us / value, 2),
        "dense_bytes_per_step": dense_bytes,
        "speedup_vs_dense_roofline": round(dense_roofline_us / value, 2),
        "wall_ms_per_step_incl_flush": round(1e3 * wall / args.steps, 3),
        "compress_ms": round(compress_ms, 3), "memory_ratio": round(ratio, 4),
        "arena_bytes": int(caches[0].arena.numel()), "arena_bytes_one_capacity": arena_one_capacity(M, params, spec, cap),
        "rotations_ms": None if rotations_ms is None else round(rotations_ms, 3),
        "channel_reorder": reorder,
        "update_path": update_path, "dyn_windows": dyn_windows, "encoding_overlap": overlap,
        "strategies": {f"{k[0]}/{k[1]}/{k[2]}": v for k, v in sorted(stats[0]["strategies"].items())},
        "cpu_baseline": cpu, "parity": parity, "datagen_s": round(t_gen, 1), "source_hash": source_hash(),
    }
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
