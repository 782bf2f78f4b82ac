#!/usr/bin/env python3
"""Benchmark of the MosaicKV decode step on one MI355X.

Workload (the metric's configuration): decode attention over a compressed
KV cache, batch 8 x 131072-token contexts, 32 query / 8 kv heads, head dim
128, bf16, ~3x compression, 5 % of segments planted to carry 80 % of the
softmax mass.  A step is one mosaic_decode_attention call (q rotation, block
scoring, top-k, split-K packed attention, reduce with back-rotation) over the
resident cache.  A >= 1 GiB buffer is overwritten before every step so that
the 256 MB MALL holds none of the step's data; only the decode itself sits
between the step's events.

Prints ONE JSON line: value = microseconds per decode step (lower is better),
plus the roofline of the dominant kernel, the dense fp16 baseline of the same
shape, the compression pass and the CPU oracle on a bounded sample.
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
    ap.add_argument("--cpu-sample-pairs", type=int, default=4)
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
    cap = spec.max_ctx
    log(f"generating {spec.name}: {spec.num_seqs} x {spec.max_ctx} tokens, {spec.hkv} kv heads")
    t0 = time.time()
    lay = gen.make_layer(spec, 0, device=dev, capacity=cap)
    torch.cuda.synchronize()
    t_gen = time.time() - t0
    q = lay["queries"] if lay["queries"] is not None else gen.make_queries(spec, 0, device=dev)
    params = M.Params(num_kv_heads=spec.hkv, group_size=spec.group, dtype=spec.dtype, rot_window=spec.rot_window,
                      tau_channel=spec.tau_channel, tau_block=spec.tau_block, select=spec.select, **extra)
    cache = M.MosaicCache(params, spec.num_seqs, cap, rotated=spec.rotate, device=dev)
    # compression pass (timed once, after one untimed pass)
    cache.compress(lay["k"], lay["v"], lay["ctx_lens"], lay["rot_k"], lay["rot_v"])
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    cache.compress(lay["k"], lay["v"], lay["ctx_lens"], lay["rot_k"], lay["rot_v"])
    e1.record()
    torch.cuda.synchronize()
    compress_ms = e0.elapsed_time(e1)
    stats = cache.stats()
    log(f"data {t_gen:.1f}s, compress {compress_ms:.2f} ms, ratio {stats['ratio']:.3f}")
    # the rotation matrices computed on the GPU from the same K/V (covariance
    # and Jacobi eigensolver; the cache above used the host's rotations)
    rotations_ms = None
    reorder = None
    if spec.rotate and not args.no_rotations:
        rws = torch.empty(0, dtype=torch.uint8, device=dev)
        rk_g, rv_g = M.compute_rotations(params, lay["k"], lay["v"], lay["ctx_lens"], cap)
        n = C.c_size_t()
        M.load().mosaic_rotation_workspace_bytes(C.byref(params.to_c()), spec.num_seqs, cap, C.byref(n))
        rws = torch.empty(n.value, dtype=torch.uint8, device=dev)
        torch.cuda.synchronize()
        e0.record()
        M.compute_rotations(params, lay["k"], lay["v"], lay["ctx_lens"], cap, ws=rws)
        e1.record()
        torch.cuda.synchronize()
        rotations_ms = e0.elapsed_time(e1)
        log(f"rotations on the GPU {rotations_ms:.2f} ms")
        # the selection-pattern reorder of those matrices, and the memory ratio of
        # the cache compressed with them before and after it
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
    overlap = None
    if not args.no_extras:
        update_path = update_path_us(M, gen, spec, params, dev)
        log(f"append {update_path}")
        overlap = encoding_overlap(cache, lay, dev, compress_ms)
        log(f"encoding overlap {overlap}")

    flush = torch.empty(args.flush_mb << 20, dtype=torch.uint8, device=dev)
    out = torch.empty((spec.num_seqs, spec.hq, D), dtype=torch.float32, device=dev)
    scale = 1.0 / math.sqrt(D)
    cache.set_timing(True)

    flush.fill_(1)
    sink = torch.zeros((), dtype=torch.int64, device=dev)

    def evict():
        # read (not write) a buffer larger than the 256 MB MALL, so that the
        # next step finds neither its data nor dirty lines to write back
        torch.sum(flush.view(torch.int64), dim=0, out=sink)

    def step():
        evict()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        cache.decode(q, scale, out=out)
        b.record()
        return a, b

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # the timed steps: plain library calls, no per-kernel events between them
    cache.set_timing(False)
    step_ms = []
    torch.cuda.synchronize()
    w0 = time.time()
    for _ in range(args.steps):
        a, b = step()
        b.synchronize()
        step_ms.append(a.elapsed_time(b))
    torch.cuda.synchronize()
    wall = time.time() - w0
    ms = float(np.mean(step_ms))
    log(f"decode {1e3 * ms:.1f} us/step over {args.steps} steps")
    ref_out = out.clone()
    # per-kernel durations: the same steps again with events on the launch stream
    cache.set_timing(True)
    kern = {k: [] for k in M.MosaicCache.KERNELS}
    for _ in range(args.steps):
        a, b = step()
        kt = cache.decode_timing()           # waits for this step's kernels
        for k, v in kt.items():
            kern[k].append(v)
    torch.cuda.synchronize()
    cache.set_timing(False)
    kern_us = {k: 1e3 * float(np.mean(v)) for k, v in kern.items()}
    # the same call captured once into a HIP graph and replayed (every replay is
    # checked against the eager output)
    def graph_replay():
        """Capture one call into a HIP graph and time its replays; every
        replay must reproduce the eager output bit for bit."""
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

    graph_us = None
    if not args.no_graph:
        try:
            graph_us = graph_replay()
            if graph_us is not None:
                log(f"graph replay {graph_us:.1f} us/step")
        except RuntimeError as exc:          # capture not supported here: no graph figure
            log(f"graph capture failed: {exc}")
            torch.cuda.synchronize()
        out.copy_(ref_out)

    # algorithmic bytes from the cache's own descriptors and selections
    lay_c, wsl = cache.layout, cache.ws_layout
    nb_list, sel_list, desc_list = [], [], []
    for p in range(cache.num_pairs):
        L = spec.ctx[p // spec.hkv]
        nd = L // 64 + (1 if L % 64 >= 32 else 0)
        raw = cache.region("desc", p, 16 * nd).cpu().numpy()
        dd = []
        for j in range(nd):
            r = raw[16 * j:16 * j + 16]
            u = r[:12].view(np.uint32)
            dd.append((int(u[0]), int(u[1]), int(u[2]), int(r[12]), int(r[13]), int(r[14]), int(r[15])))
        desc_list.append(dd)
        nw = lay_c.num_windows
        wsel = cache.ws_region("wsel", p, 4 * (nw + 2)).cpu().numpy().view(np.int32)
        k = int(wsel[nw])
        sel_list.append(cache.ws_region("sel", p, 4 * max(k, 1)).cpu().numpy().view(np.int32)[:k].tolist())
        nb_list.append(int(wsel[nw + 1]))
    ab, selected = algorithmic_bytes(cache, spec, nb_list, sel_list, desc_list)
    dom = max(("score", "attn"), key=lambda k: kern_us[k])
    achieved = ab[dom] / (kern_us[dom] * 1e-6) / 1e9
    traffic = None
    tf = os.path.join(ROOT, "profiles", f"traffic_{args.config}.json")
    if os.path.exists(tf) and not args.ctx and args.mode == "mosaic" and args.trunc == D and not args.force_default \
            and not args.fp8:
        t = json.load(open(tf))
        if t.get("source_hash") == source_hash() and t.get("kernel") == dom:
            traffic = t.get("bytes_per_launch")

    # dense fp16 attention of the same shape (own split-K kernel), same flush protocol
    dense_us = None
    if not args.no_dense:
        kd = lay["k"].to(torch.float16)
        vd = lay["v"].to(torch.float16)
        qd = q.to(torch.float16)
        ctx = torch.tensor(lay["ctx_lens"], dtype=torch.int32, device=dev)
        dout = M.dense_decode(qd, kd, vd, ctx, scale, spec.max_ctx, spec.group)
        ws = torch.empty(1 << 20, dtype=torch.uint8, device=dev)
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
        dense_us = 1e3 * float(np.mean(dts))
        log(f"dense fp16 {dense_us:.1f} us/step")
        del kd, vd

    # CPU oracle on a bounded sample (decode of a few pairs, scaled to the workload)
    cpu = None
    parity = None
    if not args.no_cpu_baseline:
        from oracle import oracle as O
        ns = min(args.cpu_sample_pairs, cache.num_pairs)
        op = O.Params(group=spec.group, dtype=spec.dtype, rot_window=spec.rot_window, tau_channel=spec.tau_channel,
                      tau_block=spec.tau_block, select=spec.select, **extra)
        qb = gen.bits(q)

        def comp(p):
            b, h = divmod(p, spec.hkv)
            L = spec.ctx[b]
            pr = O.Pair(op, cap, lay["rot_k"][b, h].cpu().numpy() if spec.rotate else None,
                        lay["rot_v"][b, h].cpu().numpy() if spec.rotate else None)
            t = time.time()
            pr.compress(gen.bits(lay["k"][b, h, :L]), gen.bits(lay["v"][b, h, :L]))
            return pr, time.time() - t

        threads = min(ns, os.cpu_count() or 1, 16)
        log(f"oracle: compressing {ns} pairs on {threads} threads")
        with cf.ThreadPoolExecutor(threads) as ex:
            res = list(ex.map(comp, range(ns)))
        pairs = [r[0] for r in res]

        def dec(p):
            b, h = divmod(p, spec.hkv)
            return pairs[p].decode(qb[b, h * spec.group:(h + 1) * spec.group], scale)

        t = time.time()
        with cf.ThreadPoolExecutor(threads) as ex:
            outs = list(ex.map(dec, range(ns)))
        t_dec = time.time() - t
        cpu = dict(value=t_dec * (cache.num_pairs / ns) * 1e6, unit="us/step", cores=threads, kind="oracle",
                   sample=f"oracle decode of {ns} of {cache.num_pairs} (sequence, kv head) pairs on {threads} "
                          f"threads, scaled x{cache.num_pairs / ns:g}; oracle compress of those pairs took "
                          f"{sum(r[1] for r in res):.1f} thread-s")
        got = out.cpu().numpy()
        err, rel, sel_ok = 0.0, 0.0, True
        for p in range(ns):
            b, h = divmod(p, spec.hkv)
            o, s_o = outs[p]
            g_ = got[b, h * spec.group:(h + 1) * spec.group]
            err = max(err, float(np.abs(g_ - o).max()))
            rel = max(rel, float(np.linalg.norm(g_ - o) / max(np.linalg.norm(o), 1e-30)))
            sel_ok &= list(s_o) == sel_list[p]
        parity = dict(pairs=ns, max_abs=err, rel_l2=rel, selected_blocks_identical=bool(sel_ok))

    value = ms * 1e3
    res = {
        "metric": METRIC, "value": round(value, 3), "unit": "us/step", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 5), "higher_is_better": False, "scaling": "weak",
        "vs_baseline": None, "dtype": spec.dtype, "data": "synthetic",
        "config": {"workload": f"{spec.name}: decode attention over a compressed KV cache, batch {spec.num_seqs} x "
                               f"{spec.max_ctx} tokens, {spec.hq} q / {spec.hkv} kv heads, d=128, {spec.dtype}, "
                               f"select 1/10 of tokens, planted 5% of segments"
                               + ("; quest mode: all channels kept, 16-token blocks, no rotation"
                                  if args.mode == "quest" else "")
                               + (f"; bitmaps of the first {args.trunc} channels" if args.trunc != D else "")
                               + ("; default strategy forced" if args.force_default else "")
                               + ("; E4M3 token values" if args.fp8 else ""),
                   "mode": args.mode,
                   "num_seqs": spec.num_seqs, "ctx": spec.max_ctx, "q_heads": spec.hq, "kv_heads": spec.hkv,
                   "head_dim": D, "select": f"{spec.select[0]}/{spec.select[1]}", "mall_flush_mb": args.flush_mb},
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": traffic,
                     "algorithmic_bytes_per_launch": ab[dom], "mean_launch_us": round(kern_us[dom], 3)},
        "effective_gbps": round(ab["total"] / (ms * 1e-3) / 1e9, 1),
        "algorithmic_bytes_per_step": ab,
        "selected": selected,
        "kernels_us": {k: round(v, 3) for k, v in kern_us.items()},
        "graph_replay_us_per_step": None if graph_us is None else round(graph_us, 3),
        "dense_us_per_step": None if dense_us is None else round(dense_us, 2),
        "speedup_vs_dense": None if dense_us is None else round(dense_us / value, 2),
        "wall_ms_per_step_incl_flush": round(1e3 * wall / args.steps, 3),
        "compress_ms": round(compress_ms, 3), "memory_ratio": round(stats["ratio"], 4),
        "rotations_ms": None if rotations_ms is None else round(rotations_ms, 3),
        "channel_reorder": reorder,
        "update_path": update_path, "encoding_overlap": overlap,
        "strategies": {f"{k[0]}/{k[1]}/{k[2]}": v for k, v in sorted(stats["strategies"].items())},
        "cpu_baseline": cpu, "parity": parity, "datagen_s": round(t_gen, 1), "source_hash": source_hash(),
    }
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
