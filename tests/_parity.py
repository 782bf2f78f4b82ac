"""Helpers of the GPU parity tests: run the oracle and the HIP library on the
same seeded inputs and compare what they produce."""
from __future__ import annotations

import concurrent.futures as cf
import math
import os

import numpy as np
import torch

import paper_2607_00760_amd as M
from oracle import oracle as O
from workloads import gen

D = 128
THREADS = min(16, os.cpu_count() or 1)
TOL_ABS, TOL_REL = 2e-3, 1e-3


def params_pair(spec: gen.WorkloadSpec, **kw):
    """The same method parameters for the library and for the oracle."""
    common = dict(rot_window=spec.rot_window, tau_channel=spec.tau_channel, tau_block=spec.tau_block,
                  select=spec.select)
    common.update(kw)
    lp = M.Params(num_kv_heads=spec.hkv, group_size=spec.group, dtype=spec.dtype, **common)
    op = O.Params(group=spec.group, dtype=spec.dtype, **common)
    return lp, op


def bits(t):
    return gen.bits(t)


def oracle_pairs(op: O.Params, spec, lay, cap):
    """Compress every (sequence, kv head) on the oracle, in parallel."""
    def one(pi):
        b, h = divmod(pi, spec.hkv)
        L = lay["ctx_lens"][b]
        rk = lay["rot_k"][b, h].cpu().numpy() if lay["rot_k"] is not None else None
        rv = lay["rot_v"][b, h].cpu().numpy() if lay["rot_v"] is not None else None
        pr = O.Pair(op, cap, rk, rv)
        pr.compress(bits(lay["k"][b, h, :L]), bits(lay["v"][b, h, :L]))
        return pr
    with cf.ThreadPoolExecutor(THREADS) as ex:
        return list(ex.map(one, range(spec.num_seqs * spec.hkv)))


def gpu_cache(lp: M.Params, spec, lay, cap, dev="cuda"):
    c = M.MosaicCache(lp, spec.num_seqs, cap, rotated=lay["rot_k"] is not None, device=dev)
    k, v = lay["k"].to(dev).contiguous(), lay["v"].to(dev).contiguous()
    rk = lay["rot_k"].to(dev).contiguous() if lay["rot_k"] is not None else None
    rv = lay["rot_v"].to(dev).contiguous() if lay["rot_v"] is not None else None
    c.compress(k, v, lay["ctx_lens"], rk, rv)
    torch.cuda.synchronize()
    return c


def gpu_state(c: M.MosaicCache, pair: int, opair: O.Pair):
    """The GPU's used bytes of every region of `pair`, sized by the oracle's counts."""
    info = opair.info()
    meta = c.region("meta", pair, 16).cpu().numpy().view(np.int32)
    st = dict(L=int(meta[0]), nblk_final=int(meta[1]), tok_tail=int(meta[2]), sc_tail=int(meta[3]))
    nd = info.n_desc
    st["desc"] = c.region("desc", pair, 16 * nd).cpu().numpy()
    tok_n = opair.token_arena().size
    sc_n = opair.score_arena().size
    st["tok"] = c.region("token", pair, tok_n).cpu().numpy()
    st["sc"] = c.region("score", pair, sc_n).cpu().numpy()
    buf = c.region("buf", pair, 2 * 32 * D * 2).cpu().numpy().view(np.uint16).reshape(2, 32, D)
    stg = c.region("stage", pair, 2 * 64 * D * 2).cpu().numpy().view(np.uint16).reshape(2, 64, D)
    st["bufk"], st["bufv"] = buf[0, :info.n_buf], buf[1, :info.n_buf]
    m = info.L % 64
    st["stgk"], st["stgv"] = stg[0, :m], stg[1, :m]
    return st


def assert_state_equal(c, pair, opair, where=""):
    g = gpu_state(c, pair, opair)
    i = opair.info()
    assert (g["L"], g["nblk_final"], g["tok_tail"], g["sc_tail"]) == (i.L, i.nblk_final, i.tok_tail, i.sc_tail), \
        f"{where} pair {pair}: meta {g} vs oracle {(i.L, i.nblk_final, i.tok_tail, i.sc_tail)}"
    od = opair.descriptor_bytes()
    assert np.array_equal(g["desc"], od), f"{where} pair {pair}: descriptors differ\n{g['desc'].reshape(-1, 16)[:4]}\n" \
                                          f"{od.reshape(-1, 16)[:4]}"
    ot, osc = opair.token_arena(), opair.score_arena()
    if not np.array_equal(g["sc"], osc):
        bad = np.nonzero(g["sc"] != osc)[0]
        raise AssertionError(f"{where} pair {pair}: score arena differs at {bad.size} bytes, first {bad[:8]}")
    if not np.array_equal(g["tok"], ot):
        bad = np.nonzero(g["tok"] != ot)[0]
        raise AssertionError(f"{where} pair {pair}: token arena differs at {bad.size} bytes, first {bad[:8]}")
    bk, bv = opair.buffer()
    sk, sv = opair.staging()
    assert np.array_equal(g["bufk"], bk) and np.array_equal(g["bufv"], bv), f"{where} pair {pair}: update buffer"
    assert np.array_equal(g["stgk"], sk) and np.array_equal(g["stgv"], sv), f"{where} pair {pair}: staging"


def oracle_decode_all(opairs, spec, q, scale):
    """-> (out [S][Hq][D] fp64, list of selected arrays, list of score arrays)."""
    G = spec.group
    qb = bits(q)
    def one(pi):
        b, h = divmod(pi, spec.hkv)
        qq = qb[b, h * G:(h + 1) * G]
        out, sel = opairs[pi].decode(qq, scale)
        return out, sel, opairs[pi].scores(qq)
    with cf.ThreadPoolExecutor(THREADS) as ex:
        res = list(ex.map(one, range(len(opairs))))
    out = np.zeros((spec.num_seqs, spec.hq, D))
    for pi, (o, _, _) in enumerate(res):
        b, h = divmod(pi, spec.hkv)
        out[b, h * G:(h + 1) * G] = o
    return out, [r[1] for r in res], [r[2] for r in res]


def gpu_scores_sel(c: M.MosaicCache, pair: int, nb: int):
    sc = c.ws_region("score", pair, 4 * nb).cpu().numpy().view(np.float32).copy()
    nw = c.layout.num_windows
    wsel = c.ws_region("wsel", pair, 4 * (nw + 2)).cpu().numpy().view(np.int32)
    k = int(wsel[nw])
    sel = c.ws_region("sel", pair, 4 * max(k, 1)).cpu().numpy().view(np.int32)[:k].copy()
    return sc, sel, wsel


def assert_close(got, want, where=""):
    """max-abs within TOL_ABS and rel-L2 within TOL_REL (the fp32 outputs
    against the oracle's fp64 ones) -> (max-abs, rel-L2)."""
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    err = np.abs(got - want)
    if err.size == 0:
        return 0.0, 0.0
    rel = np.linalg.norm(got - want) / max(np.linalg.norm(want), 1e-30)
    assert err.max() <= TOL_ABS and rel <= TOL_REL, \
        f"{where}: max-abs {err.max():.3e} rel-L2 {rel:.3e}"
    return err.max(), rel


def scale_of():
    return 1.0 / math.sqrt(D)
