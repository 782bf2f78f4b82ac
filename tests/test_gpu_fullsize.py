"""GPU parity at the workloads' full sizes, in the launch configuration the
benchmark times (one library call per step over every sequence and kv head).

The GPU runs the whole workload; the oracle recomputes a seeded sample of
(sequence, kv head) pairs one by one and must agree with it exactly on the
packed bytes, descriptors, block scores and selections of those pairs, and
within 2e-3 max-abs / 1e-3 rel-L2 on their outputs.  The 1M-token, 32-layer
case is too large for the oracle to compress whole in a test.  Every layer is
built on the GPU and a seeded 1 % of its (pair, segment) positions is checked
byte for byte against the oracle's compression of that one segment (with its
window's rotation), together with one kv head's selection per layer (the
token budget of the GPU's own scores).  One layer is further checked on a
prefix of the cache byte for byte, the scores of that prefix, and the
attention output against an independent fp64 evaluation over the GPU's
selection (packed records decoded here, rotation merged back by R_v).
"""
import concurrent.futures as cf
import math

import numpy as np
import pytest
import torch

from _parity import (D, assert_close, assert_state_equal, bits, gpu_cache, gpu_scores_sel, params_pair,
                     scale_of)
from oracle import oracle as O
from workloads import gen

pytestmark = pytest.mark.gpu


def _sample(n_pairs, k, seed):
    rng = np.random.default_rng(seed)
    return sorted(int(x) for x in rng.choice(n_pairs, size=min(k, n_pairs), replace=False))


def _spread(spec, per_seq, seed):
    """per_seq seeded kv heads of every sequence (all pairs when per_seq >= hkv)."""
    rng = np.random.default_rng(seed)
    out = []
    for b in range(spec.num_seqs):
        hs = rng.choice(spec.hkv, size=min(per_seq, spec.hkv), replace=False)
        out += [b * spec.hkv + int(h) for h in hs]
    return sorted(out)


def _oracle_pair(op, spec, lay, cap, pi, L=None):
    b, h = divmod(pi, spec.hkv)
    L = lay["ctx_lens"][b] if L is None else L
    rk = lay["rot_k"][b, h].cpu().numpy() if lay["rot_k"] is not None else None
    rv = lay["rot_v"][b, h].cpu().numpy() if lay["rot_v"] is not None else None
    pr = O.Pair(op, cap, rk, rv)
    pr.compress(bits(lay["k"][b, h, :L]), bits(lay["v"][b, h, :L]))
    return pr


def _oracle_pairs(op, spec, lay, cap, pairs):
    with cf.ThreadPoolExecutor(min(len(pairs), 16)) as ex:
        return dict(zip(pairs, ex.map(lambda pi: _oracle_pair(op, spec, lay, cap, pi), pairs)))


def _check_decode(c, spec, ops, q, out, where):
    G, sc = spec.group, scale_of()
    qb = bits(q)
    got = out.cpu().numpy()
    for pi, pr in ops.items():
        b, h = divmod(pi, spec.hkv)
        qq = qb[b, h * G:(h + 1) * G]
        want, sel = pr.decode(qq, sc)
        nb = pr.info().nblk
        gs, gsel, _ = gpu_scores_sel(c, pi, nb)
        assert np.array_equal(gs.view(np.uint32), pr.scores(qq).view(np.uint32)), f"{where} pair {pi}: block scores"
        assert np.array_equal(gsel, sel), f"{where} pair {pi}: selected blocks"
        assert_close(got[b, h * G:(h + 1) * G], want, f"{where} pair {pi}")


def test_c3_full_size_sampled():
    """8 x 131072 tokens, 32 q / 8 kv heads, bf16, planted segments: the bench workload."""
    spec = gen.spec("c3")
    print(f"[fullsize] c3 {spec.num_seqs}x{spec.max_ctx}", flush=True)
    cap = spec.capacity
    lay = gen.make_layer(spec, 0, device="cuda", capacity=cap)
    lp, op = params_pair(spec)
    c = gpu_cache(lp, spec, lay, cap)
    q = lay["queries"]
    out = c.decode(q, scale_of())
    torch.cuda.synchronize()
    pairs = _spread(spec, 2, 3)                     # 16 of the 64 pairs, two per sequence
    ops = _oracle_pairs(op, spec, lay, cap, pairs)
    for pi, pr in ops.items():
        assert_state_equal(c, pi, pr, where="c3")
    _check_decode(c, spec, ops, q, out, "c3")


@pytest.mark.parametrize("name, per_seq, check_every", [("c2", 8, 4), ("c5", 1, 16)])
def test_append_decode_full_size_sampled(name, per_seq, check_every):
    """c2: 4 x 32768 fp16 with 16 x (append + decode); c5: 16 ragged sequences
    (16K..98K) of G = 7 Student-t bf16 with 64 x (append + decode), which
    crosses provisional flushes and segment finalizations."""
    spec = gen.spec(name)
    print(f"[fullsize] {name} ctx={spec.ctx[:4]}... steps={spec.appends}", flush=True)
    cap = spec.capacity
    lay = gen.make_layer(spec, 0, device="cuda", capacity=cap)
    lp, op = params_pair(spec)
    # c5: a capacity per sequence (its context plus the appends), so each
    # pair's regions are sized for its own sequence
    c = gpu_cache(lp, spec, lay, [L + spec.appends for L in spec.ctx] if name == "c5" else cap)
    pairs = _spread(spec, per_seq, 7)               # c2: all 32 pairs; c5: one per sequence (16 of 64)
    ops = _oracle_pairs(op, spec, lay, cap, pairs)
    for pi, pr in ops.items():
        assert_state_equal(c, pi, pr, where=f"{name} prefill")
    for t in range(spec.appends):
        kn, vn = gen.make_appends(spec, t)
        c.append(kn.cuda(), vn.cuda())
        kb, vb = bits(kn), bits(vn)
        for pi, pr in ops.items():
            b, h = divmod(pi, spec.hkv)
            pr.append(kb[b, h], vb[b, h])
        q = gen.make_queries(spec, t + 1)
        out = c.decode(q.cuda(), scale_of())
        if t % check_every == check_every - 1 or t == spec.appends - 1:
            torch.cuda.synchronize()
            for pi, pr in ops.items():
                assert_state_equal(c, pi, pr, where=f"{name} step {t}")
            _check_decode(c, spec, ops, q, out, f"{name} step {t}")


def _unpack_blocks(c, pi, descs, blocks, dtype):
    """Independent decoder of the selected blocks' packed K/V records of one
    pair -> (K, V) [tokens][D] fp64 in the rotated space (zeros on dropped
    channels), token counts per block."""
    npdt = np.float16 if dtype == "fp16" else None
    tok = c.region("token", pi).cpu().numpy()
    fb = np.array([d[2] for d in descs])
    Ks, Vs = [], []
    for blk in blocks:
        i = int(np.searchsorted(fb, blk, side="right") - 1)
        off, _, first, r, l2g, l2b, _ = descs[i]
        g, B = 1 << l2g, 1 << l2b
        bmb, vb = D // (8 * g), 2 * r
        base = off + (blk - first) * B * 2 * (bmb + vb)
        for half, dst in ((0, Ks), (1, Vs)):
            h0 = base + half * B * (bmb + vb)
            for j in range(B):
                bm = np.unpackbits(tok[h0 + j * bmb: h0 + (j + 1) * bmb], bitorder="little")[:D // g]
                raw = tok[h0 + B * bmb + j * vb: h0 + B * bmb + (j + 1) * vb].view(np.uint16)
                if npdt is not None:
                    vals = raw.view(np.float16).astype(np.float64)
                else:
                    vals = (raw.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
                x = np.zeros(D)
                ch = np.nonzero(np.repeat(bm, g))[0]
                x[ch] = vals
                dst.append(x)
    return np.array(Ks), np.array(Vs)


def test_c4_one_layer_full_size_properties():
    """One layer of the 1M-token workload (1 x 1,048,576 tokens, 8 kv heads, fp16)."""
    spec = gen.spec("c4", layers=1)
    print(f"[fullsize] c4 one layer {spec.max_ctx}", flush=True)
    cap = spec.capacity
    lay = gen.make_layer(spec, 0, device="cuda", capacity=cap)
    lp, op = params_pair(spec)
    c = gpu_cache(lp, spec, lay, cap)
    q = gen.make_queries(spec, 0)
    out = c.decode(q.cuda(), scale_of())
    torch.cuda.synchronize()
    pi = _sample(spec.hkv, 1, 11)[0]
    b, h = divmod(pi, spec.hkv)
    G, sc = spec.group, scale_of()
    # (1) a 2-window prefix, compressed by the oracle, equals the GPU's first bytes
    Lp = 2 * spec.rot_window
    pr = _oracle_pair(op, spec, lay, cap, pi, L=Lp)
    nd = pr.info().n_desc
    gd = c.region("desc", pi, 16 * nd).cpu().numpy()
    assert np.array_equal(gd, pr.descriptor_bytes()), "c4 prefix descriptors"
    ot, osc = pr.token_arena(), pr.score_arena()
    assert np.array_equal(c.region("token", pi, ot.size).cpu().numpy(), ot), "c4 prefix token arena"
    assert np.array_equal(c.region("score", pi, osc.size).cpu().numpy(), osc), "c4 prefix score arena"
    # (2) the prefix blocks' scores equal the oracle's
    qq = bits(q)[b, h * G:(h + 1) * G]
    nbp = pr.info().nblk
    nb = int(c.ws_region("wsel", pi, 4 * (c.layout.num_windows + 2)).cpu().numpy().view(np.int32)[-1])
    gs, gsel, _ = gpu_scores_sel(c, pi, nb)
    assert np.array_equal(gs[:nbp].view(np.uint32), pr.scores(qq).view(np.uint32)), "c4 prefix scores"
    # (3) the selection is the token budget over the GPU's scores: blocks in
    # (score desc, index asc) order while fewer than ceil(rho * tokens) are taken
    L = spec.ctx[b]
    nd_all = L // 64 + (1 if L % 64 >= 32 else 0)
    raw = c.region("desc", pi, 16 * nd_all).cpu().numpy()
    descs = []
    for j in range(nd_all):
        rr = raw[16 * j:16 * j + 16]
        u = rr[:12].view(np.uint32)
        descs.append((int(u[0]), int(u[1]), int(u[2]), int(rr[12]), int(rr[13]), int(rr[14]), int(rr[15])))
    sizes = np.concatenate([np.full((32 if d[6] & 1 else 64) >> d[5], 1 << d[5]) for d in descs])
    assert sizes.size == nb
    budget = -(-int(sizes.sum()) * spec.select[0] // spec.select[1])
    key = np.where(gs == 0, 0.0, gs)
    order = np.lexsort((np.arange(nb), -key.astype(np.float64)))
    before = np.cumsum(sizes[order]) - sizes[order]
    assert np.array_equal(gsel, np.sort(order[before < budget])), "c4 selection is not the token budget of the scores"
    # (4) attention over that selection, evaluated here in fp64
    K, V = _unpack_blocks(c, pi, descs, gsel, spec.dtype)
    fb = np.array([d[2] for d in descs])
    win = []
    for blk in gsel:
        i = int(np.searchsorted(fb, blk, side="right") - 1)
        win += [(i * 64) // spec.rot_window] * (1 << descs[i][5])
    win = np.array(win)
    rk = lay["rot_k"][b, h].double().cpu().numpy()
    rv = lay["rot_v"][b, h].double().cpu().numpy()
    qf = q[b, h * G:(h + 1) * G].double().numpy()
    logits = np.empty((G, len(K)))
    for w in np.unique(win):
        m = win == w
        logits[:, m] = (qf @ rk[w].T) @ K[m].T
    logits *= sc
    nbuf = L % 64 - (32 if L % 64 >= 32 else 0)
    assert nbuf == 0
    mx = logits.max(1, keepdims=True)
    p = np.exp(logits - mx)
    acc = np.zeros((G, D))
    for w in np.unique(win):
        m = win == w
        acc += (p[:, m] @ V[m]) @ rv[w]
    want = acc / p.sum(1, keepdims=True)
    assert_close(out.cpu().numpy()[b, h * G:(h + 1) * G], want, "c4 attention over the GPU selection")


@pytest.mark.parametrize("first", [0, 8, 16, 24])
def test_c4_every_layer_sampled_segments(first):
    """Eight of the 32 layers of the 1M-token workload per test, each built,
    compressed and decoded on the GPU as the benchmark does: for each layer a
    seeded 1 % of its segments (over all kv heads) are compressed by the oracle
    as one-segment sequences under the segment's window rotation and must equal
    the GPU's descriptor strategy, packed token records and block keys byte for
    byte (a segment's records depend only on its tokens and rotation); and the
    decode's selection of one kv head per layer is the token budget of the
    GPU's own scores."""
    spec = gen.spec("c4")
    lp, op = params_pair(spec)
    cap = spec.capacity
    W = spec.rot_window
    for layer in range(first, first + 8):
        lay = gen.make_layer(spec, layer, device="cuda", capacity=cap)
        c = gpu_cache(lp, spec, lay, cap)
        q = gen.make_queries(spec, 0, layer).cuda()
        c.decode(q, scale_of())
        torch.cuda.synchronize()
        nseg = spec.ctx[0] // 64
        rng = np.random.default_rng(4040 + layer)
        picks = sorted((int(pi), int(sg)) for pi, sg in zip(rng.integers(0, spec.hkv, nseg * spec.hkv // 100),
                                                             rng.integers(0, nseg, nseg * spec.hkv // 100)))
        descs = {pi: c.region("desc", pi, 16 * nseg).cpu().numpy().reshape(nseg, 16) for pi in set(p for p, _ in picks)}
        kk, vv = lay["k"], lay["v"]

        def one(job):
            pi, sg = job
            h = pi % spec.hkv
            w = (sg * 64) // W
            rk = lay["rot_k"][0, h, w:w + 1].cpu().numpy()
            rv = lay["rot_v"][0, h, w:w + 1].cpu().numpy()
            pr = O.Pair(op, 64, rk, rv)
            pr.compress(bits(kk[0, h, sg * 64:(sg + 1) * 64]), bits(vv[0, h, sg * 64:(sg + 1) * 64]))
            return pr.descriptor_bytes().reshape(-1, 16)[0], pr.token_arena(), pr.score_arena()

        with cf.ThreadPoolExecutor(16) as ex:
            want = list(ex.map(one, picks))
        for (pi, sg), (od, ot, osc) in zip(picks, want):
            d = descs[pi][sg]
            assert np.array_equal(d[12:15], od[12:15]), f"c4 layer {layer} pair {pi} segment {sg}: strategy"
            tok_off, sc_off = (int(x) for x in d[:8].view(np.uint32))
            got_t = c.arena[c.layout.token_off + c.pair_regions[pi][2] + tok_off:][:ot.size].cpu().numpy()
            got_s = c.arena[c.layout.score_off + c.pair_regions[pi][1] + sc_off:][:osc.size].cpu().numpy()
            assert np.array_equal(got_t, ot), f"c4 layer {layer} pair {pi} segment {sg}: token records"
            assert np.array_equal(got_s, osc), f"c4 layer {layer} pair {pi} segment {sg}: block keys"
        # the selection of one kv head is the token budget of the GPU's scores
        pi = int(rng.integers(0, spec.hkv))
        nb = int(c.ws_region("wsel", pi, 4 * (c.layout.num_windows + 2)).cpu().numpy().view(np.int32)[-1])
        gs, gsel, _ = gpu_scores_sel(c, pi, nb)
        bs = 1 << c.ws_region("bsize", pi, nb).cpu().numpy().astype(np.int64)
        budget = -(-int(bs.sum()) * spec.select[0] // spec.select[1])
        key = np.where(gs == 0, 0.0, gs)
        order = np.lexsort((np.arange(nb), -key.astype(np.float64)))
        before = np.cumsum(bs[order]) - bs[order]
        assert np.array_equal(gsel, np.sort(order[before < budget])), f"c4 layer {layer}: selection"
        print(f"[fullsize] c4 layer {layer}: {len(picks)} segments byte-exact, selection ok", flush=True)
        del c, lay
        torch.cuda.empty_cache()


def test_c3_quest_mode_full_size_sampled():
    """The quest mode (every channel kept, 16-token blocks, no rotation) on the
    full 8 x 131072 bf16 workload: sampled pairs against the oracle."""
    spec = gen.spec("c3", rotate=False)
    print(f"[fullsize] c3 quest mode {spec.num_seqs}x{spec.max_ctx}", flush=True)
    cap = spec.capacity
    lay = gen.make_layer(spec, 0, device="cuda", capacity=cap)
    lp, op = params_pair(spec, force_default=True, default=(D, 1, 16))
    c = gpu_cache(lp, spec, lay, cap)
    q = lay["queries"]
    out = c.decode(q, scale_of())
    torch.cuda.synchronize()
    pairs = _spread(spec, 1, 5)                     # one pair per sequence
    ops = _oracle_pairs(op, spec, lay, cap, pairs)
    for pi, pr in ops.items():
        assert_state_equal(c, pi, pr, where="c3 quest")
    _check_decode(c, spec, ops, q, out, "c3 quest")


def test_c3_fp8_full_size_sampled():
    """E4M3 token values on the full 8 x 131072 bf16 workload with the
    strategy search: sampled pairs against the oracle (bytes, scores,
    selections, outputs)."""
    spec = gen.spec("c3")
    print(f"[fullsize] c3 fp8 {spec.num_seqs}x{spec.max_ctx}", flush=True)
    cap = spec.capacity
    lay = gen.make_layer(spec, 0, device="cuda", capacity=cap)
    lp, op = params_pair(spec, fp8=True)
    c = gpu_cache(lp, spec, lay, cap)
    q = lay["queries"]
    out = c.decode(q, scale_of())
    torch.cuda.synchronize()
    pairs = _spread(spec, 1, 6)                     # one pair per sequence
    ops = _oracle_pairs(op, spec, lay, cap, pairs)
    for pi, pr in ops.items():
        assert_state_equal(c, pi, pr, where="c3 fp8")
    _check_decode(c, spec, ops, q, out, "c3 fp8")


def test_c3_gpu_rotations_full_size_sampled():
    """GPU rotation matrices of the full c3 cache (256 matrices of 65536
    tokens): sampled windows against the fp64 oracle (orthonormal rows,
    diagonalized covariance, eigenvalues, sign rule)."""
    import paper_2607_00760_amd as M
    from oracle import rotation as RO
    spec = gen.spec("c3")
    print(f"[fullsize] c3 rotations {spec.num_seqs}x{spec.max_ctx}", flush=True)
    cap = spec.capacity
    lay = gen.make_layer(spec, 0, device="cuda", capacity=cap)
    lp, _ = params_pair(spec)
    rk, rv, ek, ev = M.compute_rotations(lp, lay["k"], lay["v"], spec.ctx, cap, evals=True)
    torch.cuda.synchronize()
    rng = np.random.default_rng(9)
    for _ in range(3):
        b, h, w = int(rng.integers(spec.num_seqs)), int(rng.integers(spec.hkv)), int(rng.integers(2))
        for which, R, E in (("k", rk, ek), ("v", rv, ev)):
            a, e = w * spec.rot_window, (w + 1) * spec.rot_window
            x = lay[which][b, h, a:e].double().cpu().numpy()
            Ro, eo = RO.window_rotation(x)
            Rg = R[b, h, w].double().cpu().numpy()
            eg = E[b, h, w].double().cpu().numpy()
            lam = float(eo[0])
            assert np.abs(Rg @ Rg.T - np.eye(D)).max() <= 3e-5, f"{which} {b} {h} {w}: orthonormal"
            Mr = Rg @ (x.T @ x) @ Rg.T
            assert np.abs(np.diag(Mr) - eo).max() <= 5e-5 * lam, f"{which} {b} {h} {w}: Rayleigh quotients"
            assert np.abs(Mr - np.diag(np.diag(Mr))).max() <= 5e-5 * lam, f"{which} {b} {h} {w}: diagonal"
            assert np.abs(eg - eo).max() <= 5e-5 * lam, f"{which} {b} {h} {w}: eigenvalues"
            top = np.argmax(np.abs(Rg), axis=1)
            assert np.all(Rg[np.arange(D), top] > 0), f"{which} {b} {h} {w}: sign rule"


def test_c3_reorder_full_size_sampled():
    """Selection-pattern reorder of the c3 workload's own rotation matrices
    (64 pairs x 2 windows of 65536 tokens, K and V) in one library call:
    sampled windows identical to the oracle's reorder of the same matrices."""
    import paper_2607_00760_amd as M
    from oracle import rotation as RO
    spec = gen.spec("c3")
    print(f"[fullsize] c3 reorder {spec.num_seqs}x{spec.max_ctx}", flush=True)
    cap = spec.capacity
    lay = gen.make_layer(spec, 0, device="cuda", capacity=cap)
    lp, _ = params_pair(spec)
    rk, rv = lay["rot_k"].clone().contiguous(), lay["rot_v"].clone().contiguous()
    M.reorder_rotations(lp, lay["k"], lay["v"], spec.ctx, cap, rk, rv)
    torch.cuda.synchronize()
    nw = rk.shape[2]
    rng = np.random.default_rng(10)
    for _ in range(2):
        b, h, w = int(rng.integers(spec.num_seqs)), int(rng.integers(spec.hkv)), int(rng.integers(nw))
        for which, R in (("k", rk), ("v", rv)):
            a, e = w * spec.rot_window, min((w + 1) * spec.rot_window, spec.ctx[b])
            R0 = lay["rot_" + which][b, h, w].cpu().numpy()
            x = lay[which][b, h, a:e].float().cpu().numpy()
            order = RO.reorder_order(RO.coselection_counts(x, R0, lp.default[0]))
            assert np.array_equal(R[b, h, w].cpu().numpy(), R0[order]), f"{which} seq {b} head {h} window {w}"
