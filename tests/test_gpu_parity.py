"""GPU parity: the HIP library against the CPU oracle on the same seeded inputs.

Bit-exact: descriptors (strategy choices, offsets), packed score and token
arenas, update buffer and staging, block scores and the selected block lists.
Within 2e-3 max-abs and 1e-3 relative L2: the fp32 attention outputs.
"""
import math

import numpy as np
import pytest
import torch

from _parity import (D, assert_close, assert_state_equal, bits, gpu_cache, gpu_scores_sel, oracle_decode_all,
                     oracle_pairs, params_pair, scale_of)
import paper_2607_00760_amd as M
from oracle import oracle as O
from workloads import gen

pytestmark = pytest.mark.gpu

CASES = {
    # name: (spec, extra params)
    "c1": (gen.spec("c1"), {}),
    "ragged_bf16_w128": (gen.spec("c3", ctx=(0, 1, 31, 32, 33, 63, 64, 100, 1000, 2049), hkv=2, kind="gauss",
                                  rot_window=128), {}),
    "g7_student": (gen.spec("c5", ctx=(300, 77, 129, 2000), appends=0), {}),
    "forced_norot_fp16": (gen.spec("c2", ctx=(700, 64, 1500), hkv=2, rotate=False), dict(force_default=True)),
    "mixed_strategies": (gen.spec("c2", ctx=(4096, 2500), hkv=4), {}),
    "keep_all_rho1": (gen.spec("c1", ctx=(333, 200), hkv=2), dict(force_default=True, default=(128, 1, 4),
                                                                  select=(1, 1))),
    # the sequence-only (quest) mode: every channel kept, 16-token blocks, no rotation
    "quest_mode": (gen.spec("c3", ctx=(2500, 700), hkv=2, rotate=False), dict(force_default=True,
                                                                              default=(128, 1, 16))),
    # channel truncation: bitmaps of the first 96 (64) channels: 12 / 6 / 3-byte bitmaps
    # at g = 1 / 2 / 4 (4 / 2 bytes at T = 64, g = 2 / 4), so g >= 2 records sit at any byte
    "truncated_96": (gen.spec("c1", ctx=(3000, 1200), hkv=2), dict(trunc=96)),
    "truncated_64_g2": (gen.spec("c2", ctx=(1500, 700), hkv=2), dict(trunc=64, force_default=True,
                                                                    default=(32, 2, 8))),
    # kept counts outside 16/32/48: the general (runtime trip count) walks
    "odd_keeps": (gen.spec("c2", ctx=(1500, 900), hkv=2), dict(keep_cand=(8, 24, 40), default=(24, 2, 8),
                                                            tau_channel=0.2)),
    # E4M3 token values: strategy search (16-byte granule and dword loads), the
    # default strategy (fixed-count walks), kept counts that are multiples of 4
    # but not of 16 (dword loads), every channel kept (the general walk), and
    # with truncated bitmaps
    "fp8_search_bf16": (gen.spec("c3", ctx=(3000, 1200), hkv=2), dict(fp8=True)),
    "fp8_default_fp16": (gen.spec("c1", ctx=(1500, 700, 64, 5), hkv=2), dict(fp8=True, force_default=True)),
    "fp8_keeps_by_4": (gen.spec("c2", ctx=(1500, 900), hkv=2), dict(fp8=True, keep_cand=(12, 20, 44),
                                                                 default=(20, 2, 8), tau_channel=0.2)),
    "fp8_keep_all": (gen.spec("c1", ctx=(333, 200), hkv=2), dict(fp8=True, force_default=True,
                                                              default=(128, 1, 4), select=(1, 1))),
    "fp8_truncated_96": (gen.spec("c1", ctx=(2000, 900), hkv=2), dict(fp8=True, trunc=96)),
    # rotations reordered by selection pattern (the oracle's reorder of the
    # workload's matrices), with 96-channel bitmaps: the use the reorder serves
    "reordered_truncated_96": (gen.spec("c2", ctx=(2500, 900), hkv=2, rot_window=1024), dict(trunc=96)),
    # E4M3 values over a wide range: tokens scaled by 2^-14 .. 2^9, so kept
    # values fall below 2^-6 (subnormal codes, zeros) and above 448 (saturation);
    # K and V for the byte-exact compression, K only for the decode (unit-scale
    # values keep the outputs O(1) under the same absolute bound)
    "fp8_wide_range": (gen.spec("c3", ctx=(1500, 700), hkv=2, kind="gauss"), dict(fp8=True)),
    # more than 32 K blocks in a pair: the multi-workgroup top-k (18 chunks of
    # 4096 blocks for the first pair, 5 for the second)
    "long_topk_b4": (gen.spec("c1", ctx=(290000, 70000), hkv=1, rotate=False), dict(force_default=True,
                                                                                   default=(32, 1, 4))),
    # 16 K to 32 K blocks in the first pair: the single-workgroup top-k with 32
    # keys per thread, beside a short pair on 16 keys per thread
    "mid_topk_b4": (gen.spec("c1", ctx=(100000, 3000), hkv=1, rotate=False), dict(force_default=True,
                                                                                 default=(32, 1, 4))),
}


def _case(name, decode=False):
    spec, extra = CASES[name]
    cap = spec.max_ctx + 130
    lay = gen.make_layer(spec, 0, capacity=cap)
    lp, op = params_pair(spec, **extra)
    if name == "fp8_wide_range":
        n = lay["k"].shape[2]
        scale = torch.pow(2.0, (torch.arange(n) % 24 - 14).float())[None, None, :, None]
        for which in (("k",) if decode else ("k", "v")):
            lay[which] = (lay[which].float() * scale).to(lay[which].dtype)     # exact: powers of two
    if name.startswith("reordered"):
        from oracle import rotation as RO
        for which in ("k", "v"):
            R = lay["rot_" + which].clone()
            for b in range(spec.num_seqs):
                for h in range(spec.hkv):
                    x = lay[which][b, h].float().numpy()
                    R[b, h] = torch.from_numpy(RO.reorder_rotations(x, spec.ctx[b], spec.rot_window,
                                                                    R[b, h].numpy(), lp.default[0])[0])
            lay["rot_" + which] = R
    return spec, lay, lp, op, cap


@pytest.mark.parametrize("name", list(CASES))
def test_compress_bit_exact(name):
    spec, lay, lp, op, cap = _case(name)
    print(f"[compress] {name} ctx={spec.ctx} hkv={spec.hkv} G={spec.group} {spec.dtype}", flush=True)
    c = gpu_cache(lp, spec, lay, cap)
    ops = oracle_pairs(op, spec, lay, cap)
    for p in range(spec.num_seqs * spec.hkv):
        assert_state_equal(c, p, ops[p], where=name)


@pytest.mark.parametrize("name", ["c1", "mixed_strategies", "forced_norot_fp16", "truncated_64_g2", "fp8_search_bf16",
                                  "ragged_bf16_w128"])
def test_single_pass_compress_equals_two_pass(name):
    """The single-pass compression (one rotation per token, records through
    the workspace slots) writes the same arena as the two-pass one."""
    spec, lay, lp, op, cap = _case(name)
    caches = []
    for single in (True, False):
        c = M.MosaicCache(lp, spec.num_seqs, cap, rotated=lay["rot_k"] is not None, device="cuda")
        c.arena.zero_()
        rk = lay["rot_k"].cuda() if lay["rot_k"] is not None else None
        rv = lay["rot_v"].cuda() if lay["rot_v"] is not None else None
        c.compress(lay["k"].cuda(), lay["v"].cuda(), lay["ctx_lens"], rk, rv, single_pass=single)
        caches.append(c)
    torch.cuda.synchronize()
    assert torch.equal(caches[0].arena, caches[1].arena), name


@pytest.mark.parametrize("name", list(CASES))
def test_decode_parity(name):
    spec, lay, lp, op, cap = _case(name, decode=True)
    print(f"[decode] {name} ctx={spec.ctx}", flush=True)
    c = gpu_cache(lp, spec, lay, cap)
    ops = oracle_pairs(op, spec, lay, cap)
    q = gen.make_queries(spec, 0)
    out = c.decode(q.cuda(), scale_of())
    torch.cuda.synchronize()
    want, sels, scores = oracle_decode_all(ops, spec, q, scale_of())
    for p in range(spec.num_seqs * spec.hkv):
        nb = ops[p].info().nblk
        gs, gsel, _ = gpu_scores_sel(c, p, nb)
        assert np.array_equal(gs.view(np.uint32), scores[p].view(np.uint32)), f"{name} pair {p}: block scores"
        assert np.array_equal(gsel, sels[p]), f"{name} pair {p}: selected blocks"
    err, rel = assert_close(out.cpu().numpy(), want, name)
    print(f"[decode] {name}: max-abs {err:.3e} rel-L2 {rel:.3e}", flush=True)


@pytest.mark.parametrize("name", ["c1", "ragged_bf16_w128", "g7_student", "fp8_search_bf16"])
def test_append_flush_finalize_parity(name):
    spec, lay, lp, op, cap = _case(name)
    steps = 100
    print(f"[append] {name} steps={steps}", flush=True)
    c = gpu_cache(lp, spec, lay, cap)
    ops = oracle_pairs(op, spec, lay, cap)
    sc = scale_of()
    for t in range(steps):
        kn, vn = gen.make_appends(spec, t)
        c.append(kn.cuda(), vn.cuda())
        kb, vb = bits(kn), bits(vn)
        for p, pr in enumerate(ops):
            b, h = divmod(p, spec.hkv)
            pr.append(kb[b, h], vb[b, h])
        if t % 33 == 32 or t == steps - 1:
            torch.cuda.synchronize()
            for p in range(len(ops)):
                assert_state_equal(c, p, ops[p], where=f"{name} step {t}")
            q = gen.make_queries(spec, t + 1)
            out = c.decode(q.cuda(), sc)
            want, _, _ = oracle_decode_all(ops, spec, q, sc)
            assert_close(out.cpu().numpy(), want, f"{name} step {t}")


@pytest.mark.parametrize("name", ["long_topk_b4", "mid_topk_b4"])
def test_long_topk_all_ties(name):
    """A zero query scores every block 0: the selection is the first blocks in
    block order up to the token budget, on the multi-workgroup top-k (where
    the equal-token prefix carries across chunks) and on the 32-key path."""
    spec, lay, lp, op, cap = _case(name)
    c = gpu_cache(lp, spec, lay, cap)
    ops = oracle_pairs(op, spec, lay, cap)
    q = torch.zeros((spec.num_seqs, spec.hq, D), dtype=spec.torch_dtype)
    out = c.decode(q.cuda(), scale_of())
    torch.cuda.synchronize()
    want, sels, scores = oracle_decode_all(ops, spec, q, scale_of())
    for p in range(spec.num_seqs * spec.hkv):
        nb = ops[p].info().nblk
        gs, gsel, _ = gpu_scores_sel(c, p, nb)
        assert not np.any(scores[p]), "a zero query scores every block 0"
        assert np.array_equal(gs.view(np.uint32), scores[p].view(np.uint32))
        L = spec.ctx[p // spec.hkv]
        scoreable = L // 64 * 64 + (32 if L % 64 >= 32 else 0)     # final segments + a provisional half
        budget = -(-scoreable * spec.select[0] // spec.select[1])
        assert np.array_equal(sels[p], np.arange(-(-budget // 4))), "oracle: the first blocks in order"
        assert np.array_equal(gsel, sels[p]), f"pair {p}: selected blocks"
    assert_close(out.cpu().numpy(), want, "long_topk_all_ties")


def test_keep_all_equals_dense_on_gpu():
    """r = D, rho = 1, identity rotation: the method is dense attention."""
    spec = gen.spec("c1", ctx=(333, 200, 64, 31), hkv=2, rotate=False)
    cap = spec.max_ctx + 130
    lay = gen.make_layer(spec, 0, capacity=cap)
    lp, _ = params_pair(spec, force_default=True, default=(128, 1, 4), select=(1, 1))
    c = gpu_cache(lp, spec, lay, cap)
    q = gen.make_queries(spec, 0).cuda()
    out = c.decode(q, scale_of()).cpu().numpy()
    kb, vb, qb = bits(lay["k"]), bits(lay["v"]), bits(q)
    for b in range(spec.num_seqs):
        L = spec.ctx[b]
        for h in range(spec.hkv):
            want = O.dense_attention(qb[b, h * spec.group:(h + 1) * spec.group], kb[b, h, :L], vb[b, h, :L],
                                     np.float32(scale_of()), spec.dtype)
            assert_close(out[b, h * spec.group:(h + 1) * spec.group], want, f"seq {b} head {h}")


@pytest.mark.parametrize("dtype,G", [("fp16", 4), ("bf16", 7)])
def test_dense_baseline(dtype, G):
    import paper_2607_00760_amd as M
    spec = gen.spec("c1", ctx=(3000, 1025, 1), hkv=2, group=G, dtype=dtype)
    lay = gen.make_layer(spec, 0)
    q = gen.make_queries(spec, 0).cuda()
    ctx = torch.tensor(spec.ctx, dtype=torch.int32, device="cuda")
    out = M.dense_decode(q, lay["k"].cuda(), lay["v"].cuda(), ctx, scale_of(), spec.max_ctx, G).cpu().numpy()
    kb, vb, qb = bits(lay["k"]), bits(lay["v"]), bits(q)
    for b in range(spec.num_seqs):
        for h in range(spec.hkv):
            L = spec.ctx[b]
            want = O.dense_attention(qb[b, h * G:(h + 1) * G], kb[b, h, :L], vb[b, h, :L], np.float32(scale_of()), dtype)
            assert_close(out[b, h * G:(h + 1) * G], want, f"dense seq {b} head {h}")


def test_decode_is_deterministic():
    spec, lay, lp, op, cap = _case("mixed_strategies")
    c = gpu_cache(lp, spec, lay, cap)
    q = gen.make_queries(spec, 3).cuda()
    a = c.decode(q, scale_of()).clone()
    b = c.decode(q, scale_of()).clone()
    c2 = gpu_cache(lp, spec, lay, cap)
    d = c2.decode(q, scale_of())
    assert torch.equal(a, b) and torch.equal(a, d)


def test_ragged_capacities_parity():
    """A capacity per sequence (context + 100): each pair's regions sized for
    its own sequence and located through the pair table.  Prefill, 100
    appends across flushes and finalizes, and decode are byte-exact /
    within tolerance against the oracle, and the arena is smaller than with
    the longest capacity everywhere."""
    spec = gen.spec("c5", ctx=(1000, 64, 3000, 257), hkv=2, appends=100, rot_window=1024)
    caps = [L + spec.appends for L in spec.ctx]
    lay = gen.make_layer(spec, 0, capacity=max(caps))
    lp, op = params_pair(spec)
    print(f"[ragged] caps={caps}", flush=True)
    c = gpu_cache(lp, spec, lay, caps)
    uni = M.MosaicCache(lp, spec.num_seqs, max(caps), rotated=True)
    tok_ragged = sum(r[3] for r in c.pair_regions)
    assert tok_ragged < 0.5 * len(c.pair_regions) * uni.layout.token_stride      # 4721 of 4 x 3100 tokens
    assert c.arena.numel() < uni.arena.numel()
    del uni
    ops = oracle_pairs(op, spec, lay, max(caps))
    for p, pr in enumerate(ops):
        assert_state_equal(c, p, pr, where="ragged prefill")
    sc = scale_of()
    for t in range(spec.appends):
        kn, vn = gen.make_appends(spec, t)
        c.append(kn.cuda(), vn.cuda())
        kb, vb = bits(kn), bits(vn)
        for p, pr in enumerate(ops):
            b, h = divmod(p, spec.hkv)
            pr.append(kb[b, h], vb[b, h])
    with pytest.raises(M.MosaicError):                          # every sequence is full now
        c.append(kn.cuda(), vn.cuda())
    torch.cuda.synchronize()
    for p, pr in enumerate(ops):
        assert_state_equal(c, p, pr, where="ragged after appends")
    q = gen.make_queries(spec, 7)
    out = c.decode(q.cuda(), sc)
    want, sels, _ = oracle_decode_all(ops, spec, q, sc)
    for p in range(len(ops)):
        _, gsel, _ = gpu_scores_sel(c, p, ops[p].info().nblk)
        assert np.array_equal(gsel, sels[p]), f"pair {p}: selected blocks"
    err = assert_close(out.cpu().numpy(), want, "ragged capacities")
    print(f"[ragged] max-abs {err[0]:.2e} rel-L2 {err[1]:.2e}", flush=True)
