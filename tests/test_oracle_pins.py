"""Pins of the CPU oracle against what the paper and mathematics fix.

Each test checks the oracle against something other than itself: library
conversions, brute force on tiny inputs, closed forms, limiting cases of the
thresholds, textbook dense attention, exact signed-permutation rotations and
numbers the paper prints (tests/golden/paper_numbers.json).
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import torch

from oracle import oracle as O

D = 128
GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_numbers.json")))


@pytest.fixture(scope="module", autouse=True)
def _built():
    O.build(force=False)


def rng(seed):
    return np.random.default_rng(seed)


def to_bits(x, dtype):
    t = torch.tensor(np.asarray(x, np.float32))
    t = t.to(torch.bfloat16 if dtype == "bf16" else torch.float16)
    return t.view(torch.int16).numpy().view(np.uint16)


def from_bits(b, dtype):
    t = torch.from_numpy(np.ascontiguousarray(b).view(np.int16))
    return t.view(torch.bfloat16 if dtype == "bf16" else torch.float16).double().numpy()


# ---------------------------------------------------------------- conversions
def test_f16_rne_matches_numpy():
    r = rng(0)
    pats = r.integers(0, 2**32, 200000, dtype=np.uint64).astype(np.uint32)
    x = pats.view(np.float32)
    x = x[np.isfinite(x)]
    edge = np.array([0.0, -0.0, 65504.0, 65519.99, 65520.0, 1e-8, 2.0**-25, 2.0**-24, 3 * 2.0**-26,
                     2.0**-14, 2.0**-14 * (1 - 2.0**-11), 1.0 + 2.0**-11, 1.0 + 3 * 2.0**-11, -3.5e-6],
                    np.float32)
    scaled = (r.standard_normal(100000) * r.choice([1e-6, 1e-3, 1, 100, 3e4], 100000)).astype(np.float32)
    for xs in (x[:50000], edge, scaled):
        got = O.f32_to_f16_bits(xs)
        with np.errstate(over="ignore"):
            want = xs.astype(np.float16).view(np.uint16)
        assert np.array_equal(got, want)


def test_bf16_rne_matches_torch():
    r = rng(1)
    pats = r.integers(0, 2**32, 100000, dtype=np.uint64).astype(np.uint32)
    x = pats.view(np.float32)
    x = x[np.isfinite(x) & (np.abs(x) < 3.3e38)]
    x = np.concatenate([x, np.array([1.0 + 2.0**-8, 1.0 + 3 * 2.0**-8, -0.0, 1e-40], np.float32)])
    got = O.f32_to_bf16_bits(x)
    want = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(got, want)


def test_16bit_to_f32_all_patterns():
    pats = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    f16 = O.f16_bits_to_f32(pats)
    ref = pats.view(np.float16).astype(np.float32)
    ok = np.isfinite(ref)
    assert np.array_equal(f16[ok].view(np.uint32), ref[ok].view(np.uint32))
    bf = O.bf16_bits_to_f32(pats)
    refb = (pats.astype(np.uint32) << 16).view(np.float32)
    okb = np.isfinite(refb)
    assert np.array_equal(bf[okb].view(np.uint32), refb[okb].view(np.uint32))


# ---------------------------------------------------------------- ordered sums
def test_tree_sum_is_pairwise():
    # exact on integers; and pairwise (not left-to-right) where rounding decides:
    # (1+1) + (1+2^24) = 2 + 2^24 -> 16777218 ; left-to-right would give 16777220
    a = np.array([1.0, 1.0, 1.0, 2.0**24], np.float32)
    assert O.tree_sum(a) == np.float32(16777218.0)
    ints = rng(2).integers(-1000, 1000, 128).astype(np.float32)
    assert O.tree_sum(ints) == np.float32(ints.astype(np.int64).sum())


# ---------------------------------------------------------------- rotation (Sec. 2.3)
def test_rotation_identity_exact():
    x = rng(3).standard_normal((5, D)).astype(np.float32)
    assert np.array_equal(O.rotate(x, np.eye(D, dtype=np.float32)), x)
    assert np.array_equal(O.rotate(x, None), x)


def test_rotation_signed_permutation_exact():
    r = rng(4)
    perm = r.permutation(D)
    sign = r.choice([-1.0, 1.0], D)
    R = np.zeros((D, D), np.float32)
    R[np.arange(D), perm] = sign            # row j picks channel perm[j]
    x = r.standard_normal((3, D)).astype(np.float32)
    y = O.rotate(x, R)
    assert np.array_equal(y, (x[:, perm] * sign).astype(np.float32))


def test_rotation_matches_matmul_and_norm():
    r = rng(5)
    Q, _ = np.linalg.qr(r.standard_normal((D, D)))
    R = Q.astype(np.float32)
    x = r.standard_normal((4, D)).astype(np.float32)
    y = O.rotate(x, R)
    ref = x.astype(np.float64) @ R.astype(np.float64).T
    assert np.max(np.abs(y - ref)) < 1e-5
    assert np.allclose(np.linalg.norm(y, axis=1), np.linalg.norm(x, axis=1), rtol=1e-5)


# ---------------------------------------------------------------- top-k rule
def _brute_topk(s, k):
    """Max-sum subset of size k; ties -> lexicographically smallest index set."""
    best, best_set = None, None
    for sub in itertools.combinations(range(len(s)), k):
        tot = sum(int(s[i]) for i in sub)
        if best is None or tot > best:
            best, best_set = tot, sub
    return set(best_set)


def test_topk_matches_brute_force():
    r = rng(6)
    for n in range(1, 10):
        for _ in range(6):
            s = r.integers(0, 4, n).astype(np.float32)   # many ties
            for k in range(0, n + 1):
                m = O.topk_mask(s, k)
                assert set(np.nonzero(m)[0].tolist()) == (_brute_topk(s, k) if k else set())


def test_topk_tie_storm_takes_lowest_indices():
    m = O.topk_mask(np.ones(128, np.float32), 32)
    assert np.array_equal(np.nonzero(m)[0], np.arange(32))
    m = O.topk_mask(np.array([0.0, -0.0, 0.0, -0.0], np.float32), 2)   # -0 == +0
    assert np.array_equal(np.nonzero(m)[0], [0, 1])


def test_group_scores_closed_form():
    y = np.zeros(D, np.float32)
    y[:8] = [1, -2, 3, -4, 0.5, 0.25, -8, 16]
    assert O.group_scores(y, 1)[:8].tolist() == [1, 2, 3, 4, 0.5, 0.25, 8, 16]
    assert O.group_scores(y, 2)[:4].tolist() == [3, 7, 0.75, 24]
    assert O.group_scores(y, 4)[:2].tolist() == [10, 24.75]


# ---------------------------------------------------------------- packed format (Sec. 5.1)
def _unpack(rec, r, g, dtype):
    """Independent decoder of one packed vector -> (kept channel mask, values at kept)."""
    nbits = D // g
    words = rec[: nbits // 8].view(np.uint32) if nbits >= 32 else None
    bits = np.array([(int(words[i // 32]) >> (i % 32)) & 1 for i in range(nbits)], bool)
    kept = np.repeat(bits, g)
    vals = rec[nbits // 8:].view(np.uint16)
    assert vals.size == r
    return kept, vals


@pytest.mark.parametrize("r,g", [(16, 4), (16, 2), (16, 1), (32, 4), (32, 2), (32, 1), (48, 4), (48, 2), (48, 1)])
@pytest.mark.parametrize("dtype", ["fp16", "bf16"])
def test_pack_vector_roundtrip(r, g, dtype):
    rr = rng(7 + r + g)
    for _ in range(5):
        y = (rr.standard_normal(D) * rr.choice([0.1, 1, 10], D)).astype(np.float32)
        rec = O.pack_vector(y, r, g, dtype)
        assert rec.size == r * 2 + D // (8 * g)
        kept, vals = _unpack(rec, r, g, dtype)
        # kept groups = top r/g by (L1 magnitude desc, index asc), computed with numpy
        a = np.abs(y).reshape(-1, g)
        sc = a[:, 0] if g == 1 else ((a[:, 0] + a[:, 1]) if g == 2 else (a[:, 0] + a[:, 1]) + (a[:, 2] + a[:, 3]))
        order = np.lexsort((np.arange(sc.size), -sc))
        want = np.zeros(sc.size, bool)
        want[order[: r // g]] = True
        assert np.array_equal(kept, np.repeat(want, g))
        assert np.array_equal(vals, to_bits(y[kept], dtype))


def test_bitmap_and_ratio_paper_numbers():
    ex = GOLD["bitmap_example"]
    e = ex["elem_bits"] // 8
    r = int(round(D * (1 - ex["compression_rate"])))
    dense = D * e
    assert r * e / dense == ex["packed_fraction"]
    assert O.bitmap_bytes(1) / dense == ex["bitmap_fraction"]
    assert O.vec_bytes(r, 1, e) == r * e + O.bitmap_bytes(1)
    full = GOLD["memory_reduction_vs_full"]
    st = full["strategy"]
    ratio = 2 * D * 2 / O.bytes_per_token(st["keep"], st["group"], st["block"], 2)
    assert abs(ratio - full["value"]) < full["abs_tol"]
    q = GOLD["memory_reduction_vs_quest"]
    assert abs(ratio * (1 + q["quest_overhead"]) - q["value"]) < q["abs_tol"]


def test_used_bytes_closed_form_forced_default():
    P = O.Params(force_default=True, dtype="bf16")
    pr = O.Pair(P, 640)
    x = to_bits(rng(8).standard_normal((640, D)), "bf16")
    pr.compress(x, x)
    inf = pr.info()
    per_seg = 64 * 2 * (32 * 2 + 16) + 8 * (32 * 2 + 16) + 16
    assert inf.used_bytes == 10 * per_seg
    assert all((d["r"], d["log2g"], d["log2b"]) == (32, 0, 3) for d in pr.descriptors())
    ratio = 640 * 2 * D * 2 / inf.used_bytes
    assert abs(ratio - 512 / (160 + 10 + 0.25)) < 1e-12


# ---------------------------------------------------------------- strategy (Sec. 4.3 / 5.5)
def test_strategy_all_ones_closed_form():
    # all-equal magnitudes: kept = lowest groups, dropped fraction = (128 - r) / 128 exactly
    y = np.ones((64, D), np.float32)
    for tau, want in [(0.9, (16, 4)), (0.8, (32, 4)), (0.7, (48, 4)), (0.6, (48, 1))]:
        r, g, B = O.choose_strategy(O.Params(tau_channel=tau, tau_block=0.5), y, y)
        assert (r, g) == want
        assert B == 16                      # identical tokens: zero intra-block variance
    r, g, B = O.choose_strategy(O.Params(tau_channel=0.9, tau_block=0.0), y, y)
    assert B == 4                           # tau 0: nothing is strictly below 0 -> fallback


def test_strategy_one_hot_is_lossless():
    y = np.zeros((64, D), np.float32)
    y[np.arange(64), (np.arange(64) * 7) % D] = 3.0
    r, g, B = O.choose_strategy(O.Params(tau_channel=1e-6), y, y)
    assert (r, g) == (16, 4)


def test_strategy_limits():
    y = rng(9).standard_normal((64, D)).astype(np.float32)
    assert O.choose_strategy(O.Params(tau_channel=np.inf, tau_block=np.inf), y, y) == (16, 4, 16)
    assert O.choose_strategy(O.Params(tau_channel=0.0, tau_block=0.0), y, y) == (48, 1, 4)


def test_strategy_needs_both_k_and_v():
    """Reading R-4: one (r, g) for the segment, accepted only if K and V both
    pass.  All-ones vectors drop (128 - r) / 128 of their energy at any group
    size; one-hot vectors drop nothing."""
    ones = np.ones((64, D), np.float32)
    hot = np.zeros((64, D), np.float32)
    hot[np.arange(64), (np.arange(64) * 5) % D] = 2.0
    P = O.Params(tau_channel=0.8, tau_block=0.5)
    assert O.choose_strategy(P, hot, ones)[:2] == (32, 4)     # a K-only rule gives (16, 4)
    assert O.choose_strategy(P, ones, hot)[:2] == (32, 4)     # a V-only rule gives (16, 4)
    assert O.choose_strategy(P, hot, hot)[:2] == (16, 4)
    assert O.choose_strategy(P, ones, ones)[:2] == (32, 4)


def test_strategy_rate_first_order():
    """Reading R-4: the rate first (r = 16 -> 32 -> 48), then g = 4 -> 2 -> 1.
    Sixteen dominant channels spaced 4 apart fit r = 16 only one per group:
    (16, 1); a group-size-first order would take (32, 2)."""
    y = np.full((64, D), 0.01, np.float32)
    y[:, 0:64:4] = 1.0
    assert O.choose_strategy(O.Params(tau_channel=0.05, tau_block=0.5), y, y)[:2] == (16, 1)


def test_block_size_looks_at_keys_only():
    """Reading R-5: the block size follows the intra-block variance of the
    rotated keys; the values do not enter."""
    ones = np.ones((64, D), np.float32)
    alt = np.stack([np.ones(D) * (1 if t % 2 == 0 else -1) for t in range(64)]).astype(np.float32)
    P = O.Params(tau_channel=0.9, tau_block=0.5)
    assert O.choose_strategy(P, ones, alt)[2] == 16           # constant keys: no variance
    assert O.choose_strategy(P, alt, ones)[2] == 4            # every block mean 0: ratio 1, fallback


def test_block_size_closed_forms():
    base = np.ones(D, np.float32)
    # constant inside each 8-token group, sign flips between groups: B=16 mean is 0
    # (variance = total energy), B=8 variance is 0
    y = np.stack([base * (1 if (t // 8) % 2 == 0 else -1) for t in range(64)]).astype(np.float32)
    assert O.choose_strategy(O.Params(tau_channel=0.9, tau_block=0.5), y, y)[2] == 8
    # alternating sign every token: every block mean is 0 -> variance ratio exactly 1
    y = np.stack([base * (1 if t % 2 == 0 else -1) for t in range(64)]).astype(np.float32)
    assert O.choose_strategy(O.Params(tau_channel=0.9, tau_block=1.0), y, y)[2] == 4
    assert O.choose_strategy(O.Params(tau_channel=0.9, tau_block=1.0001), y, y)[2] == 16


def test_strategy_monotone_in_tau():
    r = rng(10)
    order = [(a, b) for a in (16, 32, 48) for b in (4, 2, 1)]
    for trial in range(4):
        scale = r.choice([1.0, 4.0, 16.0], D)
        yk = (r.standard_normal((64, D)) * scale).astype(np.float32)
        yv = (r.standard_normal((64, D)) * scale[::-1]).astype(np.float32)
        prev_c, prev_b = None, None
        for tau in (0.05, 0.1, 0.2, 0.3, 0.5, 0.8):
            rr, g, B = O.choose_strategy(O.Params(tau_channel=tau, tau_block=tau + 0.4), yk, yv)
            c = order.index((rr, g))
            if prev_c is not None:
                assert c <= prev_c and B >= prev_b
            prev_c, prev_b = c, B


def test_block_key_of_identical_tokens_is_the_token():
    x = np.zeros(D, np.float32)
    x[:40] = np.arange(40) * 0.25 - 3.0          # dyadic: block sums are exact
    toks = np.tile(x, (64, 1))
    bits = to_bits(toks, "fp16")
    pr = O.Pair(O.Params(force_default=True), 64)
    pr.compress(bits, bits)
    sc = pr.score_arena()
    rec = O.pack_vector(x, 32, 1, "fp16")
    assert np.array_equal(sc.reshape(8, -1), np.tile(rec, (8, 1)))


# ---------------------------------------------------------------- top-k count (Sec. 4.2 / 6.1)
def test_select_count():
    assert O.select_count(0, 1, 10) == 0
    assert O.select_count(1, 1, 10) == 1
    assert O.select_count(10, 1, 10) == 1
    assert O.select_count(11, 1, 10) == 2
    assert O.select_count(16384, 1, 10) == 1639
    assert O.select_count(131072, 1, 10) == 13108
    assert O.select_count(7, 1, 1) == 7


# ---------------------------------------------------------------- decode vs dense attention
def _numpy_attention(q, k, v, scale, dtype):
    scale = float(np.float32(scale))            # the scale is an fp32 argument
    qd, kd, vd = from_bits(q, dtype), from_bits(k, dtype), from_bits(v, dtype)
    if kd.shape[0] == 0:
        return np.zeros_like(qd)
    z = (qd @ kd.T) * scale
    z = z - z.max(axis=1, keepdims=True)
    p = np.exp(z)
    return (p @ vd) / p.sum(axis=1, keepdims=True)


@pytest.mark.parametrize("dtype", ["fp16", "bf16"])
@pytest.mark.parametrize("G", [4, 7])
def test_everything_kept_equals_dense(dtype, G):
    """r = D, rho = 1, identity rotation: the method reduces to dense attention."""
    r = rng(11 + G)
    for L in (0, 1, 31, 32, 33, 63, 64, 65, 100, 200, 257):
        for B in (4, 16):
            P = O.Params(group=G, dtype=dtype, force_default=True, default=(128, 1, B), select=(1, 1),
                         rot_window=128)
            k = to_bits(r.standard_normal((L, D)), dtype)
            v = to_bits(r.standard_normal((L, D)), dtype)
            q = to_bits(r.standard_normal((G, D)) * 2, dtype)
            pr = O.Pair(P, max(L, 1))
            pr.compress(k, v)
            out, sel = pr.decode(q, 1 / math.sqrt(D))
            ref = _numpy_attention(q, k, v, 1 / math.sqrt(D), dtype)
            assert np.max(np.abs(out - ref)) < 1e-12, (L, B)
            assert len(sel) == pr.info().nblk


def test_signed_permutation_rotation_equals_dense():
    """Exact rotations (signed permutations, one per window): the q rotation,
    the packed rotated K/V and the back-rotation of the output must cancel."""
    r = rng(12)
    G, L, W = 4, 300, 128
    nw = 3
    Rk = np.zeros((nw, D, D), np.float32)
    Rv = np.zeros((nw, D, D), np.float32)
    for w in range(nw):
        for R in (Rk[w], Rv[w]):
            R[np.arange(D), r.permutation(D)] = r.choice([-1.0, 1.0], D)
    P = O.Params(group=G, dtype="fp16", force_default=True, default=(128, 1, 8), select=(1, 1), rot_window=W)
    k = to_bits(r.standard_normal((L, D)), "fp16")
    v = to_bits(r.standard_normal((L, D)), "fp16")
    q = to_bits(r.standard_normal((G, D)) * 2, "fp16")
    pr = O.Pair(P, L, Rk, Rv)
    pr.compress(k, v)
    out, _ = pr.decode(q, 0.125)
    ref = _numpy_attention(q, k, v, 0.125, "fp16")
    assert np.max(np.abs(out - ref)) < 1e-12


def test_orthogonal_rotation_close_to_dense():
    r = rng(13)
    G, L = 4, 256
    Q1, _ = np.linalg.qr(r.standard_normal((D, D)))
    Q2, _ = np.linalg.qr(r.standard_normal((D, D)))
    P = O.Params(group=G, dtype="fp16", force_default=True, default=(128, 1, 8), select=(1, 1))
    k = to_bits(r.standard_normal((L, D)), "fp16")
    v = to_bits(r.standard_normal((L, D)), "fp16")
    q = to_bits(r.standard_normal((G, D)), "fp16")
    pr = O.Pair(P, L, Q1[None].astype(np.float32), Q2[None].astype(np.float32))
    pr.compress(k, v)
    out, _ = pr.decode(q, 1 / math.sqrt(D))
    ref = _numpy_attention(q, k, v, 1 / math.sqrt(D), "fp16")
    assert np.max(np.abs(out - ref)) < 3e-3        # only the fp16 rounding of rotated values


def _ahead_tokens(s, sizes, b):
    """Tokens of the blocks ranked ahead of block b: higher score, or the same
    score and a lower index."""
    return sum(int(sizes[j]) for j in range(len(s)) if s[j] > s[b] or (s[j] == s[b] and j < b))


def test_select_budget_closed_forms():
    # Sec. 6.1: 10 % of tokens, ceil in integers, at least one when any is scoreable
    assert [O.select_budget(n, 1, 10) for n in (0, 1, 10, 11, 64, 131072)] == [0, 1, 1, 2, 7, 13108]
    assert O.select_budget(100, 1, 16) == 7 and O.select_budget(100, 1, 8) == 13 and O.select_budget(9, 1, 1) == 9


def test_select_blocks_pairwise_definition():
    """Brute force: a block is taken iff the blocks ranked ahead of it hold
    fewer tokens than the budget (mixed block sizes, tie storms)."""
    r = rng(42)
    for n in range(1, 11):
        for _ in range(12):
            s = r.integers(0, 4, n).astype(np.float32)
            sizes = r.choice([4, 8, 16], n)
            for budget in range(1, int(sizes.sum()) + 2):
                m = O.select_blocks(s, sizes, budget)
                assert m.tolist() == [_ahead_tokens(s, sizes, b) < budget for b in range(n)], (s, sizes, budget)


def test_select_blocks_uniform_size_is_block_topk():
    """One block size B: ceil(ceil(rho B n) / B) = ceil(rho n), so the token
    budget takes the top ceil(rho n) blocks."""
    r = rng(43)
    for B in (4, 8, 16):
        for nb in (1, 5, 10, 11, 64, 1000):
            s = r.standard_normal(nb).astype(np.float32)
            s[r.integers(0, nb, nb // 3)] = 0.5
            m = O.select_blocks(s, np.full(nb, B), O.select_budget(nb * B, 1, 10))
            assert np.array_equal(m, O.topk_mask(s, O.select_count(nb, 1, 10))), (B, nb)


def test_selection_is_token_budget_of_scores():
    """Decode selects by the token budget over its own block scores: a block is
    selected iff the blocks ranked ahead of it hold fewer than ceil(rho *
    scoreable tokens) tokens; here segments of identical tokens take 16-token
    blocks, the others 8 or 4, so the sizes are mixed."""
    r = rng(14)
    G, L = 4, 64 * 40 + 45
    P = O.Params(group=G, dtype="bf16", tau_channel=0.3, tau_block=0.9)
    Q, _ = np.linalg.qr(r.standard_normal((D, D)))
    R = Q.astype(np.float32)[None]
    x = r.standard_normal((L, D))
    for seg in range(0, 40, 3):
        x[64 * seg:64 * seg + 64] = x[64 * seg] * 3.0        # zero block variance -> B = 16
    k = to_bits(x, "bf16")
    v = to_bits(r.standard_normal((L, D)), "bf16")
    q = to_bits(r.standard_normal((G, D)), "bf16")
    pr = O.Pair(P, L, R, R)
    pr.compress(k, v)
    s = pr.scores(q)
    assert s.size == pr.info().nblk
    sizes = []
    for d in pr.descriptors():
        n = 32 if d["flags"] & 1 else 64
        sizes += [1 << d["log2b"]] * (n >> d["log2b"])
    sizes = np.array(sizes)
    assert len(set(sizes.tolist())) >= 2 and sizes.sum() == L - pr.info().n_buf
    budget = -(-int(sizes.sum()) // 10)
    _, sel = pr.decode(q, 0.1)
    want = [b for b in range(s.size) if _ahead_tokens(s, sizes, b) < budget]
    assert np.array_equal(sel, want)
    assert budget <= sizes[sel].sum() < budget + 16


def test_block_score_closed_form():
    """Integer data, identity rotation, r = D: the chain is an exact integer
    dot product, and the block score is the max over the group's heads."""
    r = rng(15)
    G = 4
    P = O.Params(group=G, force_default=True, default=(128, 1, 4), select=(1, 1))
    k = r.integers(-3, 4, (64, D)).astype(np.float32)
    q = r.integers(-3, 4, (G, D)).astype(np.float32)
    pr = O.Pair(P, 64)
    pr.compress(to_bits(k, "fp16"), to_bits(k, "fp16"))
    s = pr.scores(to_bits(q, "fp16"))
    means = k.reshape(16, 4, D).mean(axis=1)           # exact (sums of small ints / 4)
    want = (q.astype(np.float64) @ means.T.astype(np.float64)).max(axis=0)
    assert np.array_equal(s.astype(np.float64), want)


def test_block_scores_multi_window_closed_form():
    """Three rotation windows, each its own signed permutation, integer data,
    every channel kept: q . R_w^T and the block means rotated by R_w cancel
    exactly, so every block score is max_h q_h . mean(block) whatever the
    window; a q rotated with another window's R would not cancel."""
    r = rng(40)
    G, W, nw = 4, 128, 3
    L = W * nw
    Rk = np.zeros((nw, D, D), np.float32)
    for w in range(nw):
        Rk[w][np.arange(D), r.permutation(D)] = r.choice([-1.0, 1.0], D)
    assert not np.array_equal(Rk[0], Rk[1])
    P = O.Params(group=G, force_default=True, default=(128, 1, 4), select=(1, 1), rot_window=W)
    k = r.integers(-3, 4, (L, D)).astype(np.float32)
    q = r.integers(-3, 4, (G, D)).astype(np.float32)
    pr = O.Pair(P, L, Rk, Rk)
    pr.compress(to_bits(k, "fp16"), to_bits(k, "fp16"))
    s = pr.scores(to_bits(q, "fp16"))
    means = k.reshape(-1, 4, D).mean(axis=1)
    want = (q.astype(np.float64) @ means.T.astype(np.float64)).max(axis=0)
    assert s.size == L // 4 and np.array_equal(s.astype(np.float64), want)


@pytest.mark.parametrize("dtype", ["fp16", "bf16"])
def test_dense_attention_matches_numpy(dtype):
    """The oracle's dense reference against numpy's softmax attention."""
    r = rng(41)
    for L, G in ((0, 4), (1, 4), (77, 7), (300, 4), (1000, 8)):
        q = to_bits(r.standard_normal((G, D)) * 2, dtype)
        k = to_bits(r.standard_normal((L, D)), dtype)
        v = to_bits(r.standard_normal((L, D)), dtype)
        out = O.dense_attention(q, k, v, 0.125, dtype)
        ref = _numpy_attention(q, k, v, 0.125, dtype)
        assert np.max(np.abs(out - ref)) < 1e-12, (L, G)


# ---------------------------------------------------------------- update buffer / double buffering
def _state(pr):
    i = pr.info()
    bk, bv = pr.buffer()
    sk, sv = pr.staging()
    return (i.L, i.n_final, i.prov, i.n_buf, i.nblk, i.used_bytes, pr.token_arena().tobytes(),
            pr.score_arena().tobytes(), pr.descriptor_bytes().tobytes(), bk.tobytes(), bv.tobytes(),
            sk.tobytes(), sv.tobytes())


@pytest.mark.parametrize("dtype", ["fp16", "bf16"])
def test_prefill_equals_prefill_plus_appends(dtype):
    r = rng(16)
    Lmax = 64 * 5 + 40
    Q, _ = np.linalg.qr(r.standard_normal((D, D)))
    R = np.stack([Q, Q[::-1]]).astype(np.float32)
    k = to_bits(r.standard_normal((Lmax, D)) * r.choice([1, 6], D), dtype)
    v = to_bits(r.standard_normal((Lmax, D)), dtype)
    P = O.Params(dtype=dtype, rot_window=128, tau_channel=0.25)
    for L0, L in [(0, 70), (5, 64), (32, 97), (64, 200), (100, 257), (150, Lmax)]:
        a = O.Pair(P, Lmax, R, R[::-1].copy())
        a.compress(k[:L], v[:L])
        b = O.Pair(P, Lmax, R, R[::-1].copy())
        b.compress(k[:L0], v[:L0])
        for t in range(L0, L):
            b.append(k[t], v[t])
        assert _state(a) == _state(b), (L0, L)


def test_state_machine_counts_and_provisional_strategy():
    r = rng(17)
    P = O.Params(dtype="fp16", tau_channel=0.3, force_default=False)
    k = to_bits(r.standard_normal((200, D)) * r.choice([1, 8], D), "fp16")
    pr = O.Pair(P, 200)
    pr.compress(k[:64], k[:64])
    prev = pr.descriptors()[0]
    for t in range(64, 200):
        pr.append(k[t], k[t])
        i = pr.info()
        m = i.L % 64
        assert (i.n_final, i.prov, i.n_buf) == (i.L // 64, int(m >= 32), m - 32 * int(m >= 32))
        ds = pr.descriptors()
        if i.prov:
            d = ds[-1]
            assert d["flags"] == 1
            assert (d["r"], d["log2g"], d["log2b"]) == (prev["r"], prev["log2g"], prev["log2b"])
            assert d["tok_off"] == i.tok_tail and d["first_block"] == i.nblk_final
        elif m == 0:
            prev = ds[-1]
            assert prev["flags"] == 0
    with pytest.raises(ValueError):
        pr.append(k[0], k[0])                 # capacity exhausted


def test_first_provisional_uses_default():
    r = rng(18)
    P = O.Params(dtype="fp16", default=(48, 2, 16))
    k = to_bits(r.standard_normal((40, D)), "fp16")
    pr = O.Pair(P, 64)
    pr.compress(k, k)
    d = pr.descriptors()
    assert len(d) == 1 and d[0]["flags"] == 1 and (d[0]["r"], d[0]["log2g"], d[0]["log2b"]) == (48, 1, 4)
    assert pr.info().n_buf == 8


# ---------------------------------------------------------------- channel truncation (Sec. 5.2)
def test_truncation_ratio_closed_form():
    # 96-bit bitmaps at the default strategy: 2 (64 + 12) + (64 + 12) / 8 bytes per token
    assert O.bitmap_bytes(1) == 16 and O.vec_bytes(32, 1, 2, 96) == 64 + 12
    # exactly T / g bits: 96 / g bits -> 12, 6, 3 bytes (Sec. 5.2: truncated channels
    # need no bitmap bit, so every group size saves a quarter of its bitmap)
    for g, T, bm in ((1, 96, 12), (2, 96, 6), (4, 96, 3), (1, 64, 8), (2, 64, 4), (4, 64, 2), (4, 128, 4),
                     (4, 32, 1), (2, 32, 2)):
        assert O.vec_bytes(32, g, 2, T) == 64 + bm
    assert abs(512 / O.bytes_per_token(32, 1, 8, 2, 96) - 512 / 161.5) < 1e-12
    # every group size gains from the truncation: (32, 2, 8) 512 / 153 -> 512 / 148.75
    assert O.bytes_per_token(32, 2, 8, 2, 128) == 2 * 72 + 72 / 8
    assert O.bytes_per_token(32, 2, 8, 2, 96) == 2 * 70 + 70 / 8
    for g in (1, 2, 4):
        assert O.bytes_per_token(32, g, 8, 2, 96) < O.bytes_per_token(32, g, 8, 2, 128)
    P = O.Params(force_default=True, dtype="bf16", trunc=96)
    pr = O.Pair(P, 640)
    x = to_bits(rng(21).standard_normal((640, D)), "bf16")
    pr.compress(x, x)
    per_seg = 64 * 2 * (32 * 2 + 12) + 8 * (32 * 2 + 12) + 16
    assert pr.info().used_bytes == 10 * per_seg


@pytest.mark.parametrize("g", [1, 2, 4])
def test_truncated_bitmap_is_brute_force_topk_of_leading_channels(g):
    """Identity rotation, forced (32, g, 4): every packed K vector keeps the
    top 32 / g groups among the first 96 / g by L1 score (lowest index on ties),
    its bitmap is exactly 96 / g bits LSB first, its values in ascending
    channel order."""
    T, r, B = 96, 32, 4
    P = O.Params(force_default=True, default=(r, g, B), dtype="fp16", trunc=T)
    x = rng(22 + g).standard_normal((64, D)) * np.linspace(0.2, 3.0, D)[None, :]   # tail channels largest
    kb = to_bits(x, "fp16")
    pr = O.Pair(P, 64)
    pr.compress(kb, kb)
    tok = pr.token_arena()
    y = from_bits(kb, "fp16")
    bmb, vb = T // g // 8, 2 * r
    for t in range(64):
        s = np.abs(y[t]).reshape(D // g, g).sum(axis=1)          # group L1 (g <= 4 adds in a pairwise order)
        order = sorted(range(T // g), key=lambda i: (-s[i], i))[: r // g]
        want_bits = np.zeros(T // g, np.uint8)
        want_bits[order] = 1
        blk = tok[(t // B) * B * 2 * (bmb + vb):]
        bm = np.unpackbits(blk[(t % B) * bmb:(t % B + 1) * bmb], bitorder="little")
        assert bm.size == T // g and np.array_equal(bm, want_bits), t
        ch = np.nonzero(np.repeat(want_bits, g))[0]
        vals = blk[B * bmb + (t % B) * vb: B * bmb + (t % B + 1) * vb].view(np.uint16)
        assert np.array_equal(vals, kb[t][ch]), t


def test_truncated_keep_everything_equals_dense_over_leading_channels():
    """r = T = 96, rho = 1, identity rotation: attention over the first 96
    channels of K and V (the truncated ones read as zero); update-buffer
    tokens stay dense, so they keep all channels."""
    r_ = rng(23)
    G, L, T = 4, 200, 96
    P = O.Params(group=G, dtype="bf16", force_default=True, default=(T, 1, 8), select=(1, 1), rot_window=128,
                 trunc=T)
    k = to_bits(r_.standard_normal((L, D)), "bf16")
    v = to_bits(r_.standard_normal((L, D)), "bf16")
    q = to_bits(r_.standard_normal((G, D)), "bf16")
    pr = O.Pair(P, L)
    pr.compress(k, v)
    out, _ = pr.decode(q, 1 / math.sqrt(D))
    kz, vz = k.copy(), v.copy()
    nc = (L // 64) * 64                        # compressed tokens; the rest is the update buffer
    kz[:nc, T:] = 0
    vz[:nc, T:] = 0
    ref = _numpy_attention(q, kz, vz, 1 / math.sqrt(D), "bf16")
    assert np.max(np.abs(out - ref)) < 1e-12


# ---------------------------------------------------------------- FP8 values (Sec. 7, reading R-20)
def _torch_e4m3(x):
    return torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def test_e4m3_decode_matches_torch():
    codes = np.arange(256, dtype=np.uint8)
    want = torch.from_numpy(codes).view(torch.float8_e4m3fn).float().numpy()
    got = O.e4m3_to_f32(codes)
    fin = np.isfinite(want)
    assert np.array_equal(np.isnan(got), ~fin) and fin.sum() == 254
    assert np.array_equal(got[fin], want[fin])
    assert np.signbit(got[0x80]) and not np.signbit(got[0x00])
    # the format's landmarks: largest finite, smallest normal and subnormal, one
    assert (got[0x7e], got[0x08], got[0x01], got[0x38]) == (448.0, 2.0**-6, 2.0**-9, 1.0)


def test_e4m3_rne_matches_torch_and_saturates():
    r = rng(30)
    scaled = (r.standard_normal(60000) * r.choice([2.0**-12, 2.0**-8, 2.0**-5, 1.0, 30.0, 300.0], 60000))
    scaled = scaled.astype(np.float32)
    vals = O.e4m3_to_f32(np.arange(0, 0x7f, dtype=np.uint8)).astype(np.float64)
    mids = (vals[:-1] + vals[1:]) / 2                      # ties: 4 significant bits, exact in fp32
    edge = np.concatenate([vals, mids, np.nextafter(mids.astype(np.float32), np.float32(0)),
                           np.nextafter(mids.astype(np.float32), np.float32(1e9)),
                           [0.0, 1e-30, 2.0**-10, 463.99, 448.0 + 8.0]]).astype(np.float32)
    for xs in (scaled[np.abs(scaled) < 464], edge, -edge):
        assert np.array_equal(O.f32_to_e4m3(xs), _torch_e4m3(xs))
    # past the largest finite value's rounding range torch gives NaN; the reading saturates
    big = np.array([464.0, 500.0, 1e6, 3e38], np.float32)
    assert np.all(O.f32_to_e4m3(big) == 0x7E) and np.all(O.f32_to_e4m3(-big) == 0xFE)


def test_fp8_record_sizes_closed_form():
    # default strategy with E4M3 token values: 2 (32 + 16) + (64 + 16) / 8 = 106 bytes per token
    assert O.vec_bytes(32, 1, 1) == 48 and O.bytes_per_token(32, 1, 8, 1) == 106.0
    assert abs(512 / O.bytes_per_token(32, 1, 8, 1) - 4.830188679245283) < 1e-12
    P = O.Params(force_default=True, dtype="bf16", fp8=True)
    pr = O.Pair(P, 640)
    x = to_bits(rng(31).standard_normal((640, D)), "bf16")
    pr.compress(x, x)
    per_seg = 64 * 2 * (32 + 16) + 8 * (32 * 2 + 16) + 16
    assert pr.info().used_bytes == 10 * per_seg


@pytest.mark.parametrize("dtype", ["fp16", "bf16"])
def test_fp8_records_hold_e4m3_of_the_kept_values(dtype):
    """Identity rotation, forced (32, 1, 8): each K and V token record is the
    16-byte bitmap of the 32 largest |x| followed by their E4M3 codes in
    ascending channel order; block keys keep 16-bit values."""
    r, B = 32, 8
    P = O.Params(force_default=True, default=(r, 1, B), dtype=dtype, fp8=True)
    x = rng(32).standard_normal((64, D)) * np.exp(rng(33).uniform(-6, 4, (64, D)))   # subnormal to saturated
    kb = to_bits(x, dtype)
    vb_bits = to_bits(-x[::-1], dtype)
    pr = O.Pair(P, 64)
    pr.compress(kb, vb_bits)
    tok, sc = pr.token_arena(), pr.score_arena()
    rec = 16 + r
    assert tok.size == 64 * 2 * rec and sc.size == (64 // B) * (16 + 2 * r)
    for which, bits_ in ((0, kb), (1, vb_bits)):
        y = from_bits(bits_, dtype)
        for t in range(64):
            ch = np.sort(sorted(range(D), key=lambda c: (-abs(y[t, c]), c))[:r])
            blk = tok[(t // B) * B * 2 * rec + which * B * rec:]
            bm = np.unpackbits(blk[(t % B) * 16:(t % B + 1) * 16], bitorder="little")
            assert np.array_equal(np.nonzero(bm)[0], ch), (which, t)
            codes = blk[B * 16 + (t % B) * r: B * 16 + (t % B + 1) * r]
            assert np.array_equal(codes, _torch_e4m3(np.clip(y[t, ch], -448, 448))), (which, t)
    # the first block key: the fp32 mean of its 8 keys (ascending adds, times 1/8),
    # the 16-byte bitmap of its 32 largest |mu|, then their 16-bit values
    yk = from_bits(kb, dtype).astype(np.float32)
    acc = yk[0].copy()
    for t in range(1, B):
        acc = (acc + yk[t]).astype(np.float32)
    mu = (acc * np.float32(1.0 / B)).astype(np.float32)
    ch = np.sort(sorted(range(D), key=lambda c: (-abs(float(mu[c])), c))[:r])
    assert np.array_equal(np.nonzero(np.unpackbits(sc[:16], bitorder="little"))[0], ch)
    assert np.array_equal(sc[16:16 + 2 * r].view(np.uint16), to_bits(mu[ch], dtype))


def test_fp8_keep_everything_equals_dense_over_e4m3_values():
    """r = D, rho = 1, identity rotation, E4M3 values: attention over K and V
    rounded to E4M3 for the compressed tokens; update-buffer tokens stay 16-bit."""
    r_ = rng(34)
    G, L = 4, 200
    P = O.Params(group=G, dtype="bf16", force_default=True, default=(D, 1, 8), select=(1, 1), rot_window=128,
                 fp8=True)
    k = to_bits(r_.standard_normal((L, D)), "bf16")
    v = to_bits(r_.standard_normal((L, D)), "bf16")
    q = to_bits(r_.standard_normal((G, D)), "bf16")
    pr = O.Pair(P, L)
    pr.compress(k, v)
    out, _ = pr.decode(q, 1 / math.sqrt(D))
    nc = (L // 64) * 64
    e4 = lambda b: torch.from_numpy(_torch_e4m3(from_bits(b, "bf16"))).view(torch.float8_e4m3fn).float().numpy()
    kq, vq = k.copy(), v.copy()
    kq[:nc] = to_bits(e4(k[:nc]), "bf16")                  # E4M3 values are exact in bf16
    vq[:nc] = to_bits(e4(v[:nc]), "bf16")
    assert not np.array_equal(kq, k)
    ref = _numpy_attention(q, kq, vq, 1 / math.sqrt(D), "bf16")
    assert np.max(np.abs(out - ref)) < 1e-12
