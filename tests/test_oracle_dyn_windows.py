"""Pins of the oracle's loss-closed windows of decode tokens (Sec. 4.3 "Dynamic
Compression Strategy", Sec. 5.5 "Incremental Strategy Generation"; reading
R-23): the per-segment compression loss, the close rule (accumulated loss
above a threshold once a minimum length is held, or the maximum length), the
close protocol (a buffer flush waits for the closed window's rotation), the
recompression of a closed window, and decode over irregular windows.

Each check is against something other than the oracle itself: closed forms on
constant and one-hot data, a numpy brute force of the loss, the oracle's own
prefill compression of the same tokens (a separately pinned path), exact
signed-permutation rotations against numpy dense attention, and an
independent numpy decoder of the packed records.
"""
import math

import numpy as np
import pytest
import torch

from oracle import oracle as O

D = 128
S = 64


@pytest.fixture(scope="module", autouse=True)
def _built():
    O.build(force=False)


def to_bits(x, dtype="fp16"):
    t = torch.tensor(np.asarray(x, np.float32)).to(torch.bfloat16 if dtype == "bf16" else torch.float16)
    return t.view(torch.int16).numpy().view(np.uint16)


def from_bits(b, dtype="fp16"):
    t = torch.from_numpy(np.ascontiguousarray(b).view(np.int16))
    return t.view(torch.bfloat16 if dtype == "bf16" else torch.float16).double().numpy()


def eye_rot(nw):
    return np.broadcast_to(np.eye(D, dtype=np.float32), (nw, D, D)).copy()


def signed_perm(r):
    R = np.zeros((D, D), np.float32)
    R[np.arange(D), r.permutation(D)] = r.choice([-1.0, 1.0], D)
    return R


def window_rotation(x):
    """Rows = eigenvectors of X^T X by descending eigenvalue (fp64), signed so
    the largest-magnitude component is positive, cast to fp32."""
    X = np.asarray(x, np.float64)
    _, vecs = np.linalg.eigh(X.T @ X)
    rows = vecs.T[::-1].copy()
    idx = np.argmax(np.abs(rows), axis=1)
    sg = np.sign(rows[np.arange(D), idx])
    sg[sg == 0] = 1.0
    return (rows * sg[:, None]).astype(np.float32)


def drive(pr, k, v, closer, L0):
    """Append tokens L0.. of k, v; when an append is refused because a closed
    window awaits its rotation, close it with closer(pair, window info) and
    append again.  Returns the closes seen: (window, first token, tokens,
    tokens in the cache when the refusal came)."""
    seen = []
    for t in range(L0, k.shape[0]):
        st = pr.append_status(k[t], v[t])
        if st == -4:
            w = pr.windows()
            assert w["pend"] >= 0
            assert t % S == S // 2 - 1, t          # refused only by the append that would flush
            a, b = w["wseg"][w["pend"]] * S, w["wseg"][w["pend"] + 1] * S
            seen.append((w["pend"], a, b - a, t))
            closer(pr, w["pend"], a, b)
            st = pr.append_status(k[t], v[t])
        assert st == 0, (t, st)
    return seen


# ---------------------------------------------------------------- the loss of a segment
def test_segment_loss_closed_forms():
    P = O.Params()
    ones = np.ones((S, D), np.float32)
    assert O.segment_loss(P, ones, ones, 32, 1) == 0.75           # 96 of 128 equal channels dropped
    assert O.segment_loss(P, ones, ones, 16, 4) == 0.875
    assert O.segment_loss(P, ones, ones, 48, 2) == 0.625
    hot = np.zeros((S, D), np.float32)
    hot[:, 3] = 2.0
    assert O.segment_loss(P, hot, hot, 16, 4) == 0.0              # one channel: lossless
    half = np.zeros((S, D), np.float32)
    half[:, :64] = 1.0
    # the larger of K's and V's loss (not K's alone, not their mean)
    assert O.segment_loss(P, hot, half, 32, 1) == 0.5
    assert O.segment_loss(P, half, hot, 32, 1) == 0.5
    assert O.segment_loss(P, ones, half, 32, 1) == 0.75
    zero = np.zeros((S, D), np.float32)
    assert O.segment_loss(P, zero, zero, 32, 1) == 0.0             # no energy: no loss
    assert O.segment_loss(P, zero, ones, 32, 1) == 0.75


@pytest.mark.parametrize("r,g", [(16, 4), (32, 2), (32, 1), (48, 1)])
def test_segment_loss_brute_force(r, g):
    rr = np.random.default_rng(3 + r + g)
    yk = (rr.standard_normal((S, D)) * rr.choice([0.2, 1, 5], D)).astype(np.float32)
    yv = (rr.standard_normal((S, D)) * rr.choice([0.2, 1, 5], D)).astype(np.float32)

    def rel_drop(y):
        y = y.astype(np.float64)
        a = np.abs(y).reshape(S, -1, g)
        sc = a[..., 0] if g == 1 else ((a[..., 0] + a[..., 1]) if g == 2 else (a[..., 0] + a[..., 1]) + (a[..., 2] + a[..., 3]))
        drop = 0.0
        for t in range(S):
            order = np.lexsort((np.arange(sc.shape[1]), -sc[t]))
            keep = np.zeros(sc.shape[1], bool)
            keep[order[: r // g]] = True
            drop += float(np.sum((y[t] ** 2)[~np.repeat(keep, g)]))
        return drop / float(np.sum(y ** 2))

    want = max(rel_drop(yk), rel_drop(yv))
    got = O.segment_loss(O.Params(), yk, yv, r, g)
    assert abs(got - want) <= 1e-5 * want


# ---------------------------------------------------------------- the close rule
def dyn_params(**kw):
    base = dict(dyn=True, rot_window=4096, tau_window=1.0, min_window=64)
    base.update(kw)
    return O.Params(**base)


def identity_closer(pr, w, a, b, k, v):
    pr.close(np.eye(D, dtype=np.float32), np.eye(D, dtype=np.float32), k[a:b], v[a:b])


def test_loss_close_every_two_segments():
    """All-ones tokens: every segment takes the fallback (48, 1), whose loss is
    80/128 = 0.625, so with a threshold of 1.0 the sum passes it at the second
    segment of each window: windows start at segments 0, 6, 8, 10, ... after a
    four-segment prefill whose window stays open."""
    P = dyn_params(tau_window=1.0, min_window=64)
    N = 1200
    k = to_bits(np.ones((N, D)))
    pr = O.Pair(P, N, eye_rot(1), eye_rot(1))
    pr.compress(k[:256], k[:256])
    assert pr.windows() == dict(nwin=1, pend=-1, wloss=0.0, wseg=[0])
    seen = drive(pr, k, k, lambda p, w, a, b: identity_closer(p, w, a, b, k, k), 256)
    w = pr.windows()
    assert w["wseg"] == [0, 6, 8, 10, 12, 14, 16, 18] and w["pend"] == -1     # segments 0..17 finalized
    assert [s[0] for s in seen] == list(range(len(seen)))
    assert seen[0][1:3] == (0, 384)
    assert all(s[2] == 128 for s in seen[1:])


def test_max_length_close_of_lossless_tokens():
    """One-hot tokens lose nothing: windows close only at the maximum length,
    rot_window tokens after their first one."""
    P = dyn_params(rot_window=512, tau_window=0.0, min_window=64)
    N = 2000
    x = np.zeros((N, D), np.float32)
    x[:, 0] = 1.0
    y = np.zeros((N, D), np.float32)
    y[:, 5] = 3.0
    k, v = to_bits(x), to_bits(y)
    pr = O.Pair(P, N, eye_rot(4), eye_rot(4))
    pr.compress(k[:100], v[:100])
    seen = drive(pr, k, v, lambda p, w, a, b: identity_closer(p, w, a, b, k, v), 100)
    w = pr.windows()
    assert w["wseg"] == [0, 8, 16, 24] and w["wloss"] == 0.0
    assert [s[1:3] for s in seen] == [(0, 512), (512, 512), (1024, 512)]


def test_min_window_holds_a_close():
    """Loss above the threshold after every segment, but a window must hold
    256 tokens first: after the prefill window (256 tokens already) closes at
    its first decode segment, windows close every four segments."""
    P = dyn_params(tau_window=0.5, min_window=256)
    N = 1300
    k = to_bits(np.ones((N, D)))
    pr = O.Pair(P, N, eye_rot(1), eye_rot(1))
    pr.compress(k[:256], k[:256])
    drive(pr, k, k, lambda p, w, a, b: identity_closer(p, w, a, b, k, k), 256)
    assert pr.windows()["wseg"][:5] == [0, 5, 9, 13, 17]


def test_prefill_windows_are_fixed_and_the_last_stays_open():
    P = dyn_params(rot_window=256, min_window=64)
    for L, want in ((0, [0]), (100, [0]), (256, [0, 4]), (600, [0, 4, 8]), (640, [0, 4, 8])):
        pr = O.Pair(P, 1000, eye_rot(4), eye_rot(4))
        k = to_bits(np.ones((L, D)))
        pr.compress(k, k)
        assert pr.windows()["wseg"] == want, L
        assert pr.windows()["pend"] == -1


def test_refused_append_changes_nothing():
    P = dyn_params(tau_window=1.0, min_window=64)
    N = 420
    k = to_bits(np.ones((N, D)))
    pr = O.Pair(P, N, eye_rot(1), eye_rot(1))
    pr.compress(k[:256], k[:256])
    for t in range(256, 415):
        assert pr.append_status(k[t], k[t]) == 0
    assert pr.windows()["pend"] == 0
    before = (pr.info().L, pr.token_arena().tobytes(), pr.score_arena().tobytes(), pr.descriptor_bytes().tobytes(),
              pr.buffer()[0].tobytes(), pr.staging()[0].tobytes())
    assert pr.append_status(k[415], k[415]) == -4
    after = (pr.info().L, pr.token_arena().tobytes(), pr.score_arena().tobytes(), pr.descriptor_bytes().tobytes(),
             pr.buffer()[0].tobytes(), pr.staging()[0].tobytes())
    assert before == after
    with pytest.raises(ValueError):
        O.Pair(P, N, eye_rot(1), eye_rot(1)).close(np.eye(D), np.eye(D), k[:64], k[:64])


# ---------------------------------------------------------------- the recompression of a closed window
def drifting_tokens(seed, N, drift=0.02):
    """Anisotropic tokens whose principal directions turn slowly: the energy
    scale of direction j decays with j, and the basis is rotated by a small
    rotation every token, so a window's rotation fits later tokens worse."""
    r = np.random.default_rng(seed)
    Q, _ = np.linalg.qr(r.standard_normal((D, D)))
    A = r.standard_normal((D, D)) * drift
    step, _ = np.linalg.qr(np.eye(D) + (A - A.T) / 2)
    scales = np.exp(-np.arange(D) / 12.0) * 4 + 0.05
    out = np.empty((N, D), np.float32)
    for t in range(N):
        out[t] = (r.standard_normal(D) * scales) @ Q.T
        if t % 16 == 15:
            Q = step @ Q
    return out


def test_close_equals_prefill_compression_of_the_window():
    """After a close, the closed window's records are those a fresh prefill of
    the window's tokens with the new rotation writes, moved to the window's
    offsets; its block numbering continues the earlier segments'."""
    P = dyn_params(tau_window=1.0, min_window=128, dtype="bf16")
    N = 1800
    xk, xv = drifting_tokens(1, N), drifting_tokens(2, N)
    k, v = to_bits(xk, "bf16"), to_bits(xv, "bf16")
    R0k, R0v = window_rotation(from_bits(k[:500], "bf16")), window_rotation(from_bits(v[:500], "bf16"))
    pr = O.Pair(P, N, R0k[None], R0v[None])
    pr.compress(k[:500], v[:500])
    checked = []

    def closer(p, w, a, b):
        desc_before = p.descriptors()
        base = desc_before[a // S]
        Rk, Rv = window_rotation(from_bits(k[a:b], "bf16")), window_rotation(from_bits(v[a:b], "bf16"))
        p.close(Rk, Rv, k[a:b], v[a:b])
        fresh = O.Pair(O.Params(dtype="bf16", rot_window=1 << 20), b - a, Rk[None], Rv[None])
        fresh.compress(k[a:b], v[a:b])
        fd = fresh.descriptors()
        d = p.descriptors()
        tok, sc, ftok, fsc = p.token_arena(), p.score_arena(), fresh.token_arena(), fresh.score_arena()
        for j, s in enumerate(range(a // S, b // S)):
            for key in ("r", "log2g", "log2b", "flags"):
                assert d[s][key] == fd[j][key], (s, key)
            assert d[s]["tok_off"] == base["tok_off"] + fd[j]["tok_off"]
            assert d[s]["sc_off"] == base["sc_off"] + fd[j]["sc_off"]
            assert d[s]["first_block"] == base["first_block"] + fd[j]["first_block"]
        assert np.array_equal(tok[base["tok_off"]:], ftok)
        assert np.array_equal(sc[base["sc_off"]:], fsc)
        checked.append((w, a, b))

    seen = drive(pr, k, v, closer, 500)
    assert len(checked) >= 2 and len(seen) == len(checked)
    # the drift makes later windows close on their loss, not at the maximum length
    assert all(b - a < P.rot_window for _, a, b in checked)


# ---------------------------------------------------------------- decode over the windows
def numpy_attention(q, k, v, scale, dtype="fp16"):
    qd, kd, vd = from_bits(q, dtype), from_bits(k, dtype), from_bits(v, dtype)
    z = (qd @ kd.T) * float(np.float32(scale))
    z = z - z.max(axis=1, keepdims=True)
    p = np.exp(z)
    return (p @ vd) / p.sum(axis=1, keepdims=True)


def test_signed_permutation_windows_decode_to_dense():
    """Keep everything, select everything, a fresh signed permutation for
    every window: decode equals dense attention exactly (in fp64) at every
    step, also while a closed window still holds its provisional encoding."""
    r = np.random.default_rng(5)
    G = 4
    P = O.Params(dyn=True, rot_window=256, tau_window=0.0, min_window=64, force_default=True,
                 default=(128, 1, 8), select=(1, 1))
    N = 1100
    k = to_bits(r.standard_normal((N, D)))
    v = to_bits(r.standard_normal((N, D)))
    q = to_bits(r.standard_normal((G, D)) * 2)
    pr = O.Pair(P, N, np.stack([signed_perm(r)]), np.stack([signed_perm(r)]))
    pr.compress(k[:300], v[:300])
    closes = 0
    for t in range(300, N):
        st = pr.append_status(k[t], v[t])
        if st == -4:
            w = pr.windows()
            out, _ = pr.decode(q, 0.125)
            assert np.max(np.abs(out - numpy_attention(q, k[:t], v[:t], 0.125))) < 1e-12
            a, b = w["wseg"][w["pend"]] * S, w["wseg"][w["pend"] + 1] * S
            pr.close(signed_perm(r), signed_perm(r), k[a:b], v[a:b])
            closes += 1
            assert pr.append_status(k[t], v[t]) == 0
        if t % 97 == 0:
            out, _ = pr.decode(q, 0.125)
            assert np.max(np.abs(out - numpy_attention(q, k[:t + 1], v[:t + 1], 0.125))) < 1e-12, t
    w = pr.windows()
    # the 300-token prefill fills window 0 (256 tokens) and opens window 1
    assert closes >= 3 and w["nwin"] == 2 + closes + (1 if w["pend"] >= 0 else 0)


def decode_records(pr, P, rk, rv, wseg, dtype):
    """Independent numpy decoder: every scoreable token's K and V from the
    packed records (bitmap of D/g bits LSB first, kept values ascending), back
    in the input space through its window's rotation (x = y . R)."""
    tok = pr.token_arena()
    ks, vs = [], []
    for s, d in enumerate(pr.descriptors()):
        w = max(i for i in range(len(wseg)) if wseg[i] <= s)
        r, g, B = d["r"], 1 << d["log2g"], 1 << d["log2b"]
        n = 32 if d["flags"] & 1 else S
        bmb, vb = D // g // 8, 2 * r
        off = d["tok_off"]
        for b0 in range(0, n, B):
            blk = tok[off + (b0 // B) * B * 2 * (bmb + vb):]
            for which, out, R in ((0, ks, rk[w]), (1, vs, rv[w])):
                base = which * B * (bmb + vb)
                for j in range(B):
                    bm = blk[base + j * bmb: base + (j + 1) * bmb]
                    vals = from_bits(blk[base + B * bmb + j * vb: base + B * bmb + (j + 1) * vb].view(np.uint16), dtype)
                    bits = np.unpackbits(bm, bitorder="little")[: D // g].astype(bool)
                    y = np.zeros(D)
                    y[np.repeat(bits, g)] = vals
                    out.append(y @ R.astype(np.float64))
    return np.array(ks).reshape(-1, D), np.array(vs).reshape(-1, D)


def test_decode_over_loss_closed_windows_matches_numpy_decoder():
    """Windows of irregular length (closed by their loss), each with its own
    rotation, every block selected: the oracle's decode (q rotated per window,
    output rotated back per window) equals numpy attention over the records
    decoded independently and rotated back token by token."""
    G = 4
    P = dyn_params(tau_window=1.5, min_window=128, select=(1, 1))
    N = 1500
    k = to_bits(drifting_tokens(7, N))
    v = to_bits(drifting_tokens(8, N))
    r = np.random.default_rng(9)
    q = to_bits(r.standard_normal((G, D)))
    R0k, R0v = window_rotation(from_bits(k[:400])), window_rotation(from_bits(v[:400]))
    rots = {0: (R0k, R0v)}

    def closer(p, w, a, b):
        Rk, Rv = window_rotation(from_bits(k[a:b])), window_rotation(from_bits(v[a:b]))
        rots[w] = rots[w + 1] = (Rk, Rv)
        p.close(Rk, Rv, k[a:b], v[a:b])

    pr = O.Pair(P, N, R0k[None], R0v[None])
    pr.compress(k[:400], v[:400])
    seen = drive(pr, k, v, closer, 400)
    lens = [s[2] for s in seen]
    assert len(seen) >= 3 and len(set(lens)) > 1 and all(n % S == 0 for n in lens)
    w = pr.windows()
    nwin = w["nwin"]
    for i in range(nwin):
        rots.setdefault(i, rots[max(j for j in rots if j <= i)])
    rk = [rots[i][0] for i in range(nwin)]
    rv = [rots[i][1] for i in range(nwin)]
    kd, vd = decode_records(pr, P, rk, rv, w["wseg"], "fp16")
    bk, bv = pr.buffer()
    kd = np.concatenate([kd, from_bits(bk)])
    vd = np.concatenate([vd, from_bits(bv)])
    qd = from_bits(q)
    z = (qd @ kd.T) * float(np.float32(0.125))
    z -= z.max(axis=1, keepdims=True)
    p = np.exp(z)
    want = (p @ vd) / p.sum(axis=1, keepdims=True)
    out, sel = pr.decode(q, 0.125)
    assert len(sel) == pr.info().nblk
    assert np.max(np.abs(out - want)) < 1e-9


# ---------------------------------------------------------------- the incremental covariance
def test_incremental_covariance_is_window_gram_matrix():
    """Integer tokens (every product and sum exact in fp64): at each close,
    the window's incrementally accumulated covariance equals X^T X of its raw
    tokens exactly -- the prefill part of the open window included (a prefill
    of two fixed windows plus a remainder), and the slot of the window before
    it untouched."""
    r = np.random.default_rng(21)
    P = dyn_params(rot_window=1024, tau_window=1.0, min_window=128)
    L0, N = 1100, 2600
    xk = r.integers(-4, 5, (N, D)).astype(np.float32)
    xv = r.integers(-4, 5, (N, D)).astype(np.float32)
    xk[:, :8] *= 3                                       # some structure: the first channels dominate
    k, v = to_bits(xk), to_bits(xv)
    pr = O.Pair(P, N, eye_rot(3), eye_rot(3))
    pr.compress(k[:L0], v[:L0])
    assert pr.windows()["wseg"] == [0, 16]               # window 1 holds tokens 1024..1087 so far
    ck, cv = pr.cov(1)
    assert np.array_equal(ck, xk[1024:1088].astype(np.float64).T @ xk[1024:1088].astype(np.float64))
    checked = []

    def closer(p, w, a, b):
        ck, cv = p.cov(w)
        X, Y = xk[a:b].astype(np.float64), xv[a:b].astype(np.float64)
        assert np.array_equal(ck, X.T @ X) and np.array_equal(cv, Y.T @ Y), (w, a, b)
        if w > 0:                                        # the previous window's slot is the other one
            pk, _ = p.cov(w - 1)
            assert not np.array_equal(pk, ck)
        identity_closer(p, w, a, b, k, v)
        checked.append((w, a, b))

    drive(pr, k, v, closer, L0)
    assert len(checked) >= 3 and checked[0][1] == 1024
