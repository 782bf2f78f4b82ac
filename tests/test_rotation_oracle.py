"""Pins of the rotation oracle (oracle/rotation.py) against closed forms and an
independent library route (singular value decomposition), CPU only."""
import numpy as np

from oracle import rotation as RO

D = 128


def test_diagonal_covariance_gives_sorted_permutation():
    # one row per channel, channel c scaled by s_c: X^T X = diag(s_c^2) exactly
    rng = np.random.default_rng(1)
    s = rng.permutation(np.arange(1, D + 1, dtype=np.float64)) * 0.5
    X = np.diag(s)
    R, ev = RO.window_rotation(X)
    order = np.argsort(-s ** 2, kind="stable")
    want = np.zeros((D, D))
    want[np.arange(D), order] = 1.0
    assert np.array_equal(R, want)
    assert np.allclose(ev, (s ** 2)[order], rtol=0, atol=1e-9)


def test_known_eigenbasis_is_recovered():
    rng = np.random.default_rng(2)
    Q, _ = np.linalg.qr(rng.standard_normal((D, D)))
    lam = np.sort(rng.uniform(1.0, 100.0, D))[::-1] + np.arange(D)[::-1] * 0.5   # distinct, descending
    X = np.diag(np.sqrt(lam)) @ Q.T                        # X^T X = Q diag(lam) Q^T
    R, ev = RO.window_rotation(X)
    assert np.allclose(ev, lam, rtol=1e-10, atol=0)
    want = RO.signed_rows(Q.T)                             # rows = eigenvectors in lam order
    assert np.allclose(R, want, atol=1e-8)
    # the sign rule: every row's largest-magnitude component is positive
    assert np.all(R[np.arange(D), np.argmax(np.abs(R), axis=1)] > 0)


def test_matches_singular_value_decomposition():
    rng = np.random.default_rng(3)
    X = rng.standard_normal((300, D)) * np.linspace(3.0, 0.5, D)[None, :]
    R, ev = RO.window_rotation(X)
    _, sv, vt = np.linalg.svd(X, full_matrices=False)
    assert np.allclose(ev, sv ** 2, rtol=1e-9)
    assert np.allclose(R, RO.signed_rows(vt), atol=1e-8)
    # invariants: orthonormal rows, diagonalizes X^T X in descending order
    assert np.allclose(R @ R.T, np.eye(D), atol=1e-12)
    C = R @ (X.T @ X) @ R.T
    assert np.allclose(C - np.diag(np.diag(C)), 0.0, atol=1e-8 * ev[0])
    assert np.all(np.diff(np.diag(C)) <= 1e-9 * ev[0])


def test_uncentered():
    # a constant offset is a direction of its own: centering would remove it
    X = np.ones((10, D)) * 3.0
    R, ev = RO.window_rotation(X)
    assert np.isclose(ev[0], 9.0 * 10 * D)
    assert np.allclose(R[0], np.full(D, 1.0 / np.sqrt(D)), atol=1e-12)


def test_windows_repeat_the_last_one_with_tokens():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((2500, D))
    R, ev = RO.rotations(x, 2500, 1024, 4)
    for w, (a, b) in enumerate([(0, 1024), (1024, 2048), (2048, 2500)]):
        Rw, ew = RO.window_rotation(x[a:b])
        assert np.array_equal(R[w], Rw) and np.array_equal(ev[w], ew)
    assert np.array_equal(R[3], R[2]) and np.array_equal(ev[3], ev[2])
    R0, ev0 = RO.rotations(x, 0, 1024, 2)
    assert np.array_equal(R0[0], np.eye(D)) and np.array_equal(R0[1], np.eye(D)) and not ev0.any()


# ---- selection-pattern reorder (reading R-21) -------------------------------
def test_selection_counts_brute_force():
    """Counts against a plain per-token loop: sorted by (-|y|, channel) on a
    signed-permutation rotation (exact in fp32), with planted ties."""
    rng = np.random.default_rng(5)
    n, r = 200, 32
    x = np.round(rng.standard_normal((n, D)) * 4) / 4          # quarter steps: many equal magnitudes
    perm = rng.permutation(D)
    sgn = rng.choice([-1.0, 1.0], D)
    R = np.zeros((D, D))
    R[np.arange(D), perm] = sgn                                # y_j = sgn_j x_perm(j), exact
    want = np.zeros(D, dtype=np.int64)
    for t in range(n):
        y = [sgn[j] * x[t, perm[j]] for j in range(D)]
        for j in sorted(range(D), key=lambda j: (-abs(y[j]), j))[:r]:
            want[j] += 1
    got = RO.selection_counts(x, R, r)
    assert np.array_equal(got, want) and got.sum() == n * r


def test_coselection_counts_brute_force():
    """Co-selection counts against a per-token loop over the selected pairs,
    on the same exact signed-permutation rotation with ties; the diagonal is
    the selection count."""
    rng = np.random.default_rng(15)
    n, r = 120, 24
    x = np.round(rng.standard_normal((n, D)) * 4) / 4
    R = np.zeros((D, D))
    R[np.arange(D), rng.permutation(D)] = rng.choice([-1.0, 1.0], D)
    want = np.zeros((D, D), dtype=np.int64)
    for t in range(n):
        y = R @ x[t]
        sel = sorted(range(D), key=lambda j: (-abs(y[j]), j))[:r]
        for i in sel:
            for j in sel:
                want[i, j] += 1
    got = RO.coselection_counts(x, R, r)
    assert np.array_equal(got, want)
    assert np.array_equal(np.diagonal(got), RO.selection_counts(x, R, r))


def _feature_tokens(n, rng, scales=None, signs=False):
    """Token t activates features t, t+5, t+11, t+19 (mod 32); feature f is
    channels f, f+32, f+64, f+96, all active together.  Every channel is
    selected equally often (identity rotation, r = 16), so only co-selection
    tells the features apart."""
    x = np.zeros((n, D))
    s = np.ones(D) if scales is None else scales
    for t in range(n):
        for f in (t % 32, (t + 5) % 32, (t + 11) % 32, (t + 19) % 32):
            for c in (f, f + 32, f + 64, f + 96):
                x[t, c] = s[c] * (rng.choice([-1.0, 1.0]) if signs else 1.0)
    return x


def test_reorder_groups_coselected_channels():
    """Equal selection counts: an order by count alone keeps the identity (and
    groups of four would mix four features); the co-selection groups are the
    features, lowest channel first: 0, 32, 64, 96, 1, 33, ..."""
    rng = np.random.default_rng(16)
    x = _feature_tokens(256, rng)
    C = RO.coselection_counts(x, np.eye(D), 16)
    n = np.diagonal(C)
    assert np.all(n == n[0])                                  # every channel selected equally often
    order = RO.reorder_order(C)
    assert np.array_equal(order, np.array([f + 32 * k for f in range(32) for k in range(4)]))


def test_reorder_order_seeds_and_tie_rules():
    """Hand-made counts: the first group starts at the most selected channel;
    a partner is the channel most co-selected with the whole group so far,
    then the more selected, then the lower; the last groups take what is left
    in index order when nothing else is co-selected."""
    C = np.zeros((D, D), dtype=np.int64)
    n = np.zeros(D, dtype=np.int64)
    n[10], n[20], n[30], n[40], n[50] = 9, 5, 5, 4, 3
    C[np.arange(D), np.arange(D)] = n
    def co(i, j, v):
        C[i, j] = C[j, i] = v
    co(10, 20, 3); co(10, 30, 3)                               # tie on C with 10: both n = 5 -> lower (20)
    co(20, 50, 2); co(10, 50, 1)                               # with {10, 20}: 50 has 3, 30 has 3 -> larger n (30)
    co(40, 50, 1)
    order = RO.reorder_order(C)
    assert order[:4].tolist() == [10, 20, 30, 50]
    assert order[4:8].tolist() == [40, 0, 1, 2]                # 40 is the most selected left; then index order
    assert np.array_equal(np.sort(order), np.arange(D))


def test_coselection_reorder_moves_the_ratio():
    """Features with random signs and scales, under a rotation (an exact
    signed permutation) that scatters each feature's channels: no group of 4
    or 2 holds a feature, and the strategy search keeps single channels,
    (16, 1); after the co-selection reorder each feature is one aligned group
    and (16, 4) holds it losslessly, with a quarter of the bitmap bytes.  The
    memory ratio rises (an order by selection count alone keeps the scattered
    order here: every channel is selected equally often)."""
    from oracle import oracle as O
    rng = np.random.default_rng(17)
    L = 1024
    x = _feature_tokens(L, rng, scales=rng.uniform(1.0, 2.0, D), signs=True)
    xb = O.f32_to_f16_bits(x).reshape(L, D)
    xf = O.f16_bits_to_f32(xb).reshape(L, D)
    R = np.zeros((D, D), np.float32)
    R[np.arange(D), rng.permutation(D)] = rng.choice([-1.0, 1.0], D)
    Rco, orders = RO.reorder_rotations(xf, L, L, R[None], 16)
    P = O.Params(rot_window=L, default=(16, 4, 8))
    used = {}
    for name, Rw in (("given", R[None]), ("coselection", Rco)):
        pr = O.Pair(P, L, Rw, Rw)
        pr.compress(xb, xb)
        used[name] = pr.info().used_bytes
        used[name + "_rg"] = sorted({(d["r"], 1 << d["log2g"]) for d in pr.descriptors()})
    assert used["given_rg"] == [(16, 1)] and used["coselection_rg"] == [(16, 4)], used
    assert used["coselection"] < 0.8 * used["given"], used
