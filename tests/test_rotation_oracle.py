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


def test_reorder_planted_frequencies():
    """Identity rotation, channel c planted large in a known number of tokens:
    the order is by descending planted count, ascending channel on ties."""
    rng = np.random.default_rng(6)
    r = 16
    freq = rng.integers(0, 40, D)
    freq[:r] = 50                                             # r channels planted in every token
    n = 50
    x = np.zeros((n, D))
    for t in range(n):
        big = [c for c in range(D) if t < freq[c]][:r]          # the first r channels planted at t
        x[t, big] = 1.0 + 0.001 * np.arange(len(big))[::-1]
    counts = RO.selection_counts(x, np.eye(D), r)
    want = np.zeros(D, dtype=np.int64)
    for t in range(n):
        big = [c for c in range(D) if t < freq[c]][:r]
        if len(big) < r:                                      # the rest are zeros: lowest channels fill in
            big += [c for c in range(D) if c not in big][: r - len(big)]
        want[big] += 1
    assert np.array_equal(counts, want)
    order = RO.reorder_order(counts)
    assert np.array_equal(order, np.array(sorted(range(D), key=lambda c: (-want[c], c))))


def test_reorder_invariants_and_degenerate_cases():
    rng = np.random.default_rng(7)
    x = rng.standard_normal((700, D)).astype(np.float32)
    Q, _ = np.linalg.qr(rng.standard_normal((D, D)))
    R = np.stack([Q, Q.T, Q]).astype(np.float32)
    Rp, orders = RO.reorder_rotations(x, 700, 256, R, 32)
    for w in range(3):
        assert np.array_equal(np.sort(orders[w]), np.arange(D))   # a permutation
        assert np.array_equal(Rp[w], R[w][orders[w]])             # of the rows
        a, b = w * 256, min((w + 1) * 256, 700)
        c = RO.selection_counts(x[a:b], R[w], 32)[orders[w]]
        assert np.all(np.diff(c) <= 0)                            # counts descend along the new order
    # keeping every channel: equal counts, identity order
    Rall, oall = RO.reorder_rotations(x, 700, 256, R, D)
    assert np.array_equal(oall, np.tile(np.arange(D), (3, 1))) and np.array_equal(Rall, R)
    # windows past the last token take the last order; no tokens at all: identity
    R4 = np.stack([Q, Q.T, Q, Q]).astype(np.float32)
    R4p, o4 = RO.reorder_rotations(x, 300, 256, R4, 32)
    assert np.array_equal(o4[2], o4[1]) and np.array_equal(o4[3], o4[1])
    R0p, o0 = RO.reorder_rotations(x, 0, 256, R4, 32)
    assert np.array_equal(R0p, R4)
