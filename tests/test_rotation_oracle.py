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
