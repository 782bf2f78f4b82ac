"""Oracle of the rotation matrices (SVD basis of each window's K or V matrix).

TEST INFRASTRUCTURE ONLY: imported by tests/ and bench.py's checks, never by
the product package; it shares no code with the HIP library.

The rotation of a window is the basis of right singular vectors of its K (or
V) matrix X (Sec. 2.3, Sec. 5.2: the rotation matrices are computed from the
KV cache once it exists): rows of R are the eigenvectors of X^T X, by
descending eigenvalue (= squared singular value), so that y = x . R^T puts
the most energetic directions first.  Readings (the paper does not fix them):
the covariance is uncentered (the rotation of Sec. 2.3 acts on raw vectors);
each row is signed so that its largest-magnitude component is positive (the
first such component on ties); a window with no token repeats the last
window that has one, and the identity stands before any.

Plain fp64: X^T X by numpy, eigenpairs by numpy.linalg.eigh.
"""
from __future__ import annotations

import numpy as np

D = 128


def signed_rows(vecs_as_rows: np.ndarray) -> np.ndarray:
    """Each row multiplied by the sign of its largest-magnitude component."""
    r = np.array(vecs_as_rows, dtype=np.float64, copy=True)
    idx = np.argmax(np.abs(r), axis=1)                      # first maximum on ties
    s = np.sign(r[np.arange(r.shape[0]), idx])
    s[s == 0] = 1.0
    return r * s[:, None]


def window_rotation(x: np.ndarray):
    """x [n][D] (any float type) -> (R [D][D] fp64 rows, eigenvalues [D] descending)."""
    X = np.asarray(x, dtype=np.float64)
    cov = X.T @ X
    evals, evecs = np.linalg.eigh(cov)                      # ascending
    order = np.argsort(-evals, kind="stable")
    return signed_rows(evecs[:, order].T), evals[order]


def rotations(x: np.ndarray, L: int, W: int, nw: int):
    """Rotations of every window of one (sequence, kv head): x [>= L][D] raw
    vectors, L tokens, window W, nw windows -> (R [nw][D][D], evals [nw][D])."""
    R = np.empty((nw, D, D))
    ev = np.zeros((nw, D))
    last = None
    for w in range(nw):
        a, b = w * W, min((w + 1) * W, L)
        if a < b:
            last = window_rotation(x[a:b])
        if last is None:
            R[w], ev[w] = np.eye(D), 0.0
        else:
            R[w], ev[w] = last
    return R, ev
