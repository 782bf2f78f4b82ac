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


# ---- selection-pattern channel reorder (Sec. 5.5) --------------------------
# Reading R-21 (the paper names the goal, not the procedure): channels are
# ordered by how often each is selected, i.e. among the r largest |y| of a
# token's rotated vector (lowest channel first on ties), over the window's
# tokens, most often first, lower current row first on equal counts; rows of R
# follow.  Channels selected alike become neighbours and the least selected
# come last, where a truncation of the bitmap drops them.  y is the
# compressor's fp32 chain (oracle.rotate); x holds the 16-bit inputs as fp32.
def selection_counts(x, R, r):
    """x [n][D] fp32 (exact 16-bit values), R [D][D] fp32 -> counts [D] int64."""
    from oracle import oracle as O
    x = np.asarray(x, dtype=np.float32).reshape(-1, D)
    counts = np.zeros(D, dtype=np.int64)
    if x.shape[0] == 0:
        return counts
    y = O.rotate(x, np.asarray(R, dtype=np.float32))
    order = np.argsort(-np.abs(y), axis=1, kind="stable")   # equal magnitudes keep ascending channels
    np.add.at(counts, order[:, :r].ravel(), 1)
    return counts


def reorder_order(counts):
    """New row order: descending count, ascending row on ties."""
    return np.argsort(-np.asarray(counts), kind="stable")


def reorder_rotations(x, L, W, R, r):
    """Rotations of one (sequence, kv head) reordered window by window: x [>= L][D]
    fp32, R [nw][D][D] fp32 -> (R' [nw][D][D], orders [nw][D]).  A window without
    tokens takes the order of the last window with tokens (identity before any)."""
    R = np.asarray(R, dtype=np.float32)
    nw = R.shape[0]
    out = np.empty_like(R)
    orders = np.empty((nw, D), dtype=np.int64)
    last = np.arange(D)
    for w in range(nw):
        a, b = w * W, min((w + 1) * W, L)
        if a < b:
            last = reorder_order(selection_counts(x[a:b], R[w], r))
        orders[w] = last
        out[w] = R[w][last]
    return out, orders
