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
# Reading R-21 (the paper names the goal -- channels with similar selection
# patterns become neighbours -- not the procedure).  A token selects the r
# largest |y| of its rotated vector (lowest channel first on ties; y is the
# compressor's fp32 chain, oracle.rotate; x holds the 16-bit inputs as fp32).
# Over the window's tokens, n_c counts the tokens selecting channel c and
# C[i][j] the tokens selecting both i and j (C[c][c] = n_c).  Channels are
# placed in groups of four, the largest element group: a group starts with
# the unplaced channel of the largest n (lowest channel on ties), then takes
# three times the unplaced channel selected most often together with the
# group so far (largest sum of C over its members), then the larger n, then
# the lower channel.  Groups follow in the order formed, members in the order
# taken; rows of R follow.  Groups of 2 and 4 then hold channels selected
# together, and the least selected channels come last, where a truncation of
# the bitmap drops them.
def selection_masks(x, R, r):
    """x [n][D] fp32 (exact 16-bit values), R [D][D] fp32 -> bool [n][D]: each
    token's selected channels."""
    from oracle import oracle as O
    x = np.asarray(x, dtype=np.float32).reshape(-1, D)
    m = np.zeros((x.shape[0], D), dtype=bool)
    if x.shape[0] == 0:
        return m
    y = O.rotate(x, np.asarray(R, dtype=np.float32))
    order = np.argsort(-np.abs(y), axis=1, kind="stable")   # equal magnitudes keep ascending channels
    np.put_along_axis(m, order[:, :r], True, axis=1)
    return m


def selection_counts(x, R, r):
    """-> n [D] int64: tokens selecting each channel."""
    return selection_masks(x, R, r).sum(axis=0).astype(np.int64)


def coselection_counts(x, R, r):
    """-> C [D][D] int64: tokens selecting both channels (a library matmul of the
    0/1 selection matrix with itself)."""
    m = selection_masks(x, R, r).astype(np.int64)
    return m.T @ m


def reorder_order(C):
    """New row order from co-selection counts C [D][D] (groups of four, above)."""
    C = np.asarray(C, dtype=np.int64)
    n = np.diagonal(C)
    placed = np.zeros(D, dtype=bool)
    order = []
    while len(order) < D:
        gsum = np.zeros(D, dtype=np.int64)
        for _ in range(4):
            j = max((c for c in range(D) if not placed[c]), key=lambda c: (gsum[c], n[c], -c))
            order.append(j)
            placed[j] = True
            gsum += C[j]
    return np.array(order, dtype=np.int64)


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
            last = reorder_order(coselection_counts(x[a:b], R[w], r))
        orders[w] = last
        out[w] = R[w][last]
    return out, orders
