"""Offline calibration (oracle; test-only).

* top-1 selection (sec. 3.1 "Top-1 PCA" and "Why the L-infinity norm"): per
  calibration sequence, the token with the largest L-infinity norm;
* C = X^T X / N and its eigendecomposition with eigenvalues descending
  (Eq. 2); the leading eigenvector is the outlier direction, and X U moves it
  onto the first channel (sec. 3.1 "Concentrate Outliers");
* sorted grouping (sec. 3.2 "Group-Wise Offsetting", sec. 4.3 "Sorted versus
  Zigzag Grouping"): the G largest channels lead the G groups in descending
  order, the others fill the groups in ascending order;
* the rotation R = U P blockdiag(H_g / sqrt(g)) fused into the weights
  (sec. 3.3 step 2(1)), and P4 as a row permutation of the producing weights
  (step 2(4)).

Readings: ties in the top-1 selection go to the first token; ties in sorting
go to the lower channel index; eigenvectors are signed so that their entry
of largest magnitude (first on ties) is positive; the statistic that orders
the channels is the eigenvalue (the variance of the rotated channel) for P1
and the per-channel maximum magnitude for P4.  The eigendecomposition is
LAPACK's (numpy.linalg.eigh) in fp64.
"""

import numpy as np

from . import hadamard


def top1_select(x):
    """x: [n_seq, L, D] -> (idx [n_seq], X fp64 [n_seq, D])."""
    x = np.asarray(x, dtype=np.float64)
    linf = np.abs(x).max(axis=-1)              # [n_seq, L]
    idx = linf.argmax(axis=-1)                 # first maximum
    return idx.astype(np.int32), x[np.arange(x.shape[0]), idx].copy()


def channel_absmax(x):
    """x: [rows, D] -> fp64 [D] = max over rows of |x|."""
    return np.abs(np.asarray(x, dtype=np.float64)).max(axis=0)


def gram(X):
    """C = X^T X / N in fp64 (Eq. 2, zero-mean activations assumed)."""
    X = np.asarray(X, dtype=np.float64)
    return X.T @ X / X.shape[0]


def sign_fix(U):
    """Sign each column so that its entry of largest magnitude is positive."""
    U = np.array(U, dtype=np.float64)
    piv = np.abs(U).argmax(axis=0)
    s = np.where(U[piv, np.arange(U.shape[1])] < 0, -1.0, 1.0)
    return U * s


def eigh_desc(C):
    """Eigenvalues descending and eigenvectors (columns), signed as above."""
    w, V = np.linalg.eigh(np.asarray(C, dtype=np.float64))
    order = np.argsort(-w, kind="stable")
    return w[order], sign_fix(V[:, order])


def desc_order(key):
    """Indices by descending key, ties by lower index."""
    key = np.asarray(key, dtype=np.float64)
    return np.lexsort((np.arange(key.size), -key))


def group_permutation(key, g):
    """perm[new slot] = original channel: sorted grouping with G = D / g groups."""
    key = np.asarray(key, dtype=np.float64)
    D = key.size
    if D % g:
        raise ValueError("D must be a multiple of g")
    G = D // g
    order = desc_order(key)
    heads, rest = order[:G], order[G:]
    rest = rest[np.lexsort((rest, key[rest]))]  # ascending, ties by index
    perm = np.empty(D, dtype=np.int32)
    for b in range(G):
        perm[b * g] = heads[b]
        perm[b * g + 1:(b + 1) * g] = rest[b * (g - 1):(b + 1) * (g - 1)]
    return perm


def build_rotation(U, D, perm=None, g=1, apply_hadamard=False):
    """R = U P blockdiag(H_g / sqrt(g)) in fp64 (U None: identity)."""
    M = np.eye(D) if U is None else np.asarray(U, dtype=np.float64)
    if perm is not None:
        M = M[:, np.asarray(perm)]
    if apply_hadamard:
        M = hadamard.rotate(M, g)  # rows times blockdiag(H_g) / sqrt(g)
    return M


def fuse_weights(W, R):
    """W R: the weights of a layer whose input is rotated by R."""
    return np.asarray(W, dtype=np.float64) @ np.asarray(R, dtype=np.float64)


def permute_rows(W, perm):
    return np.asarray(W)[np.asarray(perm)]


def calibrate_rotation(x_calib, g):
    """The top-1 PCA rotation of one linear-layer input (U1 P1 H1): returns
    (idx, X, C, evals, U, perm, R)."""
    idx, X = top1_select(x_calib)
    C = gram(X)
    w, U = eigh_desc(C)
    perm = group_permutation(w, g)
    R = build_rotation(U, U.shape[0], perm, g, True)
    return idx, X, C, w, U, perm, R
