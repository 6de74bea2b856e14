"""Sylvester Hadamard matrix and the online block rotation (oracle; test-only).

Follows sec. 3.2 of OffQ: an orthogonal +/-1 matrix whose first row is all ones
(offsetting technique), applied as ``X_had = X_rot H / sqrt(D)`` (Eq. 4), and
the group-wise variant that applies it independently inside contiguous groups
of ``g`` channels (sec. 3.2, "Group-Wise Offsetting").  Reading: the Sylvester
construction ``H_1 = [1]``, ``H_2n = [[H_n, H_n], [H_n, -H_n]]``, whose first row
and column are all ones; any sign randomisation of the "partially random"
matrix is fused into upstream weights offline and is not part of the online
path.
"""

import numpy as np


def sylvester(n):
    """Return the n x n Sylvester Hadamard matrix (int64), n a power of two."""
    if n < 1 or n & (n - 1):
        raise ValueError("n must be a power of two")
    h = np.ones((1, 1), dtype=np.int64)
    while h.shape[0] < n:
        h = np.block([[h, h], [h, -h]])
    return h


def fwht(x):
    """Unnormalised Walsh-Hadamard transform along the last axis, in fp64.

    ``fwht(x) == x @ sylvester(n)`` (H is symmetric), computed with the same
    recursion that defines the matrix: split the last axis in halves ``a, b``
    and return ``[T(a) + T(b), T(a) - T(b)]``.
    """
    x = np.asarray(x, dtype=np.float64)
    n = x.shape[-1]
    if n & (n - 1):
        raise ValueError("length must be a power of two")
    if n == 1:
        return x.copy()
    a = fwht(x[..., : n // 2])
    b = fwht(x[..., n // 2:])
    return np.concatenate([a + b, a - b], axis=-1)


def rotate(x, g):
    """Block-diagonal online rotation ``y = x (I_{K/g} (x) H_g) / sqrt(g)`` in fp64.

    ``x``: [..., K] with K a multiple of ``g``; groups are contiguous channel
    blocks ``[b*g, (b+1)*g)`` (sec. 3.2, group-wise offsetting: the first
    channel of each group is the one turned into a constant offset).
    """
    x = np.asarray(x, dtype=np.float64)
    K = x.shape[-1]
    if K % g:
        raise ValueError("K must be a multiple of g")
    xb = x.reshape(x.shape[:-1] + (K // g, g))
    y = fwht(xb) / np.sqrt(np.float64(g))
    return y.reshape(x.shape)


def offset(x, g):
    """The constant offset each group receives: ``x[..., b*g] / sqrt(g)``.

    Sec. 3.2 / Eq. 5: the first channel of a group is spread uniformly over all
    channels of that group as ``x_1 / sqrt(D)``.  Returns [..., K/g] in fp64.
    """
    x = np.asarray(x, dtype=np.float64)
    K = x.shape[-1]
    return x[..., ::g][..., : K // g] / np.sqrt(np.float64(g))
