"""Exact integer GEMM of 4-bit codes and the dequantising epilogue (oracle; test-only).

From Eq. 1: an activation is reconstructed as x_hat = s_{m,b} (q_a - z_{m,b})
(per row m and group b) and a weight as w_hat = sw_n q_w (symmetric, per
output channel).  Hence

    sum_k x_hat[m,k] w_hat[n,k]
        = sw_n * sum_b s_{m,b} * (acc_b[m,n] - z_{m,b} * colsum_b[n]),
    acc_b[m,n]  = sum_{k in b} q_a[m,k] q_w[n,k]   (exact integers),
    colsum_b[n] = sum_{k in b} q_w[n,k].

The integer products use float64 BLAS: every partial sum is an integer of
magnitude <= g * 15 * 8 < 2^53, so any summation order is exact.
"""

import numpy as np


def int_gemm_groups(q_a, q_w, g):
    """acc[b, m, n] = sum_{k in group b} q_a[m,k] * q_w[n,k]  (int64 [G, M, N])."""
    q_a = np.asarray(q_a)
    q_w = np.asarray(q_w)
    M, K = q_a.shape
    N, K2 = q_w.shape
    if K != K2 or K % g:
        raise ValueError("shape mismatch")
    G = K // g
    acc = np.empty((G, M, N), dtype=np.int64)
    for b in range(G):
        a = q_a[:, b * g:(b + 1) * g].astype(np.float64)
        w = q_w[:, b * g:(b + 1) * g].astype(np.float64)
        acc[b] = np.rint(a @ w.T).astype(np.int64)
    return acc


def int_gemm_bruteforce(q_a, q_w, g):
    """Same as ``int_gemm_groups`` with explicit int64 loops (tiny shapes only)."""
    q_a = np.asarray(q_a).astype(np.int64)
    q_w = np.asarray(q_w).astype(np.int64)
    M, K = q_a.shape
    N = q_w.shape[0]
    G = K // g
    acc = np.zeros((G, M, N), dtype=np.int64)
    for b in range(G):
        for m in range(M):
            for n in range(N):
                t = 0
                for k in range(b * g, (b + 1) * g):
                    t += int(q_a[m, k]) * int(q_w[n, k])
                acc[b, m, n] = t
    return acc


def epilogue(acc, a_scale, a_zero, w_scale, w_colsum):
    """Y[m,n] = sw_n * sum_b s_{m,b} (acc_b[m,n] - z_{m,b} colsum_b[n])  in fp64.

    acc [G, M, N] ints; a_scale [M, G] (fp16 values); a_zero [M, G];
    w_scale [N] (fp16 values); w_colsum [G, N].
    """
    acc = np.asarray(acc).astype(np.float64)
    s = np.asarray(a_scale).astype(np.float64)            # [M, G]
    z = np.asarray(a_zero).astype(np.float64)             # [M, G]
    sw = np.asarray(w_scale).astype(np.float64)           # [N]
    cs = np.asarray(w_colsum).astype(np.float64)          # [G, N]
    G = acc.shape[0]
    y = np.zeros(acc.shape[1:], dtype=np.float64)
    for b in range(G):
        y += s[:, b:b + 1] * (acc[b] - z[:, b:b + 1] * cs[b][None, :])
    return y * sw[None, :]


def epilogue_magnitude(acc, a_scale, a_zero, w_scale, w_colsum):
    """E[m,n] = |sw_n| * sum_b |s_{m,b} (acc_b - z_{m,b} colsum_b)|  (fp64).

    The size of the terms the epilogue adds; an fp32 fold of G terms has an
    absolute error bounded by a small multiple of 2^-24 * E (used as the
    cancellation floor of the output tolerance).
    """
    acc = np.asarray(acc).astype(np.float64)
    s = np.asarray(a_scale).astype(np.float64)
    z = np.asarray(a_zero).astype(np.float64)
    sw = np.asarray(w_scale).astype(np.float64)
    cs = np.asarray(w_colsum).astype(np.float64)
    e = np.zeros(acc.shape[1:], dtype=np.float64)
    for b in range(acc.shape[0]):
        e += np.abs(s[:, b:b + 1] * (acc[b] - z[:, b:b + 1] * cs[b][None, :]))
    return e * np.abs(sw)[None, :]


def dequant_matmul(q_a, a_scale, a_zero, q_w, w_scale, g):
    """Brute-force reference: (s (q_a - z)) @ (sw q_w)^T in fp64."""
    q_a = np.asarray(q_a).astype(np.float64)
    M, K = q_a.shape
    G = K // g
    s = np.repeat(np.asarray(a_scale).astype(np.float64), g, axis=1)
    z = np.repeat(np.asarray(a_zero).astype(np.float64), g, axis=1)
    xa = s * (q_a - z)
    wq = np.asarray(q_w).astype(np.float64) * np.asarray(w_scale).astype(np.float64)[:, None]
    assert G * g == K
    return xa @ wq.T


def bf16_round(x):
    """Round fp64 values to bfloat16 (round-to-nearest-even), returned as fp64."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    u = (u + 0x7FFF + lsb) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def bf16_ulp(x):
    """Unit in the last place of bfloat16 at |x| (fp64)."""
    a = np.abs(np.asarray(x, dtype=np.float64))
    a = np.maximum(a, 2.0 ** -126)
    e = np.floor(np.log2(a))
    return 2.0 ** (e - 7)
