"""GPU parity: offline calibration (offq_top1_select, offq_channel_absmax,
offq_gram, offq_eigh, offq_group_permutation, offq_build_rotation,
offq_fuse_weights, offq_permute_rows) against oracle/calibration.py.

Bars: selections, permutations, gathers and maxima bit-exact; the fp64
covariance within a summation bound; eigenvalues within 1e-10 of the
largest; eigenvectors of eigenvalues separated from their neighbours equal
to the oracle's (same sign convention) within 1e-8, every eigenvector with a
residual |C u - lambda u| below 1e-9 |C| and U orthogonal to 1e-10 (several
bases are correct inside a degenerate eigenspace, e.g. the null space when
N < D); rotations and fused weights within fp32 rounding bounds.
"""
import math

import numpy as np
import pytest
import torch

import paper_2606_07116_amd as offq
from oracle import calibration as OC
from paper_2606_07116_amd import inputs
from tests import parity as P

pytestmark = pytest.mark.gpu


def _calib_acts(n_seq, L, D, seed, n_dirs=1):
    """Calibration activations with outlier tokens along shared directions."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((n_seq, L, D)).astype(np.float32)
    for _ in range(n_dirs):
        d = rng.standard_normal(D)
        d /= np.linalg.norm(d)
        t = rng.integers(0, L, n_seq)
        x[np.arange(n_seq), t] += (rng.uniform(20, 60, (n_seq, 1)) * d).astype(np.float32)
    return inputs.round_to_bf16(x)


@pytest.mark.parametrize("n_seq,L,D", [(8, 300, 4096), (3, 1, 8), (16, 64, 1024)])
def test_top1_select_and_absmax(n_seq, L, D):
    x = _calib_acts(n_seq, L, D, seed=D + L)
    xd = P.to_dev_bf16(x.reshape(-1, D)).reshape(n_seq, L, D)
    idx, X = offq.offq_top1_select(xd)
    am = offq.offq_channel_absmax(xd.reshape(-1, D))
    torch.cuda.synchronize()
    idx_ref, X_ref = OC.top1_select(x)
    assert np.array_equal(P.host(idx), idx_ref)
    assert np.array_equal(P.host(X), X_ref)
    assert np.array_equal(P.host(am), OC.channel_absmax(x.reshape(-1, D)))


def test_top1_select_strided_sequences():
    n_seq, L, D = 4, 20, 64
    x = _calib_acts(n_seq, 2 * L, D, seed=2)           # take every other token
    xd = P.to_dev_bf16(x.reshape(-1, D)).reshape(n_seq, 2 * L, D)[:, ::2]
    idx, X = offq.offq_top1_select(xd)
    torch.cuda.synchronize()
    idx_ref, X_ref = OC.top1_select(x[:, ::2])
    assert np.array_equal(P.host(idx), idx_ref) and np.array_equal(P.host(X), X_ref)


@pytest.mark.parametrize("N,D", [(128, 1024), (37, 100), (300, 64)])
def test_gram(N, D):
    X = np.random.default_rng(N).standard_normal((N, D)).astype(np.float32)
    C = P.host(offq.offq_gram(torch.from_numpy(X).to(P.DEV)))
    C_ref = OC.gram(X)
    assert np.array_equal(C, C.T)
    a = np.abs(X.astype(np.float64))
    bound = (N + 2) * 2.0 ** -53 * (a.T @ a) / N
    assert np.all(np.abs(C - C_ref) <= bound + 1e-300)


def _check_eig(C, ev, U, gap_tol=1e-6):
    w_ref, U_ref = OC.eigh_desc(C)
    D = C.shape[0]
    scale = np.abs(w_ref).max()
    assert np.all(np.abs(ev - w_ref) <= 1e-10 * scale)
    assert np.all(np.diff(ev) <= 0)
    res = np.linalg.norm(C @ U - U * ev[None, :], axis=0)
    assert np.all(res <= 1e-9 * np.linalg.norm(C)), res.max()
    assert np.abs(U.T @ U - np.eye(D)).max() <= 1e-10
    gaps = np.minimum(np.r_[np.inf, -np.diff(w_ref)], np.r_[-np.diff(w_ref), np.inf])
    sep = gaps > gap_tol * scale
    assert np.abs(U[:, sep] - U_ref[:, sep]).max(initial=0.0) <= 1e-8
    return sep.sum()


@pytest.mark.parametrize("D,N", [(64, 200), (256, 64), (1024, 256), (130, 300), (2, 5)])
def test_eigh(D, N):
    x = _calib_acts(N, 1, D, seed=D, n_dirs=3).reshape(N, D)
    C = OC.gram(x)
    ev, U, sweeps, rel = offq.offq_eigh(torch.from_numpy(C).to(P.DEV))
    torch.cuda.synchronize()
    assert rel <= D * 2.0 ** -52 and sweeps < 30
    n_sep = _check_eig(C, P.host(ev), P.host(U))
    assert n_sep >= min(N, D) // 2  # most eigenvectors are compared one by one


def test_eigh_closed_forms():
    D = 16
    v = np.arange(1.0, D + 1)
    C = np.outer(v, v) + np.diag(np.linspace(0.0, 1.0, D))
    ev, U, _, _ = offq.offq_eigh(torch.from_numpy(C).to(P.DEV))
    torch.cuda.synchronize()
    _check_eig(C, P.host(ev), P.host(U))
    # a diagonal matrix is already converged: zero sweeps, sorted diagonal
    Dg = np.diag(np.array([3.0, -1.0, 7.0, 0.5]))
    ev, U, sweeps, _ = offq.offq_eigh(torch.from_numpy(Dg).to(P.DEV))
    torch.cuda.synchronize()
    assert sweeps == 0 and np.array_equal(P.host(ev), [7.0, 3.0, 0.5, -1.0])
    assert np.array_equal(np.abs(P.host(U)), np.eye(4)[:, [2, 0, 3, 1]])


@pytest.mark.parametrize("D,g", [(6, 3), (4096, 128), (1024, 1024), (512, 1)])
def test_group_permutation(D, g):
    rng = np.random.default_rng(D + g)
    key = np.round(rng.standard_normal(D), 2) if D > 6 else np.array([1.0, 2, 3, 4, 50, 60])
    perm = P.host(offq.offq_group_permutation(torch.from_numpy(key).to(P.DEV), g))
    torch.cuda.synchronize()
    assert np.array_equal(perm, OC.group_permutation(key, g))


@pytest.mark.parametrize("D,g,had,use_u,use_p", [(256, 64, True, True, True), (128, 128, True, False, True),
                                                 (512, 16, False, True, False), (64, 8, True, False, False)])
def test_build_rotation(D, g, had, use_u, use_p):
    rng = np.random.default_rng(D)
    U = np.ascontiguousarray(OC.eigh_desc(OC.gram(rng.standard_normal((D + 5, D))))[1]) if use_u else None
    perm = OC.group_permutation(rng.standard_normal(D), g) if use_p else None
    R = offq.offq_build_rotation(torch.from_numpy(U).to(P.DEV) if use_u else None, D,
                                 torch.from_numpy(perm).to(P.DEV) if use_p else None, g, had)
    torch.cuda.synchronize()
    R_ref = OC.build_rotation(U, D, perm, g, had)
    got = P.host(R).astype(np.float64)
    # fp64 butterflies (log2 g stages) rounded once to fp32
    bound = 2.0 ** -23 * np.abs(R_ref) + 1e-13
    assert np.all(np.abs(got - R_ref) <= bound)


@pytest.mark.parametrize("N,K", [(300, 512), (64, 128), (1000, 96)])
def test_fuse_and_permute_weights(N, K):
    rng = np.random.default_rng(N + K)
    W = rng.standard_normal((N, K)).astype(np.float32)
    R = np.ascontiguousarray(
        OC.build_rotation(OC.eigh_desc(OC.gram(rng.standard_normal((K + 1, K))))[1], K), dtype=np.float32)
    Wd = torch.from_numpy(W).to(P.DEV)
    Wf = P.host(offq.offq_fuse_weights(Wd, torch.from_numpy(R).to(P.DEV)))
    perm = rng.permutation(N).astype(np.int32)
    Wp = P.host(offq.offq_permute_rows(Wd, torch.from_numpy(perm).to(P.DEV)))
    torch.cuda.synchronize()
    ref = OC.fuse_weights(W, R)
    bound = (K + 2) * 2.0 ** -24 * (np.abs(W.astype(np.float64)) @ np.abs(R.astype(np.float64)))
    assert np.all(np.abs(Wf - ref) <= bound)
    assert np.array_equal(Wp, OC.permute_rows(W, perm))


def test_calibration_pipeline_moves_the_outlier_to_the_group_heads():
    """top-1 selection -> covariance -> eigh -> grouping -> rotation on the GPU
    for one 512-channel layer input with one shared outlier direction: the
    selected tokens and the group heads match the oracle, the rest of the
    permutation is the oracle's grouping of the GPU's eigenvalues (the order
    inside the null space of C is not unique), and after R the outlier is the
    per-token offset of group 0 (sec. 3.1, sec. 3.2)."""
    n_seq, L, D, g = 64, 40, 512, 128
    x = _calib_acts(n_seq, L, D, seed=11)
    xd = P.to_dev_bf16(x.reshape(-1, D)).reshape(n_seq, L, D)
    idx, X = offq.offq_top1_select(xd)
    C = offq.offq_gram(X)
    ev, U, _, _ = offq.offq_eigh(C)
    perm = offq.offq_group_permutation(ev, g)
    R = offq.offq_build_rotation(U, D, perm, g, True)
    torch.cuda.synchronize()
    idx_r, X_r, C_r, w_r, U_r, perm_r, R_r = OC.calibrate_rotation(x, g)
    assert np.array_equal(P.host(idx), idx_r)
    perm_h, ev_h = P.host(perm), P.host(ev)
    assert np.array_equal(perm_h[::g], perm_r[::g])
    assert np.array_equal(perm_h, OC.group_permutation(ev_h, g))
    Xh = P.host(X).astype(np.float64)
    proj = Xh @ P.host(U)[:, 0]
    Xr = Xh @ P.host(R).astype(np.float64)
    assert np.allclose(Xr[:, :g].mean(axis=1) * math.sqrt(g), proj, rtol=1e-4, atol=1e-4)
    assert (proj ** 2).sum() > 0.6 * (Xh ** 2).sum()
