"""Pins of the calibration oracle (oracle/calibration.py): the paper's sorted
grouping example, its L-infinity example, brute-force top-1 selection and
covariance, the eigendecomposition's defining identities and a rank-1 closed
form, the concentration of a planted outlier direction onto the first
channel, and the rotation / weight-fusion identities."""
import math
import os

import numpy as np
import pytest

from oracle import calibration as OC
from oracle import hadamard as OH


def _golden(golden_dir, name):
    out = {}
    for line in open(os.path.join(golden_dir, name)):
        line = line.strip()
        if line and not line.startswith("#"):
            k, v = line.split(":")
            out[k.strip()] = [float(t) for t in v.split()]
    return out


def test_sorted_grouping_matches_the_papers_example(golden_dir):
    gold = _golden(golden_dir, "sorted_grouping.txt")
    vals = np.array(gold["values"])
    perm = OC.group_permutation(vals, int(gold["group_size"][0]))
    assert list(vals[perm]) == gold["sorted"]
    assert list(vals[perm]) != gold["zigzag"]
    assert sorted(perm) == list(range(6))


def test_group_permutation_properties():
    rng = np.random.default_rng(0)
    key = np.round(rng.standard_normal(64), 1)  # with ties
    perm = OC.group_permutation(key, 8)
    assert sorted(perm) == list(range(64))
    heads = key[perm[::8]]
    assert np.all(np.diff(heads) <= 0)  # heads descending
    assert np.min(heads) >= np.max(np.delete(key, perm[::8]))  # the 8 largest lead
    rest = [perm[b * 8 + t] for b in range(8) for t in range(1, 8)]
    assert np.all(np.diff(key[rest]) >= 0)  # the rest ascending across the groups
    # ties: lower index first
    for a, b in zip(rest[:-1], rest[1:]):
        if key[a] == key[b]:
            assert a < b
    # g = D: one group, its head the largest
    assert OC.group_permutation(key, 64)[0] == int(np.argmax(key))


def test_top1_prefers_the_spiky_token():
    # sec. 3.1: on the unit sphere [1, 0, 0] has the larger L-inf norm than [0.58]*3
    x = np.array([[[0.58, 0.58, 0.58], [1.0, 0.0, 0.0], [0.0, 0.6, 0.8]]])
    idx, X = OC.top1_select(x)
    assert idx[0] == 1 and np.array_equal(X[0], [1.0, 0.0, 0.0])


def test_top1_and_gram_brute_force():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((3, 5, 4))
    x[1, 2, 0] = 9.0
    x[1, 4, 3] = -9.0  # tie in |.|: the first token wins
    idx, X = OC.top1_select(x)
    for s in range(3):
        best, bi = -1.0, -1
        for t in range(5):
            m = max(abs(v) for v in x[s, t])
            if m > best:
                best, bi = m, t
        assert idx[s] == bi
        assert np.array_equal(X[s], x[s, bi])
    assert idx[1] == 2
    C = OC.gram(X)
    for i in range(4):
        for j in range(4):
            assert abs(C[i, j] - sum(X[n, i] * X[n, j] for n in range(3)) / 3) < 1e-14
    assert np.array_equal(C, C.T)


def test_channel_absmax():
    x = np.array([[1.0, -3.0], [-2.0, 0.5]])
    assert np.array_equal(OC.channel_absmax(x), [2.0, 3.0])


@pytest.mark.parametrize("D,N", [(16, 40), (32, 8)])
def test_eigh_identities(D, N):
    rng = np.random.default_rng(D)
    C = OC.gram(rng.standard_normal((N, D)))
    w, U = OC.eigh_desc(C)
    assert np.all(np.diff(w) <= 1e-12)
    assert np.allclose(U @ np.diag(w) @ U.T, C, atol=1e-12)
    assert np.allclose(U.T @ U, np.eye(D), atol=1e-12)
    piv = np.abs(U).argmax(axis=0)
    assert np.all(U[piv, np.arange(D)] > 0)


def test_eigh_rank_one_closed_form():
    v = np.array([3.0, -4.0, 0.0, 12.0])
    w, U = OC.eigh_desc(np.outer(v, v))
    assert abs(w[0] - 169.0) < 1e-12 and np.all(np.abs(w[1:]) < 1e-12)
    assert np.allclose(U[:, 0], v / 13.0 * np.sign(v[3]), atol=1e-14)


def test_top1_pca_concentrates_a_planted_outlier_direction():
    # sec. 3.1: activations with an outlier along one direction shared by
    # tokens; after X U the outlier sits on the first channel
    rng = np.random.default_rng(3)
    D, n_seq, L = 64, 32, 50
    d = rng.standard_normal(D)
    d /= np.linalg.norm(d)
    x = rng.standard_normal((n_seq, L, D)) * 0.1
    spikes = rng.integers(0, L, n_seq)
    x[np.arange(n_seq), spikes] += 30.0 * d * rng.choice([-1, 1], n_seq)[:, None]
    idx, X, C, w, U, perm, R = OC.calibrate_rotation(x, 16)
    assert np.array_equal(idx, spikes)
    assert abs(abs(U[:, 0] @ d) - 1.0) < 1e-3
    Xr = X @ U
    energy = (Xr ** 2).sum(axis=0)
    assert energy[0] > 0.99 * energy.sum()
    # P1 puts it on the first channel of group 0, and H1 spreads it as an offset
    assert perm[0] == 0
    xr = X @ R
    mean0 = xr[:, :16].mean(axis=1)
    assert np.allclose(mean0 * math.sqrt(16), (X @ U)[:, 0], atol=1e-9)


def test_rotation_is_orthogonal_and_fusion_preserves_the_layer():
    rng = np.random.default_rng(4)
    D, N = 32, 10
    _, U = OC.eigh_desc(OC.gram(rng.standard_normal((50, D))))
    perm = OC.group_permutation(rng.standard_normal(D), 8)
    R = OC.build_rotation(U, D, perm, 8, True)
    assert np.allclose(R @ R.T, np.eye(D), atol=1e-12)
    # column block b of R = U[:, perm] restricted to the block, times H_8 / sqrt 8
    H = OH.sylvester(8) / math.sqrt(8)
    assert np.allclose(R[:, 8:16], U[:, perm[8:16]] @ H, atol=1e-14)
    x = rng.standard_normal((3, D))
    W = rng.standard_normal((N, D))
    assert np.allclose((x @ R) @ OC.fuse_weights(W, R).T, x @ W.T, atol=1e-12)
    # identity rotation without Hadamard
    assert np.array_equal(OC.build_rotation(None, D), np.eye(D))
    assert np.array_equal(OC.permute_rows(W, np.arange(N)[::-1]), W[::-1])
