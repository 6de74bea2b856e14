"""Pins of the oracle rotation against facts the paper and mathematics fix."""
import numpy as np
import pytest
from scipy.linalg import hadamard as scipy_hadamard

from oracle import hadamard as H


@pytest.mark.parametrize("n", [1, 2, 4, 8, 64, 256, 1024])
def test_sylvester_matches_library(n):
    # scipy.linalg.hadamard is the Sylvester construction (independent code).
    assert np.array_equal(H.sylvester(n), scipy_hadamard(n))


@pytest.mark.parametrize("n", [2, 16, 128, 512])
def test_sylvester_orthogonal_first_row_ones(n):
    h = H.sylvester(n)
    # +/-1 entries, orthogonal (H H^T = n I), first row all ones (sec. 3.2).
    assert set(np.unique(h)) == {-1, 1}
    assert np.array_equal(h @ h.T, n * np.eye(n, dtype=np.int64))
    assert np.all(h[0] == 1)


@pytest.mark.parametrize("g", [2, 8, 64, 256])
def test_fwht_equals_library_matrix_product(g):
    rng = np.random.default_rng(1)
    x = rng.standard_normal((5, 3 * g))
    ref = np.concatenate([x[:, b * g:(b + 1) * g] @ scipy_hadamard(g) for b in range(3)], axis=1)
    ref /= np.sqrt(g)
    assert np.allclose(H.rotate(x, g), ref, rtol=1e-13, atol=1e-12)


def test_eq5_worked_example(golden_dir):
    rows = np.loadtxt(f"{golden_dir}/eq5_two_point.txt", ndmin=2)
    for x1, x2, y1, y2, off, r1, r2 in rows:
        y = H.rotate(np.array([[x1, x2]]), 2)[0]
        assert np.allclose(y, [y1, y2], rtol=1e-15, atol=0)
        assert np.isclose(H.offset(np.array([[x1, x2]]), 2)[0, 0], off, rtol=1e-15)
        residual = H.rotate(np.array([[0.0, x2]]), 2)[0]
        assert np.allclose(residual, [r1, r2], rtol=1e-15)
        assert np.allclose(y, off + residual, rtol=1e-15)


@pytest.mark.parametrize("g", [4, 128, 4096])
def test_rotation_is_orthogonal_involution(g):
    rng = np.random.default_rng(2)
    x = rng.standard_normal((3, 2 * g)) * 10
    y = H.rotate(x, g)
    assert np.allclose(np.linalg.norm(y, axis=1), np.linalg.norm(x, axis=1), rtol=1e-12)
    # Sylvester H is symmetric with H H = g I: applying the rotation twice returns x.
    assert np.allclose(H.rotate(y, g), x, rtol=1e-12, atol=1e-11)


@pytest.mark.parametrize("g", [8, 512])
def test_offset_invariants(g):
    rng = np.random.default_rng(3)
    G = 3
    x = rng.standard_normal((4, G * g))
    x[:, ::g] += 300.0  # structured outlier on the first channel of each group
    y = H.rotate(x, g).reshape(4, G, g)
    # (i) the group mean of y is exactly the constant offset x_{b*g} / sqrt(g) ...
    off = H.offset(x, g)
    assert np.allclose(y.mean(axis=-1), off, rtol=1e-12)
    # ... i.e. sqrt(g) * mean = the first channel of the group (Eq. 5, sec. 3.2).
    assert np.allclose(np.sqrt(g) * y.mean(axis=-1), x[:, ::g], rtol=1e-12)
    # (ii) y minus its offset is the rotation of x with the first channels zeroed.
    x0 = x.copy()
    x0[:, ::g] = 0.0
    y0 = H.rotate(x0, g).reshape(4, G, g)
    assert np.allclose(y - off[..., None], y0, rtol=1e-12, atol=1e-10)
    # (iii) a pure first-channel input becomes a constant a / sqrt(g).
    a = np.zeros((1, g))
    a[0, 0] = 7.0
    assert np.allclose(H.rotate(a, g), 7.0 / np.sqrt(g), rtol=1e-15)


def test_group_layout_is_block_diagonal():
    rng = np.random.default_rng(4)
    g, G = 16, 4
    x = rng.standard_normal((2, g * G))
    full = np.kron(np.eye(G), scipy_hadamard(g)) / np.sqrt(g)
    assert np.allclose(H.rotate(x, g), x @ full, rtol=1e-13, atol=1e-13)


def test_rejects_bad_sizes():
    with pytest.raises(ValueError):
        H.sylvester(12)
    with pytest.raises(ValueError):
        H.rotate(np.zeros((1, 10)), 4)
