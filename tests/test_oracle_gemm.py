"""Pins of the oracle integer GEMM and epilogue (algebra of Eq. 1)."""
import numpy as np
import pytest

from oracle import gemm as Gm
from oracle import hadamard as H
from oracle import kv as KV
from oracle import quantizer as Q


def _tiny(M, N, K, g, seed):
    rng = np.random.default_rng(seed)
    q_a = rng.integers(0, 16, size=(M, K)).astype(np.uint8)
    q_w = rng.integers(-8, 8, size=(N, K)).astype(np.int8)
    s = rng.uniform(0.01, 2.0, size=(M, K // g)).astype(np.float16)
    z = rng.integers(-300, 300, size=(M, K // g)).astype(np.int16)
    sw = rng.uniform(0.001, 0.01, size=N).astype(np.float16)
    return q_a, q_w, s, z, sw


@pytest.mark.parametrize("M,N,K,g", [(3, 5, 16, 16), (4, 3, 32, 8), (2, 2, 64, 64)])
def test_blas_equals_int64_bruteforce(M, N, K, g):
    q_a, q_w, *_ = _tiny(M, N, K, g, 0)
    assert np.array_equal(Gm.int_gemm_groups(q_a, q_w, g), Gm.int_gemm_bruteforce(q_a, q_w, g))


def test_blas_exact_at_extreme_codes():
    # largest possible partial sums: all codes 15 x -8 over a long group
    K = 8192
    q_a = np.full((2, K), 15, np.uint8)
    q_w = np.full((3, K), -8, np.int8)
    acc = Gm.int_gemm_groups(q_a, q_w, K)
    assert np.all(acc == -120 * K)


@pytest.mark.parametrize("g", [8, 32])
def test_epilogue_equals_dequantized_matmul(g):
    M, N, K = 5, 7, 64
    q_a, q_w, s, z, sw = _tiny(M, N, K, g, 1)
    acc = Gm.int_gemm_groups(q_a, q_w, g)
    cs = Q.colsum(q_w, g)
    y = Gm.epilogue(acc, s, z, sw, cs)
    ref = Gm.dequant_matmul(q_a, s, z, q_w, sw, g)
    assert np.allclose(y, ref, rtol=1e-12, atol=1e-12 * np.abs(ref).max())
    e = Gm.epilogue_magnitude(acc, s, z, sw, cs)
    assert np.all(e >= np.abs(y) * (1 - 1e-12))


def test_end_to_end_approximates_float_layer():
    """Rotate -> quantize -> integer GEMM -> epilogue approximates x W'^T where W'
    is the weight with the same rotation fused in (sec. 3.3, step 2: rotations are
    fused into the weights so the product is unchanged)."""
    rng = np.random.default_rng(2)
    M, N, K, g = 32, 48, 256, 256
    x = rng.standard_normal((M, K))
    x[:, 0] += 150.0
    w = rng.standard_normal((N, K)) * 0.02
    y = H.rotate(x, g).astype(np.float32)
    wr = H.rotate(w, g).astype(np.float32)    # W' = W H/sqrt(g) (H symmetric)
    q_a, s, z = Q.quantize_groups(y, g)
    q_w, sw = Q.quantize_weights(wr)
    acc = Gm.int_gemm_groups(q_a, q_w, g)
    out = Gm.epilogue(acc, s, z, sw, Q.colsum(q_w, g))
    ref = x @ w.T
    rel = np.linalg.norm(out - ref) / np.linalg.norm(ref)
    assert rel < 0.15


def test_kv_quantizer_is_group_per_row():
    rng = np.random.default_rng(3)
    rows = rng.standard_normal((10, 128)).astype(np.float32)
    rows[:, 5] += 40
    y = KV.kv_rotate(rows, True)
    assert np.allclose(y, H.rotate(rows, 128))
    assert np.array_equal(KV.kv_rotate(rows, False), rows.astype(np.float64))
    c, s, z = KV.kv_quantize(y.astype(np.float32))
    c2, s2, z2 = Q.quantize_groups(y.astype(np.float32), 128)
    assert np.array_equal(c, c2) and np.array_equal(s, s2[:, 0]) and np.array_equal(z, z2[:, 0])


def test_bf16_helpers():
    assert Gm.bf16_round(np.array([1.0 + 2 ** -9]))[0] == 1.0        # tie -> even
    assert Gm.bf16_round(np.array([1.0 + 3 * 2 ** -9]))[0] == 1.0 + 2 ** -7
    assert Gm.bf16_ulp(np.array([1.0]))[0] == 2 ** -7
