"""Pins of the oracle integer GEMM and epilogue (algebra of Eq. 1)."""
import os
from fractions import Fraction

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


def _golden_epilogue(golden_dir):
    rows = [ln.split() for ln in open(os.path.join(golden_dir, "epilogue_cancellation.txt"))
            if ln.strip() and not ln.startswith("#")]
    q_a = np.array([rows[0]], dtype=np.int64)
    q_w = np.array([rows[1]], dtype=np.int64)
    s = np.array([rows[2]], dtype=np.float16)
    z = np.array([rows[3]], dtype=np.int64)
    sw = np.array(rows[4], dtype=np.float16)
    acc0, acc1, cs0, cs1 = (int(v) for v in rows[5])
    y, e = (float(v) for v in rows[6])
    return q_a, q_w, s, z, sw, (acc0, acc1), (cs0, cs1), y, e


def test_epilogue_hand_worked_cancellation(golden_dir):
    """Eq. 1's epilogue on a hand-worked case whose two group terms nearly
    cancel: the output and its magnitude E (the sum of the absolute terms,
    which sets the cancellation floor of the output tolerance) both equal the
    values worked out by hand, so an E that is too large or too small fails."""
    q_a, q_w, s, z, sw, acc_h, cs_h, y_h, e_h = _golden_epilogue(golden_dir)
    acc = Gm.int_gemm_bruteforce(q_a, q_w, 2)
    assert acc[:, 0, 0].tolist() == list(acc_h)
    cs = Q.colsum(q_w.astype(np.int8), 2)
    assert cs[:, 0].tolist() == list(cs_h)
    assert Gm.epilogue(acc, s, z, sw, cs)[0, 0] == y_h
    assert Gm.epilogue_magnitude(acc, s, z, sw, cs)[0, 0] == e_h
    assert Gm.dequant_matmul(q_a, s, z, q_w, sw, 2)[0, 0] == y_h


@pytest.mark.parametrize("G,seed", [(1, 0), (3, 1), (8, 2), (28, 3)])
def test_epilogue_and_magnitude_match_exact_rationals(G, seed):
    """Y and E against their definitions evaluated in exact rational
    arithmetic (fp16 scales are dyadic rationals; codes, zero-points and
    column sums are integers).  The fp64 oracle may differ only by its own
    rounding: at most (G + 2) * 2^-53 * E for both."""
    g = 4
    M, N = 3, 4
    rng = np.random.default_rng(seed)
    q_a = rng.integers(0, 16, size=(M, G * g))
    q_w = rng.integers(-8, 8, size=(N, G * g))
    s = rng.uniform(0.01, 3.0, size=(M, G)).astype(np.float16)
    z = rng.integers(-32768, 32768, size=(M, G))
    sw = rng.uniform(-0.02, 0.02, size=N).astype(np.float16)
    acc = Gm.int_gemm_bruteforce(q_a, q_w, g)
    cs = Q.colsum(q_w.astype(np.int8), g)
    y = Gm.epilogue(acc, s, z, sw, cs)
    e = Gm.epilogue_magnitude(acc, s, z, sw, cs)
    for m in range(M):
        for n in range(N):
            terms = []
            for b in range(G):
                a_b = sum(int(q_a[m, k]) * int(q_w[n, k]) for k in range(b * g, (b + 1) * g))
                c_b = sum(int(q_w[n, k]) for k in range(b * g, (b + 1) * g))
                terms.append(Fraction(float(s[m, b])) * (a_b - int(z[m, b]) * c_b))
            swf = Fraction(float(sw[n]))
            y_ex = swf * sum(terms)
            e_ex = abs(swf) * sum(abs(t) for t in terms)
            tol = (G + 2) * 2.0 ** -53 * float(e_ex)
            assert abs(Fraction(float(y[m, n])) - y_ex) <= tol
            assert abs(Fraction(float(e[m, n])) - e_ex) <= tol
            assert e[m, n] >= abs(y[m, n]) * (1 - 1e-15)


def test_bf16_ulp_binades():
    """ulp of bfloat16 (8 significant bits, fp32's exponent range) at chosen
    values: powers of two take the spacing above them, subnormals 2^-133."""
    cases = {1.0: 2 ** -7, 1.9921875: 2 ** -7, 2.0: 2 ** -6, 3.0: 2 ** -6, 0.75: 2 ** -8,
             -3.0: 2 ** -6, 65504.0: 2.0 ** 8, 1e30: 2.0 ** 92, 2.0 ** -126: 2.0 ** -133,
             2.0 ** -127: 2.0 ** -133, 2.0 ** -133: 2.0 ** -133, 0.0: 2.0 ** -133,
             3.0e38: 2.0 ** 120}
    got = Gm.bf16_ulp(np.array(list(cases)))
    assert got.tolist() == list(cases.values())


def test_bf16_ulp_equals_bit_increment():
    """ulp of bf16 at x = the gap between the bf16 value below |x| (|x|'s fp32
    bit pattern truncated to 16 bits) and the next bf16 pattern, over random
    normal and subnormal inputs."""
    rng = np.random.default_rng(7)
    hi = rng.integers(0, 0x7F7F, size=20000).astype(np.uint32)      # finite, next also finite
    lo = rng.integers(0, 1 << 16, size=hi.size).astype(np.uint32)
    x = ((hi << 16) | lo).view(np.float32)
    x = np.where(rng.random(hi.size) < 0.5, -x, x)
    b = (np.abs(x).view(np.uint32) >> 16).astype(np.uint32)
    below = (b << 16).view(np.float32).astype(np.float64)
    above = ((b + 1) << 16).view(np.float32).astype(np.float64)
    assert np.array_equal(Gm.bf16_ulp(x.astype(np.float64)), above - below)
