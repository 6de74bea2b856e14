"""Pins of the oracle quantizers (Eq. 1; sec. 3.4; sec. 4 implementation)."""
import numpy as np
import pytest

from oracle import hadamard as H
from oracle import quantizer as Q


def _load3(path):
    with open(path) as f:
        rows = [l.split() for l in f if l.strip() and not l.startswith("#")]
    return [np.array(r, dtype=np.float64) for r in rows]


def test_ties_round_half_to_even(golden_dir):
    y, codes, meta = _load3(f"{golden_dir}/quantizer_ties.txt")
    q, s, z = Q.quantize_groups(y[None, :].astype(np.float32), len(y))
    assert np.array_equal(q[0], codes.astype(np.uint8))
    assert float(s[0, 0]) == meta[0] and int(z[0, 0]) == meta[1]


def test_offset_absorbed_into_zero_point(golden_dir):
    y, codes, meta = _load3(f"{golden_dir}/quantizer_offset_group.txt")
    q, s, z = Q.quantize_groups(y[None, :].astype(np.float32), len(y))
    assert np.array_equal(q[0], codes.astype(np.uint8))
    assert float(s[0, 0]) == meta[0] and int(z[0, 0]) == meta[1]
    # exact reconstruction s (q - z) of the offset group
    assert np.array_equal(Q.dequantize(q, s, z, len(y))[0], y)


def test_metadata_cost(golden_dir):
    g, sb, zb, bits = np.loadtxt(f"{golden_dir}/metadata_bits.txt")
    assert Q.metadata_bits_per_element(int(g), int(sb), int(zb)) == bits
    # storage of the actual arrays: codes packed 2/byte + fp16 scale + int16 zero
    M, K = 4, 1024
    q, s, z = Q.quantize_groups(np.random.default_rng(0).standard_normal((M, K)).astype(np.float32), int(g))
    nbytes = Q.pack_nibbles(q).nbytes + s.nbytes + z.nbytes
    assert nbytes * 8 / (M * K) == bits


@pytest.mark.parametrize("g", [16, 128, 4096])
def test_code_range_scale_zero_types(g):
    rng = np.random.default_rng(5)
    y = (rng.standard_normal((8, 2 * g)) * 3 + rng.standard_normal((8, 1)) * 50).astype(np.float32)
    q, s, z = Q.quantize_groups(y, g)
    assert q.dtype == np.uint8 and q.min() >= 0 and q.max() <= 15
    assert s.dtype == np.float16 and z.dtype == np.int16
    # min and max of every group hit the end codes unless fp16 rounding of s moves them
    qg = q.reshape(8, 2, g)
    assert np.all(qg.min(-1) == 0)
    assert np.all(qg.max(-1) >= 14)


@pytest.mark.parametrize("g", [32, 512])
def test_nearest_level_property(g):
    """Each unclamped code is the nearest grid level s (q - z) to y (Eq. 1), checked
    with exact fp64 division independent of the reciprocal used by the quantizer."""
    rng = np.random.default_rng(6)
    y = rng.standard_normal((16, 4 * g)) * rng.uniform(0.1, 20)
    y += rng.uniform(-300, 300, size=(16, 1))   # offsets -> large |z|
    y = y.astype(np.float32)
    q, s, z = Q.quantize_groups(y, g)
    assert np.abs(z.astype(np.int64)).max() > 50
    sq = np.repeat(s.astype(np.float64), g, axis=1)
    zz = np.repeat(z.astype(np.float64), g, axis=1)
    xh = sq * (q.astype(np.float64) - zz)
    inside = (q > 0) & (q < 15)
    err = np.abs(xh - y.astype(np.float64))[inside]
    assert np.all(err <= sq[inside] / 2 * (1 + 2.0 ** -20))


@pytest.mark.parametrize("g", [16, 256])
def test_reconstruction_error_bound(g):
    """|x_hat - y| <= sq/2 + 15 |s - sq| + 2^-23 max|y| for every element."""
    rng = np.random.default_rng(7)
    y = (rng.standard_normal((32, 2 * g)) * 5 + 40).astype(np.float32)
    q, s16, z = Q.quantize_groups(y, g)
    yg = y.reshape(32, 2, g).astype(np.float64)
    s_exact = (yg.max(-1) - yg.min(-1)) / 15.0
    sq = s16.astype(np.float64)
    xh = Q.dequantize(q, s16, z, g).reshape(32, 2, g)
    bound = sq / 2 + 15 * np.abs(s_exact - sq) + 2.0 ** -23 * np.abs(yg).max(-1)
    assert np.all(np.abs(xh - yg).max(-1) <= bound * (1 + 1e-9))


def test_degenerate_group_reconstructs_offset():
    # A pure first-channel input (x = a e_0) rotates to a constant a/sqrt(g);
    # the constant group takes the degenerate branch: codes 0, x_hat ~ a/sqrt(g),
    # and rotating back returns a e_0 up to the fp16 rounding of s.
    g = 64
    x = np.zeros((1, g))
    x[0, 0] = 37.0
    y = H.rotate(x, g).astype(np.float32)
    q, s, z = Q.quantize_groups(y, g)
    assert np.all(q == 0) and int(z[0, 0]) == -1
    xh = Q.dequantize(q, s, z, g)
    assert np.allclose(xh, 37.0 / 8.0, rtol=2.0 ** -11)
    back = H.rotate(xh, g)
    assert np.isclose(back[0, 0], 37.0, rtol=2.0 ** -11) and np.allclose(back[0, 1:], 0, atol=1e-12)
    # all-zero group: s = 1, z = 0, codes 0
    q0, s0, z0 = Q.quantize_groups(np.zeros((1, g), np.float32), g)
    assert np.all(q0 == 0) and float(s0[0, 0]) == 1.0 and int(z0[0, 0]) == 0


def test_offset_only_shifts_zero_point():
    """Adding a constant to a group (what the rotation does with the outlier
    channel, Eq. 5) leaves the scale unchanged and moves only the zero-point:
    with an offset that is an even number of (exact) steps, codes are identical
    (ties round to even, so an odd number of steps may flip a tie)."""
    base = np.array([[0.0, 1.25, 3.5, 7.5, 2.0, 6.0, 0.5, 4.75]], dtype=np.float32)
    q0, s0, z0 = Q.quantize_groups(base, 8)
    assert float(s0[0, 0]) == 0.5
    for shift in (10.0, -64.0, 1000.0):
        q1, s1, z1 = Q.quantize_groups(base + np.float32(shift), 8)
        assert np.array_equal(q0, q1)
        assert float(s1[0, 0]) == 0.5
        assert int(z1[0, 0]) == int(z0[0, 0]) - int(round(shift / 0.5))


def test_offsetting_reduces_error_vs_plain_outlier():
    """The method's claim (abstract, sec. 3.2): with the outlier concentrated in
    the first channel, the Hadamard turns it into an offset and the 4-bit error of
    the remaining channels drops versus quantizing with the outlier elsewhere."""
    rng = np.random.default_rng(8)
    g = 256
    x = rng.standard_normal((64, g))
    x_first = x.copy()
    x_first[:, 0] += 200.0
    x_other = x.copy()
    x_other[:, 3] += 200.0
    def err(xx):
        y = H.rotate(xx, g).astype(np.float32)
        q, s, z = Q.quantize_groups(y, g)
        return np.sqrt(np.mean((Q.dequantize(q, s, z, g) - y.astype(np.float64)) ** 2))
    assert err(x_first) < 0.2 * err(x_other)


def test_pack_unpack_roundtrip():
    rng = np.random.default_rng(9)
    u = rng.integers(0, 16, size=(3, 64)).astype(np.uint8)
    p = Q.pack_nibbles(u)
    assert p.shape == (3, 32)
    assert np.array_equal(p[:, 0], (u[:, 0] | (u[:, 1] << 4)).astype(np.uint8))
    assert np.array_equal(Q.unpack_nibbles(p), u)
    s = rng.integers(-8, 8, size=(3, 64)).astype(np.int8)
    assert np.array_equal(Q.unpack_nibbles(Q.pack_nibbles(s), signed=True), s)
    assert Q.pack_nibbles(np.array([[-1, -8]], np.int8))[0, 0] == 0x8F


def test_weight_quantizer():
    rng = np.random.default_rng(10)
    w = (rng.standard_normal((32, 256)) * 0.02).astype(np.float32)
    w[5] = 0.0
    q, sw = Q.quantize_weights(w)
    assert q.dtype == np.int8 and q.min() >= -8 and q.max() <= 7
    amax = np.abs(w).max(axis=1)
    assert np.array_equal(sw[:5], (amax[:5] / np.float32(7)).astype(np.float16))
    assert float(sw[5]) == 1.0 and np.all(q[5] == 0)
    # the largest-magnitude weight of each row maps to +/-7
    idx = np.abs(w).argmax(axis=1)
    rows = np.arange(32) != 5
    assert np.all(np.abs(q[np.arange(32), idx])[rows] == 7)
    # symmetric rounding to nearest: |w - sw q| <= sw/2 (+ tiny) inside the range
    err = np.abs(w.astype(np.float64) - sw.astype(np.float64)[:, None] * q)
    assert np.all(err[rows] <= sw.astype(np.float64)[rows, None] / 2 * (1 + 2.0 ** -20) + 1e-12)
    cs = Q.colsum(q, 64)
    assert cs.shape == (4, 32) and cs.dtype == np.int32
    assert cs[2, 7] == int(q[7, 128:192].astype(np.int64).sum())
