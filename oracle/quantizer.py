"""Uniform 4-bit quantizers of OffQ (oracle; test-only).

Activations / KV (sec. 3, Eq. 1; sec. 4 implementation: per-group asymmetric;
sec. 3.4: 16-bit scale and 16-bit zero-point per group):

    x_q = clamp(round(x / s) + z, 0, 2^b - 1),  b = 4,  z an integer.

The paper leaves the choice of s and z, the rounding rule and the storage
types open.  Readings used here (the GPU library implements the same ones):

1. Range: min-max over the group, no clipping; the range is not widened to
   include 0 (the footnote to Eq. 5: asymmetric quantization need not keep 0 in
   range, the offset shifts it away).
       mx = max(y), mn = min(y)                        (fp32)
       s  = fl32(fl32(mx - mn) / 15)                   (IEEE fp32)
   Degenerate group (mx == mn): s = |mn|, or 1 if mn == 0 (all codes 0 and
   x_hat = mn up to the fp16 rounding of s: a pure offset reconstructs).
2. 16-bit scale: s16 = fp16_rne(clamp(s, 2^-24, 65504)); the quantizer uses the
   stored value, sq = f32(s16), so that codes and metadata agree; r = fl32(1/sq).
3. 16-bit zero-point: z = clamp(rne(-mn * r), -32768, 32767), the product being
   the exact real product of the two fp32 numbers.
4. Codes: q = clamp(rne(y * r) + z, 0, 15), again with the exact product y*r
   (one rounding, to the nearest integer, ties to even).
5. Packing: two codes per byte, even channel in the low nibble.

Weights (sec. 4 implementation: per-channel symmetric 4-bit):
    sw  = fp16_rne(clamp(max_k |w| / 7, 2^-24, 65504))   (1 for an all-zero row)
    q_w = clamp(rne(w / f32(sw)), -8, 7)                  (exact quotient)
    colsum_b[n] = sum_{k in group b} q_w[n, k]
"""

import numpy as np

QMAX = 15  # 2^4 - 1 (Eq. 1 with b = 4)
FP16_MIN_SUB = np.float32(2.0 ** -24)
FP16_MAX = np.float32(65504.0)


def quantize_groups(y, g):
    """Quantize fp32 ``y`` [M, K] per (row, group of g channels).

    Returns ``(codes, scale, zero)``: codes uint8 [M, K] (values 0..15, one per
    byte, unpacked), scale float16 [M, K/g], zero int16 [M, K/g].
    """
    y = np.ascontiguousarray(y, dtype=np.float32)
    M, K = y.shape
    if K % g:
        raise ValueError("K must be a multiple of g")
    G = K // g
    yg = y.reshape(M, G, g)

    mx = yg.max(axis=-1)
    mn = yg.min(axis=-1)
    s = (mx - mn) / np.float32(QMAX)                      # fp32 ops
    degenerate = mx == mn
    s_deg = np.where(mn != 0, np.abs(mn), np.float32(1)).astype(np.float32)
    s = np.where(degenerate, s_deg, s).astype(np.float32)
    s = np.minimum(np.maximum(s, FP16_MIN_SUB), FP16_MAX).astype(np.float32)
    s16 = s.astype(np.float16)                            # RNE
    sq = s16.astype(np.float32)
    r = (np.float32(1) / sq).astype(np.float32)           # IEEE fp32

    r64 = r.astype(np.float64)
    z = np.rint(-mn.astype(np.float64) * r64)             # exact product, RNE
    z = np.clip(z, -32768, 32767)
    t = np.rint(yg.astype(np.float64) * r64[..., None])   # exact product, RNE
    q = np.clip(t + z[..., None], 0, QMAX)
    return (q.reshape(M, K).astype(np.uint8), s16, z.astype(np.int16))


def dequantize(codes, scale, zero, g):
    """x_hat = s (x_q - z) in fp64 (inverse of Eq. 1)."""
    codes = np.asarray(codes)
    M, K = codes.shape
    G = K // g
    q = codes.reshape(M, G, g).astype(np.float64)
    s = np.asarray(scale).astype(np.float64)[..., None]
    z = np.asarray(zero).astype(np.float64)[..., None]
    return (s * (q - z)).reshape(M, K)


def pack_nibbles(q):
    """Pack 4-bit values [.., K] (uint8 0..15 or int8 -8..7) two per byte.

    Channel 2j goes to the low nibble of byte j, channel 2j+1 to the high one;
    signed values are stored as 4-bit two's complement.
    """
    q = np.asarray(q).astype(np.int64) & 0xF
    lo = q[..., 0::2]
    hi = q[..., 1::2]
    return (lo | (hi << 4)).astype(np.uint8)


def unpack_nibbles(p, signed=False):
    """Inverse of ``pack_nibbles``: [.., K/2] bytes -> [.., K] values."""
    p = np.asarray(p, dtype=np.uint8).astype(np.int64)
    lo = p & 0xF
    hi = (p >> 4) & 0xF
    q = np.stack([lo, hi], axis=-1).reshape(p.shape[:-1] + (2 * p.shape[-1],))
    if signed:
        q = np.where(q >= 8, q - 16, q)
        return q.astype(np.int8)
    return q.astype(np.uint8)


def quantize_weights(w):
    """Per-output-channel symmetric 4-bit quantization of fp32 ``w`` [N, K].

    Returns ``(q_w int8 [N, K] in -8..7, sw float16 [N])``.
    """
    w = np.ascontiguousarray(w, dtype=np.float32)
    amax = np.abs(w).max(axis=1)
    s = amax / np.float32(7)                              # fp32 IEEE
    s = np.where(amax == 0, np.float32(1), s).astype(np.float32)
    s = np.minimum(np.maximum(s, FP16_MIN_SUB), FP16_MAX).astype(np.float32)
    sw = s.astype(np.float16)
    sq = sw.astype(np.float64)
    q = np.clip(np.rint(w.astype(np.float64) / sq[:, None]), -8, 7)
    return q.astype(np.int8), sw


def colsum(q_w, g):
    """Per-group weight code sums colsum[b, n] = sum_{k in group b} q_w[n, k] (int32)."""
    q_w = np.asarray(q_w).astype(np.int64)
    N, K = q_w.shape
    return q_w.reshape(N, K // g, g).sum(axis=-1).T.astype(np.int32).copy()


def metadata_bits_per_element(g, scale_bits=16, zero_bits=16, code_bits=4):
    """Storage cost per activation element of per-group codes plus (s, z) (sec. 3.4)."""
    return (code_bits * g + scale_bits + zero_bits) / g
