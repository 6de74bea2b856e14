"""Attention over the 4-bit KV cache: one decode step, and the causal prefill
of a chunk of tokens (oracle; test-only).

Sec. 3.3, step 2(3): the RoPE-encoded query and key of every head receive the
same per-head online Hadamard H3, so their dot product is unchanged (H3 is
orthogonal) while the key cache is quantized in the rotated basis.  Step 2(2):
the value cache carries the offline per-head rotation R2, which the output
projection undoes; if the values were instead quantized after the online
Hadamard as well, the attention output is rotated back by the same H3.  The
cache holds one quantizer group per (batch, head, position): 4-bit codes, an
fp16 scale and an int16 zero-point (sec. 4.2, "Number of Groups"; Eq. 1), so
the dequantized row is s (c - z).

Readings (the paper leaves the arithmetic of this step open):
* the query enters the scores in bf16 after an fp32 rotation:
  q_r = bf16_rne(fl32(fl32(1/sqrt(Dh)) * fl32(sum_i q_i H[i, d])));
* scores, softmax and the value sum are exact (fp64) on the dequantized cache;
  the result is returned unrounded (the kernel rounds it to bf16 once).
"""

import numpy as np

from . import hadamard, quantizer


def _bf16(x):
    """Round fp32 values to bfloat16, nearest-even (returned as fp64)."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def rotate_query(q):
    """q [..., Dh] (bf16 values) -> q_r [..., Dh] (bf16 values, fp64 array)."""
    q = np.asarray(q, dtype=np.float64)
    dh = q.shape[-1]
    s = hadamard.fwht(q).astype(np.float32)          # exact sum, rounded once
    c = np.float32(1.0 / np.sqrt(np.float64(dh)))
    return _bf16(c * s)


def dequantize_rows(codes_packed, scale, zero):
    """[..., S, Dh/2] packed codes with [..., S] scale and zero -> [..., S, Dh] fp64."""
    c = quantizer.unpack_nibbles(np.asarray(codes_packed)).astype(np.float64)
    s = np.asarray(scale, dtype=np.float64)[..., None]
    z = np.asarray(zero, dtype=np.float64)[..., None]
    return s * (c - z)


def softmax(x):
    """Numerically safe softmax along the last axis (fp64)."""
    x = np.asarray(x, dtype=np.float64)
    e = np.exp(x - x.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def decode_attention(q, k_codes, k_scale, k_zero, v_codes, v_scale, v_zero, seq_len, sm_scale,
                     v_hadamard=False):
    """One decode step for every (b, h).

    q: [B, Hq, Dh] bf16 values; k_codes, v_codes: uint8 [B, Hkv, S_cap, Dh/2];
    k_scale, v_scale: fp16 [B, Hkv, S_cap]; k_zero, v_zero: int16 [B, Hkv, S_cap],
    Hq a multiple of Hkv (query head h reads key/value head h // (Hq / Hkv)).
    Returns fp64 [B, H, Dh]:  softmax_j(sm_scale * q_r . K_j) @ V  over the
    positions j < seq_len, followed by the inverse rotation of V if
    ``v_hadamard``.
    """
    qr = rotate_query(q)
    k = dequantize_rows(k_codes[:, :, :seq_len], k_scale[:, :, :seq_len], k_zero[:, :, :seq_len])
    v = dequantize_rows(v_codes[:, :, :seq_len], v_scale[:, :, :seq_len], v_zero[:, :, :seq_len])
    group = qr.shape[1] // k.shape[1]
    if group > 1:
        # grouped-query attention: query head h reads key/value head h // group
        k = np.repeat(k, group, axis=1)
        v = np.repeat(v, group, axis=1)
    scores = np.float64(sm_scale) * np.einsum("bhd,bhsd->bhs", qr, k)
    p = softmax(scores)
    o = np.einsum("bhs,bhsd->bhd", p, v)
    if v_hadamard:
        o = hadamard.rotate(o, o.shape[-1])
    return o


def prefill_attention(q, k_codes, k_scale, k_zero, v_codes, v_scale, v_zero, past, sm_scale,
                      v_hadamard=False, rows=None):
    """Causal attention of T new tokens per sequence over the cache.

    q: [B, T, Hq, Dh] bf16 values (the queries after RoPE); the cache arrays as
    for decode_attention, holding the ``past`` earlier positions followed by
    the T new ones.  Query t of a sequence sits at position past + t and
    attends to positions 0 .. past + t (sec. 3.3 step 2(3) for the rotations;
    the mask is ordinary causal self-attention), so row t is the decode step
    of that token with seq_len = past + t + 1.  ``rows`` (optional) lists the
    t to compute.  Returns fp64 [B, len(rows) or T, Hq, Dh].
    """
    q = np.asarray(q)
    T = q.shape[1]
    ts = np.arange(T) if rows is None else np.asarray(rows)
    n = past + int(ts.max()) + 1
    qr = rotate_query(q[:, ts])                                  # [B, R, Hq, Dh]
    k = dequantize_rows(k_codes[:, :, :n], k_scale[:, :, :n], k_zero[:, :, :n])
    v = dequantize_rows(v_codes[:, :, :n], v_scale[:, :, :n], v_zero[:, :, :n])
    group = qr.shape[2] // k.shape[1]
    if group > 1:
        k = np.repeat(k, group, axis=1)
        v = np.repeat(v, group, axis=1)
    scores = np.float64(sm_scale) * np.einsum("brhd,bhsd->bhrs", qr, k)
    allowed = np.arange(n)[None, :] <= (past + ts)[:, None]      # [R, n]
    scores = np.where(allowed[None, None], scores, -np.inf)
    p = softmax(scores)
    o = np.einsum("bhrs,bhsd->brhd", p, v)
    if v_hadamard:
        o = hadamard.rotate(o, o.shape[-1])
    return o


def output_bound(v_codes, v_scale, v_zero, seq_len):
    """Per-(b, h) max_j,d |V_j[d]| over the attended positions (fp64 [B, H, 1]):
    the scale against which absolute errors of the output are measured."""
    v = dequantize_rows(v_codes[:, :, :seq_len], v_scale[:, :, :seq_len], v_zero[:, :, :seq_len])
    return np.abs(v).max(axis=(2, 3))[..., None]
