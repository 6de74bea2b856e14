"""A quantized decoder layer: one decode step, or the prefill of a chunk of
tokens (oracle; test-only).

The pipeline of sec. 3.3 / Fig. 2 (decode: one new token per sequence;
prefill: T new tokens per sequence, the attention causal over them):

    h  = x (+ residual);  y = RMSNorm(h)            (norm scale fused offline)
    quantize y (no online rotation: U1 P1 H1 are fused offline, step 2(1))
    qkv = y W_qkv^T   (4-bit x 4-bit, Eq. 1 dequantization)
    RoPE on the query and key heads; H3 on the key (step 2(3)); KV4 quantize
    (group = head dim, sec. 4.2) into the cache at the token's position
    o  = attention(H3 q, cache)                      (oracle.attention)
    quantize o (R2 is fused offline, step 2(2)); h1 = h + o W_o^T
    y1 = RMSNorm(h1); quantize; gu = y1 W_ug^T  (gate | up; P4 fused offline)
    a  = SwiGLU(gu); H4 + quantize (online, step 2(4)); h2 = h1 + a W_d^T

Readings (the paper fixes none of this arithmetic): activations between the
steps are bf16, rounded once from the fp32 value a kernel holds (fp64 here
rounded to fp32, then to bf16); the residual add rounds fl32(x + r) to bf16;
RMSNorm divides by sqrt(mean(h^2) + eps); RoPE rotates dims (i, i + 64) of a
head by the fp32 angle fl32(pos * fl32(base^(-2i/128))); the key is rounded
to bf16 after RoPE, before H3; SwiGLU is silu(gate) * up.
"""

import numpy as np

from . import attention, gemm, hadamard, kv, quantizer


def bf16(x):
    """Round to bfloat16 through fp32 (nearest-even both times); fp64 result."""
    return gemm.bf16_round(np.asarray(x, dtype=np.float64))


def add_rmsnorm(x, res, eps):
    """x, res: bf16 values [M, D] (res may be None) -> (h, y) bf16 values (fp64)."""
    x = np.asarray(x, dtype=np.float64)
    if res is None:
        h = x.copy()
    else:
        h = bf16(np.asarray(x, np.float32) + np.asarray(res, np.float32))
    ms = np.mean(h * h, axis=-1, keepdims=True)
    y = bf16(h / np.sqrt(ms + np.float64(eps)))
    return h, y


def rope_inv_freq(base, dh=128):
    """fl32(base^(-2i/dh)) for i < dh/2."""
    i = np.arange(dh // 2, dtype=np.float64)
    return np.power(np.float64(base), -2.0 * i / dh).astype(np.float32)


def rope(x, pos, base):
    """x: [..., 128] (any float values), pos: int array broadcast over the
    leading axes -> fp64 [..., 128] rotated by the fp32 angles."""
    x = np.asarray(x, dtype=np.float64)
    dh = x.shape[-1]
    inv = rope_inv_freq(base, dh)
    ang = (np.asarray(pos, dtype=np.float32)[..., None] * inv).astype(np.float64)  # fl32 product
    c, s = np.cos(ang), np.sin(ang)
    a, b = x[..., : dh // 2], x[..., dh // 2:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def swiglu(gu):
    """gu: [M, 2F] (gate | up) -> fp64 silu(gate) * up, unrounded."""
    gu = np.asarray(gu, dtype=np.float64)
    F = gu.shape[-1] // 2
    g, u = gu[..., :F], gu[..., F:]
    return g / (1.0 + np.exp(-g)) * u


def kv_rows(qkv, Hq, Hkv, pos, base, k_hadamard=True, v_hadamard=False):
    """The rows the KV step quantizes: (q [M, Hq, 128] unrounded,
    k_y [M, Hkv, 128], v_y [M, Hkv, 128]) in fp64 (k_y, v_y before the
    quantizer's fp32 conversion)."""
    qkv = np.asarray(qkv, dtype=np.float64)
    M = qkv.shape[0]
    heads = qkv.reshape(M, Hq + 2 * Hkv, 128)
    p = np.asarray(pos)[:, None]
    q = rope(heads[:, :Hq], p, base)
    k = bf16(rope(heads[:, Hq:Hq + Hkv], p, base))
    v = heads[:, Hq + Hkv:]
    k_y = kv.kv_rotate(k.reshape(-1, 128), k_hadamard).reshape(M, Hkv, 128)
    v_y = kv.kv_rotate(v.reshape(-1, 128), v_hadamard).reshape(M, Hkv, 128)
    return q, k_y, v_y


def quantized_linear(y, w_q, w_scale, g, hadamard_online=False):
    """bf16 activations y [M, K] -> bf16 output of the W4A4 linear layer
    (optional online block Hadamard, quantizer of Eq. 1 per group of g,
    exact integer GEMM, fp64 epilogue, bf16 rounding)."""
    yr = hadamard.rotate(y, g) if hadamard_online else np.asarray(y, np.float64)
    q, s, z = quantizer.quantize_groups(yr.astype(np.float32), g)
    acc = gemm.int_gemm_groups(q, w_q, g)
    return bf16(gemm.epilogue(acc, s, z, w_scale, quantizer.colsum(w_q, g)))


def decode_layer(x, weights, cache, pos, seq_len, cfg):
    """One decode step.  x: bf16 [M, D]; weights: dict of (q_w int8, sw fp16)
    for "qkv", "o", "ug", "down"; cache: dict of the 4-bit K/V cache arrays
    [M, Hkv, s_cap, ...] (copied, the new position written); pos: [M] ints;
    seq_len: positions attended after the write; cfg: Hq, Hkv, g, eps,
    rope_base.  Returns (out bf16 [M, D], dict of intermediates, new cache)."""
    Hq, Hkv, g, eps, base = cfg["Hq"], cfg["Hkv"], cfg["g"], cfg["eps"], cfg["rope_base"]
    M = x.shape[0]
    cache = {k: v.copy() for k, v in cache.items()}
    _, y0 = add_rmsnorm(x, None, eps)
    qkv = quantized_linear(y0, *weights["qkv"], g)
    q, k_y, v_y = kv_rows(qkv, Hq, Hkv, pos, base)
    for name, rows in (("k", k_y), ("v", v_y)):
        codes, s, z = kv.kv_quantize(rows.reshape(-1, 128).astype(np.float32))
        packed = quantizer.pack_nibbles(codes).reshape(M, Hkv, 64)
        for m in range(M):
            cache[name + "_codes"][m, :, pos[m]] = packed[m]
            cache[name + "_scale"][m, :, pos[m]] = s.reshape(M, Hkv)[m]
            cache[name + "_zero"][m, :, pos[m]] = z.reshape(M, Hkv)[m]
    o = bf16(attention.decode_attention(bf16(q), cache["k_codes"], cache["k_scale"],
                                        cache["k_zero"], cache["v_codes"], cache["v_scale"],
                                        cache["v_zero"], seq_len, 1.0 / np.sqrt(128.0)))
    attn_out = quantized_linear(o.reshape(M, Hq * 128), *weights["o"], g)
    h1, y1 = add_rmsnorm(x, attn_out, eps)
    gu = quantized_linear(y1, *weights["ug"], g)
    a = bf16(swiglu(gu))
    down = quantized_linear(a, *weights["down"], g, hadamard_online=True)
    out, _ = add_rmsnorm(h1, down, eps)
    inter = dict(y0=y0, qkv=qkv, q=bf16(q), o=o, attn_out=attn_out, h1=h1, y1=y1, gu=gu, a=a,
                 down=down)
    return out, inter, cache


def prefill_layer(x, weights, cache, past, cfg):
    """The prefill of T tokens per sequence.  x: bf16 [B * T, D], row
    b * T + t the token at position past + t of sequence b; cache: the 4-bit
    K/V cache [B, Hkv, s_cap, ...] holding ``past`` positions per sequence
    (copied, the T new positions written); weights and cfg as for
    decode_layer.  Returns (out bf16 [B * T, D], dict of intermediates, new
    cache)."""
    Hq, Hkv, g, eps, base = cfg["Hq"], cfg["Hkv"], cfg["g"], cfg["eps"], cfg["rope_base"]
    B = cache["k_codes"].shape[0]
    M = x.shape[0]
    T = M // B
    pos = past + np.tile(np.arange(T), B)
    cache = {k: v.copy() for k, v in cache.items()}
    _, y0 = add_rmsnorm(x, None, eps)
    qkv = quantized_linear(y0, *weights["qkv"], g)
    q, k_y, v_y = kv_rows(qkv, Hq, Hkv, pos, base)
    for name, rows in (("k", k_y), ("v", v_y)):
        codes, s, z = kv.kv_quantize(rows.reshape(-1, 128).astype(np.float32))
        packed = quantizer.pack_nibbles(codes).reshape(B, T, Hkv, 64)
        cache[name + "_codes"][:, :, past:past + T] = packed.transpose(0, 2, 1, 3)
        cache[name + "_scale"][:, :, past:past + T] = s.reshape(B, T, Hkv).transpose(0, 2, 1)
        cache[name + "_zero"][:, :, past:past + T] = z.reshape(B, T, Hkv).transpose(0, 2, 1)
    qb = bf16(q).reshape(B, T, Hq, 128)
    o = bf16(attention.prefill_attention(qb, cache["k_codes"], cache["k_scale"], cache["k_zero"],
                                         cache["v_codes"], cache["v_scale"], cache["v_zero"],
                                         past, 1.0 / np.sqrt(128.0)))
    attn_out = quantized_linear(o.reshape(M, Hq * 128), *weights["o"], g)
    h1, y1 = add_rmsnorm(x, attn_out, eps)
    gu = quantized_linear(y1, *weights["ug"], g)
    a = bf16(swiglu(gu))
    down = quantized_linear(a, *weights["down"], g, hadamard_online=True)
    out, _ = add_rmsnorm(h1, down, eps)
    inter = dict(y0=y0, qkv=qkv, q=qb.reshape(M, Hq, 128), o=o.reshape(M, Hq, 128),
                 attn_out=attn_out, h1=h1, y1=y1, gu=gu, a=a, down=down)
    return out, inter, cache
