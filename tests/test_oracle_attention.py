"""Pins of the decode-attention oracle (oracle/attention.py) against facts fixed
by the mathematics: closed forms (one position, identical keys, a dominant
key), an independent implementation of softmax attention (torch's fp64 SDPA),
the explicit Hadamard matrix, and invariances of the dequantized cache."""
import math

import numpy as np
import pytest
import torch

from oracle import attention as OA
from oracle import hadamard as OH
from oracle import quantizer as OQ
from paper_2606_07116_amd import inputs


def _case(B=2, H=3, S=40, Dh=128, seed=1):
    q = inputs.queries(B, H, Dh, seed=seed)
    kc, ks, kz = inputs.kv4_cache(B, H, S, Dh, seed=seed)
    vc, vs, vz = inputs.kv4_cache(B, H, S, Dh, seed=seed + 1)
    return q, kc, ks, kz, vc, vs, vz


def _deq_loops(codes, scale, zero):
    """Dequantize one row with explicit loops (low nibble = even dimension)."""
    out = []
    for byte in codes:
        out.append(float(scale) * ((int(byte) & 15) - int(zero)))
        out.append(float(scale) * ((int(byte) >> 4) - int(zero)))
    return np.array(out)


def test_dequantize_rows_matches_loops():
    _, kc, ks, kz, _, _, _ = _case(B=1, H=2, S=5, Dh=16)
    d = OA.dequantize_rows(kc, ks, kz)
    for h in range(2):
        for j in range(5):
            assert np.array_equal(d[0, h, j], _deq_loops(kc[0, h, j], ks[0, h, j], kz[0, h, j]))


def test_rotate_query_is_bf16_of_normalised_hadamard():
    q = inputs.queries(3, 4, 128, seed=2)
    qr = OA.rotate_query(q)
    exact = q.astype(np.float64) @ OH.sylvester(128).astype(np.float64) / math.sqrt(128)
    # bf16 values: low 16 bits of the fp32 pattern are zero
    assert np.all((qr.astype(np.float32).view(np.uint32) & 0xFFFF) == 0)
    # nearest bf16 of the exact rotation (up to the fp32 steps before rounding)
    assert np.all(np.abs(qr - exact) <= 2.0 ** -8 * np.abs(exact) * (1 + 2.0 ** -12) + 1e-30)
    # an orthogonal map keeps the norm (to bf16 precision)
    n0 = np.linalg.norm(q.astype(np.float64), axis=-1)
    assert np.allclose(np.linalg.norm(qr, axis=-1), n0, rtol=2.0 ** -8)


def test_rotate_query_tiny_closed_form():
    # Dh = 2: H = [[1, 1], [1, -1]] / sqrt(2); q = (1, 0) -> (c, c) with c = bf16(fl32(1/sqrt 2))
    qr = OA.rotate_query(np.array([[[1.0, 0.0]]], np.float32))
    c = float(np.float32(1.0 / math.sqrt(2.0)))
    c_bf16 = 0.70703125  # nearest bf16 to 0.70710678
    assert abs(c - 0.70710678) < 1e-7
    assert np.array_equal(qr[0, 0], [c_bf16, c_bf16])
    qr = OA.rotate_query(np.array([[[0.0, 2.0]]], np.float32))
    assert np.array_equal(qr[0, 0], [2 * c_bf16, -2 * c_bf16])


def test_single_position_returns_its_value_row():
    q, kc, ks, kz, vc, vs, vz = _case(S=8)
    o = OA.decode_attention(q, kc, ks, kz, vc, vs, vz, 1, 1 / math.sqrt(128))
    assert np.array_equal(o, OA.dequantize_rows(vc[:, :, :1], vs[:, :, :1], vz[:, :, :1])[:, :, 0])


def test_identical_keys_average_the_values():
    q, kc, ks, kz, vc, vs, vz = _case(S=17)
    kc[:] = kc[:, :, :1]
    ks[:] = ks[:, :, :1]
    kz[:] = kz[:, :, :1]
    o = OA.decode_attention(q, kc, ks, kz, vc, vs, vz, 17, 1 / math.sqrt(128))
    mean = OA.dequantize_rows(vc, vs, vz).mean(axis=2)
    assert np.allclose(o, mean, rtol=0, atol=1e-12)


def test_dominant_key_selects_its_value():
    q, kc, ks, kz, vc, vs, vz = _case(S=30)
    o = OA.decode_attention(q, kc, ks, kz, vc, vs, vz, 30, 1e4)
    qr = OA.rotate_query(q)
    k = OA.dequantize_rows(kc, ks, kz)
    best = np.einsum("bhd,bhsd->bhs", qr, k).argmax(axis=-1)
    v = OA.dequantize_rows(vc, vs, vz)
    want = np.take_along_axis(v, best[..., None, None], axis=2)[:, :, 0]
    assert np.all(np.isfinite(o))
    assert np.allclose(o, want, rtol=0, atol=1e-9)


@pytest.mark.parametrize("seq_len", [1, 7, 40])
def test_matches_torch_sdpa(seq_len):
    q, kc, ks, kz, vc, vs, vz = _case(S=40)
    sm = 1 / math.sqrt(128)
    o = OA.decode_attention(q, kc, ks, kz, vc, vs, vz, seq_len, sm)
    qr = torch.from_numpy(OA.rotate_query(q))[:, :, None, :]
    k = torch.from_numpy(OA.dequantize_rows(kc, ks, kz)[:, :, :seq_len])
    v = torch.from_numpy(OA.dequantize_rows(vc, vs, vz)[:, :, :seq_len])
    ref = torch.nn.functional.scaled_dot_product_attention(qr, k, v, scale=sm)[:, :, 0].numpy()
    assert np.allclose(o, ref, rtol=1e-12, atol=1e-12)


def test_positions_past_seq_len_are_ignored():
    q, kc, ks, kz, vc, vs, vz = _case(S=40)
    o = OA.decode_attention(q, kc, ks, kz, vc, vs, vz, 25, 0.1)
    kc2, vc2 = kc.copy(), vc.copy()
    kc2[:, :, 25:] = 255 - kc2[:, :, 25:]
    vc2[:, :, 25:] = 0
    assert np.array_equal(o, OA.decode_attention(q, kc2, ks, kz, vc2, vs, vz, 25, 0.1))


def test_zero_point_shift_leaves_output_unchanged():
    q, kc, ks, kz, vc, vs, vz = _case(S=12, Dh=64)
    # shift every code of the rows that avoid 15 by one level, and their zero-points too
    codes = OQ.unpack_nibbles(kc)
    ok = codes.max(axis=-1) < 15
    codes2 = codes + ok[..., None].astype(np.uint8)
    kz2 = kz + ok.astype(np.int16)
    o1 = OA.decode_attention(q, kc, ks, kz, vc, vs, vz, 12, 0.2)
    o2 = OA.decode_attention(q, OQ.pack_nibbles(codes2), ks, kz2, vc, vs, vz, 12, 0.2)
    assert np.allclose(o1, o2, rtol=0, atol=1e-12)


def test_value_rotation_is_undone_with_the_explicit_matrix():
    q, kc, ks, kz, vc, vs, vz = _case(S=20)
    sm = 0.3
    o_rot = OA.decode_attention(q, kc, ks, kz, vc, vs, vz, 20, sm, v_hadamard=True)
    o_plain = OA.decode_attention(q, kc, ks, kz, vc, vs, vz, 20, sm, v_hadamard=False)
    h = OH.sylvester(128).astype(np.float64) / math.sqrt(128)
    assert np.allclose(o_rot, o_plain @ h, rtol=0, atol=1e-12)
    # and with values that really were rotated before quantization, the
    # rotated-back output approximates attention over the unrotated values
    v = inputs.kv_rows(2 * 3 * 20, 128, seed=9).reshape(2, 3, 20, 128)
    from oracle import kv as OKV
    codes, s, z = OKV.kv_quantize(OKV.kv_rotate(v.reshape(-1, 128), True).astype(np.float32))
    vc_r = OQ.pack_nibbles(codes).reshape(2, 3, 20, 64)
    o = OA.decode_attention(q, kc, ks, kz, vc_r, s.reshape(2, 3, 20), z.reshape(2, 3, 20), 20, sm,
                            v_hadamard=True)
    qr = OA.rotate_query(q)
    p = OA.softmax(sm * np.einsum("bhd,bhsd->bhs", qr, OA.dequantize_rows(kc, ks, kz)))
    want = np.einsum("bhs,bhsd->bhd", p, v.astype(np.float64))
    # 4-bit quantization error of each value row: at most half a step (s/2) per
    # rotated coordinate, so at most sqrt(128) s / 2 in norm after rotating back
    err = np.linalg.norm(o - want, axis=-1)
    bound = np.sqrt(128) * 0.5 * s.reshape(2, 3, 20).astype(np.float64).max(axis=-1) * 1.001
    assert np.all(err <= bound)


# ---------------------------------------------------------------- prefill form
def _prefill_case(B=2, T=9, Hq=4, Hkv=2, past=5, S=None, seed=3):
    S = S or past + T + 3
    q = inputs.queries(B * T, Hq, 128, seed=seed).reshape(B, T, Hq, 128)
    kc, ks, kz = inputs.kv4_cache(B, Hkv, S, 128, seed=seed)
    vc, vs, vz = inputs.kv4_cache(B, Hkv, S, 128, seed=seed + 1)
    return q, kc, ks, kz, vc, vs, vz


@pytest.mark.parametrize("B,T,Hq,Hkv,past", [(2, 9, 4, 2, 5), (1, 12, 2, 2, 0), (2, 5, 8, 2, 30)])
def test_prefill_matches_torch_sdpa_with_an_explicit_causal_mask(B, T, Hq, Hkv, past):
    """torch's fp64 SDPA on the dequantized cache, the grouped heads expanded
    by repeat_interleave and the mask built as a boolean matrix."""
    q, kc, ks, kz, vc, vs, vz = _prefill_case(B, T, Hq, Hkv, past)
    sm = 1 / math.sqrt(128)
    o = OA.prefill_attention(q, kc, ks, kz, vc, vs, vz, past, sm)
    n = past + T
    qr = torch.from_numpy(OA.rotate_query(q)).permute(0, 2, 1, 3)          # [B, Hq, T, D]
    k = torch.from_numpy(OA.dequantize_rows(kc, ks, kz)[:, :, :n]).repeat_interleave(Hq // Hkv, 1)
    v = torch.from_numpy(OA.dequantize_rows(vc, vs, vz)[:, :, :n]).repeat_interleave(Hq // Hkv, 1)
    mask = torch.zeros(T, n, dtype=torch.bool)
    for t in range(T):
        mask[t, :past + t + 1] = True
    ref = torch.nn.functional.scaled_dot_product_attention(qr, k, v, attn_mask=mask, scale=sm)
    assert np.allclose(o, ref.permute(0, 2, 1, 3).numpy(), rtol=1e-12, atol=1e-12)


def test_prefill_first_token_of_an_empty_context_returns_its_value_row():
    q, kc, ks, kz, vc, vs, vz = _prefill_case(past=0)
    o = OA.prefill_attention(q, kc, ks, kz, vc, vs, vz, 0, 0.7)
    v0 = OA.dequantize_rows(vc[:, :, :1], vs[:, :, :1], vz[:, :, :1])[:, :, 0]   # [B, Hkv, D]
    want = np.repeat(v0, 2, axis=1)
    assert np.allclose(o[:, 0], want, rtol=0, atol=1e-12)


def test_prefill_rows_are_decode_steps_over_their_prefixes():
    """Row t of the prefill is the decode step of that token with
    seq_len = past + t + 1 (the other path of the oracle), and a subset of
    rows computes the same values."""
    q, kc, ks, kz, vc, vs, vz = _prefill_case(past=4, T=7)
    o = OA.prefill_attention(q, kc, ks, kz, vc, vs, vz, 4, 0.2)
    for t in range(7):
        d = OA.decode_attention(q[:, t], kc, ks, kz, vc, vs, vz, 4 + t + 1, 0.2)
        assert np.allclose(o[:, t], d, rtol=1e-13, atol=1e-13)
    sub = OA.prefill_attention(q, kc, ks, kz, vc, vs, vz, 4, 0.2, rows=[6, 2])
    assert np.array_equal(sub, o[:, [6, 2]])


def test_prefill_later_positions_do_not_reach_earlier_queries():
    """Changing the cache row at position j changes exactly the queries that
    attend to it (t >= j - past)."""
    past, T = 3, 8
    q, kc, ks, kz, vc, vs, vz = _prefill_case(past=past, T=T)
    o = OA.prefill_attention(q, kc, ks, kz, vc, vs, vz, past, 0.5)
    j = past + 4
    kc2, vc2 = kc.copy(), vc.copy()
    kc2[:, :, j] = 255 - kc2[:, :, j]
    vc2[:, :, j] = 255 - vc2[:, :, j]
    o2 = OA.prefill_attention(q, kc2, ks, kz, vc2, vs, vz, past, 0.5)
    assert np.array_equal(o[:, :4], o2[:, :4])
    assert np.all(np.abs(o[:, 4:] - o2[:, 4:]).max(axis=(2, 3)) > 1e-6)
