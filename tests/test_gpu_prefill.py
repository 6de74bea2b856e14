"""GPU parity: the prefill form of the decoder-layer chain.

offq_kv_attention_prefill (causal attention of T new tokens per sequence over
the 4-bit cache) against oracle.attention.prefill_attention, and
offq_rope_kv_prefill (RoPE, H3 and the KV4 quantizer for T tokens per
sequence) against the oracle's KV rows and quantizer.

The attention bar is the decode kernel's (tests/test_gpu_kv_attention.py),
per query row:
  |out - ref| <= 2^-8 (1 + 2^-5) |ref| + 2^-11 E,
  E = sum_j p_j max_d |V_j[d]| over the row's attended positions.
The kernel does the decode arithmetic on the matrix cores: exact products of
fp16 operands (the 4-bit codes enter as fp16 values c 2^-24), fp32 sums, the
weights p sv rounded to fp16 once, and one bf16 rounding of the output.
"""
import math

import numpy as np
import pytest
import torch

import paper_2606_07116_amd as offq
from oracle import attention as OA
from oracle import gemm as OG
from oracle import kv as OKV
from oracle import layer as OL
from oracle import quantizer as OQ
from paper_2606_07116_amd import inputs
from tests import parity as P

pytestmark = pytest.mark.gpu

SM = 1.0 / math.sqrt(128.0)


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(P.DEV)


def _magnitude(q, kc, ks, kz, vc, vs, vz, past, sm, rows):
    """E per (b, row, head) for the rows listed: sum_j p_j max_d |V_j[d]|."""
    n = past + int(max(rows)) + 1
    qr = OA.rotate_query(q[:, rows])
    k = OA.dequantize_rows(kc[:, :, :n], ks[:, :, :n], kz[:, :, :n])
    vmax = np.abs(OA.dequantize_rows(vc[:, :, :n], vs[:, :, :n], vz[:, :, :n])).max(-1)
    g = qr.shape[2] // k.shape[1]
    k, vmax = np.repeat(k, g, axis=1), np.repeat(vmax, g, axis=1)
    s = sm * np.einsum("brhd,bhsd->bhrs", qr, k)
    s = np.where(np.arange(n)[None, :] <= (past + np.asarray(rows))[:, None], s, -np.inf)
    p = OA.softmax(s)
    return np.einsum("bhrs,bhs->brh", p, vmax)[..., None]


def check(out, ref, mag):
    out = out.astype(np.float64)
    tol = 2.0 ** -8 * (1 + 2.0 ** -5) * np.abs(ref) + 2.0 ** -11 * mag
    bad = np.abs(out - ref) > tol
    assert not bad.any(), (
        f"prefill attention mismatch at {np.argwhere(bad)[:5].tolist()} (of {bad.sum()}): "
        f"gpu {out[bad][:5]} ref {ref[bad][:5]}")


def _host_cache(B, Hkv, S, seed, poison_from=None):
    kc, ks, kz = inputs.kv4_cache(B, Hkv, S, 128, seed=seed)
    vc, vs, vz = inputs.kv4_cache(B, Hkv, S, 128, seed=seed + 1)
    if poison_from is not None and poison_from < S:
        # rows past the last attended position: codes that would dominate
        # every score and huge values (never read)
        kc[:, :, poison_from:] = 0xFF
        ks[:, :, poison_from:] = np.float16(60000.0)
        kz[:, :, poison_from:] = -30000
        vs[:, :, poison_from:] = np.float16(np.inf)
    return kc, ks, kz, vc, vs, vz


def _cache_dict(kc, ks, kz, vc, vs, vz):
    return dict(k_codes=_dev(kc), k_scale=_dev(ks), k_zero=_dev(kz), v_codes=_dev(vc),
                v_scale=_dev(vs), v_zero=_dev(vz))


def _run(B, T, Hq, Hkv, past, S=None, v_had=False, seed=0, rows=None, sm=SM, cache=None):
    S = S or past + T + 5
    q = inputs.queries(B * T, Hq, 128, seed=seed).reshape(B, T, Hq, 128)
    c = cache if cache is not None else _host_cache(B, Hkv, S, seed, poison_from=past + T)
    out = offq.offq_kv_attention_prefill(P.to_dev_bf16(q), _cache_dict(*c), past, sm_scale=sm,
                                         v_hadamard=v_had)
    torch.cuda.synchronize()
    got = P.host(out.float())
    rows = list(range(T)) if rows is None else rows
    ref = OA.prefill_attention(q, *c, past, sm, v_hadamard=v_had, rows=rows)
    check(got[:, rows], ref, _magnitude(q, *c, past, sm, rows))
    return out


@pytest.mark.parametrize("B,T,Hq,Hkv,past", [
    (1, 1, 4, 1, 0), (1, 1, 4, 1, 37),        # one token, with and without context
    (2, 37, 4, 1, 0), (1, 64, 4, 1, 0),       # a ragged and a whole 64-position workgroup
    (1, 100, 8, 2, 5),                        # two workgroups, ragged, a short context
    (2, 65, 2, 2, 0), (1, 300, 2, 2, 0),      # G = 1 (256 positions per workgroup)
    (1, 130, 4, 2, 3),                        # G = 2 (128 positions per workgroup)
    (1, 40, 8, 1, 0), (1, 33, 16, 2, 70),     # G = 8 (32 positions per workgroup)
    (2, 300, 8, 2, 200),                      # many key blocks, a context longer than a block
])
def test_prefill_attention_shapes(B, T, Hq, Hkv, past):
    _run(B, T, Hq, Hkv, past, seed=B * 1000 + T + past)


@pytest.mark.parametrize("v_had", [False, True])
def test_prefill_attention_value_rotation(v_had):
    _run(2, 70, 4, 1, 9, v_had=v_had, seed=7)


@pytest.mark.parametrize("sm", [0.01, 0.3])
def test_prefill_attention_score_scales(sm):
    """Flat and peaked softmax rows."""
    _run(1, 90, 4, 2, 40, sm=sm, seed=8)


@pytest.mark.parametrize("past,T", [(0, 2048), (1536, 512)])
def test_prefill_attention_full_size_sampled(past, T):
    """A Llama-3-8B layer's shape (32 query heads, 8 kv heads), two sequences:
    a 2048-token prefill, and a 512-token chunk after 1536 cached positions.
    Every output is computed; rows at tile edges and spread over the range
    are compared."""
    rows = sorted({0, 1, 31, 32, 63, 64, 127, 128, T // 2 - 1, T // 2, T - 33, T - 32, T - 2,
                   T - 1, 777 % T, 1500 % T})
    _run(2, T, 32, 8, past, S=past + T, rows=rows, seed=past + T)


@pytest.mark.parametrize("case", ["offset_keys", "int16_range"])
def test_prefill_attention_large_zero_points(case):
    """Attended rows with large zero-points, the regime the method creates
    (Eq. 1, Eq. 5): rows quantized by the oracle from keys and values whose
    first channel carries an offset of 300..3000, and zero-points drawn over
    the int16 range with small scales."""
    from tests.test_gpu_kv_attention import _offset_key_cache
    B, Hkv, T, past = 2, 2, 150, 60
    S = past + T
    if case == "offset_keys":
        kc, ks, kz = _offset_key_cache(B, Hkv, S, 21, 300.0, 3000.0)
        vc, vs, vz = _offset_key_cache(B, Hkv, S, 22, 300.0, 3000.0)
        assert np.abs(kz).max() >= 100
        sm = 0.002
    else:
        rng = np.random.default_rng(5)
        kc, _, _ = inputs.kv4_cache(B, Hkv, S, 128, seed=23)
        vc, _, _ = inputs.kv4_cache(B, Hkv, S, 128, seed=24)
        ks = rng.uniform(0.005, 0.02, size=(B, Hkv, S)).astype(np.float16)
        vs = rng.uniform(0.005, 0.02, size=(B, Hkv, S)).astype(np.float16)
        kz = rng.integers(-32768, 32768, size=(B, Hkv, S)).astype(np.int16)
        vz = rng.integers(-32768, 32768, size=(B, Hkv, S)).astype(np.int16)
        sm = SM
    _run(B, T, 8, Hkv, past, S=S, seed=25, sm=sm, cache=(kc, ks, kz, vc, vs, vz))


@pytest.mark.parametrize("sm", [0.05, 1.0])
def test_prefill_attention_large_value_scales(sm):
    """Value scales up to 60000 (fp16's top binade): a weight p sv must stay
    finite in fp16, so the reference maximum of a row may lag its true
    maximum by less there (sm = 1: peaked rows whose maximum keeps moving)."""
    B, Hkv, T, past = 1, 2, 200, 30
    S = past + T
    rng = np.random.default_rng(int(sm * 100))
    kc, ks, kz, vc, _, vz = _host_cache(B, Hkv, S, 31)
    vs = rng.uniform(2000.0, 60000.0, size=(B, Hkv, S)).astype(np.float16)
    _run(B, T, 8, Hkv, past, S=S, seed=32, sm=sm, cache=(kc, ks, kz, vc, vs, vz))


def test_prefill_attention_deterministic_and_out_buffer():
    B, T, Hq, Hkv, past = 1, 80, 4, 1, 10
    q = inputs.queries(B * T, Hq, 128, seed=3).reshape(B, T, Hq, 128)
    cache = _cache_dict(*_host_cache(B, Hkv, past + T, 3))
    qd = P.to_dev_bf16(q)
    a = offq.offq_kv_attention_prefill(qd, cache, past)
    out = torch.full_like(a, 5.0)
    b = offq.offq_kv_attention_prefill(qd, cache, past, out=out)
    torch.cuda.synchronize()
    assert b.data_ptr() == out.data_ptr() and torch.equal(a, b)


def test_prefill_attention_refuses_bad_arguments():
    B, T, Hkv, past = 1, 8, 1, 0
    cache = _cache_dict(*_host_cache(B, Hkv, 8, 4))
    q3 = torch.zeros((B, T, 3, 128), dtype=torch.bfloat16, device=P.DEV)
    with pytest.raises(offq.OffqError, match="UNSUPPORTED"):
        offq.offq_kv_attention_prefill(q3, cache, past)        # Hq / Hkv = 3
    q4 = torch.zeros((B, T, 4, 128), dtype=torch.bfloat16, device=P.DEV)
    with pytest.raises(offq.OffqError, match="INVALID"):
        offq.offq_kv_attention_prefill(q4, cache, 1)           # past + T > s_cap
    with pytest.raises(offq.OffqError, match="INVALID"):
        offq.offq_kv_attention_prefill(q4, cache, past, out=q4)  # out overlaps q
    e = offq.offq_kv_attention_prefill(torch.zeros((B, 0, 4, 128), dtype=torch.bfloat16,
                                                   device=P.DEV), cache, past)
    assert e.shape == (B, 0, 4, 128)


def _zero_cache(B, Hkv, s_cap, fill):
    z = lambda *s, dt: torch.full(s, fill, dtype=dt, device=P.DEV)
    return dict(k_codes=z(B, Hkv, s_cap, 64, dt=torch.uint8), v_codes=z(B, Hkv, s_cap, 64, dt=torch.uint8),
                k_scale=z(B, Hkv, s_cap, dt=torch.float16), v_scale=z(B, Hkv, s_cap, dt=torch.float16),
                k_zero=z(B, Hkv, s_cap, dt=torch.int16), v_zero=z(B, Hkv, s_cap, dt=torch.int16))


@pytest.mark.parametrize("B,T,Hq,Hkv,past,s_cap", [(2, 37, 8, 2, 5, 50), (1, 300, 32, 8, 0, 300),
                                                  (2, 150, 5, 1, 20, 170)])
def test_rope_kv_prefill(B, T, Hq, Hkv, past, s_cap):
    """Row b T + t lands at position past + t of sequence b's cache, as the
    oracle's RoPE + H3 + KV quantizer writes it; nothing else changes."""
    M = B * T
    rng = np.random.default_rng(T)
    qkv = inputs.round_to_bf16(rng.standard_normal((M, (Hq + 2 * Hkv) * 128)).astype(np.float32) * 2)
    pos = (past + np.tile(np.arange(T), B)).astype(np.int32)
    cache = _zero_cache(B, Hkv, s_cap, 7)
    q, ky, vy = offq.offq_rope_kv_prefill(P.to_dev_bf16(qkv), B, Hq, Hkv, _dev(pos), cache,
                                          debug=True)
    # the same rows through the decode form (one token per sequence, T = 1)
    dcache = _zero_cache(M, Hkv, s_cap, 7)
    q1, ky1, vy1 = offq.offq_rope_kv_append(P.to_dev_bf16(qkv), Hq, Hkv, _dev(pos), dcache,
                                            debug=True)
    torch.cuda.synchronize()
    assert torch.equal(q, q1) and torch.equal(ky, ky1) and torch.equal(vy, vy1)
    q_ref, ky_ref, vy_ref = OL.kv_rows(qkv, Hq, Hkv, pos, 500000.0)
    assert np.array_equal(P.host(vy), vy_ref)
    # the query within one bf16 ulp of the oracle's RoPE; the key rows within
    # the rotation bound of the decode form's test (fp32 RoPE, a bf16 rounding
    # of the key before H3, the 7-stage fp32 butterfly)
    qg = P.host(q.float()).astype(np.float64)
    qr = OL.bf16(q_ref)
    assert np.all(np.abs(qg - qr) <= OG.bf16_ulp(qr) * (1 + 1e-9) + 1e-6 * np.abs(q_ref).max())
    k_in = OL.bf16(OL.rope(qkv.reshape(M, Hq + 2 * Hkv, 128)[:, Hq:Hq + Hkv], pos[:, None], 500000.0))
    kb = (7 + 2) * 2.0 ** -24 * np.abs(k_in).sum(-1, keepdims=True) / math.sqrt(128) + \
        OG.bf16_ulp(k_in).sum(-1, keepdims=True) / math.sqrt(128) + 1e-5 * np.abs(k_in).max(-1, keepdims=True)
    assert np.all(np.abs(P.host(ky) - ky_ref) <= kb)
    for name, rows in (("k", P.host(ky)), ("v", P.host(vy))):
        codes, s, z = OKV.kv_quantize(rows.reshape(-1, 128))
        packed = OQ.pack_nibbles(codes).reshape(B, T, Hkv, 64).transpose(0, 2, 1, 3)
        c = P.host(cache[name + "_codes"])
        sc = P.fp16_bits(P.host(cache[name + "_scale"]))
        zz = P.host(cache[name + "_zero"])
        assert np.array_equal(c[:, :, past:past + T], packed), name
        assert np.array_equal(sc[:, :, past:past + T],
                              P.fp16_bits(s.reshape(B, T, Hkv).transpose(0, 2, 1))), name
        assert np.array_equal(zz[:, :, past:past + T], z.reshape(B, T, Hkv).transpose(0, 2, 1)), name
        others = np.r_[0:past, past + T:s_cap]
        assert np.all(c[:, :, others] == 7) and np.all(zz[:, :, others] == 7), name
