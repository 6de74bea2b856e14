"""Host-only checks of the C ABI: the library loads, exports every symbol the
header declares, and rejects bad arguments before touching a device."""
import ctypes
import os
import re

import numpy as np
import pytest
import torch

from paper_2606_07116_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _header_functions():
    src = open(os.path.join(ROOT, "include", "offq.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(offq_[a-z0-9_]+)\s*\(", src)))


def test_exports_every_declared_symbol():
    names = _header_functions()
    assert "offq_rotate_quantize" in names and "offq_w4a4_gemm" in names
    assert "offq_kv_quantize" in names and "offq_pack_weights" in names
    lib = ctypes.CDLL(_lib.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(_lib.EXPORTED) == names


def test_version_and_status_strings():
    assert _lib.ABI_VERSION == 1
    assert _lib.status_name(0) == "OFFQ_OK"
    assert _lib.status_name(1) == "OFFQ_ERR_INVALID"
    assert _lib.status_name(2) == "OFFQ_ERR_UNSUPPORTED"
    assert _lib.status_name(3) == "OFFQ_ERR_HIP"
    assert _lib.status_name(99) == "OFFQ_ERR_UNKNOWN"


P = 0x10000  # a fake, 64 KiB-aligned address: never dereferenced (validation fails first)


@pytest.mark.parametrize("args,expect", [
    # (x, M, K, ldx, g, had, codes, scale, zero, ydbg)
    ((P, 4, 256, 256, 100, 1, P, P, P, None), _lib.OFFQ_ERR_INVALID),      # g not power of 2
    ((P, 4, 256, 256, 8, 1, P, P, P, None), _lib.OFFQ_ERR_UNSUPPORTED),    # g too small
    ((P, 4, 32768, 32768, 16384, 1, P, P, P, None), _lib.OFFQ_ERR_UNSUPPORTED),  # g too large
    ((P, 4, 384, 384, 256, 1, P, P, P, None), _lib.OFFQ_ERR_INVALID),      # K % g
    ((P, 4, 256, 200, 256, 1, P, P, P, None), _lib.OFFQ_ERR_INVALID),      # ldx < K
    ((P, 4, 256, 260, 256, 1, P, P, P, None), _lib.OFFQ_ERR_INVALID),      # ldx % 8
    ((P, 4, 256, 256, 256, 2, P, P, P, None), _lib.OFFQ_ERR_INVALID),      # bad flag
    ((None, 4, 256, 256, 256, 1, P, P, P, None), _lib.OFFQ_ERR_INVALID),   # null x
    ((P + 8, 4, 256, 256, 256, 1, P, P, P, None), _lib.OFFQ_ERR_INVALID),  # misaligned x
    ((P, 4, 256, 256, 256, 1, P + 2, P, P, None), _lib.OFFQ_ERR_INVALID),  # misaligned codes
    ((P, -1, 256, 256, 256, 1, P, P, P, None), _lib.OFFQ_ERR_INVALID),     # M < 0
    ((P, 0, 256, 256, 256, 1, P, P, P, None), _lib.OFFQ_OK),               # empty: no-op
])
def test_rotate_quantize_validation(args, expect):
    st = _lib.offq_rotate_quantize_raw(*args, None)
    assert st == expect, _lib.last_error()
    if st != _lib.OFFQ_OK:
        assert _lib.last_error()


@pytest.mark.parametrize("args,expect", [
    # (a, as, az, w, ws, cs, M, N, K, g, y, ldy, acc)
    ((P, P, P, P, P, P, 4, 8, 256, 32, P, 8, None), _lib.OFFQ_ERR_UNSUPPORTED),  # g < 64
    ((P, P, P, P, P, P, 4, 8, 256, 96, P, 8, None), _lib.OFFQ_ERR_INVALID),      # g not pow2
    ((P, P, P, P, P, P, 4, 8, 320, 256, P, 8, None), _lib.OFFQ_ERR_INVALID),     # K % g
    ((P, P, P, P, P, P, 4, 8, 256, 256, P, 4, None), _lib.OFFQ_ERR_INVALID),     # ldy < N
    ((P, P, P, P, P, P, 4, 0, 256, 256, P, 8, None), _lib.OFFQ_ERR_INVALID),     # N = 0
    ((P, P, P, None, P, P, 4, 8, 256, 256, P, 8, None), _lib.OFFQ_ERR_INVALID),  # null w
    ((P + 4, P, P, P, P, P, 4, 8, 256, 256, P, 8, None), _lib.OFFQ_ERR_INVALID), # misaligned
    ((P, P, P, P, P, P, 0, 8, 256, 256, P, 8, None), _lib.OFFQ_OK),              # M = 0
])
def test_gemm_validation(args, expect):
    st = _lib.offq_w4a4_gemm_raw(*args, None)
    assert st == expect, _lib.last_error()


@pytest.mark.parametrize("args,expect", [
    # (kv, rows, Dh, stride, had, codes, scale, zero, ydbg)
    ((P, 10, 96, 96, 1, P, P, P, None), _lib.OFFQ_ERR_INVALID),
    ((P, 10, 128, 120, 1, P, P, P, None), _lib.OFFQ_ERR_INVALID),
    ((P, 10, 128, 132, 1, P, P, P, None), _lib.OFFQ_ERR_INVALID),
    ((P, 10, 8, 8, 1, P, P, P, None), _lib.OFFQ_ERR_UNSUPPORTED),
    ((P, 0, 128, 128, 1, P, P, P, None), _lib.OFFQ_OK),
])
def test_kv_validation(args, expect):
    st = _lib.offq_kv_quantize_raw(*args, None)
    assert st == expect, _lib.last_error()


@pytest.mark.parametrize("args,expect", [
    ((P, 8, 256, 48, P, P, P), _lib.OFFQ_ERR_INVALID),
    ((P, 8, 65536, 64, P, P, P), _lib.OFFQ_ERR_UNSUPPORTED),   # K/g > 512
    ((P, 0, 256, 64, P, P, P), _lib.OFFQ_ERR_INVALID),
    ((P + 4, 8, 256, 64, P, P, P), _lib.OFFQ_ERR_INVALID),
])
def test_pack_weights_validation(args, expect):
    st = _lib.offq_pack_weights_raw(*args, None)
    assert st == expect, _lib.last_error()


def test_valid_call_without_gpu_reports_hip_error():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    st = _lib.offq_rotate_quantize_raw(P, 4, 256, 256, 256, 1, P, P, P, None, None)
    assert st == _lib.OFFQ_ERR_HIP


@pytest.mark.parametrize("args,expect", [
    # (B, H, s_cap, seq_len, head_dim, sm_scale, v_had, workspace_bytes)
    ((2, 4, 100, 0, 128, 0.1, 0, 1 << 20), _lib.OFFQ_ERR_INVALID),        # seq_len = 0
    ((2, 4, 100, 101, 128, 0.1, 0, 1 << 20), _lib.OFFQ_ERR_INVALID),      # seq_len > s_cap
    ((2, 4, 100, 100, 64, 0.1, 0, 1 << 20), _lib.OFFQ_ERR_UNSUPPORTED),   # head_dim 64
    ((0, 4, 100, 100, 128, 0.1, 0, 1 << 20), _lib.OFFQ_ERR_INVALID),      # B = 0
    ((2, 4, 100, 100, 128, 0.1, 2, 1 << 20), _lib.OFFQ_ERR_INVALID),      # bad flag
    ((2, 4, 100, 100, 128, float("nan"), 0, 1 << 20), _lib.OFFQ_ERR_INVALID),
    ((2, 4, 2048, 2048, 128, 0.1, 0, 8 * 4 * 130 * 4 - 4), _lib.OFFQ_ERR_INVALID),  # small ws
    ((1 << 12, 1 << 12, 1 << 20, 1 << 20, 128, 0.1, 0, 1 << 60), _lib.OFFQ_ERR_UNSUPPORTED),
])
def test_kv_attention_validation(args, expect):
    B, H, s_cap, seq_len, dh, sm, vh, wsb = args
    st = _lib.offq_kv_attention_decode_raw(P, P, P, P, P, P, P, B, H, s_cap, seq_len, dh, sm, vh, P,
                                           P, wsb, None)
    assert st == expect, _lib.last_error()
    assert _lib.last_error()


def test_kv_attention_misaligned_and_null():
    args = [P] * 7 + [2, 4, 100, 100, 128, 0.1, 0, P, P, 1 << 20, None]
    for i, bad in ((1, P + 4), (4, P + 2), (0, None), (15, None)):
        a = list(args)
        a[i] = bad
        assert _lib.offq_kv_attention_decode_raw(*a) == _lib.OFFQ_ERR_INVALID, i


def test_kv_attention_quantize_validation():
    # q, 6 cache arrays, B, Hq, Hkv, s_cap, seq_len, head_dim, sm_scale, v_had,
    # out, out_codes, out_scale, out_zero, workspace, workspace_bytes, stream
    names = ["q", "kc", "ks", "kz", "vc", "vs", "vz", "B", "Hq", "Hkv", "s_cap", "seq_len",
             "head_dim", "sm", "v_had", "out", "codes", "scale", "zero", "ws", "wsb", "stream"]
    base = dict(zip(names, [P] * 7 + [2, 8, 2, 100, 100, 128, 0.1, 0, None, P, P, P, P, 1 << 20,
                                      None]))
    f = _lib.offq_kv_attention_decode_quantize_raw
    for k, bad in (("codes", None), ("scale", None), ("zero", None), ("scale", P + 1),
                   ("zero", P + 1), ("q", None), ("seq_len", 101), ("Hkv", 3), ("v_had", 2)):
        a = dict(base)
        a[k] = bad
        assert f(*[a[n] for n in names]) == _lib.OFFQ_ERR_INVALID, k
    a = dict(base)
    a["head_dim"] = 64
    assert f(*[a[n] for n in names]) == _lib.OFFQ_ERR_UNSUPPORTED
    # the plain entry point still requires its output
    assert _lib.offq_kv_attention_decode_gqa_raw(P, P, P, P, P, P, P, 2, 8, 2, 100, 100, 128, 0.1, 0,
                                                 None, P, 1 << 20, None) == _lib.OFFQ_ERR_INVALID


def test_kv_attention_workspace_bytes():
    # one record of 2 + 128 floats per (b, h, chunk of up to 512 positions)
    assert _lib.offq_kv_attention_workspace_bytes(2, 4, 1) == 8 * 130 * 4
    assert _lib.offq_kv_attention_workspace_bytes(2, 4, 512) == 8 * 130 * 4
    assert _lib.offq_kv_attention_workspace_bytes(2, 4, 1025) == 8 * 3 * 130 * 4
    assert _lib.offq_kv_attention_workspace_bytes(8, 32, 32768) == 256 * 64 * 130 * 4
    assert _lib.offq_kv_attention_workspace_bytes(0, 4, 10) == 0
    assert _lib.offq_kv_attention_workspace_bytes(1, 1, 0) == 0


def test_layer_and_calibration_validation():
    L = _lib
    # add_rmsnorm: D not a multiple of 8; no output
    assert L.offq_add_rmsnorm_raw(P, 16, None, 0, 4, 12, 1e-5, P, 16, P, 16, None) == L.OFFQ_ERR_INVALID
    assert L.offq_add_rmsnorm_raw(P, 16, None, 0, 4, 16, 1e-5, None, 0, None, 0, None) == L.OFFQ_ERR_INVALID
    assert L.offq_add_rmsnorm_raw(P, 16, None, 0, 0, 16, 1e-5, P, 16, None, 0, None) == L.OFFQ_OK
    # swiglu: ldg < 2F
    assert L.offq_swiglu_raw(P, 16, 2, 16, P, 16, None) == L.OFFQ_ERR_INVALID
    # rope: head_dim 64, bad flag
    args = [P, 768, 2, 2, 2, 128, P, 500000.0, 1, 0, P, P, P, P, P, P, P, 100, None, None, None]
    a = list(args); a[5] = 64
    assert L.offq_rope_kv_append_raw(*a) == L.OFFQ_ERR_UNSUPPORTED
    a = list(args); a[8] = 3
    assert L.offq_rope_kv_append_raw(*a) == L.OFFQ_ERR_INVALID
    a = list(args); a[1] = 700
    assert L.offq_rope_kv_append_raw(*a) == L.OFFQ_ERR_INVALID
    # gqa: Hq not a multiple of Hkv
    assert L.offq_kv_attention_decode_gqa_raw(P, P, P, P, P, P, P, 2, 6, 4, 100, 100, 128, 0.1, 0, P,
                                              P, 1 << 20, None) == L.OFFQ_ERR_INVALID
    # eigh: odd D, too large, small workspace
    f = lambda D, wsb: L.lib.offq_eigh(P, D, D, P, P, D, P, wsb, 30, 1e-14, None, None, None)
    assert f(7, 1 << 30) == L.OFFQ_ERR_INVALID
    assert f(16384, 1 << 40) == L.OFFQ_ERR_UNSUPPORTED
    assert f(64, 100) == L.OFFQ_ERR_INVALID
    assert L.lib.offq_eigh_workspace_bytes(64) >= 4 * 64 * 64 * 8
    # grouping: D not a multiple of g
    assert L.lib.offq_group_permutation(P, 100, 64, P, P, 400, None) == L.OFFQ_ERR_INVALID
    # rotation: g not a power of two with the Hadamard
    assert L.lib.offq_build_rotation(None, 0, 96, None, 24, 1, P, 96, None) == L.OFFQ_ERR_INVALID
    # top-1: D not a multiple of 8
    assert L.lib.offq_top1_select(P, 2, 3, 12, 16, 48, P, P, 12, P, 1 << 10, None) == L.OFFQ_ERR_INVALID


def test_package_import_does_not_load_the_library():
    """The oracle's CPU pins use the seeded generators of the package; importing
    them must not need the HIP build (the library loads on first use)."""
    import subprocess
    import sys
    code = ("import sys; import paper_2606_07116_amd.inputs, oracle.gemm; "
            "assert 'paper_2606_07116_amd._lib' not in sys.modules")
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


@pytest.mark.parametrize("change,expect", [
    ({}, None),                                             # valid: reaches the device check
    ({"head_dim": 64}, _lib.OFFQ_ERR_UNSUPPORTED),
    ({"Hq": 12, "Hkv": 4}, _lib.OFFQ_ERR_UNSUPPORTED),      # group of 3
    ({"Hq": 6, "Hkv": 4}, _lib.OFFQ_ERR_INVALID),           # not a multiple
    ({"past": 70}, _lib.OFFQ_ERR_INVALID),                  # past + T > s_cap
    ({"T": -1}, _lib.OFFQ_ERR_INVALID),
    ({"v_had": 2}, _lib.OFFQ_ERR_INVALID),
    ({"sm": 0.0}, _lib.OFFQ_ERR_INVALID),
    ({"q": None}, _lib.OFFQ_ERR_INVALID),
    ({"out": P + 8}, _lib.OFFQ_ERR_INVALID),                # misaligned (16 B)
    ({"out": P + 64}, _lib.OFFQ_ERR_INVALID),               # overlaps q
    ({"past": (1 << 30) - 10, "s_cap": 1 << 31}, _lib.OFFQ_ERR_UNSUPPORTED),
    ({"T": 0, "q": None, "out": None}, _lib.OFFQ_OK),       # empty: nothing to do
])
def test_kv_attention_prefill_validation(change, expect):
    names = ["q", "B", "T", "Hq", "Hkv", "head_dim", "past", "kc", "ks", "kz", "vc", "vs", "vz",
             "s_cap", "sm", "v_had", "out", "stream"]
    a = dict(zip(names, [P, 2, 64, 8, 2, 128, 0, P, P, P, P, P, P, 100, 0.1, 0, P + (1 << 24),
                         None]))
    a.update(change)
    st = _lib.offq_kv_attention_prefill_raw(*[a[n] for n in names])
    import torch
    if expect is None:
        if torch.cuda.is_available():
            pytest.skip("a GPU is present")
        expect = _lib.OFFQ_ERR_HIP
    assert st == expect, _lib.last_error()


def test_rope_kv_prefill_validation():
    L = _lib
    # qkv, ldq, B, T, Hq, Hkv, head_dim, positions, base, k_had, v_had, q_out,
    # 6 cache arrays, s_cap, k_dbg, v_dbg, stream
    args = [P, 768, 2, 3, 2, 2, 128, P, 500000.0, 1, 0, P, P, P, P, P, P, P, 100, None, None, None]
    for i, bad, expect in ((6, 64, L.OFFQ_ERR_UNSUPPORTED), (3, 0, L.OFFQ_ERR_INVALID),
                           (9, 2, L.OFFQ_ERR_INVALID), (1, 700, L.OFFQ_ERR_INVALID),
                           (7, None, L.OFFQ_ERR_INVALID)):
        a = list(args)
        a[i] = bad
        assert L.offq_rope_kv_prefill_raw(*a) == expect, (i, L.last_error())
    a = list(args)
    a[2] = 0  # no sequences: nothing to do
    assert L.offq_rope_kv_prefill_raw(*a) == L.OFFQ_OK


@pytest.mark.parametrize("N,K", [(1, 64), (16, 128), (17, 192), (300, 4096), (33, 8320)])
def test_blocked_weight_layout(N, K):
    """The blocked operand layout of the packed weights (include/offq.h,
    offq_pack_weights): byte kk of row n at ((n / 16) KB + kk / 64) 1024 +
    (n % 16) 64 + kk % 64, KB = ceil(K / 128), zero padding, and the
    conversions to and from row-major codes are inverse."""
    rng = np.random.default_rng(N * 7 + K)
    rows = rng.integers(0, 256, size=(N, K // 2), dtype=np.uint8)
    blk = _lib.blocked_weight_codes(rows)
    KB = -(-K // 128)
    assert blk.shape == _lib.weight_codes_shape(N, K) == (-(-N // 16), KB, 16, 64)
    assert blk.size == _lib.offq_weight_codes_bytes(N, K) == -(-N // 16) * KB * 1024
    flat = blk.reshape(-1)
    for n, kk in [(0, 0), (N - 1, K // 2 - 1), (N // 2, K // 4), (min(15, N - 1), min(63, K // 2 - 1))]:
        assert flat[((n // 16) * KB + kk // 64) * 1024 + (n % 16) * 64 + kk % 64] == rows[n, kk]
    assert int(flat.astype(np.int64).sum()) == int(rows.astype(np.int64).sum())  # zero padding
    assert np.array_equal(_lib.row_major_weight_codes(blk, N, K), rows)
    t = torch.from_numpy(rows)
    assert np.array_equal(_lib.blocked_weight_codes(t).numpy(), blk)
    assert _lib.offq_weight_codes_bytes(0, K) == 0 and _lib.offq_weight_codes_bytes(N, 0) == 0
