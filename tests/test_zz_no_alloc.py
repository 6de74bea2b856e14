"""offq_kv_attention_decode_noalloc (the decode attention with its chunk
records in the library's static scratch instead of a caller workspace)
through the C ABI: its outputs equal those of the workspace entry point
(the same kernels and arithmetic, so bit for bit) on two calls in a row, the
second with a smaller input, and sizes beyond the scratch are refused before
anything is enqueued."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2606_07116_amd import _lib, inputs
from tests import parity as P

pytestmark = pytest.mark.gpu

SM = 1.0 / 128 ** 0.5


def _case(B, Hq, Hkv, S, seed):
    kc, ks, kz = inputs.kv4_cache_device(B, Hkv, S, 128, seed=seed, device=P.DEV)
    vc, vs, vz = inputs.kv4_cache_device(B, Hkv, S, 128, seed=seed + 1, device=P.DEV)
    q = P.to_dev_bf16(inputs.queries(B, Hq, 128, seed=seed))
    return q, kc, ks, kz, vc, vs, vz


def _ptrs(ts):
    return [ctypes.c_void_p(t.data_ptr()) for t in ts]


def _both(B, Hq, Hkv, S, seq_len, v_had, seed):
    ops = _case(B, Hq, Hkv, S, seed)
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    ref = torch.full((B, Hq, 128), float("nan"), dtype=torch.bfloat16, device=P.DEV)
    wsb = _lib.offq_kv_attention_workspace_bytes(B, Hq, seq_len)
    ws = torch.empty(wsb // 4, dtype=torch.float32, device=P.DEV)
    st = _lib.offq_kv_attention_decode_gqa_raw(*_ptrs(ops), B, Hq, Hkv, S, seq_len, 128, SM,
                                               v_had, ctypes.c_void_p(ref.data_ptr()),
                                               ctypes.c_void_p(ws.data_ptr()), wsb, stream)
    assert st == _lib.OFFQ_OK, _lib.last_error()
    out = torch.full((B, Hq, 128), float("nan"), dtype=torch.bfloat16, device=P.DEV)
    st = _lib.offq_kv_attention_decode_noalloc_raw(*_ptrs(ops), B, Hq, Hkv, S, seq_len, 128, SM,
                                                   v_had, ctypes.c_void_p(out.data_ptr()), stream)
    assert st == _lib.OFFQ_OK, _lib.last_error()
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), ref.view(torch.int16))
    return out


@pytest.mark.parametrize("shapes", [
    # (B, Hq, Hkv, s_cap, seq_len, v_hadamard) of the first and the second call
    ((8, 32, 32, 32768, 32768, 0), (2, 4, 4, 3000, 2049, 1)),  # the attention workload, then small
    ((4, 32, 8, 4097, 4097, 0), (1, 8, 2, 700, 513, 0)),       # grouped heads
])
def test_noalloc_matches_workspace_call(shapes):
    for i, (B, Hq, Hkv, S, n, vh) in enumerate(shapes):
        _both(B, Hq, Hkv, S, n, vh, seed=100 + 10 * i + B)


def test_noalloc_refuses_sizes_beyond_scratch():
    # 64 query heads x 8 sequences at 65536 positions need 32 MiB of records
    B, Hq, S = 8, 64, 65536
    dummy = torch.zeros(64, dtype=torch.uint8, device=P.DEV)
    p = ctypes.c_void_p(dummy.data_ptr())
    st = _lib.offq_kv_attention_decode_noalloc_raw(p, p, p, p, p, p, p, B, Hq, Hq, S, S, 128, SM, 0,
                                                   p, None)
    assert st == _lib.OFFQ_ERR_UNSUPPORTED
    assert "scratch" in _lib.last_error()
