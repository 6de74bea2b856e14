"""GPU parity at the full sizes of the five workloads, in the launch
configuration the benchmark times (no debug outputs), plus debug launches for
the exact integer accumulators.  Where the oracle cannot recompute everything
in seconds, it checks sampled rows one by one."""
import numpy as np
import pytest
import torch

import paper_2606_07116_amd as offq
from oracle import gemm as OG
from oracle import quantizer as OQ
from paper_2606_07116_amd import inputs
from tests import parity as P

pytestmark = pytest.mark.gpu

W = inputs.WORKLOADS


def _spec(cfg, layout="raw"):
    d = dict(n_outliers=cfg["n_outliers"], lo=cfg["lo"], hi=cfg["hi"], layout=layout, g=cfg.get("g"))
    for k in ("spike_frac", "spike_mult", "channels"):
        if k in cfg:
            d[k] = cfg[k]
    return d


def _weights(N, K, g, seed):
    w = inputs.weights(N, K, seed=seed)
    q_w, sw, cs, packed = P.oracle_weights(w, g)
    del w
    return q_w, sw, cs, P.upload_weights(packed, sw, cs)


def _layer_full(M, K, N, g, seed, spec, sample_rows=None, wts=None):
    """rotate-quantize (full parity) + GEMM in the benchmark's launch shape;
    outputs on all or sampled rows, and the accumulators of the same rows
    bit-exact from a debug launch of the same shape (an accumulator-only pass
    of the kernel the dispatcher picks for M x N x K, then the regular pass,
    whose output must equal the plain launch's)."""
    x = inputs.activations(M, K, seed=seed, **spec)
    (q, s, z), (codes, scale, zero) = P.rotate_quantize_and_check(x, g, True)
    del x
    q_w, sw, cs, (wc, ws, wcs) = wts if wts is not None else _weights(N, K, g, seed)
    y, _ = offq.offq_w4a4_gemm(codes, scale, zero, wc, ws, wcs, g)
    y2, accd = offq.offq_w4a4_gemm(codes, scale, zero, wc, ws, wcs, g, debug=True)
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16), y2.view(torch.int16))
    del y2
    rows = np.arange(M) if sample_rows is None else np.sort(
        np.random.default_rng(seed).choice(M, size=sample_rows, replace=False))
    acc = OG.int_gemm_groups(q[rows], q_w, g)
    got = P.host(accd[:, torch.as_tensor(rows, device=P.DEV)])
    del accd
    if not np.array_equal(got, acc):
        bad = np.argwhere(got != acc)
        raise AssertionError(f"accumulator mismatch at {bad[:5].tolist()} (of {len(bad)})")
    P.check_output(P.host(y.float())[rows], acc, s, z, sw, cs, rows=rows)
    return q_w, sw, cs, (wc, ws, wcs)


def test_tiny_layer():
    c = W["tiny_layer"]
    _layer_full(c["M"], c["K"], c["N"], c["g"], c["seed"], _spec(c))


@pytest.mark.parametrize("layout", ["raw", "concentrated"])
def test_attn_proj_prefill(layout):
    c = W["attn_proj_prefill"]
    _layer_full(c["M"], c["K"], c["N"], c["g"], c["seed"], _spec(c, layout))


def test_mlp_up_gate_prefill():
    c = W["mlp_up_gate_prefill"]
    # up and gate projections stacked as one N = 2 * 14336 GEMM
    _layer_full(c["M"], c["K"], 2 * c["N"], c["g"], c["seed"], _spec(c), sample_rows=96)


def test_mlp_down_prefill():
    c = W["mlp_down_prefill"]
    _layer_full(c["M"], c["K"], c["N"], c["g"], c["seed"], _spec(c, "concentrated"),
                sample_rows=96)


@pytest.mark.parametrize("name", ["decode_up", "decode_down"])
def test_decode(name):
    c = W[name]
    wts = _weights(c["N"], c["K"], c["g"], c["seed"])
    for M in (1, 4, 16):
        _layer_full(M, c["K"], c["N"], c["g"], c["seed"] + M, _spec(c), wts=wts)


def test_kv_cache_and_projection_chain():
    c = W["kv_cache"]
    B, H, S, Dh = c["B"], c["H"], c["S"], c["Dh"]
    rng = np.random.default_rng(0)
    rows = np.sort(rng.choice(B * H * S, size=2048, replace=False))
    ridx = torch.as_tensor(rows, device=P.DEV)
    for j in range(2):   # K then V cache, each [8, 32, 32768, 128]
        kv = inputs.kv_cache_device(B, H, S, Dh, seed=c["seed"] + j, device=P.DEV,
                                    n_outliers=c["n_outliers"], lo=c["lo"], hi=c["hi"])
        codes, scale, zero, _ = offq.offq_kv_quantize(kv, apply_hadamard=True)
        flat = kv.reshape(-1, Dh)
        sub = flat[ridx].contiguous()
        c2, s2, z2, y2 = offq.offq_kv_quantize(sub, apply_hadamard=True, debug=True)
        torch.cuda.synchronize()
        # the full-tensor launch agrees with the debug launch on the sampled rows
        assert torch.equal(codes[ridx], c2) and torch.equal(scale[ridx], s2) and torch.equal(zero[ridx], z2)
        x = P.host(sub.float())
        y = P.host(y2)
        P.check_rotation(x, y, Dh, True)
        P.check_quant(y, P.host(c2), P.host(s2)[:, None], P.host(z2)[:, None], Dh)
        del kv, codes, scale, zero, flat
        torch.cuda.empty_cache()
    p = W["kv_chain_proj"]
    _layer_full(p["M"], p["K"], p["N"], p["g"], p["seed"], _spec(p), sample_rows=128)


# The paper's default group of 128 channels on every layer (32, 112 and 224
# groups per row): full-size parity of the attention projection, the MLP down
# projection and the decode down GEMV.
def test_attn_proj_prefill_g128():
    c = dict(W["attn_proj_prefill"], g=128)
    _layer_full(c["M"], c["K"], c["N"], c["g"], c["seed"], _spec(c, "concentrated"),
                sample_rows=256)


def test_mlp_down_prefill_g128():
    c = dict(W["mlp_down_prefill"], g=128)
    _layer_full(c["M"], c["K"], c["N"], c["g"], c["seed"], _spec(c, "concentrated"),
                sample_rows=96)


def test_decode_down_g128():
    c = dict(W["decode_down"], g=128)
    wts = _weights(c["N"], c["K"], c["g"], c["seed"])
    for M in (1, 16):
        _layer_full(M, c["K"], c["N"], c["g"], c["seed"] + M, _spec(c), wts=wts)
