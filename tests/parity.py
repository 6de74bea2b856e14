"""Helpers shared by the GPU parity tests: run the HIP path through the C ABI
binding, run the CPU oracle on the same seeded inputs, compare.

Comparison rules
* codes, scale bits, zero-points, integer accumulators, packed weights:
  bit-exact;
* the fp32 rotation y (which the oracle quantizer is fed, as the GPU's
  rounding order of the butterflies is not the oracle's): within the
  recursive-summation bound of an L = log2(g)-stage fp32 Walsh-Hadamard
  transform, |y - y64| <= (L + 2) * 2^-24 * sum_group |x| / sqrt(g);
* bf16 outputs: |Y - Y_ref| <= max(1e-2 |Y_ref|, 2 ulp_bf16(Y_ref), 1e-5 E),
  E = sw sum_b |s_b (acc_b - z_b colsum_b)| (an fp32 fold of G terms errs by
  a small multiple of 2^-24 E; for one group E = |Y_ref| and the floor is
  inactive); with one group the output must also be one of the two bf16
  neighbours of Y_ref (|Y - Y_ref| <= 1 ulp).
"""

import numpy as np
import torch

import paper_2606_07116_amd as offq
from oracle import gemm as OG
from oracle import hadamard as OH
from oracle import quantizer as OQ

DEV = "cuda:0"


def to_dev_bf16(x_np):
    """fp32 numpy holding bf16 values -> device bf16 tensor (exact)."""
    return torch.from_numpy(np.ascontiguousarray(x_np, dtype=np.float32)).to(torch.bfloat16).to(DEV)


def host(t):
    return t.detach().cpu().numpy()


def fp16_bits(a):
    return np.ascontiguousarray(a).view(np.uint16)


def check_rotation(x, y_gpu, g, hadamard):
    """x: fp32 [M, K] host (bf16 values); y_gpu: fp32 [M, K] host."""
    if not hadamard:
        assert np.array_equal(y_gpu, x.astype(np.float32)), "quantize-only y must equal x"
        return
    M, K = x.shape
    y64 = OH.rotate(x.astype(np.float64), g)
    L = int(np.log2(g))
    absx = np.abs(x.astype(np.float64)).reshape(M, K // g, g).sum(-1) / np.sqrt(g)
    bound = (L + 2) * 2.0 ** -24 * np.repeat(absx, g, axis=1) * 1.01 + 1e-30
    err = np.abs(y_gpu.astype(np.float64) - y64)
    bad = err > bound
    assert not bad.any(), (
        f"rotation error above bound at {np.argwhere(bad)[:5].tolist()}; max ratio "
        f"{(err / bound).max():.3g}")


def check_quant(y_gpu, codes_gpu, scale_gpu, zero_gpu, g):
    """Oracle quantizer on the GPU's own y; codes / scale / zero bit-exact."""
    q, s, z = OQ.quantize_groups(y_gpu, g)
    packed = OQ.pack_nibbles(q)
    M = y_gpu.shape[0]
    scale_gpu = np.asarray(scale_gpu).reshape(M, -1)
    zero_gpu = np.asarray(zero_gpu).reshape(M, -1)
    if not np.array_equal(fp16_bits(scale_gpu), fp16_bits(s)):
        bad = np.argwhere(fp16_bits(scale_gpu) != fp16_bits(s))
        raise AssertionError(f"scale mismatch at {bad[:5].tolist()} (of {len(bad)})")
    if not np.array_equal(zero_gpu, z):
        bad = np.argwhere(zero_gpu != z)
        raise AssertionError(f"zero mismatch at {bad[:5].tolist()} (of {len(bad)})")
    if not np.array_equal(codes_gpu, packed):
        bad = np.argwhere(codes_gpu != packed)
        raise AssertionError(f"codes mismatch at {bad[:5].tolist()} (of {len(bad)})")
    return q, s, z


def rotate_quantize_and_check(x, g, hadamard=True):
    """Run the GPU rotate-quantize on host x (debug mode), check it against the
    oracle, and return the oracle's (q, s, z) (identical to the GPU's)."""
    xd = to_dev_bf16(x)
    codes, scale, zero, y = offq.offq_rotate_quantize(xd, g, apply_hadamard=hadamard, debug=True)
    codes2, scale2, zero2, _ = offq.offq_rotate_quantize(xd, g, apply_hadamard=hadamard, debug=False)
    torch.cuda.synchronize()
    y = host(y)
    check_rotation(x, y, g, hadamard)
    out = check_quant(y, host(codes), host(scale), host(zero), g)
    # the launch without debug output (the one the benchmark times) agrees
    assert torch.equal(codes, codes2) and torch.equal(scale, scale2) and torch.equal(zero, zero2)
    return out, (codes, scale, zero)


def oracle_weights(w, g):
    q_w, sw = OQ.quantize_weights(w)
    return q_w, sw, OQ.colsum(q_w, g), OQ.pack_nibbles(q_w)


def upload_weights(packed, sw, cs):
    """Row-major oracle codes [N, K/2] uploaded in the blocked operand layout."""
    from paper_2606_07116_amd import _lib
    return (torch.from_numpy(_lib.blocked_weight_codes(packed)).to(DEV), torch.from_numpy(sw).to(DEV),
            torch.from_numpy(cs).to(DEV))


def check_output(y_gpu, acc, s, z, sw, cs, rows=None):
    """y_gpu: bf16 host values (fp32 numpy) [m, N]; acc: oracle int [G, m, N]."""
    y_ref = OG.epilogue(acc, s if rows is None else s[rows], z if rows is None else z[rows], sw, cs)
    e = OG.epilogue_magnitude(acc, s if rows is None else s[rows], z if rows is None else z[rows], sw, cs)
    y = y_gpu.astype(np.float64)
    tol = np.maximum(np.maximum(1e-2 * np.abs(y_ref), 2 * OG.bf16_ulp(y_ref)), 1e-5 * e)
    err = np.abs(y - y_ref)
    bad = err > tol
    assert not bad.any(), (
        f"output mismatch at {np.argwhere(bad)[:5].tolist()} (of {bad.sum()}): "
        f"gpu {y[bad][:5]} ref {y_ref[bad][:5]}")
    if acc.shape[0] == 1:
        strict = err > OG.bf16_ulp(y_ref) * (1 + 1e-9)
        assert not strict.any(), (
            f"single-group output not a bf16 neighbour of the exact value at "
            f"{np.argwhere(strict)[:5].tolist()}")
    return y_ref
