"""GPU parity: fused rotate + quantize (offq_rotate_quantize) vs the oracle."""
import numpy as np
import pytest
import torch

import paper_2606_07116_amd as offq
from paper_2606_07116_amd import inputs
from tests import parity as P

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("g", [16, 32, 64, 128, 256, 512, 1024, 2048, 4096, 8192])
@pytest.mark.parametrize("had", [True, False])
def test_every_group_size(g, had):
    G = 3 if g <= 2048 else 1
    M = 7  # ragged: not a multiple of the groups per tile
    x = inputs.activations(M, G * g, seed=g, n_outliers=2, lo=30, hi=90, layout="concentrated", g=g)
    P.rotate_quantize_and_check(x, g, had)


@pytest.mark.parametrize("M,K,g", [(1, 4096, 4096), (33, 1024, 128), (5, 14336, 512),
                                   (300, 256, 64), (129, 512, 512)])
def test_ragged_rows(M, K, g):
    x = inputs.activations(M, K, seed=M + K, n_outliers=3, lo=50, hi=200, layout="raw")
    P.rotate_quantize_and_check(x, g, True)


def test_strided_rows():
    M, K, g, ldx = 40, 1024, 256, 1536
    big = inputs.activations(M, ldx, seed=11, n_outliers=2, lo=40, hi=60)
    xd = P.to_dev_bf16(big)[:, :K]
    assert xd.stride(0) == ldx
    codes, scale, zero, y = offq.offq_rotate_quantize(xd, g, debug=True)
    torch.cuda.synchronize()
    x = big[:, :K]
    P.check_rotation(x, P.host(y), g, True)
    P.check_quant(P.host(y), P.host(codes), P.host(scale), P.host(zero), g)


@pytest.mark.parametrize("M,K,g,pad,had", [(3, 4096, 4096, 128, True), (5, 8192, 8192, 64, True),
                                            (1, 8192, 8192, 8, False), (2, 4096, 4096, 8, False)])
def test_strided_rows_whole_row_groups(M, K, g, pad, had):
    """One group per row of 4096 or 8192 channels (rows split over 2 or 4
    waves) with a row stride above K."""
    big = inputs.activations(M, K + pad, seed=K + pad, n_outliers=2, lo=40, hi=120)
    xd = P.to_dev_bf16(big)[:, :K]
    assert xd.stride(0) == K + pad
    codes, scale, zero, y = offq.offq_rotate_quantize(xd, g, apply_hadamard=had, debug=True)
    codes2, scale2, zero2, _ = offq.offq_rotate_quantize(xd, g, apply_hadamard=had)
    torch.cuda.synchronize()
    x = big[:, :K]
    P.check_rotation(x, P.host(y), g, had)
    P.check_quant(P.host(y), P.host(codes), P.host(scale), P.host(zero), g)
    assert torch.equal(codes, codes2) and torch.equal(scale, scale2) and torch.equal(zero, zero2)


def test_offset_channel_absorbed():
    """A pure first-channel outlier per group becomes a constant group (Eq. 5):
    the quantizer takes the degenerate branch, codes 0, and s (0 - z) ~ a/sqrt(g)."""
    g, G, M = 512, 4, 8
    x = np.zeros((M, G * g), np.float32)
    x[:, ::g] = np.float32(96.0)
    (q, s, z), _ = P.rotate_quantize_and_check(x, g, True)
    assert np.all(q == 0)
    xh = s.astype(np.float64) * (0 - z.astype(np.float64))
    assert np.allclose(xh, 96.0 / np.sqrt(g), rtol=2.0 ** -10)


def test_degenerate_and_zero_rows():
    g = 256
    x = np.zeros((6, 2 * g), np.float32)
    x[1] = 3.0
    x[2] = -5.5
    x[3, :g] = 1e-30   # tiny: scale clamps to the fp16 subnormal minimum
    x[4] = inputs.round_to_bf16(np.linspace(-1e4, 1e4, 2 * g, dtype=np.float32))
    x = inputs.round_to_bf16(x)
    P.rotate_quantize_and_check(x, g, True)
    P.rotate_quantize_and_check(x, g, False)


def test_rounding_ties_on_device():
    """Hand-built groups whose y * r lands exactly on k + 1/2 (quantize-only path)."""
    vals = np.array([0, 15, 0.5, 1.5, 2.5, 3.5, 4.5, 5.5, 6.5, 7.5, 8.5, 9.5, 10.5, 11.5, 12.5, 13.5],
                    np.float32)
    x = np.tile(vals, (3, 4))  # g = 16 groups of the same values
    x[1] += 100.0              # offset group: z = -100, ties shift parity with z
    x[2] += 101.0
    (q, s, z), _ = P.rotate_quantize_and_check(inputs.round_to_bf16(x), 16, False)
    assert list(q[0, :16]) == [0, 15, 0, 2, 2, 4, 4, 6, 6, 8, 8, 10, 10, 12, 12, 14]


def test_empty_input_is_noop():
    x = torch.empty((0, 256), dtype=torch.bfloat16, device=P.DEV)
    codes, scale, zero, _ = offq.offq_rotate_quantize(x, 256)
    assert codes.shape == (0, 128)


def test_rejects_bad_arguments_with_status():
    x = torch.zeros((4, 256), dtype=torch.bfloat16, device=P.DEV)
    with pytest.raises(offq.OffqError) as e:
        offq.offq_rotate_quantize(x, 96)
    assert e.value.status == 1
    with pytest.raises(offq.OffqError) as e:
        offq.offq_rotate_quantize(x, 8)
    assert e.value.status == 2
