"""GPU parity: W4A4 GEMM / GEMV (offq_w4a4_gemm) and weight packing vs the oracle."""
import numpy as np
import pytest
import torch

import paper_2606_07116_amd as offq
from oracle import gemm as OG
from oracle import quantizer as OQ
from paper_2606_07116_amd import inputs
from tests import parity as P

pytestmark = pytest.mark.gpu


def _layer(M, N, K, g, seed, layout="concentrated", n_out=4):
    x = inputs.activations(M, K, seed=seed, n_outliers=n_out, lo=50, hi=200, layout=layout, g=g)
    w = inputs.weights(N, K, seed=seed)
    (q, s, z), (codes, scale, zero) = P.rotate_quantize_and_check(x, g, True)
    q_w, sw, cs, packed = P.oracle_weights(w, g)
    wc, ws, wcs = P.upload_weights(packed, sw, cs)
    y, acc = offq.offq_w4a4_gemm(codes, scale, zero, wc, ws, wcs, g, debug=True)
    y2, _ = offq.offq_w4a4_gemm(codes, scale, zero, wc, ws, wcs, g, debug=False)
    torch.cuda.synchronize()
    assert torch.equal(y, y2)
    acc_ref = OG.int_gemm_groups(q, q_w, g)
    acc_gpu = P.host(acc)
    if not np.array_equal(acc_gpu, acc_ref):
        bad = np.argwhere(acc_gpu != acc_ref)
        raise AssertionError(f"accumulator mismatch at {bad[:5].tolist()} (of {len(bad)})")
    P.check_output(P.host(y.float()), acc_ref, s, z, sw, cs)
    return y


@pytest.mark.parametrize("M,N,K,g", [
    (17, 8, 256, 256), (128, 128, 512, 512), (130, 136, 1024, 256), (200, 250, 256, 64),
    (257, 384, 2048, 512), (64, 512, 4096, 4096), (40, 96, 8192, 8192), (33, 64, 512, 128),
    # groups of 8 and 16 stages of 128 k; more groups than the grouped kernel
    # keeps in LDS (G = 32); g = 512 over a ragged 2-tile-row x 3-tile-column grid
    (100, 136, 4096, 1024), (77, 64, 8192, 2048), (40, 64, 4096, 128), (300, 260, 3584, 512),
    # more groups than fit in LDS (parameters streamed with the stages): one,
    # two, four and sixteen stages per group, an odd number of groups
    (257, 200, 14336, 128), (300, 136, 8192, 256), (100, 520, 16384, 512),
    (33, 130, 3712, 128), (64, 96, 65536, 2048),
])
def test_gemm_shapes(M, N, K, g):
    _layer(M, N, K, g, seed=M * 7 + N)


@pytest.mark.parametrize("M,N,K", [(4096, 6144, 4096), (4000, 6100, 1024)])
def test_wide_tile_gemm_accumulators(M, N, K):
    """One group per row on at least 384 tiles of 256 x 256: the wide-tile
    kernel that the MLP up/gate projection and the 8192-row projection run.
    Every accumulator bit-exact, once on whole tiles and once ragged in M and
    N (384 tiles again)."""
    _layer(M, N, K, K, seed=M + N)


@pytest.mark.parametrize("M,N,K,g", [
    (4096, 8192, 1024, 1024), (4000, 8104, 512, 512),      # one group: 512 tiles of 256 x 256
    (4000, 8100, 512, 512),                                # ragged in M and N, N not a multiple of 8
    (4096, 4096, 2048, 256), (4001, 4000, 1024, 512),      # groups: 512 tiles of 256 x 128
    (4096, 4100, 3584, 512), (3900, 4096, 8192, 2048),     # odd group count; 16 stages per group
])
def test_large_gemm_shapes(M, N, K, g):
    """Prefill-sized grids (at least 512 tiles, several tiles per CU): every
    accumulator bit-exact and the output within the bar, on whole and ragged
    tile grids, with one group per row, 2 to 8 groups, an odd number of groups
    and long groups."""
    _layer(M, N, K, g, seed=M + N + g)


def test_out_must_cover_the_output():
    """The GEMM writes M x N values at the output's row stride: a short or a
    transposed output is refused before any launch."""
    M, N, K, g = 32, 64, 256, 256
    codes = torch.zeros((M, K // 2), dtype=torch.uint8, device=P.DEV)
    sc = torch.ones((M, 1), dtype=torch.float16, device=P.DEV)
    zp = torch.zeros((M, 1), dtype=torch.int16, device=P.DEV)
    wc = torch.zeros(offq.weight_codes_shape(N, K), dtype=torch.uint8, device=P.DEV)
    ws = torch.ones(N, dtype=torch.float16, device=P.DEV)
    cs = torch.zeros((1, N), dtype=torch.int32, device=P.DEV)
    short = torch.empty((M - 1, N), dtype=torch.bfloat16, device=P.DEV)
    trans = torch.empty((N, M), dtype=torch.bfloat16, device=P.DEV).t()
    for bad in (short, trans):
        with pytest.raises(ValueError):
            offq.offq_w4a4_gemm(codes, sc, zp, wc, ws, cs, g, out=bad)


@pytest.mark.parametrize("M", [1, 2, 4, 5, 16])
@pytest.mark.parametrize("K,g", [(256, 256), (2048, 512), (8192, 8192), (1024, 64),
                                 (4096, 128), (1536, 512), (2048, 1024)])
def test_gemv_shapes(M, K, g):
    _layer(M, 200, K, g, seed=M + K)


@pytest.mark.parametrize("N", [16, 33, 1030, 5000, 9000, 16400])
def test_gemv_channel_counts(N):
    """Single and ragged 16-channel tiles; one, two and four tiles per wave
    (the last with a ragged final workgroup)."""
    _layer(3, N, 4096, 512, seed=N)


@pytest.mark.parametrize("M,N,K,g", [(4, 4096, 14336, 128), (16, 4096, 14336, 512),
                                     (1, 20000, 5120, 128), (3, 8192, 6144, 256),
                                     (5, 8192, 6144, 1024)])
def test_gemv_parts_of_k(M, N, K, g):
    """K not a multiple of 4096: each wave's part of K is an odd number of
    batches, and with g = 1024 a part ends inside a group (the group's
    zero-point term is added once)."""
    _layer(M, N, K, g, seed=K + g)


def test_raw_layout_and_spikes():
    _layer(150, 192, 1024, 1024, seed=5, layout="raw", n_out=6)


@pytest.mark.parametrize("M,N,ld,off", [
    (140, 72, 100, 10),   # GEMM
    (16, 72, 100, 10),    # decode GEMV, output start not 8-byte aligned
    (16, 70, 101, 3),     # GEMV: odd row stride, N not a multiple of 4
    (5, 66, 99, 1),
])
def test_output_row_stride(M, N, ld, off):
    """The output is a view inside a larger matrix: the M x N values land at
    its row stride and offset, nothing around them is written."""
    K, g = 512, 256
    x = inputs.activations(M, K, seed=3, n_outliers=2, lo=50, hi=60, layout="concentrated", g=g)
    w = inputs.weights(N, K, seed=3)
    (q, s, z), (codes, scale, zero) = P.rotate_quantize_and_check(x, g, True)
    q_w, sw, cs, packed = P.oracle_weights(w, g)
    wc, ws, wcs = P.upload_weights(packed, sw, cs)
    big = torch.full((M, ld), 7.0, dtype=torch.bfloat16, device=P.DEV)
    offq.offq_w4a4_gemm(codes, scale, zero, wc, ws, wcs, g, out=big[:, off:off + N])
    torch.cuda.synchronize()
    yb = P.host(big.float())
    assert np.all(yb[:, :off] == 7.0) and np.all(yb[:, off + N:] == 7.0)
    P.check_output(yb[:, off:off + N], OG.int_gemm_groups(q, q_w, g), s, z, sw, cs)


def test_extreme_codes_and_zero_points():
    """All-15 activation codes against all -8 weights with large zero-points."""
    M, N, K, g = 130, 66, 1024, 512
    codes = torch.full((M, K // 2), 0xFF, dtype=torch.uint8, device=P.DEV)
    scale = torch.full((M, K // g), 0.5, dtype=torch.float16, device=P.DEV)
    zero = torch.full((M, K // g), -32768, dtype=torch.int16, device=P.DEV)
    q_w = np.full((N, K), -8, np.int8)
    sw = np.full(N, 0.25, np.float16)
    cs = OQ.colsum(q_w, g)
    wc, ws, wcs = P.upload_weights(OQ.pack_nibbles(q_w), sw, cs)
    y, acc = offq.offq_w4a4_gemm(codes, scale, zero, wc, ws, wcs, g, debug=True)
    torch.cuda.synchronize()
    acc_ref = OG.int_gemm_groups(np.full((M, K), 15, np.uint8), q_w, g)
    assert np.array_equal(P.host(acc), acc_ref)
    P.check_output(P.host(y.float()), acc_ref, P.host(scale), P.host(zero), sw, cs)


def test_empty_m_is_noop():
    g, K, N = 256, 256, 8
    e = torch.empty((0, K // 2), dtype=torch.uint8, device=P.DEV)
    y, _ = offq.offq_w4a4_gemm(e, torch.empty((0, 1), dtype=torch.float16, device=P.DEV),
                               torch.empty((0, 1), dtype=torch.int16, device=P.DEV),
                               torch.zeros(offq.weight_codes_shape(N, K), dtype=torch.uint8,
                                           device=P.DEV),
                               torch.ones(N, dtype=torch.float16, device=P.DEV),
                               torch.zeros((1, N), dtype=torch.int32, device=P.DEV), g)
    assert y.shape == (0, N)


@pytest.mark.parametrize("N,K,g", [(7, 256, 64), (300, 4096, 4096), (64, 28672, 512), (33, 8192, 8192)])
def test_pack_weights(N, K, g):
    w = inputs.weights(N, K, seed=N)
    w[0] = 0.0                      # all-zero row -> scale 1
    w[1, 5] = 3.0                   # one large weight
    q_w, sw, cs, packed = P.oracle_weights(w, g)
    wc, ws, wcs = offq.offq_pack_weights(torch.from_numpy(w).to(P.DEV), g)
    torch.cuda.synchronize()
    assert np.array_equal(P.fp16_bits(P.host(ws)), P.fp16_bits(sw))
    assert tuple(wc.shape) == offq.weight_codes_shape(N, K)
    assert np.array_equal(offq.row_major_weight_codes(P.host(wc), N, K), packed)
    # the padding rows and k of the blocked layout hold zero codes
    assert int(P.host(wc).astype(np.int64).sum()) == int(packed.astype(np.int64).sum())
    assert np.array_equal(P.host(wcs), cs)
