"""Seeded synthetic inputs for the OffQ online path (no quantization arithmetic here).

These generators stand in for the activations and weights of the Llama-class
models the paper evaluates (sec. 4: Llama 2/3/3.2, Qwen 2.5; hidden sizes 4096,
8192, MLP sizes 14336 / 28672, head_dim 128).  No model, checkpoint or dataset
is read.  The same generators feed both the GPU library and the CPU oracle; they
only draw random numbers and place them, they never rotate or quantize.

Activation recipe (structured outliers, sec. 3.1: sparse, very large, sharing
one direction across tokens):
  * bulk ~ N(0, 1);
  * ``n_outliers`` channels each get a magnitude m_c ~ U(lo, hi), drawn once,
    with a sign fixed per channel, added on every token (rank-1 structure);
  * optionally a fraction of tokens (whole rows) is multiplied by ``spike_mult``
    ("massive activation" tokens);
  * the result is rounded to bfloat16, the dtype the online kernel reads.

Two placements of the outlier channels:
  * ``layout="raw"``: at the channels the workload names, or at seeded random
    channels -- the tensor as described, before any offline transform;
  * ``layout="concentrated"``: as the offline top-1 PCA rotation and grouping
    permutation (fused into upstream weights, sec. 3.3 step 2) deliver it to
    the online rotation: with one group the rank-1 outlier lies on channel 0
    with magnitude ||m||; with G groups the i-th largest outlier channel sits
    on the first channel of group i.

Weights: W ~ N(0, std^2) fp32 [N, K], drawn directly in the rotated basis
(same distribution as W Q for any orthogonal Q).
"""

import math

import numpy as np

# Workload registry: the five shapes of the online path, as (name -> dict).
WORKLOADS = {
    "tiny_layer": dict(M=16, K=256, N=256, g=256, n_outliers=2, channels=(3, 97),
                       lo=100.0, hi=100.0, seed=0),
    "attn_proj_prefill": dict(M=2048, K=4096, N=4096, g=4096, n_outliers=4,
                              lo=50.0, hi=200.0, seed=2),
    "mlp_up_gate_prefill": dict(M=4096, K=4096, N=14336, g=4096, n_outliers=6,
                                lo=50.0, hi=500.0, spike_frac=1e-3, spike_mult=20.0,
                                seed=3),
    "mlp_down_prefill": dict(M=4096, K=14336, N=4096, g=512, n_outliers=6,
                             lo=50.0, hi=500.0, spike_frac=1e-3, spike_mult=20.0,
                             seed=33),
    "decode_up": dict(M=16, K=8192, N=28672, g=8192, n_outliers=8,
                      lo=50.0, hi=200.0, seed=4),
    "decode_down": dict(M=16, K=28672, N=8192, g=512, n_outliers=8,
                        lo=50.0, hi=200.0, seed=44),
    "kv_cache": dict(B=8, H=32, S=32768, Dh=128, n_outliers=2, lo=20.0, hi=80.0,
                     seed=5),
    "kv_decode_attention": dict(B=8, H=32, S=32768, Dh=128, seed=6),
    # one decode step of a Llama-3-8B-shaped layer: 16 sequences at context 4096
    "decode_layer": dict(M=16, D=4096, Hq=32, Hkv=8, F=14336, g=128, ctx=4096, seed=7),
    # the prefill of the same layer: 2 sequences of 2048 tokens (4096 rows
    # through the projections), causal attention over the tokens just written
    "prefill_layer": dict(B=2, T=2048, past=0, D=4096, Hq=32, Hkv=8, F=14336, g=128, seed=9),
    # offline calibration of one 4096-channel layer input (U1 P1 H1): 128
    # calibration sequences of 2048 tokens; the rotation fused into the QKV
    # and up/gate weights of a Llama-3-8B-shaped layer
    "calibration": dict(n_seq=128, L=2048, D=4096, g=128, n_outliers=6, lo=50.0, hi=500.0,
                        spike_frac=1e-3, spike_mult=20.0, seed=8,
                        layers={"qkv": 6144, "up_gate": 28672}),
    "kv_chain_proj": dict(M=8192, K=4096, N=4096, g=4096, n_outliers=4,
                          lo=50.0, hi=200.0, seed=55),
}


def _structure(rng, M, K, n_outliers, lo, hi, channels, spike_frac):
    """Draw outlier channels, magnitudes, signs and spike rows (host RNG)."""
    if channels is None:
        channels = np.sort(rng.choice(K, size=n_outliers, replace=False))
    channels = np.asarray(channels, dtype=np.int64)
    mags = rng.uniform(lo, hi, size=len(channels)) if hi > lo else np.full(len(channels), lo)
    signs = np.where(rng.random(len(channels)) < 0.5, -1.0, 1.0)
    n_spk = int(math.ceil(spike_frac * M)) if spike_frac > 0 else 0
    spike_rows = np.sort(rng.choice(M, size=n_spk, replace=False)) if n_spk else np.zeros(0, np.int64)
    return channels, mags, signs, spike_rows


def _placement(layout, K, g, channels, mags, signs):
    """Channels and signed values to add on every token, per layout."""
    if layout == "raw":
        return channels, mags * signs
    if layout != "concentrated":
        raise ValueError("layout must be 'raw' or 'concentrated'")
    G = K // g
    order = np.argsort(-mags, kind="stable")
    if len(channels) <= G:
        # i-th largest outlier on the first channel of group i.
        pos = np.arange(len(channels), dtype=np.int64) * g
        return pos, (mags * signs)[order]
    # More outlier channels than groups: the rank-1 direction lands on channel 0
    # with its full norm (positive orientation).
    return np.zeros(1, np.int64), np.array([float(np.sqrt(np.sum(mags ** 2)))])


def activations(M, K, *, seed, n_outliers=0, lo=0.0, hi=0.0, channels=None,
                spike_frac=0.0, spike_mult=20.0, layout="raw", g=None):
    """Host activations: fp32 numpy [M, K] whose values are exact bfloat16 numbers."""
    rng = np.random.Generator(np.random.PCG64(seed))
    x = rng.standard_normal((M, K), dtype=np.float32)
    ch, mags, signs, spk = _structure(rng, M, K, n_outliers, lo, hi, channels, spike_frac)
    pos, vals = _placement(layout, K, g or K, ch, mags, signs)
    x[:, pos] += vals.astype(np.float32)[None, :]
    if len(spk):
        x[spk, :] *= np.float32(spike_mult)
    return round_to_bf16(x)


def activations_device(M, K, *, seed, device, n_outliers=0, lo=0.0, hi=0.0,
                       channels=None, spike_frac=0.0, spike_mult=20.0,
                       layout="raw", g=None):
    """Device activations (torch bfloat16 [M, K]); bulk drawn by torch's device RNG.

    Same recipe as ``activations``; used where a host draw would be too slow.
    """
    import torch

    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    x = torch.randn((M, K), generator=gen, device=device, dtype=torch.float32)
    rng = np.random.Generator(np.random.PCG64(seed))
    ch, mags, signs, spk = _structure(rng, M, K, n_outliers, lo, hi, channels, spike_frac)
    pos, vals = _placement(layout, K, g or K, ch, mags, signs)
    x[:, torch.as_tensor(pos, device=device)] += torch.as_tensor(
        vals, dtype=torch.float32, device=device)[None, :]
    if len(spk):
        x[torch.as_tensor(spk, device=device)] *= spike_mult
    return x.to(torch.bfloat16)


def weights(N, K, *, seed, std=0.02):
    """Host weights ~ N(0, std^2), fp32 numpy [N, K]."""
    rng = np.random.Generator(np.random.PCG64(seed + 1000))
    w = rng.standard_normal((N, K), dtype=np.float32)
    w *= np.float32(std)
    return w


def weights_device(N, K, *, seed, device, std=0.02):
    """Device weights ~ N(0, std^2), torch fp32 [N, K]."""
    import torch

    gen = torch.Generator(device=device)
    gen.manual_seed(seed + 1000)
    return torch.randn((N, K), generator=gen, device=device, dtype=torch.float32) * std


def kv_cache_device(B, H, S, Dh, *, seed, device, n_outliers=2, lo=20.0, hi=80.0):
    """Device K or V cache, torch bfloat16 [B, H, S, Dh]: N(0,1) bulk plus, per
    head, ``n_outliers`` dims with a fixed signed magnitude U(lo, hi) on every
    position (the per-head structured outliers of the key cache, sec. 3.1)."""
    import torch

    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    x = torch.randn((B, H, S, Dh), generator=gen, device=device, dtype=torch.float32)
    rng = np.random.Generator(np.random.PCG64(seed))
    for h in range(H):
        dims = rng.choice(Dh, size=n_outliers, replace=False)
        vals = rng.uniform(lo, hi, size=n_outliers) * np.where(rng.random(n_outliers) < 0.5, -1.0, 1.0)
        for d, v in zip(dims, vals):
            x[:, h, :, int(d)] += float(v)
    return x.to(torch.bfloat16)


def kv4_cache(B, H, S, Dh, *, seed, s_lo=0.05, s_hi=0.6, z_lo=3, z_hi=12):
    """Host 4-bit cache in the layout the KV quantizer writes: packed code bytes
    uint8 [B, H, S, Dh/2] (both nibbles uniform on 0..15), fp16 scales
    [B, H, S] ~ U(s_lo, s_hi) and int16 zero-points [B, H, S] uniform on
    z_lo..z_hi.  Drawn directly (no rotation or quantization happens here): a
    Hadamard-rotated row spans its 16 levels around a zero-point near the
    middle of the grid."""
    rng = np.random.Generator(np.random.PCG64(seed + 7000))
    codes = rng.integers(0, 256, size=(B, H, S, Dh // 2), dtype=np.uint8)
    scale = rng.uniform(s_lo, s_hi, size=(B, H, S)).astype(np.float16)
    zero = rng.integers(z_lo, z_hi + 1, size=(B, H, S)).astype(np.int16)
    return codes, scale, zero


def kv4_cache_device(B, H, S, Dh, *, seed, device, s_lo=0.05, s_hi=0.6, z_lo=3, z_hi=12):
    """Device version of ``kv4_cache`` (same distributions, torch's device RNG)."""
    import torch

    gen = torch.Generator(device=device)
    gen.manual_seed(seed + 7000)
    codes = torch.randint(0, 256, (B, H, S, Dh // 2), generator=gen, device=device,
                          dtype=torch.uint8)
    scale = (torch.rand((B, H, S), generator=gen, device=device) * (s_hi - s_lo) + s_lo
             ).to(torch.float16)
    zero = torch.randint(z_lo, z_hi + 1, (B, H, S), generator=gen, device=device,
                         dtype=torch.int16)
    return codes, scale, zero


def queries(B, H, Dh, *, seed, std=1.0):
    """Host decode queries [B, H, Dh] ~ N(0, std^2), rounded to bfloat16
    (fp32 numpy holding the bf16 values)."""
    rng = np.random.Generator(np.random.PCG64(seed + 9000))
    q = rng.standard_normal((B, H, Dh), dtype=np.float32) * np.float32(std)
    return round_to_bf16(q)


def kv_rows(R, Dh, *, seed, n_outliers=2, lo=20.0, hi=80.0, heads=4):
    """Host KV rows [R, Dh] (fp32 holding exact bf16 values); rows cycle over
    ``heads`` heads, each with its own fixed outlier dims."""
    rng = np.random.Generator(np.random.PCG64(seed))
    x = rng.standard_normal((R, Dh), dtype=np.float32)
    for h in range(heads):
        dims = rng.choice(Dh, size=n_outliers, replace=False)
        vals = rng.uniform(lo, hi, size=n_outliers) * np.where(rng.random(n_outliers) < 0.5, -1.0, 1.0)
        x[h::heads, dims] += vals.astype(np.float32)[None, :]
    return round_to_bf16(x)


def round_to_bf16(x):
    """Round fp32 to the nearest bfloat16 (ties to even); returns fp32 numpy."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def bf16_bits(x):
    """fp32 numpy holding bf16 values -> uint16 numpy of their bf16 bit patterns."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    return (x.view(np.uint32) >> 16).astype(np.uint16)
