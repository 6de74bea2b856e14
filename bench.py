#!/usr/bin/env python3
"""Benchmark of the OffQ W4A4 online path on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]
                    [--no-components]

One step = the whole online path of the MLP of a Llama-3-8B-shaped layer at
prefill (the largest single-GPU workload): fused rotate + quantize of the
bf16 up/gate input X [4096, 4096] (offq_rotate_quantize, 4096-point
Hadamard), the int4 x int4 GEMM with the dequantising epilogue against the
stacked up and gate weights [28672, 4096] (offq_w4a4_gemm), then rotate +
quantize of the down input [4096, 14336] (block-diagonal Hadamard, 28 blocks
of 512) and the down GEMM [4096, 14336] x [4096, 14336]^T.  Inputs are
synthetic (seeded), resident in HBM before the timed region; several
input/weight sets whose total exceeds the 256 MB last-level cache are cycled
so that every step reads from HBM.

Prints ONE JSON line: the step throughput (integer TOP/s of the GEMM work per
step time), per-kernel times, the roofline of the dominant kernel, and the
CPU oracle timed on the host.  With the default workload the line also
carries, as "configs", every other workload's kernels measured the same way:
the attention-projection prefill layer, the decode GEMVs at M = 1, 4, 16 and
the KV4 cache quantize of K and V [8, 32, 32768, 128] with the 8192-row
projection after it.

Timing.  The timed region runs the K steps kernel by kernel -- the first
kernel of the step for steps 1..K, then the second for steps 1..K, and so on
(step i's kernels still run in their order on step i's buffers) -- with one
HIP event between these phases on the launch stream, so that each kernel's
mean duration ("us") is its phase time / K with no event between two
launches of it.  Then every kernel is launched again max(100, K) times with
an event after each launch ("median_us", "p10_us", "p90_us": cold, cycling
the buffer sets; "warm_median_us": one set, so inputs may sit in the
last-level cache); "event_gap_us" is the median gap between two events with
nothing between them, which each of those per-launch times includes.
"""

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "W4A4 offset-GEMM int TOPS (prefill) + quantize/decode HBM GB/s vs peak"
PEAK_INT8_TOPS = 5000.0     # MI355X dense int8 MFMA, 5.0 POP/s
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E, 8 TB/s
PEAK_FP16_TFLOPS = 2500.0   # MI355X dense fp16 / bf16 MFMA, 2.5 PFLOP/s
LLC_BYTES = 256 << 20       # MI355X Infinity Cache


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--workload", default="mlp_prefill",
                   choices=["attn_proj_prefill", "mlp_prefill", "decode", "kv_chain",
                            "kv_decode_attention", "decode_layer", "prefill_layer",
                            "calibration"])
    p.add_argument("--decode-m", type=int, default=16)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-components", action="store_true",
                   help="default workload: skip the other workloads' kernels")
    p.add_argument("--group-size", type=int, default=0,
                   help="quantization group (= Hadamard block) size for every layer of the "
                        "workload, e.g. 128 (the paper's default); 0 keeps the workload's own")
    return p.parse_args()


def rq_bytes(M, K, g):
    """Algorithmic HBM bytes of rotate-quantize: bf16 read, 4-bit codes, fp16 scale + int16 zero."""
    return M * K * 2 + M * K // 2 + 4 * M * (K // g)


def gemv_bytes(M, N, K, g):
    """Algorithmic HBM bytes of the decode GEMV (weights dominate)."""
    G = K // g
    return N * K // 2 + 2 * N + 4 * G * N + M * K // 2 + 4 * M * G + 2 * M * N


def attn_bytes(BH, S, Dh=128):
    """Algorithmic HBM bytes of one decode-attention step: the 4-bit K and V
    rows of every attended position with their fp16 scale and int16 zero-point,
    plus the bf16 query and output of each (b, h)."""
    return BH * (S * (2 * (Dh // 2) + 2 * 4) + 2 * 2 * Dh)


def weight_bytes(N, K, g):
    """Packed int4 weights with fp16 scales and int32 per-group column sums."""
    return N * K // 2 + 2 * N + 4 * (K // g) * N


def source_hash(paths):
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def traffic_for(kernel_key):
    """HBM bytes per launch measured with rocprofv3 counters (profiles/traffic.json),
    or None when the kernel source changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    e = d.get(kernel_key)
    if not e:
        return None
    if e.get("source_hash") != source_hash(e["sources"]):
        return None
    return e.get("bytes_per_launch")


class Sets:
    """Several independent input/output buffer sets, cycled per step."""

    def __init__(self, make, bytes_per_set):
        self.n = max(3, -(-2 * LLC_BYTES // max(bytes_per_set, 1)))
        self.n = min(self.n, 16)
        self.sets = [make(i) for i in range(self.n)]

    def __getitem__(self, i):
        return self.sets[i % self.n]


def make_layer_set(offq, inputs, torch, M, K, N, g, seed, spec):
    x = inputs.activations_device(M, K, seed=seed, device="cuda", **spec)
    w = inputs.weights_device(N, K, seed=seed, device="cuda")
    wc, ws, wcs = offq.offq_pack_weights(w, g)
    del w
    return dict(x=x, wc=wc, ws=ws, wcs=wcs,
                codes=torch.empty((M, K // 2), dtype=torch.uint8, device="cuda"),
                scale=torch.empty((M, K // g), dtype=torch.float16, device="cuda"),
                zero=torch.empty((M, K // g), dtype=torch.int16, device="cuda"),
                y=torch.empty((M, N), dtype=torch.bfloat16, device="cuda"),
                M=M, K=K, N=N, g=g)


def run_rq(lib, s, stream):
    return lib.offq_rotate_quantize_raw(s["x"].data_ptr(), s["M"], s["K"], s["K"], s["g"], 1,
                                        s["codes"].data_ptr(), s["scale"].data_ptr(),
                                        s["zero"].data_ptr(), None, stream)


def run_gemm(lib, s, stream):
    return lib.offq_w4a4_gemm_raw(s["codes"].data_ptr(), s["scale"].data_ptr(), s["zero"].data_ptr(),
                                  s["wc"].data_ptr(), s["ws"].data_ptr(), s["wcs"].data_ptr(),
                                  s["M"], s["N"], s["K"], s["g"], s["y"].data_ptr(), s["N"], None,
                                  stream)


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_layer_prep(np, inputs, OQ, K, N, g, spec, seed, n_cols=None):
    """Offline weight preparation of one layer (not timed): the oracle's
    symmetric weight quantizer and column sums, on the first n_cols output
    channels when given."""
    w = inputs.weights(N, K, seed=seed)
    if n_cols is not None:
        w = np.ascontiguousarray(w[:n_cols])
    q_w, sw = OQ.quantize_weights(w)
    del w
    return q_w, sw, OQ.colsum(q_w, g)


def _oracle_stages(np, OH, OQ, OG, x, g, q_w, sw, cs, t):
    """One pass of the oracle over a layer: rotate (fp64), quantize (fp32),
    integer GEMM (fp64 BLAS), epilogue (fp64); seconds added to t."""
    t0 = time.perf_counter()
    y = OH.rotate(x, g).astype(np.float32)
    t1 = time.perf_counter()
    q, s_, z = OQ.quantize_groups(y, g)
    t2 = time.perf_counter()
    acc = OG.int_gemm_groups(q, q_w, g)
    t3 = time.perf_counter()
    OG.epilogue(acc, s_, z, sw, cs)
    t4 = time.perf_counter()
    for k, v in (("rotate", t1 - t0), ("quantize", t2 - t1), ("int_gemm", t3 - t2),
                 ("epilogue", t4 - t3)):
        t[k] = t.get(k, 0.0) + v


def cpu_baseline(layers, sample_rows, min_s=10.0, per_config=None):
    """The CPU oracle, as it stands, on a bounded sample of the workload: the
    first ``sample_rows`` token rows of each layer (full K and N), the whole
    step repeated until ``min_s`` seconds; per-stage seconds; the rate in the
    metric's unit (integer TOP/s of the sampled GEMM work).  ``per_config``:
    other workloads, one pass each on their own samples, per-stage."""
    import numpy as np
    from threadpoolctl import threadpool_info, threadpool_limits

    from oracle import gemm as OG
    from oracle import hadamard as OH
    from oracle import quantizer as OQ
    from paper_2606_07116_amd import inputs

    ncpu = len(os.sched_getaffinity(0))
    with threadpool_limits(limits=ncpu):
        prepped = []
        for (name, M, K, N, g, spec, seed, n_cols) in layers:
            x = inputs.activations(sample_rows, K, seed=seed, **spec)
            prepped.append((name, x, g) + _oracle_layer_prep(np, inputs, OQ, K, N, g, spec, seed,
                                                             n_cols))
        stages = {}
        reps, t0 = 0, time.perf_counter()
        while True:
            for (name, x, g, q_w, sw, cs) in prepped:
                _oracle_stages(np, OH, OQ, OG, x, g, q_w, sw, cs, stages)
            reps += 1
            el = time.perf_counter() - t0
            if el >= min_s or reps >= 50:
                break
        del prepped
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
        ops = sum(2.0 * sample_rows * (nc or N) * K for (_, M, K, N, g, _, _, nc) in layers) * reps
        desc = ", ".join(f"{n}: K={K}, N={N}" + (f" (first {nc} output channels)" if nc else "")
                         + f", g={g}" for (n, _, K, N, g, _, _, nc) in layers)
        out = {"value": round(ops / el / 1e12, 4), "unit": "TOPS", "cores": int(threads),
               "kind": "oracle",
               "sample": f"first {sample_rows} of the {layers[0][1]} token rows of each layer "
                         f"({desc}), whole step {reps} time(s) in {el:.1f} s; rate = sampled GEMM "
                         "ops / s",
               "stage_seconds": {k: round(v, 3) for k, v in stages.items()},
               "cpu_model": _cpu_model(), "host_cpus": ncpu,
               "threads_note": "BLAS (the integer GEMM via fp64 matmul) uses the threads above; "
                               "the rotate, quantize and epilogue stages are single-threaded numpy"}
        if per_config:
            out["per_config"] = {}
            for cname, fn in per_config.items():
                out["per_config"][cname] = fn(np, inputs, OH, OQ, OG)
    return out


def cpu_prefill_layer(lc, tokens, min_s=10.0):
    """The oracle's prefill of the layer (oracle.layer.prefill_layer: every
    stage, the causal attention over the 4-bit cache included) on a bounded
    sample: the first ``tokens`` tokens of one sequence with the full-width
    weights, repeated until ``min_s`` seconds; the rate in the metric's unit
    (integer TOP/s of the sampled projections) and in tokens per second.  The
    weight quantization is setup, not timed."""
    import numpy as np
    from threadpoolctl import threadpool_info, threadpool_limits

    from oracle import layer as OL
    from oracle import quantizer as OQ
    from paper_2606_07116_amd import inputs

    D, Hq, Hkv, F, g = lc["D"], lc["Hq"], lc["Hkv"], lc["F"], lc["g"]
    shapes = {"qkv": ((Hq + 2 * Hkv) * 128, D), "o": (D, Hq * 128), "ug": (2 * F, D), "down": (D, F)}
    ncpu = len(os.sched_getaffinity(0))
    with threadpool_limits(limits=ncpu):
        weights = {k: OQ.quantize_weights(inputs.weights(n, k_, seed=lc["seed"] + j,
                                                         std=1.0 / k_ ** 0.5))
                   for j, (k, (n, k_)) in enumerate(shapes.items())}
        rng = np.random.default_rng(lc["seed"])
        x = inputs.round_to_bf16(rng.standard_normal((tokens, D)).astype(np.float32))
        kc, ks, kz = inputs.kv4_cache(1, Hkv, tokens, 128, seed=lc["seed"])
        vc, vs, vz = inputs.kv4_cache(1, Hkv, tokens, 128, seed=lc["seed"] + 1)
        cache = dict(k_codes=kc, k_scale=ks, k_zero=kz, v_codes=vc, v_scale=vs, v_zero=vz)
        cfg = dict(Hq=Hq, Hkv=Hkv, g=g, eps=1e-5, rope_base=500000.0)
        reps, t0 = 0, time.perf_counter()
        while True:
            OL.prefill_layer(x, weights, cache, 0, cfg)
            reps += 1
            el = time.perf_counter() - t0
            if el >= min_s or reps >= 50:
                break
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    ops = sum(2.0 * tokens * n * k_ for n, k_ in shapes.values()) * reps
    return {"value": round(ops / el / 1e12, 4), "unit": "TOPS", "cores": int(threads),
            "kind": "oracle", "tokens_per_s": round(tokens * reps / el, 2),
            "sample": f"the first {tokens} tokens of one sequence through the whole layer "
                      f"(D {D}, {Hq}/{Hkv} heads, MLP {F}, g = {g}, causal attention over the "
                      f"{tokens} cached positions), {reps} time(s) in {el:.1f} s; rate = "
                      "projection int ops / s",
            "cpu_model": _cpu_model(), "host_cpus": ncpu,
            "threads_note": "BLAS (the integer GEMMs via fp64 matmul) uses the threads above; "
                            "the other stages are numpy"}


def _cpu_layer_config(layers, rows, n_cols=None, unit="TOPS"):
    """One oracle pass over each layer of a workload on its first ``rows``
    rows (and first ``n_cols`` output channels when given), per-stage
    seconds and the rate in the workload's unit."""
    def run(np, inputs, OH, OQ, OG):
        t, ops, nbytes = {}, 0.0, 0.0
        for (name, M, K, N, g, spec, seed) in layers:
            x = inputs.activations(rows, K, seed=seed, **spec)
            q_w, sw, cs = _oracle_layer_prep(np, inputs, OQ, K, N, g, spec, seed, n_cols)
            nc = N if n_cols is None else n_cols
            _oracle_stages(np, OH, OQ, OG, x, g, q_w, sw, cs, t)
            ops += 2.0 * rows * nc * K
            nbytes += gemv_bytes(rows, nc, K, g) + rq_bytes(rows, K, g)
        el = sum(t.values())
        r = {"stage_seconds": {k: round(v, 4) for k, v in t.items()},
             "sample": f"first {rows} rows" + (f", first {n_cols} output channels" if n_cols else "")
             + " of " + ", ".join(f"{n}: M={M}, K={K}, N={N}, g={g}" for (n, M, K, N, g, _, _) in layers)}
        if unit == "TOPS":
            r["TOPS"] = round(ops / el / 1e12, 5)
        else:
            r["GBs"] = round(nbytes / el / 1e9, 3)
        return r
    return run


def _cpu_kv_config(rows, Dh=128):
    """The oracle's KV quantizer (128-point H3 in fp64, then the quantizer)
    on ``rows`` cache rows drawn as the KV workload's; per-stage seconds and
    algorithmic GB/s."""
    def run(np, inputs, OH, OQ, OG):
        from oracle import kv as OKV
        kc = inputs.WORKLOADS["kv_cache"]
        x = inputs.kv_rows(rows, Dh, seed=kc["seed"], n_outliers=kc["n_outliers"], lo=kc["lo"],
                           hi=kc["hi"], heads=kc["H"])
        t0 = time.perf_counter()
        y = OKV.kv_rotate(x, True).astype(np.float32)
        t1 = time.perf_counter()
        OKV.kv_quantize(y)
        t2 = time.perf_counter()
        return {"stage_seconds": {"rotate": round(t1 - t0, 4), "quantize": round(t2 - t1, 4)},
                "GBs": round(rq_bytes(rows, Dh, Dh) / (t2 - t0) / 1e9, 3),
                "sample": f"{rows} rows [.., 128] of the KV cache recipe"}
    return run


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: one GPU only (asked for --gpus {args.gpus}); the kernels run on one "
              "GPU's share of a layer and no multi-GPU path exists", file=sys.stderr)
        sys.exit(2)
    import torch

    import paper_2606_07116_amd as offq
    from paper_2606_07116_amd import _lib, inputs

    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream
    wl = args.workload

    def regroup(cfg):
        """The workload's layer with --group-size applied (outliers then sit at
        the first channel of each group of that size)."""
        if not args.group_size:
            return cfg
        g = args.group_size
        if g & (g - 1) or g < 64 or cfg["K"] % g:
            raise SystemExit(f"bench.py: --group-size {g} must be a power of two >= 64 dividing K")
        return dict(cfg, g=g)

    def check(st, what):
        if st != 0:
            raise RuntimeError(f"{what}: {_lib.status_name(st)}: {_lib.last_error()}")


    if wl in ("attn_proj_prefill", "kv_chain"):
        cfg = regroup(inputs.WORKLOADS["attn_proj_prefill" if wl == "attn_proj_prefill"
                                       else "kv_chain_proj"])
        M, K, N, g = cfg["M"], cfg["K"], cfg["N"], cfg["g"]
        spec = dict(n_outliers=cfg["n_outliers"], lo=cfg["lo"], hi=cfg["hi"])
        per_set = M * K * 2 + N * K // 2 + M * K // 2 + M * N * 2
        sets = Sets(lambda i: make_layer_set(offq, inputs, torch, M, K, N, g, cfg["seed"] + 100 * i,
                                             spec), per_set)
        layers = [("rotate_quantize", "w4a4_gemm", sets)]
        work_ops = 2.0 * M * N * K
        config = {"workload": wl, "M": M, "K": K, "N": N, "g": g,
                  "step": "rotate_quantize + w4a4_gemm", "input_sets": sets.n}
        if wl == "kv_chain":
            kc = inputs.WORKLOADS["kv_cache"]
            B, H, S, Dh = kc["B"], kc["H"], kc["S"], kc["Dh"]
            kv = [inputs.kv_cache_device(B, H, S, Dh, seed=kc["seed"] + j, device="cuda",
                                         n_outliers=kc["n_outliers"], lo=kc["lo"], hi=kc["hi"])
                  for j in range(2)]
            R = B * H * S
            kvo = [dict(codes=torch.empty((R, Dh // 2), dtype=torch.uint8, device="cuda"),
                        scale=torch.empty((R,), dtype=torch.float16, device="cuda"),
                        zero=torch.empty((R,), dtype=torch.int16, device="cuda")) for _ in range(2)]
            config.update({"kv_shape": [B, H, S, Dh], "step": "kv_quantize(K) + kv_quantize(V) + "
                           "rotate_quantize + w4a4_gemm"})
    elif wl == "mlp_prefill":
        up = regroup(inputs.WORKLOADS["mlp_up_gate_prefill"])
        dn = regroup(inputs.WORKLOADS["mlp_down_prefill"])
        spec_u = dict(n_outliers=up["n_outliers"], lo=up["lo"], hi=up["hi"],
                      spike_frac=up["spike_frac"], spike_mult=up["spike_mult"])
        spec_d = dict(n_outliers=dn["n_outliers"], lo=dn["lo"], hi=dn["hi"],
                      spike_frac=dn["spike_frac"], spike_mult=dn["spike_mult"])
        per_u = up["M"] * up["K"] * 2 + up["N"] * up["K"] + up["M"] * up["N"] * 4
        per_d = dn["M"] * dn["K"] * 2 + dn["N"] * dn["K"] // 2 + dn["M"] * dn["N"] * 2
        su = Sets(lambda i: make_layer_set(offq, inputs, torch, up["M"], up["K"], 2 * up["N"], up["g"],
                                           up["seed"] + 100 * i, spec_u), per_u)
        sd = Sets(lambda i: make_layer_set(offq, inputs, torch, dn["M"], dn["K"], dn["N"], dn["g"],
                                           dn["seed"] + 100 * i, spec_d), per_d)
        layers = [("rotate_quantize_up", "w4a4_gemm_upgate", su),
                  ("rotate_quantize_down", "w4a4_gemm_down", sd)]
        work_ops = 2.0 * up["M"] * 2 * up["N"] * up["K"] + 2.0 * dn["M"] * dn["N"] * dn["K"]
        config = {"workload": wl, "up_gate": [up["M"], up["K"], 2 * up["N"], up["g"]],
                  "down": [dn["M"], dn["K"], dn["N"], dn["g"]],
                  "step": "rotate_quantize + gemm(up|gate, N=28672) + rotate_quantize(g=512) + gemm(down)",
                  "input_sets": [su.n, sd.n]}
    elif wl == "kv_decode_attention":
        ac = inputs.WORKLOADS["kv_decode_attention"]
        B, H, S, Dh = ac["B"], ac["H"], ac["S"], ac["Dh"]

        def make_attn(i):
            kc_, ks_, kz_ = inputs.kv4_cache_device(B, H, S, Dh, seed=ac["seed"] + 10 * i,
                                                     device="cuda")
            vc_, vs_, vz_ = inputs.kv4_cache_device(B, H, S, Dh, seed=ac["seed"] + 10 * i + 1,
                                                     device="cuda")
            q_ = torch.from_numpy(inputs.queries(B, H, Dh, seed=ac["seed"] + i)).to(
                torch.bfloat16).cuda()
            wsb = offq.offq_kv_attention_workspace_bytes(B, H, S)
            return dict(q=q_, kc=kc_, ks=ks_, kz=kz_, vc=vc_, vs=vs_, vz=vz_,
                        out=torch.empty((B, H, Dh), dtype=torch.bfloat16, device="cuda"),
                        ws=torch.empty(wsb // 4, dtype=torch.float32, device="cuda"), wsb=wsb)

        asets = Sets(make_attn, attn_bytes(B * H, S, Dh))
        layers = []
        work_ops = None
        config = {"workload": wl, "kv_shape": [B, H, S, Dh], "seq_len": S,
                  "step": "kv_attention_decode (split-sequence pass + combine pass)",
                  "input_sets": asets.n}
    elif wl == "calibration":
        cc = inputs.WORKLOADS["calibration"]
        n_seq, L, D, g = cc["n_seq"], cc["L"], cc["D"], cc["g"]
        x_cal = inputs.activations_device(n_seq * L, D, seed=cc["seed"], device="cuda",
                                          n_outliers=cc["n_outliers"], lo=cc["lo"], hi=cc["hi"],
                                          spike_frac=cc["spike_frac"],
                                          spike_mult=cc["spike_mult"]).view(n_seq, L, D)
        w_in = {name: inputs.weights_device(n_, D, seed=cc["seed"] + j, device="cuda")
                for j, (name, n_) in enumerate(cc["layers"].items())}
        cal = {}
        layers = []
        work_ops = None
        args.steps, args.warmup = min(args.steps, 1), 0  # seconds per step
        config = {"workload": wl, "calibration": [n_seq, L, D], "g": g,
                  "fused_layers": {k: [v, D] for k, v in cc["layers"].items()},
                  "step": "top-1 selection, covariance, Jacobi eigendecomposition, sorted "
                          "grouping, rotation U P H, weight fusion and packing"}
    elif wl == "decode_layer":
        lc = inputs.WORKLOADS["decode_layer"]
        M, D, Hq, Hkv, F, g = lc["M"], lc["D"], lc["Hq"], lc["Hkv"], lc["F"], lc["g"]
        ctx = lc["ctx"]
        s_cap, seq_len = ctx + 1, ctx + 1
        NQKV = (Hq + 2 * Hkv) * 128
        lshapes = {"qkv": (NQKV, D), "o": (D, Hq * 128), "ug": (2 * F, D), "down": (D, F)}
        bf, u8, f16, i16 = torch.bfloat16, torch.uint8, torch.float16, torch.int16

        def make_layer(i):
            sd = lc["seed"] + 100 * i
            st = {"x": torch.from_numpy(inputs.queries(1, M, D, seed=sd)[0]).to(bf).cuda()}
            for j, (k, (n_, k_)) in enumerate(lshapes.items()):
                w = inputs.weights_device(n_, k_, seed=sd + j, device="cuda", std=1.0 / k_ ** 0.5)
                st["w_" + k] = offq.offq_pack_weights(w, g)
                del w
            kc_, ks_, kz_ = inputs.kv4_cache_device(M, Hkv, s_cap, 128, seed=sd, device="cuda")
            vc_, vs_, vz_ = inputs.kv4_cache_device(M, Hkv, s_cap, 128, seed=sd + 1, device="cuda")
            st.update(kc=kc_, ks=ks_, kz=kz_, vc=vc_, vs=vs_, vz=vz_,
                      pos=torch.full((M,), ctx, dtype=torch.int32, device="cuda"))
            e = lambda *sh, dt=bf: torch.empty(sh, dtype=dt, device="cuda")
            st.update(y0=e(M, D), qkv=e(M, NQKV), q=e(M, Hq, 128), o=e(M, Hq, 128),
                      ao=e(M, D), h0=e(M, D), h1=e(M, D), y1=e(M, D), gu=e(M, 2 * F), a=e(M, F),
                      dn=torch.zeros((M, D), dtype=bf, device="cuda"))
            for name, K_ in (("c_in", D), ("c_o", Hq * 128), ("c_d", F)):
                st[name] = (e(M, K_ // 2, dt=u8), e(M, K_ // g, dt=f16), e(M, K_ // g, dt=i16))
            st["wsb"] = offq.offq_kv_attention_workspace_bytes(M, Hq, seq_len)
            st["ws"] = e(st["wsb"] // 4, dt=torch.float32)
            return st

        lbytes = sum(weight_bytes(n_, k_, g) for n_, k_ in lshapes.values())
        kvbytes = M * Hkv * seq_len * 136
        step_bytes = lbytes + kvbytes + M * (D * 2 * 8 + NQKV * 2 + F * 6)
        lsets = Sets(make_layer, lbytes + kvbytes)
        layers = []
        work_ops = None
        config = {"workload": wl, "M": M, "D": D, "heads": [Hq, Hkv], "mlp": F, "g": g,
                  "context": ctx, "step": "add (the previous layer's residual) + RMSNorm + "
                  "quantize, QKV GEMV, RoPE + H3 + KV4 append, GQA decode attention with the "
                  "output quantized in its combine pass, O GEMV, add + RMSNorm + quantize, "
                  "up/gate GEMV, SwiGLU + H4 + quantize, down GEMV (its residual add is the next "
                  "layer's first add)", "input_sets": lsets.n}
    elif wl == "prefill_layer":
        lc = inputs.WORKLOADS["prefill_layer"]
        Bp, Tp, past = lc["B"], lc["T"], lc["past"]
        M, D, Hq, Hkv, F, g = Bp * Tp, lc["D"], lc["Hq"], lc["Hkv"], lc["F"], lc["g"]
        s_cap = past + Tp
        NQKV = (Hq + 2 * Hkv) * 128
        lshapes = {"qkv": (NQKV, D), "o": (D, Hq * 128), "ug": (2 * F, D), "down": (D, F)}
        bf, u8, f16, i16 = torch.bfloat16, torch.uint8, torch.float16, torch.int16

        def make_prefill(i):
            sd = lc["seed"] + 100 * i
            gen = torch.Generator(device="cuda")
            gen.manual_seed(sd)
            st = {"x": torch.randn((M, D), generator=gen, device="cuda").to(bf)}
            for j, (k, (n_, k_)) in enumerate(lshapes.items()):
                w = inputs.weights_device(n_, k_, seed=sd + j, device="cuda", std=1.0 / k_ ** 0.5)
                st["w_" + k] = offq.offq_pack_weights(w, g)
                del w
            kc_, ks_, kz_ = inputs.kv4_cache_device(Bp, Hkv, s_cap, 128, seed=sd, device="cuda")
            vc_, vs_, vz_ = inputs.kv4_cache_device(Bp, Hkv, s_cap, 128, seed=sd + 1, device="cuda")
            st.update(kc=kc_, ks=ks_, kz=kz_, vc=vc_, vs=vs_, vz=vz_,
                      pos=(past + torch.arange(Tp, dtype=torch.int32, device="cuda")).repeat(Bp))
            e = lambda *sh, dt=bf: torch.empty(sh, dtype=dt, device="cuda")
            st.update(qkv=e(M, NQKV), q=e(M, Hq, 128), o=e(M, Hq, 128), ao=e(M, D), h0=e(M, D),
                      h1=e(M, D), gu=e(M, 2 * F), dn=torch.zeros((M, D), dtype=bf, device="cuda"))
            for name, K_ in (("c_in", D), ("c_o", Hq * 128), ("c_d", F)):
                st[name] = (e(M, K_ // 2, dt=u8), e(M, K_ // g, dt=f16), e(M, K_ // g, dt=i16))
            return st

        lbytes = sum(weight_bytes(n_, k_, g) for n_, k_ in lshapes.values())
        lsets = Sets(make_prefill, lbytes + M * (D * 2 * 8 + NQKV * 2 + F * 6))
        layers = []
        gemm_shapes = {"w4a4_gemm_qkv": (NQKV, D), "w4a4_gemm_o": (D, Hq * 128),
                       "w4a4_gemm_upgate": (2 * F, D), "w4a4_gemm_down": (D, F)}
        work_ops = sum(2.0 * M * n_ * k_ for n_, k_ in gemm_shapes.values())
        # causal attention: 2 * 128 multiply-adds per (query, attended key) for
        # the scores and as many for the values
        attn_flops = 4.0 * 128 * Bp * Hq * (Tp * past + Tp * (Tp + 1) / 2)
        config = {"workload": wl, "B": Bp, "T": Tp, "past": past, "D": D, "heads": [Hq, Hkv],
                  "mlp": F, "g": g, "step": "add (the previous layer's residual) + RMSNorm + "
                  "quantize, QKV GEMM, RoPE + H3 + KV4 write of the T tokens, causal attention "
                  "over the 4-bit cache, quantize, O GEMM, add + RMSNorm + quantize, up/gate GEMM, "
                  "SwiGLU + H4 + quantize, down GEMM", "input_sets": lsets.n}
    else:  # decode
        up = regroup(inputs.WORKLOADS["decode_up"])
        dn = regroup(inputs.WORKLOADS["decode_down"])
        Md = args.decode_m
        spec = dict(n_outliers=up["n_outliers"], lo=up["lo"], hi=up["hi"])
        per = up["N"] * up["K"] // 2 * 2
        su = Sets(lambda i: make_layer_set(offq, inputs, torch, Md, up["K"], up["N"], up["g"],
                                           up["seed"] + 100 * i, spec), per)
        sd = Sets(lambda i: make_layer_set(offq, inputs, torch, Md, dn["K"], dn["N"], dn["g"],
                                           dn["seed"] + 100 * i, spec), per)
        layers = [("rotate_quantize_up", "w4a4_gemv_up", su), ("rotate_quantize_down", "w4a4_gemv_down", sd)]
        work_ops = None
        gbytes = gemv_bytes(Md, up["N"], up["K"], up["g"]) + gemv_bytes(Md, dn["N"], dn["K"], dn["g"])
        config = {"workload": wl, "M": Md, "up": [up["K"], up["N"], up["g"]],
                  "down": [dn["K"], dn["N"], dn["g"]], "step": "(rotate_quantize + w4a4_gemv) x2",
                  "input_sets": [su.n, sd.n]}

    torch.cuda.synchronize()

    # the step's launches in order: (kernel name, launch of step i)
    phases = []
    if wl == "kv_chain":
        for j in range(2):
            phases.append(("kv_quantize", lambda i, j=j: _lib.offq_kv_quantize_raw(
                kv[j].data_ptr(), R, Dh, Dh, 1, kvo[j]["codes"].data_ptr(), kvo[j]["scale"].data_ptr(),
                kvo[j]["zero"].data_ptr(), None, sp)))
    if wl == "calibration":
        def c_top1(i):
            cal["idx"], cal["X"] = offq.offq_top1_select(x_cal)
            return 0

        def c_gram(i):
            cal["C"] = offq.offq_gram(cal["X"])
            return 0

        def c_eigh(i):
            cal["ev"], cal["U"], cal["sweeps"], cal["rel"] = offq.offq_eigh(cal["C"])
            return 0

        def c_group(i):
            cal["perm"] = offq.offq_group_permutation(cal["ev"], g)
            cal["R"] = offq.offq_build_rotation(cal["U"], D, cal["perm"], g, True)
            return 0

        def c_fuse(i):
            cal["W"] = {k: offq.offq_fuse_weights(w, cal["R"]) for k, w in w_in.items()}
            return 0

        def c_pack(i):
            cal["packed"] = {k: offq.offq_pack_weights(w, g) for k, w in cal["W"].items()}
            return 0
        phases += [("top1_select", c_top1), ("gram", c_gram), ("eigh", c_eigh),
                   ("grouping_rotation", c_group), ("fuse_weights", c_fuse),
                   ("pack_weights", c_pack)]
    if wl == "decode_layer":
        eps, base, sm = 1e-5, 500000.0, 1.0 / 128 ** 0.5
        P_ = lambda t: t.data_ptr()

        def gemm(st, cname, K_, N_, wname, dst):
            c_, s_, z_ = st[cname]
            wc_, ws_, wcs_ = st[wname]
            return _lib.offq_w4a4_gemm_raw(P_(c_), P_(s_), P_(z_), P_(wc_), P_(ws_), P_(wcs_), M,
                                           N_, K_, g, P_(dst), N_, None, sp)

        def lin(st, cname, src, K_, N_, wname, dst, had):
            c_, s_, z_ = st[cname]
            check(_lib.offq_rotate_quantize_raw(P_(src), M, K_, K_, g, had, P_(c_), P_(s_), P_(z_),
                                                None, sp), "rotate_quantize")
            return gemm(st, cname, K_, N_, wname, dst)

        def norm_quant(st, xname, res, h_out):
            c_, s_, z_ = st["c_in"]
            check(_lib.offq_add_rmsnorm_quantize_raw(
                P_(st[xname]), D, P_(res) if res is not None else None, D, M, D, eps, g,
                P_(h_out) if h_out is not None else None, D, P_(c_), P_(s_), P_(z_), None, 0, sp),
                "add_rmsnorm_quantize")

        def step_layer(i):
            st = lsets[i]
            # steady state: the previous layer's residual add (its h1 + down)
            # is this layer's first add (x stands for that h1, dn holds the
            # down output of the set's previous step), as the next layer would
            # take this one's h1 and dn
            norm_quant(st, "x", st["dn"], st["h0"])
            check(gemm(st, "c_in", D, NQKV, "w_qkv", st["qkv"]), "gemv qkv")
            check(_lib.offq_rope_kv_append_raw(
                P_(st["qkv"]), NQKV, M, Hq, Hkv, 128, P_(st["pos"]), base, 1, 0, P_(st["q"]),
                P_(st["kc"]), P_(st["ks"]), P_(st["kz"]), P_(st["vc"]), P_(st["vs"]), P_(st["vz"]),
                s_cap, None, None, sp), "rope_kv_append")
            co_, so_, zo_ = st["c_o"]  # attention output quantized in its combine pass
            check(_lib.offq_kv_attention_decode_quantize_raw(
                P_(st["q"]), P_(st["kc"]), P_(st["ks"]), P_(st["kz"]), P_(st["vc"]), P_(st["vs"]),
                P_(st["vz"]), M, Hq, Hkv, s_cap, seq_len, 128, sm, 0, None, P_(co_), P_(so_),
                P_(zo_), P_(st["ws"]), st["wsb"], sp), "attention")
            check(gemm(st, "c_o", Hq * 128, D, "w_o", st["ao"]), "gemv o")
            norm_quant(st, "h0", st["ao"], st["h1"])
            check(gemm(st, "c_in", D, 2 * F, "w_ug", st["gu"]), "gemv up/gate")
            c_, s_, z_ = st["c_d"]
            check(_lib.offq_swiglu_rotate_quantize_raw(P_(st["gu"]), 2 * F, M, F, P_(c_), P_(s_),
                                                       P_(z_), None, sp), "swiglu_rotate_quantize")
            return gemm(st, "c_d", F, D, "w_down", st["dn"])
        # the whole layer is one phase: its kernels depend on each other
        phases.append(("decode_layer", step_layer))
    if wl == "prefill_layer":
        eps, base, sm = 1e-5, 500000.0, 1.0 / 128 ** 0.5
        P_ = lambda t: t.data_ptr()

        def pgemm(name, cname, K_, N_, wname, dst):
            def f(i):
                st = lsets[i]
                c_, s_, z_ = st[cname]
                wc_, ws_, wcs_ = st[wname]
                return _lib.offq_w4a4_gemm_raw(P_(c_), P_(s_), P_(z_), P_(wc_), P_(ws_), P_(wcs_),
                                               M, N_, K_, g, P_(st[dst]), N_, None, sp)
            return (name, f)

        def pnorm(name, xname, rname, hname):
            def f(i):
                st = lsets[i]
                c_, s_, z_ = st["c_in"]
                return _lib.offq_add_rmsnorm_quantize_raw(
                    P_(st[xname]), D, P_(st[rname]), D, M, D, eps, g, P_(st[hname]), D, P_(c_),
                    P_(s_), P_(z_), None, 0, sp)
            return (name, f)

        def p_rope(i):
            st = lsets[i]
            return _lib.offq_rope_kv_prefill_raw(
                P_(st["qkv"]), NQKV, Bp, Tp, Hq, Hkv, 128, P_(st["pos"]), base, 1, 0, P_(st["q"]),
                P_(st["kc"]), P_(st["ks"]), P_(st["kz"]), P_(st["vc"]), P_(st["vs"]), P_(st["vz"]),
                s_cap, None, None, sp)

        def p_attn(i):
            st = lsets[i]
            return _lib.offq_kv_attention_prefill_raw(
                P_(st["q"]), Bp, Tp, Hq, Hkv, 128, past, P_(st["kc"]), P_(st["ks"]), P_(st["kz"]),
                P_(st["vc"]), P_(st["vs"]), P_(st["vz"]), s_cap, sm, 0, P_(st["o"]), sp)

        def p_quant_o(i):
            st = lsets[i]
            c_, s_, z_ = st["c_o"]
            return _lib.offq_rotate_quantize_raw(P_(st["o"]), M, Hq * 128, Hq * 128, g, 0, P_(c_),
                                                 P_(s_), P_(z_), None, sp)

        def p_swiglu(i):
            st = lsets[i]
            c_, s_, z_ = st["c_d"]
            return _lib.offq_swiglu_rotate_quantize_raw(P_(st["gu"]), 2 * F, M, F, P_(c_), P_(s_),
                                                        P_(z_), None, sp)
        # steady state as in the decode layer: the previous layer's residual
        # add (x + dn) is this layer's first step
        phases += [pnorm("add_rmsnorm_quantize_in", "x", "dn", "h0"),
                   pgemm("w4a4_gemm_qkv", "c_in", D, NQKV, "w_qkv", "qkv"),
                   ("rope_kv_prefill", p_rope), ("kv_attention_prefill", p_attn),
                   ("rotate_quantize_o", p_quant_o),
                   pgemm("w4a4_gemm_o", "c_o", Hq * 128, D, "w_o", "ao"),
                   pnorm("add_rmsnorm_quantize_post", "h0", "ao", "h1"),
                   pgemm("w4a4_gemm_upgate", "c_in", D, 2 * F, "w_ug", "gu"),
                   ("swiglu_rotate_quantize", p_swiglu),
                   pgemm("w4a4_gemm_down", "c_d", F, D, "w_down", "dn")]
    if wl == "kv_decode_attention":
        def run_attn(i):
            a_ = asets[i]
            return _lib.offq_kv_attention_decode_raw(
                a_["q"].data_ptr(), a_["kc"].data_ptr(), a_["ks"].data_ptr(), a_["kz"].data_ptr(),
                a_["vc"].data_ptr(), a_["vs"].data_ptr(), a_["vz"].data_ptr(), B, H, S, S, Dh,
                1.0 / Dh ** 0.5, 0, a_["out"].data_ptr(), a_["ws"].data_ptr(), a_["wsb"], sp)
        phases.append(("kv_attention_decode", run_attn))
    for rq_name, mm_name, sets_ in layers:
        phases.append((rq_name, lambda i, s_=sets_: run_rq(_lib, s_[i], sp)))
        phases.append((mm_name, lambda i, s_=sets_: run_gemm(_lib, s_[i], sp)))

    # library launches per step (the spin below covers the host's enqueue time)
    launches_per_step = 10 if wl == "decode_layer" else len(phases)
    ms, comp = run_phases(torch, stream, phases, args.steps, args.warmup, check,
                          launches_per_step)
    n_dist = max(100, args.steps)
    if wl != "calibration":
        add_dist(torch, stream, phases, comp, n_dist, check)
    gap = event_gap(torch, stream)

    # counter-measured HBM bytes are keyed by workload (and group size when
    # --group-size overrides the workload's own)
    tkey = wl if not args.group_size else f"{wl}:g{args.group_size}"
    if wl in ("attn_proj_prefill", "kv_chain"):
        ann_rq(comp["rotate_quantize"], M, K, g)
        ann_mm(comp["w4a4_gemm"], M, N, K)
        if wl == "kv_chain":
            ann_rq(comp["kv_quantize"], R, Dh, Dh)
        value = work_ops / (ms * 1e-3) / 1e12
        unit = "TOPS"
        roof = mfma_roof(comp, "w4a4_gemm", traffic_for(f"w4a4_gemm:{tkey}"))
    elif wl == "mlp_prefill":
        ann_rq(comp["rotate_quantize_up"], up["M"], up["K"], up["g"])
        ann_rq(comp["rotate_quantize_down"], dn["M"], dn["K"], dn["g"])
        ann_mm(comp["w4a4_gemm_upgate"], up["M"], 2 * up["N"], up["K"])
        ann_mm(comp["w4a4_gemm_down"], dn["M"], dn["N"], dn["K"])
        value = work_ops / (ms * 1e-3) / 1e12
        unit = "TOPS"
        roof = mfma_roof(comp, "w4a4_gemm_upgate", traffic_for(f"w4a4_gemm:{tkey}"))
    elif wl == "calibration":
        tb = n_seq * L * D * 2
        comp["top1_select"]["alg_bytes"] = tb
        comp["top1_select"]["GBs"] = round(tb / (comp["top1_select"]["us"] * 1e-6) / 1e9, 1)
        gf = n_seq * D * D  # fp64 multiply-adds of the upper triangle, x2 flops
        comp["gram"]["fp64_TFLOPs"] = round(2 * gf / (comp["gram"]["us"] * 1e-6) / 1e12, 3)
        nf = sum(2.0 * n_ * D * D for n_ in cc["layers"].values())
        comp["fuse_weights"]["fp32_TFLOPs"] = round(nf / (comp["fuse_weights"]["us"] * 1e-6) / 1e12, 2)
        # every Jacobi step reads and writes the upper triangle of the
        # symmetric A (8 D (D + 1) bytes); V is read and written once per
        # batch of 64 steps (16 D^2 bytes)
        eb = (8.0 * D * (D + 1) * (D - 1) + 16.0 * D * D * -(-(D - 1) // 64)) * cal["sweeps"]
        comp["eigh"].update({"sweeps": cal["sweeps"], "rel_offdiag": cal["rel"], "alg_bytes": eb,
                             "GBs": round(eb / (comp["eigh"]["us"] * 1e-6) / 1e9, 1)})
        comp["eigh"]["frac_hbm"] = round(comp["eigh"]["GBs"] / PEAK_HBM_GBS, 4)
        value = round(ms / 1e3, 3)
        unit = "s per layer-input calibration"
        roof = {"bound": "hbm", "achieved": comp["eigh"]["GBs"], "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": comp["eigh"]["frac_hbm"], "traffic": None, "kernel": "eigh",
                "alg_bytes_per_launch": eb, "avg_launch_us": comp["eigh"]["us"]}
    elif wl == "decode_layer":
        name = "decode_layer"
        ann_bytes(comp[name], step_bytes)
        comp[name]["tokens_per_s"] = round(M / (comp[name]["us"] * 1e-6), 1)
        value = comp[name]["GBs"]
        unit = "GB/s"
        roof = hbm_roof(comp, name, None)
    elif wl == "prefill_layer":
        for name, (n_, k_) in gemm_shapes.items():
            ann_mm(comp[name], M, n_, k_)
        ca = comp["kv_attention_prefill"]
        ca["alg_flops"] = attn_flops
        ca["TFLOPs"] = round(attn_flops / (ca["us"] * 1e-6) / 1e12, 1)
        ca["frac_fp16_peak"] = round(ca["TFLOPs"] / PEAK_FP16_TFLOPS, 4)
        if "median_us" in ca:
            ca["TFLOPs_median"] = round(attn_flops / (ca["median_us"] * 1e-6) / 1e12, 1)
        value = work_ops / (ms * 1e-3) / 1e12
        unit = "TOPS"
        config["tokens_per_s"] = round(M / (ms * 1e-3), 1)
        roof = mfma_roof(comp, "w4a4_gemm_upgate", None)
    elif wl == "kv_decode_attention":
        name = "kv_attention_decode"
        ann_bytes(comp[name], attn_bytes(B * H, S, Dh))
        value = comp[name]["GBs"]
        unit = "GB/s"
        roof = hbm_roof(comp, name, traffic_for(f"kv_attention:{tkey}"))
    else:
        ann_rq(comp["rotate_quantize_up"], Md, up["K"], up["g"])
        ann_rq(comp["rotate_quantize_down"], Md, dn["K"], dn["g"])
        for name, c in (("w4a4_gemv_up", up), ("w4a4_gemv_down", dn)):
            ann_bytes(comp[name], gemv_bytes(Md, c["N"], c["K"], c["g"]))
        value = gbytes / (ms * 1e-3) / 1e9
        unit = "GB/s"
        roof = hbm_roof(comp, "w4a4_gemv_up", traffic_for(f"w4a4_gemv:{tkey}"))

    # measured HBM bytes per launch of the other kernels, where counters exist
    tnames = {"rotate_quantize": "rotate_quantize", "w4a4_gemm": "w4a4_gemm",
              "kv_quantize": "kv_quantize", "rotate_quantize_up": "rotate_quantize_up",
              "rotate_quantize_down": "rotate_quantize_down", "w4a4_gemm_upgate": "w4a4_gemm",
              "w4a4_gemm_down": "w4a4_gemm_down", "w4a4_gemv_up": "w4a4_gemv",
              "w4a4_gemv_down": "w4a4_gemv_down", "kv_attention_decode": "kv_attention"}
    for name, c in comp.items():
        if name in tnames:
            tb = traffic_for(f"{tnames[name]}:{tkey}")
            if tb is not None:
                c["traffic_bytes"] = tb
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": unit, "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": wl != "calibration", "scaling": "weak", "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic (seeded Llama-shaped activations with structured outliers; random weights)",
        "config": config, "roofline": roof, "components": comp, "event_gap_us": round(gap, 3),
        "timing": f"us = phase mean over {args.steps} launches with no event between them; "
                  f"median/p10/p90 over {n_dist} launches with an event after each "
                  "(cold: buffer sets cycled; warm: one set)",
    }
    if wl == "mlp_prefill" and not args.no_components and not args.group_size:
        for sets_ in (su, sd):
            sets_.sets.clear()
        torch.cuda.empty_cache()
        out["configs"] = other_configs(torch, offq, _lib, inputs, stream, sp, check, args, n_dist)
    if not args.no_cpu_baseline and wl == "mlp_prefill":
        lay = [("up_gate", up["M"], up["K"], 2 * up["N"], up["g"], spec_u, up["seed"], 8192),
               ("down", dn["M"], dn["K"], dn["N"], dn["g"], spec_d, dn["seed"], None)]
        per_config = None
        if not args.group_size:
            ap = inputs.WORKLOADS["attn_proj_prefill"]
            du = inputs.WORKLOADS["decode_up"]
            dd = inputs.WORKLOADS["decode_down"]
            sp2 = dict(n_outliers=ap["n_outliers"], lo=ap["lo"], hi=ap["hi"])
            sp4 = dict(n_outliers=du["n_outliers"], lo=du["lo"], hi=du["hi"])
            per_config = {
                "attn_proj_prefill": _cpu_layer_config(
                    [("proj", ap["M"], ap["K"], ap["N"], ap["g"], sp2, ap["seed"])], 128),
                "decode_M16": _cpu_layer_config(
                    [("up", 16, du["K"], du["N"], du["g"], sp4, du["seed"]),
                     ("down", 16, dd["K"], dd["N"], dd["g"], sp4, dd["seed"])], 16, n_cols=2048,
                    unit="GBs"),
                "kv_quantize": _cpu_kv_config(1 << 16),
            }
        out["cpu_baseline"] = cpu_baseline(lay, 256, 10.0, per_config)
    elif not args.no_cpu_baseline and wl == "prefill_layer":
        out["cpu_baseline"] = cpu_prefill_layer(inputs.WORKLOADS["prefill_layer"], 64, 10.0)
    elif not args.no_cpu_baseline and wl == "attn_proj_prefill":
        out["cpu_baseline"] = cpu_baseline([("proj", M, K, N, g, spec, cfg["seed"], None)], 512, 10.0)
    print(json.dumps(out), flush=True)


# ------------------------------------------------------------------ timing
def run_phases(torch, stream, phases, steps, warmup, check, launches_per_step):
    """Warm-up, then the K steps phase by phase (one event between phases)."""
    for i in range(warmup):
        for name, fn in phases:
            check(fn(i), name)
    torch.cuda.synchronize()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(len(phases) + 1)]
    # The GPU first spins (about 50 us per launch to come) while the host
    # enqueues the whole timed region, so that no kernel waits for its launch
    # call (a launch from Python takes longer than the shortest kernels here).
    if hasattr(torch.cuda, "_sleep"):
        torch.cuda._sleep(100_000 * launches_per_step * steps)
    evs[0].record(stream)
    for p, (name, fn) in enumerate(phases):
        for i in range(steps):
            check(fn(warmup + i), name)
        evs[p + 1].record(stream)
    torch.cuda.synchronize()
    ms = evs[0].elapsed_time(evs[-1]) / steps
    comp = {}
    for p, (name, fn) in enumerate(phases):
        us = 1000.0 * evs[p].elapsed_time(evs[p + 1]) / steps
        if name in comp:  # a kernel launched twice per step (K and V): per launch
            c = comp[name]
            c["us"] = round((c["us"] * c["launches"] + us) / (c["launches"] + 1), 3)
            c["launches"] += 1
        else:
            comp[name] = {"us": round(us, 3), "launches": 1}
    return ms, comp


def launch_times(torch, stream, fn, n, check, name, warm):
    """n launches with an event after each; per-launch microseconds, sorted."""
    torch.cuda.synchronize()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
    if hasattr(torch.cuda, "_sleep"):
        torch.cuda._sleep(100_000 * n)
    evs[0].record(stream)
    for i in range(n):
        check(fn(0 if warm else i), name)
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    return sorted(1000.0 * evs[i].elapsed_time(evs[i + 1]) for i in range(n))


def _pct(t, q):
    return round(t[min(len(t) - 1, int(round(q * (len(t) - 1))))], 3)


def add_dist(torch, stream, phases, comp, n, check):
    """Per-launch median, p10 and p90 over n cold launches and the median of
    n warm launches of every phase (a phase launched twice per step, K and V,
    is measured on its first launch function)."""
    seen = set()
    for name, fn in phases:
        if name in seen:
            continue
        seen.add(name)
        t = launch_times(torch, stream, fn, n, check, name, warm=False)
        tw = launch_times(torch, stream, fn, n, check, name, warm=True)
        comp[name].update({"median_us": _pct(t, 0.5), "p10_us": _pct(t, 0.1),
                           "p90_us": _pct(t, 0.9), "n_dist": n, "warm_median_us": _pct(tw, 0.5)})


def event_gap(torch, stream, n=64):
    """Median time between two events recorded back to back on the stream."""
    torch.cuda.synchronize()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
    for e in evs:
        e.record(stream)
    torch.cuda.synchronize()
    t = sorted(1000.0 * evs[i].elapsed_time(evs[i + 1]) for i in range(n))
    return t[n // 2]


def ann_bytes(c, b):
    """Algorithmic bytes per launch and the rates of the mean and median."""
    c["alg_bytes"] = b
    c["GBs"] = round(b / (c["us"] * 1e-6) / 1e9, 1)
    c["frac_hbm"] = round(c["GBs"] / PEAK_HBM_GBS, 4)
    if "median_us" in c:
        c["GBs_median"] = round(b / (c["median_us"] * 1e-6) / 1e9, 1)


def ann_rq(c, M, K, g, n=1):
    ann_bytes(c, rq_bytes(M, K, g) * n)


def ann_mm(c, M, N, K):
    ops = 2.0 * M * N * K
    c["alg_ops"] = ops
    c["TOPS"] = round(ops / (c["us"] * 1e-6) / 1e12, 1)
    c["frac_int8_peak"] = round(c["TOPS"] / PEAK_INT8_TOPS, 4)
    if "median_us" in c:
        c["TOPS_median"] = round(ops / (c["median_us"] * 1e-6) / 1e12, 1)


def mfma_roof(comp, dom, traffic):
    c = comp[dom]
    return {"bound": "mfma", "achieved": c["TOPS"], "peak": PEAK_INT8_TOPS, "unit": "TOP/s",
            "frac": c["frac_int8_peak"], "traffic": traffic, "kernel": dom,
            "alg_ops_per_launch": c["alg_ops"], "avg_launch_us": c["us"]}


def hbm_roof(comp, dom, traffic):
    c = comp[dom]
    return {"bound": "hbm", "achieved": c["GBs"], "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": c["frac_hbm"], "traffic": traffic, "kernel": dom,
            "alg_bytes_per_launch": c["alg_bytes"], "avg_launch_us": c["us"]}


# ------------------------------------------------- the other workloads' kernels
def other_configs(torch, offq, _lib, inputs, stream, sp, check, args, n_dist):
    """Every other workload's kernels, timed like the main step (phase mean
    over max(20, K) launches, then the per-launch distributions): the
    attention-projection prefill layer, the decode GEMVs at M = 1, 4, 16 and
    the KV4 cache quantize with the 8192-row projection."""
    steps = max(20, args.steps)
    W = inputs.WORKLOADS
    res = {}

    def layer(name_rq, name_mm, cfg, M, N, seed_off=0):
        spec = dict(n_outliers=cfg["n_outliers"], lo=cfg["lo"], hi=cfg["hi"])
        K, g = cfg["K"], cfg["g"]
        per = M * K * 2 + N * K // 2 + M * K // 2 + M * N * 2
        sets = Sets(lambda i: make_layer_set(offq, inputs, torch, M, K, N, g,
                                             cfg["seed"] + seed_off + 100 * i, spec), per)
        return sets, [(name_rq, lambda i, s_=sets: run_rq(_lib, s_[i], sp)),
                      (name_mm, lambda i, s_=sets: run_gemm(_lib, s_[i], sp))]

    def measure(phases):
        _, comp = run_phases(torch, stream, phases, steps, 3, check, len(phases))
        add_dist(torch, stream, phases, comp, n_dist, check)
        return comp

    ap = W["attn_proj_prefill"]
    sets, ph = layer("rotate_quantize", "w4a4_gemm", ap, ap["M"], ap["N"])
    comp = measure(ph)
    ann_rq(comp["rotate_quantize"], ap["M"], ap["K"], ap["g"])
    ann_mm(comp["w4a4_gemm"], ap["M"], ap["N"], ap["K"])
    for k, t in (("rotate_quantize", "rotate_quantize"), ("w4a4_gemm", "w4a4_gemm")):
        tb = traffic_for(f"{t}:attn_proj_prefill")
        if tb is not None:
            comp[k]["traffic_bytes"] = tb
    res["attn_proj_prefill"] = {"shape": [ap["M"], ap["K"], ap["N"], ap["g"]], "kernels": comp}
    del sets, ph
    torch.cuda.empty_cache()

    du, dd = W["decode_up"], W["decode_down"]
    for Md in (16, 4, 1):
        su, pu = layer("rotate_quantize_up", "w4a4_gemv_up", du, Md, du["N"], Md)
        sd, pd = layer("rotate_quantize_down", "w4a4_gemv_down", dd, Md, dd["N"], Md)
        comp = measure(pu + pd)
        ann_rq(comp["rotate_quantize_up"], Md, du["K"], du["g"])
        ann_rq(comp["rotate_quantize_down"], Md, dd["K"], dd["g"])
        ann_bytes(comp["w4a4_gemv_up"], gemv_bytes(Md, du["N"], du["K"], du["g"]))
        ann_bytes(comp["w4a4_gemv_down"], gemv_bytes(Md, dd["N"], dd["K"], dd["g"]))
        if Md == 16:
            for k, t in (("w4a4_gemv_up", "w4a4_gemv"), ("w4a4_gemv_down", "w4a4_gemv_down")):
                tb = traffic_for(f"{t}:decode")
                if tb is not None:
                    comp[k]["traffic_bytes"] = tb
        res[f"decode_M{Md}"] = {"up": [Md, du["K"], du["N"], du["g"]],
                                "down": [Md, dd["K"], dd["N"], dd["g"]], "kernels": comp}
        del su, sd, pu, pd
        torch.cuda.empty_cache()

    kc = W["kv_cache"]
    B, H, S, Dh = kc["B"], kc["H"], kc["S"], kc["Dh"]
    R = B * H * S
    kv = [inputs.kv_cache_device(B, H, S, Dh, seed=kc["seed"] + j, device="cuda",
                                 n_outliers=kc["n_outliers"], lo=kc["lo"], hi=kc["hi"])
          for j in range(2)]
    kvo = [dict(codes=torch.empty((R, Dh // 2), dtype=torch.uint8, device="cuda"),
                scale=torch.empty((R,), dtype=torch.float16, device="cuda"),
                zero=torch.empty((R,), dtype=torch.int16, device="cuda")) for _ in range(2)]

    def kvq(i):  # K and V tensors alternate (2 GiB each, far beyond the cache)
        j = i % 2
        return _lib.offq_kv_quantize_raw(kv[j].data_ptr(), R, Dh, Dh, 1, kvo[j]["codes"].data_ptr(),
                                         kvo[j]["scale"].data_ptr(), kvo[j]["zero"].data_ptr(),
                                         None, sp)
    pc = W["kv_chain_proj"]
    sets, ph = layer("rotate_quantize", "w4a4_gemm", pc, pc["M"], pc["N"])
    comp = measure([("kv_quantize", kvq)] + ph)
    ann_rq(comp["kv_quantize"], R, Dh, Dh)
    ann_rq(comp["rotate_quantize"], pc["M"], pc["K"], pc["g"])
    ann_mm(comp["w4a4_gemm"], pc["M"], pc["N"], pc["K"])
    for k, t in (("kv_quantize", "kv_quantize"), ("rotate_quantize", "rotate_quantize"),
                 ("w4a4_gemm", "w4a4_gemm")):
        tb = traffic_for(f"{t}:kv_chain")
        if tb is not None:
            comp[k]["traffic_bytes"] = tb
    res["kv_chain"] = {"kv_shape": [B, H, S, Dh], "proj": [pc["M"], pc["K"], pc["N"], pc["g"]],
                       "kernels": comp,
                       "note": "kv_quantize: one [8, 32, 32768, 128] tensor per launch (K and V "
                               "alternate); the step quantizes both"}
    del sets, ph, kv, kvo
    torch.cuda.empty_cache()
    return res


if __name__ == "__main__":
    main()
