"""ctypes binding of liboffq.so (argument marshalling only).

Every entry point of ``include/offq.h`` is exposed under the same name.  The
``*_raw`` functions take plain integers (device addresses, sizes, a stream
handle) exactly like the C functions; the tensor-level wrappers take torch
device tensors, check dtype/shape/contiguity, allocate outputs with torch and
pass ``data_ptr()`` and the current HIP stream.  All arithmetic happens in the
HIP kernels of the library; if the library is missing, importing this module
raises -- there is no fallback path.
"""

import ctypes
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "liboffq.so")

OFFQ_OK = 0
OFFQ_ERR_INVALID = 1
OFFQ_ERR_UNSUPPORTED = 2
OFFQ_ERR_HIP = 3

EXPORTED = (
    "offq_abi_version",
    "offq_status_string",
    "offq_last_error",
    "offq_rotate_quantize",
    "offq_w4a4_gemm",
    "offq_kv_quantize",
    "offq_pack_weights",
    "offq_weight_codes_bytes",
    "offq_kv_attention_decode",
    "offq_kv_attention_workspace_bytes",
    "offq_kv_attention_decode_gqa",
    "offq_kv_attention_decode_quantize",
    "offq_kv_attention_decode_noalloc",
    "offq_add_rmsnorm",
    "offq_swiglu",
    "offq_rope_kv_append",
    "offq_rope_kv_prefill",
    "offq_kv_attention_prefill",
    "offq_add_rmsnorm_quantize",
    "offq_swiglu_rotate_quantize",
    "offq_top1_workspace_bytes",
    "offq_top1_select",
    "offq_channel_absmax",
    "offq_gram",
    "offq_eigh_workspace_bytes",
    "offq_eigh",
    "offq_group_permutation",
    "offq_build_rotation",
    "offq_fuse_weights",
    "offq_permute_rows",
)


class OffqError(RuntimeError):
    def __init__(self, status, fn, msg):
        super().__init__(f"{fn}: {status_name(status)}: {msg}")
        self.status = status


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it with `python paper_2606_07116_amd/build.py` "
            "(there is no non-HIP fallback)")
    # torch ships its own HIP runtime (SONAME libamdhip64.so.7).  Import it
    # first so that the library binds to that same runtime: a second runtime in
    # the process would not understand torch's stream handles or allocations.
    import torch  # noqa: F401

    lib = ctypes.CDLL(LIB_PATH)
    i64, i32, vp = ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p
    lib.offq_abi_version.restype = ctypes.c_int
    lib.offq_abi_version.argtypes = []
    lib.offq_status_string.restype = ctypes.c_char_p
    lib.offq_status_string.argtypes = [ctypes.c_int]
    lib.offq_last_error.restype = ctypes.c_char_p
    lib.offq_last_error.argtypes = []
    lib.offq_rotate_quantize.restype = ctypes.c_int
    lib.offq_rotate_quantize.argtypes = [vp, i64, i64, i64, i32, i32, vp, vp, vp, vp, vp]
    lib.offq_w4a4_gemm.restype = ctypes.c_int
    lib.offq_w4a4_gemm.argtypes = [vp, vp, vp, vp, vp, vp, i64, i64, i64, i32, vp, i64, vp, vp]
    lib.offq_kv_quantize.restype = ctypes.c_int
    lib.offq_kv_quantize.argtypes = [vp, i64, i32, i64, i32, vp, vp, vp, vp, vp]
    lib.offq_pack_weights.restype = ctypes.c_int
    lib.offq_pack_weights.argtypes = [vp, i64, i64, i32, vp, vp, vp, vp]
    lib.offq_weight_codes_bytes.restype = i64
    lib.offq_weight_codes_bytes.argtypes = [i64, i64]
    lib.offq_kv_attention_decode.restype = ctypes.c_int
    lib.offq_kv_attention_decode.argtypes = [vp, vp, vp, vp, vp, vp, vp, i64, i64, i64, i64, i32,
                                             ctypes.c_float, i32, vp, vp, i64, vp]
    lib.offq_kv_attention_workspace_bytes.restype = i64
    lib.offq_kv_attention_workspace_bytes.argtypes = [i64, i64, i64]
    lib.offq_kv_attention_decode_gqa.restype = ctypes.c_int
    lib.offq_kv_attention_decode_gqa.argtypes = [vp, vp, vp, vp, vp, vp, vp, i64, i64, i64, i64, i64,
                                                 i32, ctypes.c_float, i32, vp, vp, i64, vp]
    lib.offq_kv_attention_decode_quantize.restype = ctypes.c_int
    lib.offq_kv_attention_decode_quantize.argtypes = [vp, vp, vp, vp, vp, vp, vp, i64, i64, i64, i64,
                                                      i64, i32, ctypes.c_float, i32, vp, vp, vp, vp,
                                                      vp, i64, vp]
    lib.offq_add_rmsnorm.restype = ctypes.c_int
    lib.offq_add_rmsnorm.argtypes = [vp, i64, vp, i64, i64, i64, ctypes.c_float, vp, i64, vp, i64,
                                     vp]
    lib.offq_swiglu.restype = ctypes.c_int
    lib.offq_swiglu.argtypes = [vp, i64, i64, i64, vp, i64, vp]
    lib.offq_rope_kv_append.restype = ctypes.c_int
    lib.offq_rope_kv_append.argtypes = [vp, i64, i64, i64, i64, i32, vp, ctypes.c_double, i32, i32,
                                        vp, vp, vp, vp, vp, vp, vp, i64, vp, vp, vp]
    lib.offq_rope_kv_prefill.restype = ctypes.c_int
    lib.offq_rope_kv_prefill.argtypes = [vp, i64, i64, i64, i64, i64, i32, vp, ctypes.c_double,
                                         i32, i32, vp, vp, vp, vp, vp, vp, vp, i64, vp, vp, vp]
    lib.offq_kv_attention_prefill.restype = ctypes.c_int
    lib.offq_kv_attention_prefill.argtypes = [vp, i64, i64, i64, i64, i32, i64, vp, vp, vp, vp,
                                              vp, vp, i64, ctypes.c_float, i32, vp, vp]
    f64 = ctypes.c_double
    sigs = {
        "offq_add_rmsnorm_quantize": (ctypes.c_int, [vp, i64, vp, i64, i64, i64, ctypes.c_float,
                                                     i32, vp, i64, vp, vp, vp, vp, i64, vp]),
        "offq_swiglu_rotate_quantize": (ctypes.c_int, [vp, i64, i64, i64, vp, vp, vp, vp, vp]),
        "offq_kv_attention_decode_noalloc": (ctypes.c_int, [vp, vp, vp, vp, vp, vp, vp, i64, i64, i64,
                                                            i64, i64, i32, ctypes.c_float, i32, vp,
                                                            vp]),
        "offq_top1_workspace_bytes": (i64, [i64, i64]),
        "offq_top1_select": (ctypes.c_int, [vp, i64, i64, i64, i64, i64, vp, vp, i64, vp, i64, vp]),
        "offq_channel_absmax": (ctypes.c_int, [vp, i64, i64, i64, vp, vp]),
        "offq_gram": (ctypes.c_int, [vp, i64, i64, i64, vp, i64, vp]),
        "offq_eigh_workspace_bytes": (i64, [i64]),
        "offq_eigh": (ctypes.c_int, [vp, i64, i64, vp, vp, i64, vp, i64, i32, f64,
                                     ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(f64), vp]),
        "offq_group_permutation": (ctypes.c_int, [vp, i64, i32, vp, vp, i64, vp]),
        "offq_build_rotation": (ctypes.c_int, [vp, i64, i64, vp, i32, i32, vp, i64, vp]),
        "offq_fuse_weights": (ctypes.c_int, [vp, i64, i64, i64, vp, i64, vp, i64, vp]),
        "offq_permute_rows": (ctypes.c_int, [vp, i64, i64, i64, vp, vp, i64, vp]),
    }
    for name, (res, args) in sigs.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


lib = _load()
ABI_VERSION = lib.offq_abi_version()


def status_name(status):
    return lib.offq_status_string(int(status)).decode()


def last_error():
    return lib.offq_last_error().decode()


def _check(status, fn):
    if status != OFFQ_OK:
        raise OffqError(status, fn, last_error())


# ---------------------------------------------------------------- raw C calls
def offq_rotate_quantize_raw(x, M, K, ldx, g, apply_hadamard, codes, scale, zero, y_debug, stream):
    return lib.offq_rotate_quantize(x, M, K, ldx, g, apply_hadamard, codes, scale, zero, y_debug, stream)


def offq_w4a4_gemm_raw(a_codes, a_scale, a_zero, w_codes, w_scale, w_colsum, M, N, K, g, y, ldy,
                       acc_debug, stream):
    return lib.offq_w4a4_gemm(a_codes, a_scale, a_zero, w_codes, w_scale, w_colsum, M, N, K, g, y,
                              ldy, acc_debug, stream)


def offq_kv_quantize_raw(kv, rows, head_dim, row_stride, apply_hadamard, codes, scale, zero,
                         y_debug, stream):
    return lib.offq_kv_quantize(kv, rows, head_dim, row_stride, apply_hadamard, codes, scale, zero,
                                y_debug, stream)


def offq_pack_weights_raw(w, N, K, g, w_codes, w_scale, w_colsum, stream):
    return lib.offq_pack_weights(w, N, K, g, w_codes, w_scale, w_colsum, stream)


def offq_kv_attention_decode_raw(q, k_codes, k_scale, k_zero, v_codes, v_scale, v_zero, B, H, s_cap,
                                 seq_len, head_dim, sm_scale, v_hadamard, out, workspace,
                                 workspace_bytes, stream):
    return lib.offq_kv_attention_decode(q, k_codes, k_scale, k_zero, v_codes, v_scale, v_zero, B, H,
                                        s_cap, seq_len, head_dim, sm_scale, v_hadamard, out,
                                        workspace, workspace_bytes, stream)


def offq_kv_attention_workspace_bytes(B, H, seq_len):
    return lib.offq_kv_attention_workspace_bytes(B, H, seq_len)


def offq_weight_codes_bytes(N, K):
    return lib.offq_weight_codes_bytes(N, K)


def weight_codes_shape(N, K):
    """Shape of the w_codes tensor offq_pack_weights returns: [bands of 16
    rows, blocks of 128 k, 16 rows, 64 bytes] (the blocked operand layout)."""
    return ((N + 15) // 16, (K + 127) // 128, 16, 64)


def blocked_weight_codes(rows):
    """Row-major packed weight codes [N, K/2] (uint8, numpy or torch) in the
    blocked operand layout, zero padded: a layout conversion for weights
    packed elsewhere."""
    N, Kh = rows.shape
    nb, kb, _, _ = weight_codes_shape(N, 2 * Kh)
    if hasattr(rows, "new_zeros"):
        pad = rows.new_zeros((16 * nb, 64 * kb))
    else:
        import numpy as np
        pad = np.zeros((16 * nb, 64 * kb), dtype=rows.dtype)
    pad[:N, :Kh] = rows
    out = pad.reshape(nb, 16, kb, 64).swapaxes(1, 2)
    return out.contiguous() if hasattr(out, "contiguous") else out.copy()


def row_major_weight_codes(blocked, N, K):
    """The inverse of blocked_weight_codes: [N, K/2] row-major codes."""
    nb, kb, _, _ = weight_codes_shape(N, K)
    rows = blocked.reshape(nb, kb, 16, 64).swapaxes(1, 2).reshape(16 * nb, 64 * kb)
    return rows[:N, :K // 2]


def offq_kv_attention_decode_gqa_raw(q, k_codes, k_scale, k_zero, v_codes, v_scale, v_zero, B, Hq,
                                     Hkv, s_cap, seq_len, head_dim, sm_scale, v_hadamard, out,
                                     workspace, workspace_bytes, stream):
    return lib.offq_kv_attention_decode_gqa(q, k_codes, k_scale, k_zero, v_codes, v_scale, v_zero, B,
                                            Hq, Hkv, s_cap, seq_len, head_dim, sm_scale, v_hadamard,
                                            out, workspace, workspace_bytes, stream)


def offq_kv_attention_decode_quantize_raw(q, k_codes, k_scale, k_zero, v_codes, v_scale, v_zero, B,
                                          Hq, Hkv, s_cap, seq_len, head_dim, sm_scale, v_hadamard,
                                          out, out_codes, out_scale, out_zero, workspace,
                                          workspace_bytes, stream):
    return lib.offq_kv_attention_decode_quantize(q, k_codes, k_scale, k_zero, v_codes, v_scale,
                                                 v_zero, B, Hq, Hkv, s_cap, seq_len, head_dim,
                                                 sm_scale, v_hadamard, out, out_codes, out_scale,
                                                 out_zero, workspace, workspace_bytes, stream)


def offq_kv_attention_decode_noalloc_raw(q, k_codes, k_scale, k_zero, v_codes, v_scale, v_zero, B,
                                         Hq, Hkv, s_cap, seq_len, head_dim, sm_scale, v_hadamard,
                                         out, stream):
    return lib.offq_kv_attention_decode_noalloc(q, k_codes, k_scale, k_zero, v_codes, v_scale,
                                                v_zero, B, Hq, Hkv, s_cap, seq_len, head_dim,
                                                sm_scale, v_hadamard, out, stream)


def offq_add_rmsnorm_raw(x, ldx, res, ldr, M, D, eps, h_out, ldh, y_out, ldy, stream):
    return lib.offq_add_rmsnorm(x, ldx, res, ldr, M, D, eps, h_out, ldh, y_out, ldy, stream)


def offq_swiglu_raw(gu, ldg, M, F, out, ldo, stream):
    return lib.offq_swiglu(gu, ldg, M, F, out, ldo, stream)


def offq_add_rmsnorm_quantize_raw(x, ldx, res, ldr, M, D, eps, g, h_out, ldh, codes, scale, zero,
                                  y_debug, ldy, stream):
    return lib.offq_add_rmsnorm_quantize(x, ldx, res, ldr, M, D, eps, g, h_out, ldh, codes, scale,
                                         zero, y_debug, ldy, stream)


def offq_swiglu_rotate_quantize_raw(gu, ldg, M, F, codes, scale, zero, y_debug, stream):
    return lib.offq_swiglu_rotate_quantize(gu, ldg, M, F, codes, scale, zero, y_debug, stream)


def offq_rope_kv_append_raw(qkv, ldq, M, Hq, Hkv, head_dim, positions, rope_base, k_hadamard,
                            v_hadamard, q_out, k_codes, k_scale, k_zero, v_codes, v_scale, v_zero,
                            s_cap, k_y_debug, v_y_debug, stream):
    return lib.offq_rope_kv_append(qkv, ldq, M, Hq, Hkv, head_dim, positions, rope_base, k_hadamard,
                                   v_hadamard, q_out, k_codes, k_scale, k_zero, v_codes, v_scale,
                                   v_zero, s_cap, k_y_debug, v_y_debug, stream)


def offq_rope_kv_prefill_raw(qkv, ldq, B, T, Hq, Hkv, head_dim, positions, rope_base, k_hadamard,
                             v_hadamard, q_out, k_codes, k_scale, k_zero, v_codes, v_scale,
                             v_zero, s_cap, k_y_debug, v_y_debug, stream):
    return lib.offq_rope_kv_prefill(qkv, ldq, B, T, Hq, Hkv, head_dim, positions, rope_base,
                                    k_hadamard, v_hadamard, q_out, k_codes, k_scale, k_zero,
                                    v_codes, v_scale, v_zero, s_cap, k_y_debug, v_y_debug, stream)


def offq_kv_attention_prefill_raw(q, B, T, Hq, Hkv, head_dim, past, k_codes, k_scale, k_zero,
                                  v_codes, v_scale, v_zero, s_cap, sm_scale, v_hadamard, out,
                                  stream):
    return lib.offq_kv_attention_prefill(q, B, T, Hq, Hkv, head_dim, past, k_codes, k_scale,
                                         k_zero, v_codes, v_scale, v_zero, s_cap, sm_scale,
                                         v_hadamard, out, stream)


# ------------------------------------------------------------ tensor wrappers
def _torch():
    import torch
    return torch


def _stream():
    torch = _torch()
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _need(t, dtype, name, ndim=None):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dims")


def offq_rotate_quantize(x, g, apply_hadamard=True, debug=False):
    """x: bf16 [M, K] (last dim contiguous).  Returns (codes u8 [M, K/2],
    scale fp16 [M, K/g], zero int16 [M, K/g], y fp32 [M, K] or None)."""
    torch = _torch()
    _need(x, torch.bfloat16, "x", 2)
    if x.stride(1) != 1:
        raise ValueError("x must have a contiguous last dimension")
    M, K = x.shape
    dev = x.device
    codes = torch.empty((M, K // 2), dtype=torch.uint8, device=dev)
    scale = torch.empty((M, K // g), dtype=torch.float16, device=dev)
    zero = torch.empty((M, K // g), dtype=torch.int16, device=dev)
    y = torch.empty((M, K), dtype=torch.float32, device=dev) if debug else None
    _check(lib.offq_rotate_quantize(_ptr(x), M, K, x.stride(0), int(g), int(bool(apply_hadamard)),
                                    _ptr(codes), _ptr(scale), _ptr(zero), _ptr(y), _stream()),
           "offq_rotate_quantize")
    return codes, scale, zero, y


def offq_w4a4_gemm(a_codes, a_scale, a_zero, w_codes, w_scale, w_colsum, g, debug=False, out=None):
    """Returns (y bf16 [M, N], acc int32 [K/g, M, N] or None)."""
    torch = _torch()
    _need(a_codes, torch.uint8, "a_codes", 2)
    _need(a_scale, torch.float16, "a_scale", 2)
    _need(a_zero, torch.int16, "a_zero", 2)
    _need(w_codes, torch.uint8, "w_codes")
    _need(w_scale, torch.float16, "w_scale", 1)
    _need(w_colsum, torch.int32, "w_colsum", 2)
    for t, n in ((a_codes, "a_codes"), (a_scale, "a_scale"), (a_zero, "a_zero"), (w_codes, "w_codes"),
                 (w_scale, "w_scale"), (w_colsum, "w_colsum")):
        if not t.is_contiguous():
            raise ValueError(f"{n} must be contiguous")
    M, Kh = a_codes.shape
    N = w_scale.shape[0]
    K = 2 * Kh
    if w_codes.numel() != lib.offq_weight_codes_bytes(N, K) or a_scale.shape != (M, K // g) \
            or a_zero.shape != (M, K // g) or w_colsum.shape != (K // g, N):
        raise ValueError("operand shapes do not match")
    dev = a_codes.device
    y = out if out is not None else torch.empty((M, N), dtype=torch.bfloat16, device=dev)
    _need(y, torch.bfloat16, "out", 2)
    # the kernels write rows 0..M-1, columns 0..N-1 at row stride y.stride(0)
    if tuple(y.shape) != (M, N) or y.stride(1) != 1 or y.stride(0) < N:
        raise ValueError(f"out must be a [{M}, {N}] tensor with a contiguous last dimension")
    acc = torch.empty((K // g, M, N), dtype=torch.int32, device=dev) if debug else None
    _check(lib.offq_w4a4_gemm(_ptr(a_codes), _ptr(a_scale), _ptr(a_zero), _ptr(w_codes), _ptr(w_scale),
                              _ptr(w_colsum), M, N, K, int(g), _ptr(y), y.stride(0), _ptr(acc),
                              _stream()), "offq_w4a4_gemm")
    return y, acc


def offq_kv_quantize(kv, apply_hadamard=True, debug=False):
    """kv: bf16 [..., head_dim] (rows contiguous in the last dim; leading dims
    flattened).  Returns (codes u8 [rows, Dh/2], scale fp16 [rows],
    zero int16 [rows], y fp32 [rows, Dh] or None)."""
    torch = _torch()
    _need(kv, torch.bfloat16, "kv")
    Dh = kv.shape[-1]
    rows2d = kv.reshape(-1, Dh)
    if rows2d.stride(1) != 1:
        raise ValueError("kv must have a contiguous last dimension")
    R = rows2d.shape[0]
    dev = kv.device
    codes = torch.empty((R, Dh // 2), dtype=torch.uint8, device=dev)
    scale = torch.empty((R,), dtype=torch.float16, device=dev)
    zero = torch.empty((R,), dtype=torch.int16, device=dev)
    y = torch.empty((R, Dh), dtype=torch.float32, device=dev) if debug else None
    _check(lib.offq_kv_quantize(_ptr(rows2d), R, Dh, rows2d.stride(0), int(bool(apply_hadamard)),
                                _ptr(codes), _ptr(scale), _ptr(zero), _ptr(y), _stream()),
           "offq_kv_quantize")
    return codes, scale, zero, y


def offq_pack_weights(w, g):
    """w: fp32 [N, K] contiguous.  Returns (w_codes u8 in the blocked operand
    layout, shape weight_codes_shape(N, K), w_scale fp16 [N], w_colsum int32
    [K/g, N])."""
    torch = _torch()
    _need(w, torch.float32, "w", 2)
    if not w.is_contiguous():
        raise ValueError("w must be contiguous")
    N, K = w.shape
    dev = w.device
    wc = torch.empty(weight_codes_shape(N, K), dtype=torch.uint8, device=dev)
    ws = torch.empty((N,), dtype=torch.float16, device=dev)
    cs = torch.empty((K // g, N), dtype=torch.int32, device=dev)
    _check(lib.offq_pack_weights(_ptr(w), N, K, int(g), _ptr(wc), _ptr(ws), _ptr(cs), _stream()),
           "offq_pack_weights")
    return wc, ws, cs


def _attention_operands(q, k_codes, k_scale, k_zero, v_codes, v_scale, v_zero, sm_scale):
    torch = _torch()
    _need(q, torch.bfloat16, "q", 3)
    for t, dt, n in ((k_codes, torch.uint8, "k_codes"), (v_codes, torch.uint8, "v_codes")):
        _need(t, dt, n, 4)
    for t, dt, n in ((k_scale, torch.float16, "k_scale"), (v_scale, torch.float16, "v_scale"),
                     (k_zero, torch.int16, "k_zero"), (v_zero, torch.int16, "v_zero")):
        _need(t, dt, n, 3)
    for t, n in ((q, "q"), (k_codes, "k_codes"), (k_scale, "k_scale"), (k_zero, "k_zero"),
                 (v_codes, "v_codes"), (v_scale, "v_scale"), (v_zero, "v_zero")):
        if not t.is_contiguous():
            raise ValueError(f"{n} must be contiguous")
    B, H, Dh = q.shape
    Hkv, s_cap = k_codes.shape[1], k_codes.shape[2]
    if k_codes.shape != (B, Hkv, s_cap, Dh // 2) or v_codes.shape != k_codes.shape \
            or k_scale.shape != (B, Hkv, s_cap) or k_zero.shape != (B, Hkv, s_cap) \
            or v_scale.shape != (B, Hkv, s_cap) or v_zero.shape != (B, Hkv, s_cap):
        raise ValueError("operand shapes do not match")
    if sm_scale is None:
        sm_scale = 1.0 / float(Dh) ** 0.5
    return B, H, Dh, Hkv, s_cap, sm_scale


def offq_kv_attention_decode(q, k_codes, k_scale, k_zero, v_codes, v_scale, v_zero, seq_len,
                             sm_scale=None, v_hadamard=False, out=None, workspace=None):
    """One decode step of attention over the 4-bit cache.

    q: bf16 [B, H, 128]; k_codes / v_codes: u8 [B, Hkv, s_cap, 64];
    k_scale / v_scale: fp16 [B, Hkv, s_cap]; k_zero / v_zero: int16
    [B, Hkv, s_cap] (all contiguous; H a multiple of Hkv: grouped-query
    attention).  Positions 0 .. seq_len-1 are attended.  sm_scale defaults to
    1/sqrt(128).  Returns out bf16 [B, H, 128]."""
    torch = _torch()
    B, H, Dh, Hkv, s_cap, sm_scale = _attention_operands(q, k_codes, k_scale, k_zero, v_codes,
                                                         v_scale, v_zero, sm_scale)
    dev = q.device
    if out is None:
        out = torch.empty((B, H, Dh), dtype=torch.bfloat16, device=dev)
    _need(out, torch.bfloat16, "out", 3)
    if not out.is_contiguous() or out.shape != (B, H, Dh):
        raise ValueError("out must be a contiguous [B, H, head_dim] tensor")
    need = lib.offq_kv_attention_workspace_bytes(B, H, int(seq_len))
    if workspace is None:
        workspace = torch.empty((max(need, 4) + 3) // 4, dtype=torch.float32, device=dev)
    _need(workspace, torch.float32, "workspace", 1)
    _check(lib.offq_kv_attention_decode_gqa(_ptr(q), _ptr(k_codes), _ptr(k_scale), _ptr(k_zero),
                                            _ptr(v_codes), _ptr(v_scale), _ptr(v_zero), B, H, Hkv,
                                            s_cap, int(seq_len), Dh, float(sm_scale),
                                            int(bool(v_hadamard)), _ptr(out), _ptr(workspace),
                                            workspace.numel() * 4, _stream()),
           "offq_kv_attention_decode")
    return out


def offq_kv_attention_decode_noalloc(q, k_codes, k_scale, k_zero, v_codes, v_scale, v_zero,
                                     seq_len, out, sm_scale=None, v_hadamard=False):
    """offq_kv_attention_decode without a workspace (the library's static
    scratch holds the chunk records; nothing is allocated, so the caller
    passes out, bf16 [B, H, 128] contiguous).  Returns out."""
    torch = _torch()
    B, H, Dh, Hkv, s_cap, sm_scale = _attention_operands(q, k_codes, k_scale, k_zero, v_codes,
                                                         v_scale, v_zero, sm_scale)
    _need(out, torch.bfloat16, "out", 3)
    if not out.is_contiguous() or out.shape != (B, H, Dh):
        raise ValueError("out must be a contiguous [B, H, head_dim] tensor")
    _check(lib.offq_kv_attention_decode_noalloc(
        _ptr(q), _ptr(k_codes), _ptr(k_scale), _ptr(k_zero), _ptr(v_codes), _ptr(v_scale),
        _ptr(v_zero), B, H, Hkv, s_cap, int(seq_len), Dh, float(sm_scale), int(bool(v_hadamard)),
        _ptr(out), _stream()), "offq_kv_attention_decode_noalloc")
    return out


def offq_kv_attention_decode_quantize(q, k_codes, k_scale, k_zero, v_codes, v_scale, v_zero,
                                      seq_len, sm_scale=None, v_hadamard=False, out=None,
                                      workspace=None):
    """offq_kv_attention_decode with each head's output row also quantized
    (one group of 128, no rotation): returns (codes u8 [B, H * 64], scale fp16
    [B, H], zero int16 [B, H], out), out being the bf16 [B, H, 128] output
    when given (it is then also written), else None."""
    torch = _torch()
    B, H, Dh, Hkv, s_cap, sm_scale = _attention_operands(q, k_codes, k_scale, k_zero, v_codes,
                                                         v_scale, v_zero, sm_scale)
    dev = q.device
    if out is not None:
        _need(out, torch.bfloat16, "out", 3)
        if not out.is_contiguous() or out.shape != (B, H, Dh):
            raise ValueError("out must be a contiguous [B, H, head_dim] tensor")
    codes = torch.empty((B, H * Dh // 2), dtype=torch.uint8, device=dev)
    scale = torch.empty((B, H), dtype=torch.float16, device=dev)
    zero = torch.empty((B, H), dtype=torch.int16, device=dev)
    need = lib.offq_kv_attention_workspace_bytes(B, H, int(seq_len))
    if workspace is None:
        workspace = torch.empty((max(need, 4) + 3) // 4, dtype=torch.float32, device=dev)
    _need(workspace, torch.float32, "workspace", 1)
    _check(lib.offq_kv_attention_decode_quantize(
        _ptr(q), _ptr(k_codes), _ptr(k_scale), _ptr(k_zero), _ptr(v_codes), _ptr(v_scale),
        _ptr(v_zero), B, H, Hkv, s_cap, int(seq_len), Dh, float(sm_scale), int(bool(v_hadamard)),
        _ptr(out) if out is not None else None, _ptr(codes), _ptr(scale), _ptr(zero),
        _ptr(workspace), workspace.numel() * 4, _stream()), "offq_kv_attention_decode_quantize")
    return codes, scale, zero, out


def _rows(t, name):
    """2-D view facts of a bf16 tensor with a contiguous last dimension."""
    if t.dim() != 2 or t.stride(1) != 1:
        raise ValueError(f"{name} must be 2-D with a contiguous last dimension")
    return t.stride(0)


def offq_add_rmsnorm(x, res=None, eps=1e-5, want_h=True, want_y=True):
    """x, res: bf16 [M, D].  Returns (h, y): h = bf16(x + res) (x if res is None),
    y = bf16(rmsnorm(h)); either may be None if not wanted."""
    torch = _torch()
    _need(x, torch.bfloat16, "x", 2)
    if res is not None:
        _need(res, torch.bfloat16, "res", 2)
        if res.shape != x.shape:
            raise ValueError("res must match x")
    M, D = x.shape
    h = torch.empty((M, D), dtype=torch.bfloat16, device=x.device) if want_h else None
    y = torch.empty((M, D), dtype=torch.bfloat16, device=x.device) if want_y else None
    _check(lib.offq_add_rmsnorm(_ptr(x), _rows(x, "x"), _ptr(res),
                                _rows(res, "res") if res is not None else 0, M, D, float(eps),
                                _ptr(h), D, _ptr(y), D, _stream()), "offq_add_rmsnorm")
    return h, y


def offq_add_rmsnorm_quantize(x, g, res=None, eps=1e-5, want_h=False, debug=False):
    """Fused add + RMSNorm + quantize (no rotation).  x, res: bf16 [M, D].
    Returns (codes u8 [M, D/2], scale fp16 [M, D/g], zero int16 [M, D/g],
    h bf16 [M, D] or None, y bf16 [M, D] or None)."""
    torch = _torch()
    _need(x, torch.bfloat16, "x", 2)
    if res is not None:
        _need(res, torch.bfloat16, "res", 2)
    M, D = x.shape
    dev = x.device
    codes = torch.empty((M, D // 2), dtype=torch.uint8, device=dev)
    scale = torch.empty((M, D // g), dtype=torch.float16, device=dev)
    zero = torch.empty((M, D // g), dtype=torch.int16, device=dev)
    h = torch.empty((M, D), dtype=torch.bfloat16, device=dev) if want_h else None
    y = torch.empty((M, D), dtype=torch.bfloat16, device=dev) if debug else None
    _check(lib.offq_add_rmsnorm_quantize(_ptr(x), _rows(x, "x"), _ptr(res),
                                         _rows(res, "res") if res is not None else 0, M, D,
                                         float(eps), int(g), _ptr(h), D, _ptr(codes), _ptr(scale),
                                         _ptr(zero), _ptr(y), D, _stream()),
           "offq_add_rmsnorm_quantize")
    return codes, scale, zero, h, y


def offq_swiglu_rotate_quantize(gu, debug=False):
    """Fused SwiGLU + 128-point Hadamard + quantize.  gu: bf16 [M, 2F].
    Returns (codes u8 [M, F/2], scale fp16 [M, F/128], zero int16 [M, F/128],
    y fp32 [M, F] or None)."""
    torch = _torch()
    _need(gu, torch.bfloat16, "gu", 2)
    M, F2 = gu.shape
    F = F2 // 2
    dev = gu.device
    codes = torch.empty((M, F // 2), dtype=torch.uint8, device=dev)
    scale = torch.empty((M, F // 128), dtype=torch.float16, device=dev)
    zero = torch.empty((M, F // 128), dtype=torch.int16, device=dev)
    y = torch.empty((M, F), dtype=torch.float32, device=dev) if debug else None
    _check(lib.offq_swiglu_rotate_quantize(_ptr(gu), _rows(gu, "gu"), M, F, _ptr(codes), _ptr(scale),
                                           _ptr(zero), _ptr(y), _stream()),
           "offq_swiglu_rotate_quantize")
    return codes, scale, zero, y


def offq_swiglu(gu):
    """gu: bf16 [M, 2F] (gate | up).  Returns bf16 [M, F]."""
    torch = _torch()
    _need(gu, torch.bfloat16, "gu", 2)
    M, F2 = gu.shape
    F = F2 // 2
    out = torch.empty((M, F), dtype=torch.bfloat16, device=gu.device)
    _check(lib.offq_swiglu(_ptr(gu), _rows(gu, "gu"), M, F, _ptr(out), F, _stream()), "offq_swiglu")
    return out


def _cache_operands(cache, B, Hkv):
    torch = _torch()
    s_cap = cache["k_codes"].shape[2]
    for n in ("k_codes", "v_codes"):
        _need(cache[n], torch.uint8, n, 4)
        if cache[n].shape != (B, Hkv, s_cap, 64) or not cache[n].is_contiguous():
            raise ValueError(f"{n} must be a contiguous [B, Hkv, s_cap, 64] tensor")
    for n, dt in (("k_scale", torch.float16), ("v_scale", torch.float16), ("k_zero", torch.int16),
                  ("v_zero", torch.int16)):
        _need(cache[n], dt, n, 3)
        if cache[n].shape != (B, Hkv, s_cap) or not cache[n].is_contiguous():
            raise ValueError(f"{n} must be a contiguous [B, Hkv, s_cap] tensor")
    return s_cap


def _rope_kv(qkv, B, T, Hq, Hkv, positions, cache, rope_base, k_hadamard, v_hadamard, debug,
             fn, name):
    torch = _torch()
    _need(qkv, torch.bfloat16, "qkv", 2)
    _need(positions, torch.int32, "positions", 1)
    M = qkv.shape[0]
    if M != B * (T or 1):
        raise ValueError("qkv must have B * T rows")
    s_cap = _cache_operands(cache, B, Hkv)
    if positions.shape != (M,):
        raise ValueError("positions must have one entry per qkv row")
    dev = qkv.device
    q = torch.empty((M, Hq, 128), dtype=torch.bfloat16, device=dev)
    ky = torch.empty((M, Hkv, 128), dtype=torch.float32, device=dev) if debug else None
    vy = torch.empty((M, Hkv, 128), dtype=torch.float32, device=dev) if debug else None
    dims = (M,) if T is None else (B, T)
    _check(fn(_ptr(qkv), _rows(qkv, "qkv"), *dims, Hq, Hkv, 128, _ptr(positions),
              float(rope_base), int(bool(k_hadamard)), int(bool(v_hadamard)), _ptr(q),
              _ptr(cache["k_codes"]), _ptr(cache["k_scale"]), _ptr(cache["k_zero"]),
              _ptr(cache["v_codes"]), _ptr(cache["v_scale"]), _ptr(cache["v_zero"]), s_cap,
              _ptr(ky), _ptr(vy), _stream()), name)
    return q, ky, vy


def offq_rope_kv_append(qkv, Hq, Hkv, positions, cache, rope_base=500000.0, k_hadamard=True,
                        v_hadamard=False, debug=False):
    """qkv: bf16 [M, (Hq + 2 Hkv) * 128]; positions: int32 [M] (device);
    cache: dict with k_codes/v_codes u8 [M, Hkv, s_cap, 64] and k_scale/v_scale
    fp16, k_zero/v_zero int16 [M, Hkv, s_cap] (written in place).  Returns
    (q bf16 [M, Hq, 128], k_y fp32 [M, Hkv, 128] or None, v_y or None)."""
    M = qkv.shape[0]
    return _rope_kv(qkv, M, None, Hq, Hkv, positions, cache, rope_base, k_hadamard, v_hadamard,
                    debug, lib.offq_rope_kv_append, "offq_rope_kv_append")


def offq_rope_kv_prefill(qkv, B, Hq, Hkv, positions, cache, rope_base=500000.0, k_hadamard=True,
                         v_hadamard=False, debug=False):
    """The prefill form: qkv bf16 [B * T, (Hq + 2 Hkv) * 128], row b * T + t
    token t of sequence b, written at positions[b * T + t] (int32, device)
    of the cache [B, Hkv, s_cap, ...] (in place).  Returns (q bf16
    [B * T, Hq, 128], k_y, v_y fp32 [B * T, Hkv, 128] or None)."""
    M = qkv.shape[0]
    if B <= 0 or M % B:
        raise ValueError("qkv rows must be a multiple of B")
    return _rope_kv(qkv, B, M // B, Hq, Hkv, positions, cache, rope_base, k_hadamard, v_hadamard,
                    debug, lib.offq_rope_kv_prefill, "offq_rope_kv_prefill")


def offq_kv_attention_prefill(q, cache, past, sm_scale=None, v_hadamard=False, out=None):
    """Causal attention of T new tokens per sequence over the 4-bit cache.

    q: bf16 [B, T, Hq, 128] contiguous (query t at position past + t);
    cache: dict of the arrays [B, Hkv, s_cap, ...] holding past + T
    positions.  Returns out bf16 [B, T, Hq, 128] (or writes ``out``)."""
    torch = _torch()
    _need(q, torch.bfloat16, "q", 4)
    if not q.is_contiguous():
        raise ValueError("q must be contiguous")
    B, T, Hq, Dh = q.shape
    Hkv = cache["k_codes"].shape[1]
    s_cap = _cache_operands(cache, B, Hkv)
    if sm_scale is None:
        sm_scale = 1.0 / float(Dh) ** 0.5
    if out is None:
        out = torch.empty((B, T, Hq, Dh), dtype=torch.bfloat16, device=q.device)
    _need(out, torch.bfloat16, "out", 4)
    if not out.is_contiguous() or out.shape != q.shape:
        raise ValueError("out must be a contiguous tensor shaped like q")
    _check(lib.offq_kv_attention_prefill(_ptr(q), B, T, Hq, Hkv, Dh, int(past),
                                         _ptr(cache["k_codes"]), _ptr(cache["k_scale"]),
                                         _ptr(cache["k_zero"]), _ptr(cache["v_codes"]),
                                         _ptr(cache["v_scale"]), _ptr(cache["v_zero"]), s_cap,
                                         float(sm_scale), int(bool(v_hadamard)), _ptr(out),
                                         _stream()), "offq_kv_attention_prefill")
    return out


# ------------------------------------------------------- offline calibration
def offq_top1_select(x):
    """x: bf16 [n_seq, L, D] (last dim contiguous).  Returns (idx int32 [n_seq],
    X fp32 [n_seq, D]): per sequence the token of largest L-infinity norm."""
    torch = _torch()
    _need(x, torch.bfloat16, "x", 3)
    if x.stride(2) != 1:
        raise ValueError("x must have a contiguous last dimension")
    n, L, D = x.shape
    dev = x.device
    idx = torch.empty((n,), dtype=torch.int32, device=dev)
    X = torch.empty((n, D), dtype=torch.float32, device=dev)
    wb = lib.offq_top1_workspace_bytes(n, L)
    ws = torch.empty((max(wb, 4) + 3) // 4, dtype=torch.float32, device=dev)
    _check(lib.offq_top1_select(_ptr(x), n, L, D, x.stride(1), x.stride(0), _ptr(idx), _ptr(X), D,
                                _ptr(ws), ws.numel() * 4, _stream()), "offq_top1_select")
    return idx, X


def offq_channel_absmax(x):
    """x: bf16 [rows, D].  Returns fp64 [D]: max over rows of |x|."""
    torch = _torch()
    _need(x, torch.bfloat16, "x", 2)
    out = torch.empty((x.shape[1],), dtype=torch.float64, device=x.device)
    _check(lib.offq_channel_absmax(_ptr(x), x.shape[0], x.shape[1], _rows(x, "x"), _ptr(out),
                                   _stream()), "offq_channel_absmax")
    return out


def offq_gram(X):
    """X: fp32 [N, D].  Returns C = X^T X / N, fp64 [D, D]."""
    torch = _torch()
    _need(X, torch.float32, "X", 2)
    N, D = X.shape
    C = torch.empty((D, D), dtype=torch.float64, device=X.device)
    _check(lib.offq_gram(_ptr(X), N, D, _rows(X, "X"), _ptr(C), D, _stream()), "offq_gram")
    return C


def offq_eigh(C, max_sweeps=30, tol=None):
    """C: fp64 [D, D] symmetric.  Returns (evals fp64 [D] descending, U fp64
    [D, D] with eigenvectors in columns, sweeps, relative off-diagonal norm).
    tol defaults to D * 2^-52 (the level fp64 rotations bottom out at)."""
    torch = _torch()
    _need(C, torch.float64, "C", 2)
    D = C.shape[0]
    if tol is None:
        tol = D * 2.0 ** -52
    if C.shape != (D, D):
        raise ValueError("C must be square")
    ev = torch.empty((D,), dtype=torch.float64, device=C.device)
    U = torch.empty((D, D), dtype=torch.float64, device=C.device)
    wb = lib.offq_eigh_workspace_bytes(D)
    ws = torch.empty((max(wb, 8) + 7) // 8, dtype=torch.float64, device=C.device)
    sw = ctypes.c_int32(0)
    ro = ctypes.c_double(0.0)
    _check(lib.offq_eigh(_ptr(C), D, _rows(C, "C"), _ptr(ev), _ptr(U), D, _ptr(ws), ws.numel() * 8,
                         int(max_sweeps), float(tol), ctypes.byref(sw), ctypes.byref(ro),
                         _stream()), "offq_eigh")
    return ev, U, sw.value, ro.value


def offq_group_permutation(key, g):
    """key: fp64 [D].  Returns perm int32 [D] (new slot -> original channel)."""
    torch = _torch()
    _need(key, torch.float64, "key", 1)
    D = key.shape[0]
    perm = torch.empty((D,), dtype=torch.int32, device=key.device)
    ws = torch.empty((D,), dtype=torch.int32, device=key.device)
    _check(lib.offq_group_permutation(_ptr(key), D, int(g), _ptr(perm), _ptr(ws), D * 4, _stream()),
           "offq_group_permutation")
    return perm


def offq_build_rotation(U, D, perm=None, g=1, apply_hadamard=False, device=None):
    """Returns R fp32 [D, D] = U P blockdiag(H_g / sqrt g) (U None: identity)."""
    torch = _torch()
    dev = U.device if U is not None else perm.device if perm is not None else (device or "cuda")
    if U is not None:
        _need(U, torch.float64, "U", 2)
    if perm is not None:
        _need(perm, torch.int32, "perm", 1)
    R = torch.empty((D, D), dtype=torch.float32, device=dev)
    _check(lib.offq_build_rotation(_ptr(U), _rows(U, "U") if U is not None else D, D, _ptr(perm),
                                   int(g), int(bool(apply_hadamard)), _ptr(R), D, _stream()),
           "offq_build_rotation")
    return R


def offq_fuse_weights(W, R):
    """W: fp32 [N, K], R: fp32 [K, K].  Returns W R (fp32 [N, K])."""
    torch = _torch()
    _need(W, torch.float32, "W", 2)
    _need(R, torch.float32, "R", 2)
    N, K = W.shape
    out = torch.empty((N, K), dtype=torch.float32, device=W.device)
    _check(lib.offq_fuse_weights(_ptr(W), _rows(W, "W"), N, K, _ptr(R), _rows(R, "R"), _ptr(out), K,
                                 _stream()), "offq_fuse_weights")
    return out


def offq_permute_rows(W, perm):
    """W: fp32 [N, K]; perm int32 [N].  Returns W[perm] (fp32 [N, K])."""
    torch = _torch()
    _need(W, torch.float32, "W", 2)
    _need(perm, torch.int32, "perm", 1)
    N, K = W.shape
    out = torch.empty((N, K), dtype=torch.float32, device=W.device)
    _check(lib.offq_permute_rows(_ptr(W), _rows(W, "W"), N, K, _ptr(perm), _ptr(out), K, _stream()),
           "offq_permute_rows")
    return out
