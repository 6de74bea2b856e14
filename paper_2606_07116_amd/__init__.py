"""MI355X-native OffQ W4A4KV4 online path (HIP kernels behind a C ABI).

The compute lives in ``liboffq.so`` (HIP, gfx950); this package only marshals
arguments.  Entry points (same names as ``include/offq.h``):

    offq_rotate_quantize(x, g, apply_hadamard=True, debug=False)
    offq_w4a4_gemm(a_codes, a_scale, a_zero, w_codes, w_scale, w_colsum, g, debug=False)
    offq_kv_quantize(kv, apply_hadamard=True, debug=False)
    offq_pack_weights(w, g)          (w_codes in the blocked operand layout;
                                      blocked_weight_codes / row_major_weight_codes
                                      convert from / to row-major [N, K/2] codes)
    offq_kv_attention_decode(q, k_codes, k_scale, k_zero, v_codes, v_scale, v_zero, seq_len, ...)
    offq_add_rmsnorm(x, res=None, eps=1e-5)
    offq_swiglu(gu)
    offq_rope_kv_append(qkv, Hq, Hkv, positions, cache, rope_base=500000.0, ...)
    offq_rope_kv_prefill(qkv, B, Hq, Hkv, positions, cache, rope_base=500000.0, ...)
    offq_kv_attention_prefill(q, cache, past, sm_scale=None, v_hadamard=False, out=None)

Offline calibration: offq_top1_select, offq_channel_absmax, offq_gram, offq_eigh,
offq_group_permutation, offq_build_rotation, offq_fuse_weights, offq_permute_rows.

The library is loaded on first use of an entry point (not by importing the
package or its seeded input generators), and that first use raises if the
library has not been built: there is no other path.
"""

_EXPORTS = frozenset((
    "ABI_VERSION",
    "EXPORTED",
    "OffqError",
    "last_error",
    "offq_build_rotation",
    "offq_channel_absmax",
    "offq_eigh",
    "offq_fuse_weights",
    "offq_gram",
    "offq_group_permutation",
    "offq_permute_rows",
    "offq_top1_select",
    "offq_add_rmsnorm",
    "offq_add_rmsnorm_quantize",
    "offq_swiglu_rotate_quantize",
    "offq_rope_kv_append",
    "offq_rope_kv_prefill",
    "offq_kv_attention_prefill",
    "offq_swiglu",
    "offq_kv_attention_decode",
    "offq_kv_attention_decode_quantize",
    "offq_kv_attention_decode_noalloc",
    "offq_kv_attention_workspace_bytes",
    "offq_kv_quantize",
    "offq_pack_weights",
    "offq_rotate_quantize",
    "offq_w4a4_gemm",
    "offq_weight_codes_bytes",
    "weight_codes_shape",
    "blocked_weight_codes",
    "row_major_weight_codes",
    "status_name",
))


def __getattr__(name):
    if name in _EXPORTS:
        from . import _lib
        return getattr(_lib, name)
    raise AttributeError(f"module {__name__!r} has no attribute {name!r}")


def __dir__():
    return sorted(set(globals()) | _EXPORTS)
