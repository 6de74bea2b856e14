"""KV4 cache quantizer (oracle; test-only).

Sec. 3.3, step 2(3): keys receive a per-head online Hadamard H3 after RoPE;
sec. 3.3 step 2(2): values receive an offline per-head rotation R2 fused into
the weights, so no online rotation is needed for V.  The cache is quantized
with the quantizer of Eq. 1 with the group size equal to the head dimension
(sec. 4.2, "Number of Groups").  One row = one (batch, head, position).
"""

import numpy as np

from . import hadamard, quantizer


def kv_rotate(kv_rows, apply_hadamard):
    """fp64 rows [R, Dh] after the optional per-head Hadamard (g = Dh)."""
    x = np.asarray(kv_rows, dtype=np.float64)
    if not apply_hadamard:
        return x.copy()
    return hadamard.rotate(x, x.shape[-1])


def kv_quantize(y_rows):
    """Quantize fp32 rows [R, Dh] with one group per row: (codes, scale[R], zero[R])."""
    y = np.asarray(y_rows, dtype=np.float32)
    codes, s, z = quantizer.quantize_groups(y, y.shape[-1])
    return codes, s[:, 0].copy(), z[:, 0].copy()
