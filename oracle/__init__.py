"""CPU oracle for the OffQ online W4A4KV4 path -- TEST INFRASTRUCTURE ONLY.

This package is a plain, slow, obviously-correct reference of what the GPU
library computes.  It exists to check the GPU kernels, nothing else:

* only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
  ``bench.py`` may import it;
* the product package (``paper_2606_07116_amd``) never imports, calls or links
  anything in here, and this package never imports the product package; the
  two share no code;
* every function takes plain numpy arrays (inputs are produced by the seeded
  generators in ``paper_2606_07116_amd.inputs``, which hold none of the
  method's arithmetic) and returns numpy arrays.

What it follows (OffQ, "Taming Structured Outliers in LLM Quantization by
Offsetting"):

* ``hadamard``  -- the Sylvester Hadamard matrix and the block-diagonal online
  rotation ``y = x (I (x) H_g) / sqrt(g)`` (sec. 3.2, Eq. 4; group-wise
  offsetting, sec. 3.2 "Group-Wise Offsetting").
* ``quantizer`` -- the uniform asymmetric quantizer of sec. 3, Eq. 1, per group,
  with 16-bit scale and 16-bit integer zero-point (sec. 3.4), and the
  per-output-channel symmetric 4-bit weight quantizer (sec. 4, implementation).
* ``gemm``      -- the exact integer GEMM of 4-bit codes and the dequantising
  epilogue that follows from Eq. 1 (x_hat = s (x_q - z)).
* ``kv``        -- the KV-cache quantizer: per-head Hadamard (sec. 3.3, step 2(3))
  and the same quantizer with group = head_dim (sec. 4.2, "Number of Groups").

Pins: every function is checked in ``tests/`` against facts fixed by the paper
or by mathematics (library Hadamard, orthogonality, the Eq. 5 worked example,
offset invariants, rounding ties, brute-force integer GEMM, the dequantised
matmul identity).  Parity is pinned for every function here; the only value
that is bounded rather than pinned bit-for-bit is the GPU's fp32 rotation
(checked against ``rotate`` within a recursive-summation error bound).
"""

from . import hadamard, quantizer, gemm, kv  # noqa: F401
