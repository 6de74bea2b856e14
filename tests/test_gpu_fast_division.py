"""The quantizer's division-free quotients (div15_rn, rcp_fp16_rn in
csrc/common.h) equal IEEE fp32 division on every input that reaches them:
an exhaustive check on the GPU (tests/gpu_checks/fast_division.hip, built by
__graft_entry__.build())."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

EXE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "gpu_checks", "fast_division")


def test_fast_division_exhaustive():
    if not os.path.exists(EXE):
        pytest.fail(f"{EXE} is not built (run __graft_entry__.build())")
    r = subprocess.run([EXE], capture_output=True, text=True, timeout=120)
    print(r.stdout)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "0 mismatches" in r.stdout
