"""Plain HBM streams on the GPU (tests/gpu_checks/hbm_stream.hip, built by
__graft_entry__.build()): the read-only, copy and read + quarter-write rates
that bound the memory-bound kernels, the last being the KV-cache quantizer's
read/write mix.  Checks the probe's own output and that every rate is
physically possible; the rates themselves are printed, not asserted."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

EXE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "gpu_checks", "hbm_stream")


def test_hbm_stream_probe():
    if not os.path.exists(EXE):
        pytest.fail(f"{EXE} is not built (run __graft_entry__.build())")
    r = subprocess.run([EXE], capture_output=True, text=True, timeout=120)
    print(r.stdout)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "0 of 4096 sampled mixed outputs wrong" in r.stdout
