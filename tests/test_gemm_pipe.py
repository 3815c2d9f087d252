"""Host-side check of the grouped GEMM's exact vmcnt waits: builds tests/pipe_check.cpp
(which includes the kernels' own gemm_pipe.h) with hipcc for the host and runs it.
Every tile shape the kernels instantiate, K lengths up to 128 stages and every
per-wave activation DMA count: the wait count before each stage must equal the
number of DMAs a one-instruction-at-a-time replay of the issue sequence has issued
after that stage's last DMA (no GPU needed)."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


def _hipcc():
    for c in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if c and os.path.exists(c):
            return c
    return None


def test_gemm_wait_counts(tmp_path):
    hipcc = _hipcc()
    if hipcc is None:
        pytest.skip("hipcc not found")
    exe = tmp_path / "pipe_check"
    r = subprocess.run([hipcc, "-O1", "-std=c++17", os.path.join(HERE, "pipe_check.cpp"), "-o", str(exe)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout[-2000:] + r.stderr[-2000:]
