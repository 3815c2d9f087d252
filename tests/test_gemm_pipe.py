"""Host-side checks of the bf16 expert GEMMs' LDS pipelines (no GPU needed), each a
small C++ program built with hipcc for the host from the kernels' own headers:
 * tests/pipe_check.cpp (gemm_pipe.h): every tile shape the kernels instantiate, K
   lengths up to 128 stages and every per-wave activation DMA count: the wait count
   before each stage must equal the number of DMAs a one-instruction-at-a-time
   replay of the issue sequence has issued after that stage's last DMA;
 * tests/swizzle_check.cpp (lds_dma.h): the chunk each DMA lane fetches and the
   offset each MFMA lane reads agree (every lane reads its own row and k chunk)."""
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


def _build_and_run(tmp_path, name):
    hipcc = _hipcc()
    if hipcc is None:
        pytest.skip("hipcc not found")
    exe = tmp_path / name
    r = subprocess.run([hipcc, "-O1", "-std=c++17", os.path.join(HERE, name + ".cpp"), "-o", str(exe)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout[-2000:] + r.stderr[-2000:]
    return r


def test_gemm_wait_counts(tmp_path):
    _build_and_run(tmp_path, "pipe_check")


def test_lds_unit_layout(tmp_path):
    _build_and_run(tmp_path, "swizzle_check")
