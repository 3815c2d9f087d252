"""Host-side checks of bench.py that need no GPU: the single-GPU refusal of
--gpus N > 1, and the source digest that keys the committed HBM-traffic record
to the kernel code (it ignores comments and blank space, and changes with code)."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def test_bench_refuses_several_gpus():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2", "--steps", "1", "--warmup", "0"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""


def test_source_digest_ignores_comments(tmp_path, monkeypatch):
    import bench

    csrc = tmp_path / "paper_2609_05228_amd" / "csrc"
    csrc.mkdir(parents=True)
    (csrc / "k.hip").write_text("int f(int x) { return x + 1; }\n")
    (csrc / "h.h").write_text("#pragma once\nconstexpr int kA = 4;\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    d0 = bench.source_digest("k.hip")
    (csrc / "k.hip").write_text("// add one\nint f(int x) {  /* the sum */\n  return x + 1;  // done\n}\n")
    assert bench.source_digest("k.hip") == d0
    (csrc / "h.h").write_text("#pragma once\n// a constant\nconstexpr int kA = 4;\n")
    assert bench.source_digest("k.hip") == d0
    (csrc / "k.hip").write_text("int f(int x) { return x + 2; }\n")
    assert bench.source_digest("k.hip") != d0
    (csrc / "k.hip").write_text("int f(int x) { return x + 1; }\n")
    (csrc / "h.h").write_text("#pragma once\nconstexpr int kA = 5;\n")
    assert bench.source_digest("k.hip") != d0
