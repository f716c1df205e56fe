"""CPU tests of bench.py's host logic: the one-GPU guard and the kernel-code hash that
decides whether the committed HBM-counter figures still apply."""

import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_exits_with_a_message():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode != 0
    assert "one GPU" in res.stderr
    assert res.stdout.strip() == ""


def test_kernel_hash_ignores_comments_and_blank_space(tmp_path, monkeypatch):
    src = tmp_path / "k.hip"
    src.write_text("// header\n__global__ void k(int *p) {  /* body */\n  p[0] = 1; // store\n}\n")
    monkeypatch.setattr(bench, "KERNEL_SOURCES", [str(src)])
    h0 = bench.kernel_source_hash()
    src.write_text("// another header\n\n__global__   void k(int *p) {\n  p[0] = 1;\n}  /* end */\n")
    assert bench.kernel_source_hash() == h0
    src.write_text("__global__ void k(int *p) { p[0] = 2; }\n")
    assert bench.kernel_source_hash() != h0
