"""bench.py's host-side contract, on the CPU: more than one GPU is refused
with a message and a non-zero status, and the kernel-source hash (which
ties recorded counters to the code they were taken on) ignores comments and
blank lines but not code."""

import os
import shutil
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode != 0
    assert "one GPU" in r.stdout + r.stderr


def test_kernel_source_hash_ignores_comments_only(tmp_path, monkeypatch):
    for p in bench.KERNEL_SOURCES:
        dst = tmp_path / p
        dst.parent.mkdir(parents=True, exist_ok=True)
        shutil.copy(os.path.join(ROOT, p), dst)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    base = bench.kernel_source_hash()
    first = tmp_path / bench.KERNEL_SOURCES[0]
    text = first.read_text()
    first.write_text("// a new comment line\n\n/* and a block\n   comment */\n" + text.replace("\n", "   \n", 3))
    assert bench.kernel_source_hash() == base
    first.write_text(text + "\nstatic int purlin_hash_probe = 1;\n")
    assert bench.kernel_source_hash() != base
