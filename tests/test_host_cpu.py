"""Host logic that needs no GPU: the benchmark's single-GPU contract and the package's
refusal to import without its compiled library."""
import os
import shutil
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 3
    assert "exactly one GPU" in r.stderr


def test_package_import_fails_without_library(tmp_path):
    # a copy of the package without libhqlss.so must raise on import (no CPU fallback)
    pkg = tmp_path / "paper_2306_11987_amd"
    pkg.mkdir()
    for f in os.listdir(os.path.join(ROOT, "paper_2306_11987_amd")):
        if f.endswith(".py"):
            shutil.copy(os.path.join(ROOT, "paper_2306_11987_amd", f), pkg / f)
    code = "import paper_2306_11987_amd"
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300,
                       cwd=str(tmp_path), env={**os.environ, "PYTHONPATH": str(tmp_path)})
    assert r.returncode != 0
    assert "ImportError" in r.stderr and "not built" in r.stderr
