"""The library's lazily filled per-device state (compute-unit count, raised LDS limits of the GEMM
kernels) under concurrent first use: a fresh process makes its first GEMM calls from four host
threads at once, on both tile paths, and compares each result with the same call made
sequentially afterwards (tests/first_call_child.py)."""
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_first_gemm_calls_from_four_threads_in_a_fresh_process():
    r = subprocess.run([sys.executable, "-u", os.path.join(ROOT, "tests", "first_call_child.py")],
                       capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 0, (r.stdout + r.stderr)[-4000:]
    assert r.stdout.strip().endswith("ok")
