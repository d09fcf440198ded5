"""Host-side helpers of the search library, compiled for the host only (no
GPU needed): the order-preserving float32 mapping that the index applies to
float32 attribute columns and the kernels to each query's bounds."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_f32_ord_preserves_float_order(tmp_path):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    exe = tmp_path / "f32_ord_check"
    subprocess.run([hipcc, "-std=c++17", "-O1", "-I" + os.path.join(ROOT, "include"),
                    "-I" + os.path.join(ROOT, "paper_2609_16175_amd", "csrc"),
                    os.path.join(ROOT, "tests", "f32_ord_check.cpp"), "-o", str(exe)],
                   check=True, capture_output=True, timeout=300)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "0 failures" in r.stdout
