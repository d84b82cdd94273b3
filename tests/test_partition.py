"""Host check of the attention work partition (even and adaptive split arithmetic shared by the
attention kernel and the merges): builds tests/partition_check.cpp against the library's
internal header with hipcc and runs it (no GPU calls)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_partition_arithmetic(tmp_path):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not found")
    exe = tmp_path / "partition_check"
    build = subprocess.run([hipcc, "-std=c++17", "-O2", "--offload-arch=gfx950", "-x", "hip",
                            os.path.join(ROOT, "tests", "partition_check.cpp"),
                            "-I", os.path.join(ROOT, "paper_2605_30351_amd", "csrc"),
                            "-o", str(exe)], capture_output=True, text=True)
    assert build.returncode == 0, build.stderr[-2000:]
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert run.returncode == 0, run.stdout[-2000:]
    assert "bad 0" in run.stdout
