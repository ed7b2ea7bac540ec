"""The scoring scratch layout (packed lower triangle when causal), checked on
the host: tests/layout_check.cpp compiled host-only against the library's own
header, every written slot distinct and inside the sized buffer."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_scratch_layout_is_a_bijection(tmp_path):
    hipcc = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    exe = tmp_path / "layout_check"
    cmd = [hipcc, "-x", "hip", "--cuda-host-only", "-O1", "-std=c++17",
           "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(ROOT, "paper_2503_16428_amd", "csrc"),
           os.path.join(ROOT, "tests", "layout_check.cpp"), "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0 and "layout ok" in out.stdout, out.stdout
