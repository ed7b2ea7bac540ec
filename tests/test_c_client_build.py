"""The C ABI from plain C: tests/c_client.c (a client that uses only
include/xattn.h and the HIP runtime API) compiles warning-free as C11 and
links against the built library. Runs on the CPU; the GPU test runs it."""
import os
import shutil
import subprocess

import pytest

from paper_2503_16428_amd import build as B


def test_c_client_compiles_and_links(tmp_path):
    if shutil.which("gcc") is None or not os.path.exists(B.LIB):
        pytest.skip("gcc or the built library is not available")
    exe = str(tmp_path / "xattn_c_client")
    cmd = B.c_client_command(os.path.join(B.ROOT, "tests", "c_client.c"), exe)
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    nm = subprocess.run(["nm", "-u", exe], capture_output=True, text=True).stdout
    for sym in ("xattn_forward", "xattn_dense_attn", "xattn_forward_layout",
                "xattn_last_error"):
        assert sym in nm, f"{sym} is not referenced by the client"
