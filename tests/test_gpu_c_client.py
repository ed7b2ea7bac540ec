"""The library driven from plain C on the GPU (tests/c_client.c, built into
paper_2503_16428_amd/lib/xattn_c_client by the package build): the chained
forward at tau = 1 is bitwise the dense mode (every causal block selected,
Fig. 1), the lists at tau = 0.9 are valid and hold each row's top block, and
an invalid shape is rejected with a message."""
import os
import subprocess

import pytest

from paper_2503_16428_amd import build as B

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)


def test_c_client_runs():
    assert os.path.exists(B.C_CLIENT), \
        "the C client is not built (run the package build: __graft_entry__.build())"
    print("c client: forward at tau 1 vs dense, lists at tau 0.9, rejected shape", flush=True)
    r = subprocess.run([B.C_CLIENT], capture_output=True, text=True, timeout=120)
    print(r.stdout, r.stderr, flush=True)
    assert r.returncode == 0, r.stderr
    assert "c client ok" in r.stdout
