"""The library through its C ABI alone: a plain C program (no Python, no
PyTorch) allocates device memory with the HIP runtime, runs decode steps and
checks them against the fp64 oracle (tests/c_client/pda_c_client.c)."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

BIN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_client", "pda_c_client")


def test_c_client():
    assert os.path.exists(BIN), "build the C client first (__graft_entry__.build())"
    r = subprocess.run([BIN], capture_output=True, text=True, timeout=90)
    print(r.stdout, r.stderr)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all checks passed" in r.stdout
