"""The library used from plain C (tests/c/abi_step.c, built by
__graft_entry__.build()): plan creation and error codes, fc_step and
fc_tree_reduce in every schedule on device buffers from the HIP runtime's C
API, then fc_sgd_step on that sum and fc_broadcast of w' (the composed
path), compared bit for bit with the oracle's C functions."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

BIN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c", "abi_step")


def test_c_client_matches_oracle(device):
    assert os.path.exists(BIN), "tests/c/abi_step is not built; run __graft_entry__.build()"
    r = subprocess.run([BIN], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "bit-exact" in r.stdout
