"""The C ABI from a plain-C program (tests/c_abi/c_smoke.c): HIP runtime for
device memory, one ts_ffn_sparse call checked against a direct fp64
evaluation, one rejected call that must leave the output untouched.  No
Python or PyTorch is involved in the program."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

BIN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_abi", "_build", "c_smoke")


def test_c_program_uses_the_abi():
    assert os.path.exists(BIN), "build first (__graft_entry__.build())"
    r = subprocess.run([BIN], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "c_smoke ok" in r.stdout
