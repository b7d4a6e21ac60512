"""The C ABI used from plain C (tests/c_abi_check.c): separate hipMalloc
buffers per rank, the caller's own HIP stream, the exact int32 sum on every
rank for a one-GPU-per-server plan and a server plan, and the error paths.
The program is built by the package build (gcc, no Python in the loop)."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BIN = os.path.join(ROOT, "tests", "c_abi_check")


def test_c_check_is_built():
    assert os.path.exists(BIN), "tests/c_abi_check is not built: run the package build"


@pytest.mark.gpu
def test_c_abi_from_plain_c():
    if not os.path.exists(BIN):
        pytest.skip("tests/c_abi_check is not built")
    r = subprocess.run([BIN], capture_output=True, text=True, timeout=120)
    print(r.stdout, r.stderr, flush=True)
    assert r.returncode == 0, r.stderr
    assert "c_abi_check: ok" in r.stdout
