"""The C-ABI from plain C: include/ii.h compiles as strict C11 with no ROCm
include path, and (on a GPU) a C program loads a table through it and checks
every byte."""
import os
import subprocess

import pytest

import c_abi


def test_c_program_builds():
    c_abi.build()
    assert os.path.exists(c_abi.BIN)


@pytest.mark.gpu
def test_c_program_loads_bit_exact():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    if not os.path.exists(c_abi.BIN):
        c_abi.build()
    r = subprocess.run([c_abi.BIN], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.startswith("OK 39 "), r.stdout
