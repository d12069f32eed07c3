"""The library driven from plain C: tests/c_abi/abi_demo.c includes only the
C header and the HIP runtime API, allocates with hipMalloc and checks the
results of gather, scatter, planned copies, digests, and the fp8 cast and
its inverse itself.  It runs as a child process; this test passes when it
exits 0."""
import os
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
EXE = os.path.join(HERE, "c_abi", "abi_demo")


@pytest.mark.gpu
def test_c_program_through_the_abi():
    assert os.path.exists(EXE), "tests/c_abi/abi_demo is missing: run __graft_entry__.build() first"
    r = subprocess.run([EXE], capture_output=True, text=True, timeout=90)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "correct" in r.stdout
