"""The C ABI from a C++ program with no Python in between
(tests/abi/abi_smoke.cpp, built by __graft_entry__.build()): hipMalloc'd
buffers, single calls and a two-matrix plan, both layouts; scores, selection
and the fused hand-over checked against host computations of their
definitions, the plan against the single calls bit for bit."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BIN = os.path.join(ROOT, "tests", "abi", "abi_smoke")


@pytest.mark.timeout(180)
def test_c_abi_from_cpp():
    assert os.path.exists(BIN), "tests/abi/abi_smoke is not built: run __graft_entry__.build()"
    run = subprocess.run([BIN], capture_output=True, text=True, timeout=150)
    assert run.returncode == 0, run.stdout + run.stderr
    assert "abi smoke ok" in run.stdout
