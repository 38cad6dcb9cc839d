"""The C ABI end to end from C++, without Python or PyTorch (GPU).

tests/c_abi_round.cpp allocates with hipMalloc, runs one round over two units
(one of them only a ragged tail), checks the decision and the new parameters
against closed forms and probes the boundary's argument checks; it prints
"ok" on success.  It is built with the library by __graft_entry__.build().
"""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

PROGRAM = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_abi_round")


def test_c_abi_round_from_cpp():
    if not os.path.exists(PROGRAM):
        raise RuntimeError(f"{PROGRAM} is not built; run __graft_entry__.build()")
    r = subprocess.run([PROGRAM], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), r.stdout + r.stderr
