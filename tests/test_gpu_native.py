"""The C ABI driven from a C program with no Python in the loop
(tests/native/abi_step.c, built by build()): a block manager's tables, a
serving step, its rows against the single-kernel entry points bit for bit, the
pools, and invalid calls."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

EXE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "native", "abi_step.bin")


def test_native_c_program():
    assert os.path.exists(EXE), "tests/native/abi_step.bin is missing: run __graft_entry__.build()"
    print("\n[case] native abi_step", flush=True)
    r = subprocess.run([EXE], capture_output=True, text=True, timeout=120)
    print(r.stdout, r.stderr, flush=True)
    assert r.returncode == 0, r.stderr
    assert r.stdout.startswith("ok")
