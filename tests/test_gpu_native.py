"""The C ABI driven from C programs with no Python in the loop (tests/native/,
built by build()):
- abi_step.c: a block manager's tables, a serving step, its rows against the
  single-kernel entry points bit for bit, the pools, and invalid calls;
- abi_offload.c: the block manager with a host pool, its swap lists run through
  cw_kv_swap_out / cw_kv_swap_in, and every step's output against the same step
  on a pool built from the sessions' own K/V, bit for bit."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

NATIVE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "native")


@pytest.mark.parametrize("name", ["abi_step", "abi_offload"])
def test_native_c_program(name):
    exe = os.path.join(NATIVE, name + ".bin")
    assert os.path.exists(exe), f"tests/native/{name}.bin is missing: run __graft_entry__.build()"
    print(f"\n[case] native {name}", flush=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    print(r.stdout, r.stderr, flush=True)
    assert r.returncode == 0, r.stderr
    assert r.stdout.startswith("ok")
