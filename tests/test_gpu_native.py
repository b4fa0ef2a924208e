"""The C ABI used from plain C++ (tests/native/cabi_smoke.cpp, built by
__graft_entry__.build()): one scheduled step through librip with HIP's own
runtime and no Python in the loop, checked against exact closed-form values."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

BIN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "native", "cabi_smoke")


def test_native_cabi_consumer():
    assert os.path.exists(BIN), "tests/native/cabi_smoke is not built; run __graft_entry__.build()"
    print("case native C-ABI smoke", flush=True)
    res = subprocess.run([BIN], capture_output=True, text=True, timeout=120)
    print(res.stdout, res.stderr, flush=True)
    assert res.returncode == 0
    assert "cabi smoke ok" in res.stdout
