"""The C ABI from plain C: tests/c/abi_consumer (built by build()) allocates
with hipMalloc, runs one cached step through the library and checks it
against closed forms -- a duplicate anchor view transports the increment
exactly (Eq. 1 with a single tap of weight 1), the DDIM step matches its
formula; the split launch over the visible-token index (with a workspace
and allocation-free) and the on-the-fly step over the foreground index give
the same bits; the coverage schedule's fused update + selection leaves no
token stale and picks view 0 -- and that argument errors return negative
codes."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu
BIN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c", "abi_consumer")


def test_plain_c_consumer():
    if not os.path.exists(BIN):
        pytest.fail(f"{BIN} is missing: run build()")
    r = subprocess.run([BIN], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "C ABI OK" in r.stdout
