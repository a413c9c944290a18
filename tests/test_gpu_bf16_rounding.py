"""The per-step kernels store bfloat16 through the hardware's pair
conversion followed by the canonical-NaN rule; tests/c/bf16_rounding
(built by build()) checks that on the GPU against the library's scalar
rule (round to nearest even, NaN -> 0x7fc0) for every float bit pattern."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu
BIN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c", "bf16_rounding")


def test_bf16_store_rule_on_every_float():
    if not os.path.exists(BIN):
        pytest.fail(f"{BIN} is missing: run build()")
    r = subprocess.run([BIN], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "0 mismatches" in r.stdout
