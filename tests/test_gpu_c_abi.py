"""The C ABI from C alone: tests/c/abi_c_check (built by build()) allocates
device memory with the HIP runtime, calls every entry point on a small 3-D
backward-Euler NS grid, checks refused calls, and compares every output with
the oracle to the parity bar.  No Python or torch in the loop."""
from __future__ import annotations

import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PROG = os.path.join(ROOT, "tests", "c", "abi_c_check")


def test_c_program_against_the_oracle():
    if not os.path.exists(PROG):  # (build() always builds it beside the library)
        pytest.skip(f"{PROG} is not built")
    print("case c-abi program", flush=True)
    r = subprocess.run([PROG], capture_output=True, text=True, timeout=120)
    print(r.stdout[-3000:], flush=True)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "c-abi: ok" in r.stdout
