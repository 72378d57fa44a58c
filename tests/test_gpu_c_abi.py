"""The library through its C ABI alone: tests/c_abi_check.c (plain C, no
Python or torch in the process) allocates with hipMalloc, calls pam_mul,
pam_gemm, pam_gemm_batched_ws, pam_gemm_batched and
pam_gemm_batched_with_plan, and compares with the C oracle (bit-exact
elementwise, the GEMM tolerance for the products)."""
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_c_abi_check_program():
    exe = os.path.join(ROOT, "tests", "c_abi_check")
    assert os.path.exists(exe), "tests/c_abi_check is not built: run __graft_entry__.build()"
    sys.stdout.write("[case] tests/c_abi_check (child process)\n")
    sys.stdout.flush()
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    sys.stdout.write(r.stdout)
    sys.stderr.write(r.stderr)
    assert r.returncode == 0, f"c_abi_check exited with {r.returncode}"
    assert "c_abi_check: OK" in r.stdout
