"""The ABI from C alone (tests/c_abi/mmi_c_check.c, built by
__graft_entry__.build()): error codes, full-window A-shape == dense bitwise,
plan statistics, sampled rows against double-precision causal attention."""
import os
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
BIN = os.path.join(HERE, "c_abi", "mmi_c_check")


def test_c_program_is_built_and_links():
    assert os.path.exists(BIN), "run __graft_entry__.build() first"
    r = subprocess.run(["ldd", BIN], capture_output=True, text=True)
    assert "libmmi.so" in r.stdout and "not found" not in r.stdout, r.stdout


@pytest.mark.gpu
def test_c_program_runs():
    r = subprocess.run([BIN], capture_output=True, text=True, timeout=300)
    print(r.stdout, r.stderr)
    assert r.returncode == 0 and "c abi ok" in r.stdout
