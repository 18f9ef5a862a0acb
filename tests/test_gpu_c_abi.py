"""The C ABI used from plain C (tests/c/abi_roundtrip.c: HIP runtime C API,
include/mezo.h and the oracle's C library only, no Python in the process): a
perturb and a fused update each within the fp32 / bf16 bars of the oracle
applied to the GPU's own input, and ChecksumMatch equal to the oracle's
checksum of the result. The program is built by __graft_entry__.build()."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

BIN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c", "abi_roundtrip")


def test_c_program_round_trip():
    assert os.path.exists(BIN), f"{BIN} is not built: run __graft_entry__.build()"
    r = subprocess.run([BIN], capture_output=True, text=True, timeout=120)
    print(r.stdout)
    assert r.returncode == 0, r.stderr + r.stdout
    assert "abi_roundtrip ok" in r.stdout
