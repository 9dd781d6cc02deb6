"""The C ABI used from a plain C program (tests/c_abi_consumer.c, built by
tests/build_c_consumer.py): HIP runtime memory, no Python binding, every
result checked against the CPU oracle inside the program."""
import os
import subprocess

import pytest

from _helpers import log

pytestmark = pytest.mark.gpu

EXE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_abi_consumer")


def test_c_program_uses_the_library_and_matches_the_oracle():
    if not os.path.exists(EXE):
        raise RuntimeError(f"{EXE} is not built; run tests/build_c_consumer.py (or __graft_entry__.build())")
    log("c_abi_consumer")
    r = subprocess.run([EXE], capture_output=True, text=True, timeout=100)
    print(r.stdout)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "PASSED: 0 failure(s)" in r.stdout
