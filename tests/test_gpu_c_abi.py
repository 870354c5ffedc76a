"""The C ABI used from C: tests/c_abi_step (built by __graft_entry__.build())
allocates with the HIP runtime, runs bf16 Weyl and E4M3 SR steps through
include/ssmq.h, checks them against the oracle library and exercises an
error path, as a child process."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu
BINARY = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_abi_step")


def test_c_program_runs_the_step():
    assert os.path.exists(BINARY), "tests/c_abi_step is missing: run __graft_entry__.build()"
    r = subprocess.run([BINARY], capture_output=True, text=True, timeout=120)
    print(r.stdout, r.stderr, flush=True)
    assert r.returncode == 0
    assert "c_abi_step: ok" in r.stdout
