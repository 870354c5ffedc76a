"""Build tests/c_abi_step, a C program that drives libssmq.so through
include/ssmq.h and checks it against the oracle library (test infrastructure)."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SOURCE = os.path.join(HERE, "c_abi_step.c")
BINARY = os.path.join(HERE, "c_abi_step")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def build(verbose: bool = False) -> str:
    tmp = BINARY + ".tmp"
    cmd = ["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(ROCM, "include"), SOURCE, "-o", tmp,
           "-L", os.path.join(ROOT, "paper_2609_39185_amd"), "-lssmq",
           "-L", os.path.join(ROOT, "oracle"), "-lssmq_oracle",
           "-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-lm",
           "-Wl,-rpath,$ORIGIN/../paper_2609_39185_amd:$ORIGIN/../oracle:" + os.path.join(ROCM, "lib")]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, BINARY)
    return BINARY


if __name__ == "__main__":
    print(build(verbose=True))
