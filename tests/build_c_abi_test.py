"""Build the test programs (test infrastructure): tests/c_abi_step, a C program
that drives libssmq.so through include/ssmq.h and checks it against the oracle
library, and tests/scale_math_check, a HIP program that checks the group-scale
division and reciprocal of the device code for every fp32 value in range."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SOURCE = os.path.join(HERE, "c_abi_step.c")
BINARY = os.path.join(HERE, "c_abi_step")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
SCALE_SOURCE = os.path.join(HERE, "scale_math_check.hip")
SCALE_BINARY = os.path.join(HERE, "scale_math_check")


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
    build_scale_check(verbose)
    return BINARY


def build_scale_check(verbose: bool = False) -> str:
    """hipcc with the library's own floating-point flags (correctly rounded fp32
    division, no contraction, denormals kept, no packed fp32)."""
    tmp = SCALE_BINARY + ".tmp"
    cmd = [os.path.join(ROCM, "bin", "hipcc"), "--offload-arch=gfx950", "-O3", "-std=c++17",
           "-ffp-contract=off", "-fno-gpu-flush-denormals-to-zero",
           "-fhip-fp32-correctly-rounded-divide-sqrt",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I", os.path.join(ROOT, "paper_2609_39185_amd", "csrc"), SCALE_SOURCE, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, SCALE_BINARY)
    return SCALE_BINARY


if __name__ == "__main__":
    print(build(verbose=True))
