"""The device's group-scale arithmetic, exhaustively: tests/scale_math_check
(built by __graft_entry__.build()) checks group_scale for every fp32 maximum in
[2^-112, FLT_MAX] and each qmax (448, 127, 7) against the device's correctly
rounded division, and recip_scale for every fp32 value in [2^-126, 2^126)
against 1 / s, as a child process."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu
BINARY = os.path.join(os.path.dirname(os.path.abspath(__file__)), "scale_math_check")


def test_scale_division_and_reciprocal_for_every_value():
    assert os.path.exists(BINARY), "tests/scale_math_check is missing: run __graft_entry__.build()"
    r = subprocess.run([BINARY], capture_output=True, text=True, timeout=120)
    print(r.stdout, r.stderr, flush=True)
    counts = {ln.split()[0]: (int(ln.split()[1]), int(ln.split()[2]))
              for ln in r.stdout.splitlines() if len(ln.split()) == 3}
    assert r.returncode == 0
    assert counts["scale_e4m3"] == (240 << 23, 0)
    assert counts["scale_int8"] == (240 << 23, 0)
    assert counts["scale_int4"] == (240 << 23, 0)
    assert counts["recip"] == (252 << 23, 0)
