"""Seeded random configurations of the fused step, each against the oracle at the
bar of the other parity tests: formats, rules, Mamba-1 and Mamba-2 shapes (rows
of 1 to 64 chunks, heads of one row to several thousand entries), scale groups
from 16 entries to one head, dither blocks from 1 to 4096, and arbitrary seed,
layer, step and (16-aligned) entry_base."""
import numpy as np
import pytest

from ._parity import check_step

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ssmq():
    import paper_2609_39185_amd as m
    m.library()
    return m

ENTRIES_PER_CHUNK = {"fp16": 8, "bf16": 8, "fp32": 4, "e4m3": 16, "int8": 16, "int4": 16}
SCALED = ("e4m3", "int8", "int4")


def _config(i):
    rng = np.random.default_rng(1000 + i)
    fmt = ["fp16", "bf16", "fp32", "e4m3", "int8", "int4"][i % 6]
    rule = ["rtn", "sr", "weyl", "philox"][(i // 6) % 4]
    if rng.random() < 0.3:
        family, headdim, dstate, ngroups = "mamba1", 1, 16, 1
        nheads = int(rng.integers(16, 400))
        batch = int(rng.integers(1, 4))
    else:
        family = "mamba2"
        v = ENTRIES_PER_CHUNK[fmt]
        dstate = int(rng.choice([d for d in (16, 32, 64, 128, 256) if d % v == 0 and d // v <= 64]))
        headdim = int(rng.choice([1, 8, 32, 64]))
        ngroups = int(rng.choice([1, 2]))
        nheads = ngroups * int(rng.integers(1, 5))
        batch = int(rng.integers(1, 4))
    head = headdim * dstate
    q = {"dither_block": int(rng.choice([1, 16, 128, 4096])),
         "dither_seed": int(rng.integers(0, 2 ** 32)), "layer": int(rng.integers(0, 64)),
         "step": int(rng.integers(0, 2 ** 32)), "entry_base": 16 * int(rng.integers(0, 2 ** 20))}
    if fmt in SCALED:
        groups = [g for g in (16, 32, 64, 128, 256, 512, 1024) if head % g == 0]
        per_head_ok = head % 16 == 0 and (
            (head <= 1024 and head & (head - 1) == 0)
            or (family == "mamba2" and head in (4096, 8192, 16384)))
        if per_head_ok:
            groups.append(0)
        q["scale_group"] = int(rng.choice(groups))
    return fmt, rule, (family, batch, nheads, headdim, dstate, ngroups), q


@pytest.mark.parametrize("i", range(96))
def test_random_config(ssmq, i):
    fmt, rule, shape, q = _config(i)
    check_step(fmt, rule, *shape, seed=int(5000 + i), what=f"random config {i}", **q)
