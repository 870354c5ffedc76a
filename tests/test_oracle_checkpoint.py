"""Pins of the oracle's checkpoint write on an fp32 state (Section 6.5 "Periodic
checkpointing"; Appendix B "Decode regime", CC = 8): one fp32 step of eq. (rec),
then every value rounded onto a format's grid and kept as fp32.

Expected values: the fp32 step (pinned against float64 in test_oracle_step.py)
followed by numpy / torch casts (RTN) or numpy's block-scale arithmetic (INT8);
dithered writes land on the grid within one step of the unrounded value.
"""
import numpy as np
import pytest
import torch

from paper_2609_39185_amd import workloads as wl

SHAPE = ("mamba2", 2, 4, 8, 32, 2)


def _inputs(seed):
    family, b, h, p, n, g = SHAPE
    A, D = wl.layer_params(family, h, n, seed)
    x, dt, B, C = wl.step_inputs(b, h, p, n, g, seed + 1)
    h0 = (np.random.default_rng(seed).standard_normal((b, h, p, n)) * 0.2).astype(np.float32)
    return h0, [t.numpy() for t in (x, dt, A, B, C, D)]


def _fp32_step(orc, h0, args):
    new, _, y, hnew = orc.state_update("fp32", "rtn", h0.view(np.uint32), None, *args)
    return hnew, y


@pytest.mark.parametrize("fmt,cast", [("fp16", torch.float16), ("bf16", torch.bfloat16)])
def test_rtn_checkpoint_is_the_cast_of_the_fp32_step(orc, fmt, cast):
    h0, args = _inputs(3)
    hnew, y = _fp32_step(orc, h0, args)
    st, sc, y2 = orc.state_update_fp32_grid(fmt, "rtn", h0, *args)
    want = torch.from_numpy(hnew).to(cast).float().numpy()
    assert sc is None
    assert np.array_equal(st, want)
    assert np.array_equal(y, y2)


def test_int8_rtn_checkpoint_block_scale(orc):
    h0, args = _inputs(5)
    hnew, _ = _fp32_step(orc, h0, args)
    st, sc, _ = orc.state_update_fp32_grid("int8", "rtn", h0, *args, group=16)
    g = hnew.reshape(-1, 16)
    s = (np.abs(g).max(axis=1) / np.float32(127)).astype(np.float32)
    r = (np.float32(1) / s).astype(np.float32)
    k = np.clip(np.rint((g * r[:, None]).astype(np.float32)), -127, 127).astype(np.float32)
    assert np.array_equal(sc, s)
    assert np.array_equal(st.reshape(-1, 16), (k * s[:, None]).astype(np.float32))


@pytest.mark.parametrize("rule", ["sr", "weyl", "philox"])
def test_dithered_checkpoint_lands_within_a_step(orc, rule):
    h0, args = _inputs(7)
    hnew, _ = _fp32_step(orc, h0, args)
    st, _, _ = orc.state_update_fp32_grid("fp16", rule, h0, *args, step=9, layer=2)
    lo = np.float16(hnew)
    f = lo.astype(np.float32)
    # on the fp16 grid, and one of the two neighbours of the unrounded value
    assert np.array_equal(st.astype(np.float16).astype(np.float32), st)
    down = np.where(f > hnew, np.nextafter(lo, np.float16(-np.inf)), lo).astype(np.float32)
    up = np.where(f < hnew, np.nextafter(lo, np.float16(np.inf)), lo).astype(np.float32)
    assert np.all((st == down) | (st == up))
    # and not always the nearer one (the dither moves some values up, some down)
    assert 0.05 < np.mean(st != f) < 0.95
