"""GPU parity of the checkpoint write on an fp32 state (SSMQ_FLAG_FP32_STATE;
Section 6.5 "Periodic checkpointing", Appendix B "Decode regime" CC = 8) against the
oracle, through the C ABI: each fp32 value rounded onto a format's grid."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_39185_amd import workloads as wl

from ._parity import DEV, MAX_DIFFER_FRACTION, code_stats, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ssmq():
    import paper_2609_39185_amd as m
    m.library()
    return m


def _codes_of(fmt, values, scale, group):
    """Grid values -> the format's codes (exact: every value is on the grid)."""
    v = np.asarray(values, np.float32).ravel()
    if fmt == "fp16":
        return v.astype(np.float16).view(np.uint16)
    if fmt == "bf16":
        return torch.from_numpy(v).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    s = np.repeat(np.asarray(scale, np.float32), group)
    q = np.where(s > 0, v / np.where(s > 0, s, 1), 0).astype(np.float32)
    if fmt == "e4m3":
        return torch.from_numpy(q).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    k = np.rint(q).astype(np.int64)
    return (k & (0xFF if fmt == "int8" else 0xF)).astype(np.uint8)


CASES = [("fp16", 0, 16), ("bf16", 0, 128), ("e4m3", 16, 16), ("e4m3", 128, 128),
         ("int8", 16, 16), ("int8", 128, 128), ("int4", 16, 16)]


@pytest.mark.parametrize("fmt,group,block", CASES)
@pytest.mark.parametrize("rule", ["rtn", "sr", "weyl", "philox"])
@pytest.mark.parametrize("family,shape", [("mamba2", (2, 4, 32, 128, 2)), ("mamba1", (3, 96, 1, 16, 1))])
def test_checkpoint_write(ssmq, fmt, group, block, rule, family, shape):
    b, h, p, n, g = shape
    if n < max(group, 16):
        group = 16
    say(f"case checkpoint {family} {fmt} g{group} {rule} {shape}")
    A, D = wl.layer_params(family, h, n, 90)
    x, dt, B, C = wl.step_inputs(b, h, p, n, g, 91)
    h0 = (np.random.default_rng(92).standard_normal((b, h, p, n)) * 0.3).astype(np.float32)
    st = torch.from_numpy(h0).to(DEV)
    sc = torch.zeros(h0.size // group, device=DEV) if fmt in oracle.SCALED else None
    y = torch.empty((b, h, p), device=DEV)
    ssmq.state_update(st, sc, x.to(DEV), dt.to(DEV), A.to(DEV), B.to(DEV), C.to(DEV), D.to(DEV), y,
                      rule=rule, fmt=fmt, dither_block=block, scale_group=group, step=5, layer=1,
                      fp32_state=True)
    torch.cuda.synchronize()
    want, wsc, wy = oracle.state_update_fp32_grid(fmt, rule, h0, x.numpy(), dt.numpy(), A.numpy(),
                                                  B.numpy(), C.numpy(), D.numpy(), step=5, layer=1,
                                                  block=block, group=group)
    got = st.cpu().numpy()
    if sc is not None:
        np.testing.assert_array_equal(sc.cpu().numpy(), wsc)
    nd, ulp = code_stats(fmt, _codes_of(fmt, got, None if sc is None else sc.cpu().numpy(), group),
                         _codes_of(fmt, want, wsc, group))
    say(f"  {nd} of {got.size} entries differ (max {ulp} steps)")
    assert nd <= MAX_DIFFER_FRACTION * got.size + 1 and ulp <= 1
    mag = np.abs(np.repeat(C.numpy().astype(np.float64), h // g, axis=1)[:, :, None, :]).sum(-1)
    assert np.all(np.abs(y.cpu().numpy() - wy) <= 1e-5 * (mag * np.abs(want).max() + np.abs(wy) + 1e-30))


def test_cc8_schedule_matches_oracle(ssmq):
    """A CC = 8 schedule on a small Mamba-1 cache: fp32 steps, every 8th a Weyl
    checkpoint onto INT8 block 16; the GPU state is reset to the oracle's after
    each step so a one-off difference cannot compound."""
    b, d, N = 1, 256, 16
    A, D = wl.layer_params("mamba1", d, N, 93)
    h = (np.random.default_rng(94).standard_normal((b, d, 1, N)) * 0.2).astype(np.float32)
    st = torch.from_numpy(h).to(DEV)
    y = torch.empty((b, d, 1), device=DEV)
    for t in range(1, 33):
        x, dt, B, C = wl.step_inputs(b, d, 1, N, 1, 200 + t)
        args = [v.to(DEV) for v in (x, dt, A, B, C, D)]
        if t % 8 == 0:
            ssmq.state_update(st, None, *args, y, rule="weyl", fmt="int8", scale_group=16, step=t,
                              fp32_state=True)
            want, _, _ = oracle.state_update_fp32_grid("int8", "weyl", h, x.numpy(), dt.numpy(),
                                                       A.numpy(), B.numpy(), C.numpy(), D.numpy(),
                                                       step=t, group=16)
        else:
            ssmq.state_update(st.view(torch.int32), None, *args, y, rule="rtn", fmt="fp32", step=t)
            new, _, _, _ = oracle.state_update("fp32", "rtn", h.view(np.uint32), None, x.numpy(),
                                               dt.numpy(), A.numpy(), B.numpy(), C.numpy(), D.numpy(),
                                               step=t)
            want = new.view(np.float32)
        torch.cuda.synchronize()
        got = st.cpu().numpy()
        differ = np.mean(got != want)
        assert differ <= 1e-3, (t, differ)
        h = want.copy()
        st.copy_(torch.from_numpy(h))
