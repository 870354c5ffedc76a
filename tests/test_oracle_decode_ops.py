"""Pins of the oracle's decode-step operations around the update (Appendix B
"Runners": conv and gating as in the Mamba reference): dt' = softplus(dt + bias),
y' = y * silu(z), and the causal depthwise conv1d state update. Expected values
come from numpy (logaddexp) and torch (silu, conv1d) in float64."""
import numpy as np
import torch

from paper_2609_39185_amd import workloads as wl


def _inputs(seed, family="mamba2", shape=(2, 4, 8, 32, 2)):
    b, h, p, n, g = shape
    A, D = wl.layer_params(family, h, n, seed)
    x, dt, B, C = wl.step_inputs(b, h, p, n, g, seed + 1)
    rng = np.random.default_rng(seed)
    h0 = (rng.standard_normal((b, h, p, n)) * 0.2).astype(np.float32)
    bias = rng.uniform(-6, 3, h).astype(np.float32)
    z = rng.standard_normal((b, h, p)).astype(np.float32)
    return h0, [t.numpy() for t in (x, dt, A, B, C, D)], bias, z


def test_softplus_dt_and_gate(orc):
    h0, (x, dt_raw, A, B, C, D), bias, z = _inputs(3)
    dt_raw = (dt_raw * 10 - 3).astype(np.float32)          # raw step sizes, both signs
    dt_raw[0, 0] = 30.0                                     # above the softplus threshold
    # softplus arguments v = dt + bias of 0.5, 5, 19.5 and 20.5 (both sides of 20)
    for (b, h), v in (((0, 1), 0.5), ((0, 2), 5.0), ((1, 0), 19.5), ((1, 3), 20.5)):
        dt_raw[b, h] = np.float32(v) - bias[h]
    v = (dt_raw + bias[None, :]).astype(np.float32)
    dt_eff = np.where(v > 20, v, np.logaddexp(0.0, v.astype(np.float64))).astype(np.float32)
    codes = h0.view(np.uint32)
    new_a, _, y_a, h_a = orc.state_update("fp32", "rtn", codes, None, x, dt_raw, A, B, C, D,
                                          dt_bias=bias, dt_softplus=True, z=z)
    new_b, _, y_b, h_b = orc.state_update("fp32", "rtn", codes, None, x, dt_eff, A, B, C, D)
    assert np.array_equal(h_a, h_b)                        # the update saw dt' exactly
    silu = torch.nn.functional.silu(torch.from_numpy(z.astype(np.float64))).numpy()
    assert np.allclose(y_a, y_b * silu, rtol=1e-13, atol=1e-300)
    # without softplus the bias is only added
    _, _, _, h_c = orc.state_update("fp32", "rtn", codes, None, x, dt_raw, A, B, C, D,
                                    dt_bias=bias)
    _, _, _, h_d = orc.state_update("fp32", "rtn", codes, None, x, v, A, B, C, D)
    assert np.array_equal(h_c, h_d)


def test_conv1d_update(orc):
    rng = np.random.default_rng(9)
    batch, channels, width = 3, 40, 4
    state = rng.standard_normal((batch, channels, width)).astype(np.float32)
    x = rng.standard_normal((batch, channels)).astype(np.float32)
    w = rng.standard_normal((channels, width)).astype(np.float32)
    bias = rng.standard_normal(channels).astype(np.float32)
    for act in (False, True):
        st, out = orc.conv1d_update(state, x, w, bias, act=act)
        window = np.concatenate([state[:, :, 1:], x[:, :, None]], axis=2)
        assert np.array_equal(st, window)
        ref = torch.nn.functional.conv1d(torch.from_numpy(window.astype(np.float64)),
                                         torch.from_numpy(w.astype(np.float64))[:, None, :],
                                         torch.from_numpy(bias.astype(np.float64)),
                                         groups=channels)[:, :, 0]
        if act:
            ref = torch.nn.functional.silu(ref)
        assert np.allclose(out, ref.numpy(), rtol=1e-13, atol=1e-13)
    st, out = orc.conv1d_update(state, x, w, None, act=False)
    assert np.allclose(out, (window.astype(np.float64) * w[None]).sum(-1), rtol=1e-13)
