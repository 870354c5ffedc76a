"""GPU parity of the decode-step operations around the update (Appendix B
"Runners"): dt' = softplus(dt + dt_bias) and y' = y * silu(z) fused into the
update (ssmq_state_update_ex), and the causal depthwise conv1d decode update
(ssmq_conv1d_update), against the oracle through the C ABI."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_39185_amd import workloads as wl

from ._parity import DEV, Bar, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ssmq():
    import paper_2609_39185_amd as m
    m.library()
    return m


CASES = [("bf16", "weyl", "mamba2", (2, 4, 64, 128, 2), {"dither_block": 128}),
         ("e4m3", "sr", "mamba2", (2, 4, 64, 128, 2), {"dither_block": 128}),
         ("int8", "weyl", "mamba2", (2, 4, 64, 128, 2), {"scale_group": 128, "dither_block": 128}),
         ("fp16", "weyl", "mamba1", (3, 200, 1, 16, 1), {}),
         ("int4", "philox", "mamba1", (2, 96, 1, 16, 1), {"scale_group": 16})]


@pytest.mark.parametrize("fmt,rule,family,shape,q", CASES)
@pytest.mark.parametrize("softplus,bias,gate", [(True, True, True), (True, False, False),
                                                (False, True, False), (False, False, True)])
def test_step_with_dt_bias_softplus_and_gate(ssmq, fmt, rule, family, shape, q, softplus, bias,
                                             gate):
    b, h, p, n, g = shape
    say(f"case decode ops {fmt} {rule} {family} {shape} softplus={softplus} bias={bias} gate={gate}")
    A, D = wl.layer_params(family, h, n, 120)
    x, dt, B, C = wl.step_inputs(b, h, p, n, g, 121)
    rng = np.random.default_rng(122)
    dt_raw = torch.from_numpy((rng.standard_normal((b, h)) * 2 - 3).astype(np.float32))
    dt_bias = torch.from_numpy(rng.uniform(-4, 1, h).astype(np.float32)) if bias else None
    z = torch.from_numpy(rng.standard_normal((b, h, p)).astype(np.float32)) if gate else None
    if not softplus:
        dt_raw = dt_raw.abs() * 0.05
    codes, scale = wl.initial_state(fmt, b, h, p, n, 123, group=q.get("scale_group", 0))
    st = codes.to(DEV)
    sc = None if scale is None else scale.to(DEV)
    y = torch.empty((b, h, p), device=DEV)
    ssmq.state_update(st, sc, x.to(DEV), dt_raw.to(DEV), A.to(DEV), B.to(DEV), C.to(DEV),
                      D.to(DEV), y, rule=rule, fmt=fmt, step=6, layer=2,
                      dt_bias=None if dt_bias is None else dt_bias.to(DEV), dt_softplus=softplus,
                      z=None if z is None else z.to(DEV), **q)
    torch.cuda.synchronize()
    r_codes, r_scale, r_y, r_h = oracle.state_update(
        fmt, rule, wl.to_numpy_codes(fmt, codes), None if scale is None else scale.numpy(),
        x.numpy(), dt_raw.numpy(), A.numpy(), B.numpy(), C.numpy(), D.numpy(), step=6, layer=2,
        block=q.get("dither_block", 16), group=q.get("scale_group", 0),
        dt_bias=None if dt_bias is None else dt_bias.numpy(), dt_softplus=softplus,
        z=None if z is None else z.numpy())
    bar = Bar(fmt, "decode ops").codes(wl.to_numpy_codes(fmt, st.cpu()), r_codes)
    if sc is not None:
        bar.scales(sc.cpu().numpy(), r_scale)
    Ch = np.repeat(C.numpy().astype(np.float64), h // g, axis=1)[:, :, None, :]
    mag = np.abs(Ch * r_h.astype(np.float64)).sum(-1) + np.abs(D.numpy()[None, :, None] * x.numpy())
    if z is not None:
        mag = mag * np.abs(torch.nn.functional.silu(z.double()).numpy())
    bar.y(y.cpu().numpy(), r_y, mag).check()


@pytest.mark.parametrize("batch,channels,width", [(1, 7, 4), (3, 1536, 4), (2, 8192 + 2 * 8 * 128, 4),
                                                  (5, 33, 1), (2, 100, 7), (0, 16, 4)])
@pytest.mark.parametrize("act", [True, False])
def test_conv1d_update(ssmq, batch, channels, width, act):
    say(f"case conv1d b{batch} c{channels} w{width} act={act}")
    rng = np.random.default_rng(channels + width)
    state = rng.standard_normal((batch, channels, width)).astype(np.float32)
    x = rng.standard_normal((batch, channels)).astype(np.float32)
    w = rng.standard_normal((channels, width)).astype(np.float32)
    bias = rng.standard_normal(channels).astype(np.float32) if width != 7 else None
    st = torch.from_numpy(state).to(DEV)
    out = torch.full((batch, channels), float("nan"), device=DEV)
    ssmq.conv1d_update(st, torch.from_numpy(x).to(DEV), torch.from_numpy(w).to(DEV),
                       None if bias is None else torch.from_numpy(bias).to(DEV), out, act=act)
    torch.cuda.synchronize()
    r_state, r_out = oracle.conv1d_update(state, x, w, bias, act=act)
    assert np.array_equal(st.cpu().numpy(), r_state)
    window = r_state.astype(np.float64)
    mag = np.abs(window * w[None].astype(np.float64)).sum(-1)
    if bias is not None:
        mag = mag + np.abs(bias.astype(np.float64))[None]
    err = np.abs(out.cpu().numpy().astype(np.float64) - r_out)
    assert np.all(err <= 1e-5 * (mag + np.abs(r_out)) + 1e-30), err.max() if err.size else 0


@pytest.mark.parametrize("fmt,rule,group", [("bf16", "weyl", 0), ("int8", "sr", 128)])
def test_composed_mamba2_decode_step(ssmq, fmt, rule, group):
    """One Mamba-2 decode step around the state (Appendix B "Runners"): the conv1d
    update over the x, B and C channels with silu, the split into x, B, C, and the
    fused update with dt + dt_bias, softplus and the z gate. Each stage is checked
    against the oracle on the inputs the GPU stage actually received."""
    b, H, P, N, G, W = 3, 8, 64, 128, 2, 4
    di = H * P
    ch = di + 2 * G * N
    rng = np.random.default_rng(140)
    conv_state = rng.standard_normal((b, ch, W)).astype(np.float32)
    xbc = rng.standard_normal((b, ch)).astype(np.float32)
    weight = (rng.standard_normal((ch, W)) * 0.5).astype(np.float32)
    bias = (rng.standard_normal(ch) * 0.1).astype(np.float32)
    dt_raw = (rng.standard_normal((b, H)) - 3).astype(np.float32)
    dt_bias = rng.uniform(-2, 0, H).astype(np.float32)
    z = rng.standard_normal((b, H, P)).astype(np.float32)
    A, D = wl.layer_params("mamba2", H, N, 141)
    codes, scale = wl.initial_state(fmt, b, H, P, N, 142, group=group)
    say(f"case composed decode step {fmt} {rule}")

    cs = torch.from_numpy(conv_state).to(DEV)
    out = torch.empty((b, ch), device=DEV)
    ssmq.conv1d_update(cs, torch.from_numpy(xbc).to(DEV), torch.from_numpy(weight).to(DEV),
                       torch.from_numpy(bias).to(DEV), out, act=True)
    x = out[:, :di].reshape(b, H, P).contiguous()
    B = out[:, di:di + G * N].reshape(b, G, N).contiguous()
    C = out[:, di + G * N:].reshape(b, G, N).contiguous()
    st = codes.to(DEV)
    sc = None if scale is None else scale.to(DEV)
    y = torch.empty((b, H, P), device=DEV)
    ssmq.state_update(st, sc, x, torch.from_numpy(dt_raw).to(DEV), A.to(DEV), B, C, D.to(DEV), y,
                      rule=rule, fmt=fmt, dither_block=128, scale_group=group, step=9, layer=1,
                      dt_bias=torch.from_numpy(dt_bias).to(DEV), dt_softplus=True,
                      z=torch.from_numpy(z).to(DEV))
    torch.cuda.synchronize()

    r_state, r_out = oracle.conv1d_update(conv_state, xbc, weight, bias, act=True)
    assert np.array_equal(cs.cpu().numpy(), r_state)
    got_out = out.cpu().numpy().astype(np.float64)
    mag = np.abs(r_state.astype(np.float64) * weight[None].astype(np.float64)).sum(-1) + np.abs(bias)
    assert np.all(np.abs(got_out - r_out) <= 1e-5 * (mag + np.abs(r_out)))
    xs, Bs, Cs = (v.cpu().numpy() for v in (x, B, C))
    r_codes, r_scale, r_y, r_h = oracle.state_update(
        fmt, rule, wl.to_numpy_codes(fmt, codes), None if scale is None else scale.numpy(), xs,
        dt_raw, A.numpy(), Bs, Cs, D.numpy(), step=9, layer=1, block=128, group=group,
        dt_bias=dt_bias, dt_softplus=True, z=z)
    bar = Bar(fmt, "composed step").codes(wl.to_numpy_codes(fmt, st.cpu()), r_codes)
    if sc is not None:
        bar.scales(sc.cpu().numpy(), r_scale)
    Ch = np.repeat(Cs.astype(np.float64), H // G, axis=1)[:, :, None, :]
    mag = (np.abs(Ch * r_h.astype(np.float64)).sum(-1) + np.abs(D.numpy()[None, :, None] * xs))
    mag = mag * np.abs(torch.nn.functional.silu(torch.from_numpy(z).double()).numpy())
    bar.y(y.cpu().numpy(), r_y, mag).check()
