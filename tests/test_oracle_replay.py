"""Pins of the oracle's open-loop replay (CPU only).

The replay (Appendix B "Open-loop replay"; Section 6.2) iterates the FP32
reference h_t = a_t h_{t-1} + w_t and the stored state hq_t = Q(a_t hq_{t-1} + w_t)
from recorded decays and writes. Expected values come from Proposition 1 and
Corollary 1 (a = 1 and a constant write: the final error is a count of
thresholds, Section 3), from the fused step's own trajectory on the same
decays and writes (a state update whose decay and write are the trace's), and
from the exact invariance of block-scaled rounding under power-of-two scaling.
"""
import numpy as np
import pytest

from paper_2609_39185_amd import workloads as wl

TWO24 = 1 << 24


def _prop1_traces(n, T, seed=0):
    """fp16 binade [1, 2): step s = 2^-10, write w_i = f_i s with f_i = k_i / 2^13,
    decay a = 1; h stays below 2 for T steps."""
    rng = np.random.default_rng(seed)
    k = rng.integers(1, 3000, n)                     # f < 0.37
    s = 2.0 ** -10
    w = (k / 8192.0 * s).astype(np.float32)          # exact: k 2^-23
    a = np.ones((T, n), np.float32)
    h0 = np.ones(n, np.float32)
    return k, s, a, np.broadcast_to(w, (T, n)).copy(), h0


@pytest.mark.parametrize("rule", ["rtn", "sr", "weyl", "philox"])
def test_proposition1_count_through_the_replay(orc, rule):
    """e_T = hq_T - h_T = -s (#{t <= T: u_t < 1 - f} - T (1 - f)) exactly; for RTN
    (u = 1/2, f < 1/2) that is -s T f: the write is erased every step."""
    n, T = 64, 1500
    k, s, a, w, h0 = _prop1_traces(n, T)
    out = orc.replay("fp16", rule, h0, a, w, block=16, seed=1, layer=3, step=100)
    hq_T = orc.dequantize("fp16", out["codes"], None, 0).astype(np.float64)
    h_T = out["h_final"].astype(np.float64)
    assert np.array_equal(h_T, 1.0 + T * k * 2.0 ** -23)   # the reference is exact here
    for i in range(n):
        if rule == "rtn":
            below = T                                       # u = 1/2 < 1 - f always
        else:
            U = np.array([orc.thresholds(rule, 1, 3, 100 + t, i, 1, 16)[0]
                          for t in range(1, T + 1)], np.int64)
            below = int(np.count_nonzero(U < (8192 - k[i]) * (TWO24 // 8192)))
        want = -s * (below - T * (1 - k[i] / 8192.0))
        assert hq_T[i] - h_T[i] == want, (i, hq_T[i] - h_T[i], want)
    # the last block's error sum holds every step's squared error
    assert np.all(out["err"][0] > 0)


def test_fp32_replay_is_the_reference(orc):
    rng = np.random.default_rng(4)
    n, T = 96, 40
    a = rng.uniform(0.5, 1.0, (T, n)).astype(np.float32)
    w = rng.standard_normal((T, n)).astype(np.float32)
    h0 = rng.standard_normal(n).astype(np.float32)
    out = orc.replay("fp32", "weyl", h0, a, w, block_steps=7)
    assert np.all(out["err"] == 0.0)
    assert np.array_equal(out["codes"].view(np.float32), out["h_final"])
    h = h0.astype(np.float64)
    ref = np.zeros(n)
    for t in range(T):                     # a h + w in double, one fp32 rounding each step
        h = (a[t].astype(np.float64) * h + w[t]).astype(np.float32).astype(np.float64)
        ref += h * h
    # fl32 of the double evaluation equals the fp32 fma unless the double sum rounded
    # on a tie of fp32: compare within one fp32 ulp per step
    assert np.allclose(out["h_final"], h, rtol=T * 2.0 ** -23)
    assert np.allclose(out["ref"].sum(0), ref, rtol=1e-5)


@pytest.mark.parametrize("fmt", ["fp16", "bf16"])
@pytest.mark.parametrize("rule", ["rtn", "sr", "weyl", "philox"])
def test_replay_follows_the_fused_step(orc, fmt, rule):
    """A Mamba-1 layer's decays a_t = exp(dt_t A) and writes w_t = dt_t x_t B_t, taken
    from the fused step itself (an fp32 state of ones with x = 0 gives a_t, a zero
    state gives w_t), replay to exactly the codes the fused step writes when it is
    iterated on the same inputs."""
    b, d, N, T = 2, 24, 16, 30
    A, D = wl.layer_params("mamba1", d, N, 3)
    A = A.numpy()
    ones = np.ones((b, d, 1, N), np.float32).view(np.uint32)
    zeros = np.zeros((b, d, 1, N), np.float32).view(np.uint32)
    a_tr, w_tr, xs = [], [], []
    for t in range(T):
        x, dt, B, C = (v.numpy() for v in wl.step_inputs(b, d, 1, N, 1, 100 + t))
        xs.append((x, dt, B, C))
        at, _, _, _ = orc.state_update("fp32", "rtn", ones, None, np.zeros_like(x), dt, A, B, C, None)
        wt, _, _, _ = orc.state_update("fp32", "rtn", zeros, None, x, dt, A, B, C, None)
        a_tr.append(at.view(np.float32).ravel())
        w_tr.append(wt.view(np.float32).ravel())
    h0 = (np.random.default_rng(9).standard_normal(b * d * N) * 0.3).astype(np.float32)
    out = orc.replay(fmt, rule, h0, np.stack(a_tr), np.stack(w_tr), block=16, seed=2, layer=5,
                     step=40, block_steps=T)
    codes, _ = orc.requantize(fmt, rule, h0, block=16, seed=2, layer=5, step=40)
    codes = codes.reshape(b, d, 1, N)
    err = np.zeros(b * d * N)
    href = h0.astype(np.float32)
    for t in range(T):
        x, dt, B, C = xs[t]
        codes, _, _, _ = orc.state_update(fmt, rule, codes, None, x, dt, A, B, C, None, block=16,
                                          seed=2, layer=5, step=40 + t + 1)
        href = np.array(orc.state_update("fp32", "rtn", href.reshape(b, d, 1, N).view(np.uint32),
                                         None, x, dt, A, B, C, None)[0]).view(np.float32).ravel()
        hq = orc.dequantize(fmt, codes, None, 0).ravel().astype(np.float64)
        err += (hq - href.astype(np.float64)) ** 2
    assert np.array_equal(out["codes"], codes.ravel())
    assert np.array_equal(out["h_final"], href)
    assert np.allclose(out["err"][0], err, rtol=1e-12, atol=0)


@pytest.mark.parametrize("fmt", ["int8", "int4", "e4m3"])
@pytest.mark.parametrize("rule", ["rtn", "weyl", "sr"])
def test_power_of_two_scaling_is_exact(orc, fmt, rule):
    """Scaling h0 and every write by 2^k scales every stored and reference value by
    2^k exactly (the block scale absorbs it, the codes relative to it do not move),
    so the codes are unchanged and the error sums scale by 4^k."""
    rng = np.random.default_rng(7)
    n, T, group = 128, 50, 16
    a = np.exp(-rng.uniform(0.0, 0.3, (T, n))).astype(np.float32)
    w = (rng.standard_normal((T, n)) * 0.1).astype(np.float32)
    h0 = rng.standard_normal(n).astype(np.float32)
    base = orc.replay(fmt, rule, h0, a, w, group=group, block=16, block_steps=10)
    for k in (-3, 4):
        f = np.float32(2.0 ** k)
        sc = orc.replay(fmt, rule, h0 * f, a, w * f, group=group, block=16, block_steps=10)
        assert np.array_equal(sc["codes"], base["codes"])
        assert np.array_equal(sc["err"], base["err"] * 4.0 ** k)
        assert np.array_equal(sc["ref"], base["ref"] * 4.0 ** k)
        assert np.array_equal(sc["scale"], base["scale"] * f)


def test_decay_zero_rounds_each_write(orc):
    """a = 0: hq_t = Q_t(w_t) and h_t = w_t, so each step's error is the requantize error."""
    rng = np.random.default_rng(8)
    n, T, group = 64, 6, 16
    a = np.zeros((T, n), np.float32)
    w = rng.standard_normal((T, n)).astype(np.float32)
    out = orc.replay("int8", "weyl", np.zeros(n, np.float32), a, w, group=group, block=16,
                     step=20, block_steps=1)
    for t in range(T):
        c, s = orc.requantize("int8", "weyl", w[t], group=group, block=16, step=20 + t + 1)
        hq = orc.dequantize("int8", c, s, group).astype(np.float64)
        assert np.array_equal(out["err"][t], (hq - w[t].astype(np.float64)) ** 2)
        assert np.array_equal(out["ref"][t], w[t].astype(np.float64) ** 2)


def test_blocks_partition_the_steps(orc):
    rng = np.random.default_rng(1)
    n, T = 32, 23
    a = rng.uniform(0.8, 1.0, (T, n)).astype(np.float32)
    w = (rng.standard_normal((T, n)) * 0.01).astype(np.float32)
    h0 = rng.standard_normal(n).astype(np.float32)
    per_step = orc.replay("bf16", "sr", h0, a, w, block=16, block_steps=1)
    blocks = orc.replay("bf16", "sr", h0, a, w, block=16, block_steps=5)
    assert blocks["err"].shape == (5, n)
    for k in range(5):
        assert np.allclose(blocks["err"][k], per_step["err"][5 * k:5 * k + 5].sum(0), rtol=1e-14)
        assert np.allclose(blocks["ref"][k], per_step["ref"][5 * k:5 * k + 5].sum(0), rtol=1e-14)
