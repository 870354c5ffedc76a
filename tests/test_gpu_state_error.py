"""The state-error study (quantized states against an FP32 twin in lockstep,
Appendix B "Open-loop replay" and "Decode regime") on the GPU.

1. On a small Mamba-1 case the study's per-block errors equal those of the same
   replay done by the oracle on the same inputs.
2. In the synthetic workload's regime (updates much larger than an fp16 step, so
   the rounded fraction f is effectively uniform and independent across steps) the
   errors follow the per-write noise lemma (Section 3): RTN's mean squared error is
   half of SR's, and two SR seeds agree. For a dither with threshold u the error of
   one write splits into a bias (u - 1/2) s, variance s^2/12 over u, and a zero-mean
   part of variance s^2/12 over f. SR's biases are independent from step to step;
   the Weyl thresholds advance by the golden increment, so consecutive biases are
   anti-correlated and largely cancel under the decay. The accumulated Weyl error
   therefore lies between RTN's (the zero-mean part alone) and SR's.
"""
import dataclasses
import os
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2609_39185_amd import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def _say(msg):
    print(msg, flush=True)


def _small(batch, d, layers, steps):
    return dataclasses.replace(wl.WORKLOADS["m1_small"], batch=batch, nheads=d, layers=layers,
                               steps=steps)


def _oracle_replay(w, L, steps, block, init, inputs, rules, fmt="fp16", group=16, cc=0):
    """The study redone by the oracle on the same inputs; returns {run: errors per block}."""
    b, d, N = w.batch, w.nheads, w.dstate
    scaled = fmt in oracle.SCALED
    g = group if scaled else 0
    runs = list(rules) + ([(r, sd, cc) for r, sd in (("rtn", 0), ("sr", 0), ("weyl", 0))]
                          if cc > 0 else [])
    codes0 = [wl.to_numpy_codes(fmt, init["codes0"][ell]) for ell in range(L)]
    scale0 = [init["scale0"][ell].numpy() if scaled else None for ell in range(L)]
    h0 = [oracle.dequantize(fmt, codes0[ell], scale0[ell], g).reshape(b, d, 1, N)
          for ell in range(L)]
    st = {r: [(h0[ell].copy() if len(r) == 3 else (codes0[ell].copy(), None if scale0[ell] is None
               else scale0[ell].copy())) for ell in range(L)] for r in runs}
    twin = [h.view(np.uint32).copy() for h in h0]
    n_blocks = (steps + block - 1) // block
    num = {r: np.zeros((n_blocks, L)) for r in runs}
    den = np.zeros((n_blocks, L))
    for t, x, dt, B, C in inputs:
        k = (t - 1) // block
        for ell in range(L):
            args = (x[ell], dt[ell], init["A"][ell].numpy(), B[ell], C[ell], init["D"][ell].numpy())
            twin[ell], _, _, _ = oracle.state_update("fp32", "rtn", twin[ell], None, *args, layer=ell,
                                                     step=t, block=w.dither_block)
            h = twin[ell].view(np.float32).astype(np.float64)
            den[k, ell] += np.sum(h * h)
            for r in runs:
                if len(r) == 3:
                    if t % r[2] == 0:
                        v, _, _ = oracle.state_update_fp32_grid(fmt, r[0], st[r][ell], *args,
                                                                seed=r[1], layer=ell, step=t,
                                                                block=w.dither_block, group=g)
                    else:
                        v, _, _, _ = oracle.state_update("fp32", "rtn", st[r][ell].view(np.uint32),
                                                         None, *args, layer=ell, step=t,
                                                         block=w.dither_block)
                        v = v.view(np.float32)
                    st[r][ell] = v
                    val = v.astype(np.float64)
                else:
                    c, sc = st[r][ell]
                    c, sc, _, _ = oracle.state_update(fmt, r[0], c, sc, *args, seed=r[1], layer=ell,
                                                      step=t, block=w.dither_block, group=g)
                    st[r][ell] = (c, sc)
                    val = oracle.dequantize(fmt, c, sc, g).reshape(h.shape).astype(np.float64)
                num[r][k, ell] += np.sum((val - h) ** 2)
    return {r: (num[r] / den).mean(-1) for r in runs}


def _name(r):
    base = r[0] if r[0] != "sr" else f"sr_seed{r[1]}"
    return base if len(r) == 2 else f"{base}_cc{r[2]}"


def test_study_matches_oracle_replay():
    L, steps, block = 2, 40, 16
    w = _small(2, 64, L, steps)
    b, d, N = w.batch, w.nheads, w.dstate
    init = {"A": [], "D": [], "codes0": []}
    for ell in range(L):
        a, dd = wl.layer_params("mamba1", d, N, seed=50 + ell)
        init["A"].append(a)
        init["D"].append(dd)
        init["codes0"].append(wl.initial_state("fp16", b, d, 1, N, seed=60 + ell)[0])
    inputs = []

    def keep(t, x, dt, B, C):
        inputs.append((t, x.cpu().numpy(), dt.cpu().numpy(), B.cpu().numpy(), C.cpu().numpy()))

    _say(f"study: batch {b}, d_inner {d}, {L} layers, {steps} steps on the GPU")
    res = bench.state_error_study(w, steps=steps, layers=L, block=block, device=DEV,
                                  on_step=keep, init=init)
    _say("oracle replay of the same inputs")
    ref = _oracle_replay(w, L, steps, block, init, inputs, bench.SE_RULES)
    for r in bench.SE_RULES:
        got = np.array(res["error"][_name(r)])
        _say(f"  {_name(r)}: gpu {got} oracle {ref[r]}")
        np.testing.assert_allclose(got, ref[r], rtol=1e-3)


@pytest.mark.parametrize("fmt", ["int8", "int4", "e4m3"])
def test_scaled_study_with_checkpoints_matches_oracle_replay(fmt):
    """Block-16 scaled formats, the trained-memory decays and CC = 4 checkpoints."""
    L, steps, block = 1, 24, 8
    w = _small(2, 64, L, steps)
    b, d, N = w.batch, w.nheads, w.dstate
    init = {"A": [], "D": [], "codes0": [], "scale0": []}
    for ell in range(L):
        a, dd = wl.layer_params_trained_memory("mamba1", d, N, seed=150 + ell)
        c0, s0 = wl.initial_state(fmt, b, d, 1, N, seed=160 + ell, group=16)
        init["A"].append(a)
        init["D"].append(dd)
        init["codes0"].append(c0)
        init["scale0"].append(s0)
    inputs = []

    def keep(t, x, dt, B, C):
        inputs.append((t, x.cpu().numpy(), dt.cpu().numpy(), B.cpu().numpy(), C.cpu().numpy()))

    res = bench.state_error_study(w, steps=steps, layers=L, block=block, device=DEV, fmt=fmt,
                                  group=16, memory="trained", cc=4, on_step=keep, init=init)
    ref = _oracle_replay(w, L, steps, block, init, inputs, bench.SE_RULES, fmt=fmt, group=16, cc=4)
    for r, want in ref.items():
        got = np.array(res["error"][_name(r)])
        _say(f"  {fmt} {_name(r)}: gpu {got} oracle {want}")
        np.testing.assert_allclose(got, want, rtol=2e-3)


def test_errors_follow_the_per_write_noise_lemma():
    w = _small(4, 1024, 2, 256)
    res = bench.state_error_study(w, steps=256, layers=2, block=128, device=DEV)
    _say(f"errors {res['error']}")
    e = {k: np.mean(v) for k, v in res["error"].items()}
    assert all(v > 0 for v in e.values())
    assert 0.35 < e["rtn"] / e["sr_seed0"] < 0.7          # s^2/12 against s^2/6
    assert 0.95 * e["rtn"] < e["weyl"] < 0.9 * e["sr_seed0"]
    assert abs(e["sr_seed1"] / e["sr_seed0"] - 1.0) < 0.1  # another seed, the same law
    # the workload holds only short memories (tau below 100 steps)
    assert res["tau_bin_share"]["<10"] + res["tau_bin_share"]["10-100"] == pytest.approx(1.0)
