"""Shared helpers of the GPU parity tests (compare the HIP path with the oracle)."""
from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_2609_39185_amd import workloads as wl

DEV = torch.device("cuda:0")

# The bar of the fused step: fp32 outputs within 1e-5 relative, at most 0.01 %
# of stored entries differing, each by at most one storage ulp.
Y_REL = 1e-5
MAX_DIFFER_FRACTION = 1e-4
MAX_ULP = 1


def say(msg: str) -> None:
    print(msg, flush=True)


def code_stats(fmt: str, got: np.ndarray, want: np.ndarray):
    """(number of differing codes, largest distance in storage ulps)."""
    got = np.asarray(oracle.entry_codes(fmt, got)).ravel()
    want = np.asarray(oracle.entry_codes(fmt, want)).ravel()
    idx = np.nonzero(got != want)[0]
    if idx.size == 0:
        return 0, 0
    if fmt == "fp32":
        a = got[idx].view(np.int32).astype(np.int64)
        b = want[idx].view(np.int32).astype(np.int64)
        return idx.size, int(np.max(np.abs(a - b)))
    ra = oracle.code_rank(fmt, got[idx])
    rb = oracle.code_rank(fmt, want[idx])
    bad = (ra < 0) | (rb < 0)
    dist = np.where(bad, 1 << 30, np.abs(ra - rb))
    return idx.size, int(dist.max())


def assert_codes(fmt, got, want, what=""):
    n, ulp = code_stats(fmt, got, want)
    size = np.asarray(got).size * oracle.entries_per_code_word(fmt)
    frac = n / max(1, size)
    say(f"  {what}: {n} of {size} stored entries differ (max {ulp} ulp)")
    assert frac <= MAX_DIFFER_FRACTION and ulp <= MAX_ULP, (what, n, ulp)


def y_magnitude(C, h_new, D, x, heads_per_group):
    """|y| scale for the relative bound: sum_n |C_n h_n| + |D x| (float64)."""
    Ch = np.repeat(np.asarray(C, np.float64), heads_per_group, axis=1)[:, :, None, :]
    mag = np.abs(Ch * np.asarray(h_new, np.float64)).sum(-1)
    if D is not None:
        mag = mag + np.abs(np.asarray(D, np.float64)[None, :, None] * np.asarray(x, np.float64))
    return mag


def assert_y(y_gpu, y_ref, mag, what=""):
    y_gpu = np.asarray(y_gpu, np.float64)
    err = np.abs(y_gpu - y_ref)
    bound = Y_REL * (mag + np.abs(y_ref))
    worst = float(np.max(err / np.maximum(bound, 1e-300))) * Y_REL
    say(f"  {what}: y max error / (|y| + sum|C h| + |D x|) = {worst:.2e}")
    assert np.all(err <= bound), what


def to_dev(*ts):
    return [None if t is None else t.to(DEV) for t in ts]


def run_update(fmt, rule, codes, scale, x, dt, A, B, C, D, **q):
    """GPU step on copies of the inputs; returns host (codes, scale, y)."""
    import paper_2609_39185_amd as ssmq
    st, sc, xd, dtd, Ad, Bd, Cd, Dd = to_dev(codes, scale, x, dt, A, B, C, D)
    y = torch.full(x.shape, float("nan"), dtype=torch.float32, device=DEV)
    ssmq.state_update(st, sc, xd, dtd, Ad, Bd, Cd, Dd, y, rule=rule, fmt=fmt, **q)
    torch.cuda.synchronize()
    return (wl.to_numpy_codes(fmt, st), None if sc is None else sc.cpu().numpy(),
            y.cpu().numpy())


def oracle_update(fmt, rule, codes, scale, x, dt, A, B, C, D, **q):
    kw = dict(seed=q.get("seed", 0), layer=q.get("layer", 0), step=q.get("step", 0),
              entry_base=q.get("entry_base", 0), block=q.get("dither_block", 16),
              group=q.get("scale_group", 0))
    return oracle.state_update(fmt, rule, wl.to_numpy_codes(fmt, codes),
                               None if scale is None else scale.numpy(), x.numpy(), dt.numpy(),
                               A.numpy(), B.numpy(), C.numpy(),
                               None if D is None else D.numpy(), **kw)


def check_step(fmt, rule, family, batch, nheads, headdim, dstate, ngroups, seed, what="",
               dither_seed=None, **q):
    """One fused step on seeded inputs: GPU vs oracle at the stated bar. seed draws
    the inputs; dither_seed, when given, is the rounding's seed (sigma)."""
    if dither_seed is not None:
        q["seed"] = dither_seed
    A, D = wl.layer_params(family, nheads, dstate, seed)
    x, dt, B, C = wl.step_inputs(batch, nheads, headdim, dstate, ngroups, seed + 1)
    codes, scale = wl.initial_state(fmt, batch, nheads, headdim, dstate, seed + 2,
                                    group=q.get("scale_group", 0))
    say(f"case {what}: {family} {fmt} {rule} b{batch} h{nheads} p{headdim} n{dstate} "
        f"g{ngroups} {q}")
    g_codes, g_scale, g_y = run_update(fmt, rule, codes, scale, x, dt, A, B, C, D, **q)
    r_codes, r_scale, r_y, r_h = oracle_update(fmt, rule, codes, scale, x, dt, A, B, C, D, **q)
    assert_codes(fmt, g_codes, r_codes, what)
    if fmt in oracle.SCALED:
        assert np.array_equal(g_scale, r_scale), f"{fmt} group scales differ"
    mag = y_magnitude(C.numpy(), r_h, None if D is None else D.numpy(), x.numpy(),
                      nheads // ngroups)
    assert_y(g_y, r_y, mag, what)
