"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Bit-exact for thresholds and for requantize (identical fp32 inputs); the fused
step at the stated bar: y within 1e-5 relative, at most 0.01 % of stored
entries differing, each by at most one storage ulp.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_39185_amd import workloads as wl

from ._parity import DEV, Bar, assert_codes, check_step, say, y_magnitude

pytestmark = pytest.mark.gpu

TWO24 = 1 << 24


@pytest.fixture(scope="module")
def ssmq():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_39185_amd as m
    m.library()
    return m


# --------------------------------------------------------------------------
# thresholds
# --------------------------------------------------------------------------
@pytest.mark.parametrize("rule", ["rtn", "sr", "weyl", "philox"])
@pytest.mark.parametrize("block", [1, 16, 128, 1 << 20])
@pytest.mark.parametrize("entry_base,n", [(0, 0), (0, 1), (3, 1000), (2 ** 33 + 7, 4099),
                                          (1 << 20, 65536)])
def test_dither_fill_bit_exact(ssmq, rule, block, entry_base, n):
    say(f"case dither_fill {rule} block {block} base {entry_base} n {n}")
    out = torch.full((max(n, 1),), -1, dtype=torch.int32, device=DEV)
    ssmq.dither_fill(out[:n] if n else out[:0], rule=rule, seed=5, layer=9, step=123456,
                     entry_base=entry_base, dither_block=block)
    torch.cuda.synchronize()
    got = out.cpu().numpy().view(np.uint32)[:n]
    want = oracle.thresholds(rule, 5, 9, 123456, entry_base, n, block)
    assert np.array_equal(got, want)
    if n == 0:
        assert out.cpu().numpy()[0] == -1


@pytest.mark.parametrize("rule", ["sr", "weyl", "philox"])
def test_dither_fill_unaligned_output(ssmq, rule):
    """An output 4-byte but not 16-byte aligned takes the word-by-word path."""
    n, base = 5003, 12
    say(f"case dither_fill {rule} output offset 4 bytes, n {n}")
    buf = torch.full((n + 1,), -1, dtype=torch.int32, device=DEV)
    ssmq.dither_fill(buf[1:], rule=rule, seed=2, layer=4, step=99, entry_base=base, dither_block=16)
    torch.cuda.synchronize()
    got = buf.cpu().numpy().view(np.uint32)
    assert got[0] == 0xFFFFFFFF
    assert np.array_equal(got[1:], oracle.thresholds(rule, 2, 4, 99, base, n, 16))


# --------------------------------------------------------------------------
# requantize: bit-exact on identical fp32 inputs, edge suites included
# --------------------------------------------------------------------------
def _edge_values(fmt, rng, n_random, entry_base, rule, block, seed, layer, step):
    """Random values over many binades plus values on and next to rounding points."""
    e = rng.integers(-40 if fmt != "bf16" else -135, 17 if fmt != "bf16" else 128, n_random)
    m = rng.integers(0, 1 << 23, n_random).astype(np.uint64)
    s = rng.integers(0, 2, n_random).astype(np.uint64)
    bits = (s << 31) | (np.clip(e + 127, 1, 254).astype(np.uint64) << 23) | m
    x = bits.astype(np.uint32).view(np.float32)
    specials = np.array([0.0, -0.0, np.inf, -np.inf, np.nan, -np.nan, 1.0, -1.0, 65504.0, 65519.0,
                         65520.0, -65520.0, 448.0, 464.0, 3.3895314e38, 3.4028235e38, 1e-45,
                         -1e-45, 5.9604645e-08, -2.9802322e-08, 1.0 + 2 ** -11, 1.0 + 2 ** -8,
                         2 ** -14, -2 ** -14, 2 ** -15 + 2 ** -25, 1e-38, -1e-40],
                        dtype=np.float32)
    x = np.concatenate([x, specials])
    # values exactly at / next to the dither's rounding point of their own entry
    U = oracle.thresholds(rule, seed, layer, step, entry_base, x.size, block)
    lo = oracle.decode(fmt, oracle.round_values(fmt, "weyl", x, np.zeros_like(U)))
    hi = oracle.decode(fmt, oracle.round_values(fmt, "weyl", x, np.full_like(U, TWO24 - 1)))
    ok = np.isfinite(lo) & np.isfinite(hi) & (hi != lo) & (rng.random(x.size) < 0.3)
    with np.errstate(invalid="ignore"):
        pt = np.where(ok, hi - (U / TWO24) * (hi - lo), 0.0)
    p32 = pt.astype(np.float32)
    sel = np.nonzero(ok)[0]
    jitter = rng.integers(-1, 2, sel.size)
    x = x.copy()
    x[sel] = np.where(jitter < 0, np.nextafter(p32[sel], np.float32(-np.inf)),
                      np.where(jitter > 0, np.nextafter(p32[sel], np.float32(np.inf)), p32[sel]))
    return x.astype(np.float32)


@pytest.mark.parametrize("fmt", ["fp16", "bf16", "fp32"])
@pytest.mark.parametrize("rule", ["rtn", "sr", "weyl", "philox"])
@pytest.mark.parametrize("n,entry_base,block", [(16 * 4096, 0, 16), (100_003, 48, 128),
                                                (15, 16, 1), (0, 0, 16)])
def test_requantize_bit_exact(ssmq, fmt, rule, n, entry_base, block):
    say(f"case requantize {fmt} {rule} n {n} base {entry_base} block {block}")
    rng = np.random.default_rng(n + block)
    x = _edge_values(fmt, rng, max(n - 27, 0), entry_base, rule, block, 3, 4, 77)[:n]
    h = torch.from_numpy(x).to(DEV)
    dt = {"fp16": torch.int16, "bf16": torch.int16, "fp32": torch.int32}[fmt]
    codes = torch.zeros(n, dtype=dt, device=DEV)
    ssmq.requantize(h, codes, None, rule=rule, fmt=fmt, dither_block=block, seed=3, layer=4,
                    step=77, entry_base=entry_base)
    torch.cuda.synchronize()
    got = wl.to_numpy_codes(fmt, codes)
    want, _ = oracle.requantize(fmt, rule, x, seed=3, layer=4, step=77, entry_base=entry_base,
                                block=block)
    if fmt == "fp32":
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32))
    else:
        assert np.array_equal(got, want), np.nonzero(got != want)[0][:10]


@pytest.mark.parametrize("rule", ["rtn", "sr", "weyl", "philox"])
@pytest.mark.parametrize("group,n_groups", [(16, 700), (128, 300), (8192, 9), (48, 33),
                                            (2048, 5), (4096, 6)])
def test_requantize_e4m3_bit_exact(ssmq, rule, group, n_groups):
    say(f"case requantize e4m3 {rule} group {group} x {n_groups}")
    rng = np.random.default_rng(group)
    n = group * n_groups
    mag = np.exp(rng.uniform(-30, 10, n_groups)).astype(np.float32)
    x = (rng.standard_normal(n).astype(np.float32) * np.repeat(mag, group)).astype(np.float32)
    x[:group] = 0.0                                       # zero group
    x[group:2 * group] *= np.float32(1e-38)              # group whose scale is subnormal
    x[2 * group + 3] = np.nan                             # NaN inside a live group
    # tiny entries next to large ones: E4M3 subnormal outputs
    x[3 * group:4 * group] = (rng.standard_normal(group) * 1e-7).astype(np.float32)
    x[3 * group] = 100.0
    h = torch.from_numpy(x).to(DEV)
    codes = torch.zeros(n, dtype=torch.uint8, device=DEV)
    scale = torch.full((n_groups,), -1.0, dtype=torch.float32, device=DEV)
    ssmq.requantize(h, codes, scale, rule=rule, fmt="e4m3", scale_group=group, seed=1, layer=2,
                    step=3, entry_base=32, dither_block=128)
    torch.cuda.synchronize()
    want, wscale = oracle.requantize("e4m3", rule, x, seed=1, layer=2, step=3, entry_base=32,
                                     block=128, group=group)
    assert np.array_equal(scale.cpu().numpy(), wscale)
    got = codes.cpu().numpy()
    assert np.array_equal(got, want), np.nonzero(got != want)[0][:10]


# --------------------------------------------------------------------------
# fused step
# --------------------------------------------------------------------------
M2_SMALL = ("mamba2", 2, 4, 64, 128, 2)


@pytest.mark.parametrize("rule", ["rtn", "sr", "weyl"])
@pytest.mark.parametrize("fmt,q", [("bf16", {"dither_block": 128}), ("fp16", {"dither_block": 16}),
                                   ("fp32", {}), ("e4m3", {"dither_block": 128}),
                                   ("e4m3", {"scale_group": 16}), ("e4m3", {"scale_group": 128}),
                                   ("e4m3", {"scale_group": 1024, "dither_block": 1})])
def test_step_head_tile(ssmq, rule, fmt, q):
    check_step(fmt, rule, *M2_SMALL, seed=10, what="head tile", step=5, layer=2, **q)


@pytest.mark.parametrize("fmt,q", [("bf16", {"dither_block": 128}), ("fp16", {"dither_block": 16}),
                                   ("e4m3", {"dither_block": 128}), ("e4m3", {"scale_group": 128}),
                                   ("int8", {"scale_group": 128}), ("int4", {"scale_group": 16})])
def test_step_head_tile_philox(ssmq, fmt, q):
    """SR driven by Philox4x32-10 (the generator behind the paper's SR)."""
    check_step(fmt, "philox", *M2_SMALL, seed=12, what="philox head tile", step=7, layer=3, **q)


@pytest.mark.parametrize("fmt,q", [("bf16", {"dither_block": 8192}), ("bf16", {"dither_block": 1 << 20}),
                                   ("e4m3", {"dither_block": 4096}), ("e4m3", {"scale_group": 128, "dither_block": 4096}),
                                   ("int8", {"scale_group": 128, "dither_block": 8192})])
def test_step_dither_block_wider_than_a_pass(ssmq, fmt, q):
    """Weyl blocks longer than one pass of a workgroup: the chunks' threshold bases
    are computed directly rather than stepped from the first."""
    check_step(fmt, "weyl", *M2_SMALL, seed=14, what="wide dither block", step=21, layer=6, **q)


def test_step_philox_mamba1_rows(ssmq):
    check_step("fp16", "philox", "mamba1", 3, 200, 1, 16, 1, seed=13, what="philox rows",
               step=11, layer=2)


SHAPES = [
    # (family, batch, nheads, headdim, dstate, ngroups)
    ("mamba1", 3, 200, 1, 16, 1),       # Mamba-1 rows, ragged grid tail
    ("mamba1", 1, 1536, 1, 16, 1),      # the small Mamba-1 workload
    ("mamba2", 3, 6, 64, 64, 3),        # head of 4096 entries
    ("mamba2", 2, 4, 32, 128, 1),       # head tile of 4096 entries
    ("mamba2", 2, 2, 64, 256, 2),       # long rows (32 / 16 lanes)
    ("mamba2", 5, 3, 8, 16, 1),         # small heads -> row kernel
    ("mamba2", 1, 2, 1, 128, 1),        # one row per head
]


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("fmt", ["fp16", "bf16", "e4m3", "fp32"])
def test_step_shapes(ssmq, shape, fmt):
    family, batch, nheads, headdim, dstate, ngroups = shape
    head = headdim * dstate
    q = {"dither_block": 16, "step": 9, "layer": 1}
    if fmt == "e4m3" and head > 1024 and not (family == "mamba2" and head % 4096 == 0):
        q["scale_group"] = 64
    for rule in ("rtn", "sr", "weyl"):
        check_step(fmt, rule, family, batch, nheads, headdim, dstate, ngroups, seed=20,
                   what=f"shape {shape}", **q)


def test_step_no_skip_term_and_entry_base(ssmq):
    """D = NULL and a nonzero entry_base (a shard of a larger tensor)."""
    A, _ = wl.layer_params("mamba2", 4, 128, 3)
    x, dt, B, C = wl.step_inputs(2, 4, 64, 128, 2, 4)
    codes, _ = wl.initial_state("bf16", 2, 4, 64, 128, 5)
    from ._parity import run_update, oracle_update
    q = dict(dither_block=128, entry_base=3 * 8192 * 4, step=11)
    g = run_update("bf16", "weyl", codes, None, x, dt, A, B, C, None, **q)
    r = oracle_update("bf16", "weyl", codes, None, x, dt, A, B, C, None, **q)
    assert_codes("bf16", g[0], r[0], "entry_base")


def test_sharding_reproduces_unsharded(ssmq):
    """Two batch halves with entry_base offsets give the unsharded result bit for bit."""
    from ._parity import run_update
    b, H, P, N, G = 4, 4, 64, 128, 2
    A, D = wl.layer_params("mamba2", H, N, 6)
    x, dt, B, C = wl.step_inputs(b, H, P, N, G, 7)
    for fmt in ("bf16", "e4m3"):
        codes, scale = wl.initial_state(fmt, b, H, P, N, 8)
        full = run_update(fmt, "weyl", codes, scale, x, dt, A, B, C, D, dither_block=128, step=3)
        half = b // 2
        parts = []
        for k in range(2):
            sl = slice(k * half, (k + 1) * half)
            sc = None if scale is None else scale[k * half * H:(k + 1) * half * H].contiguous()
            parts.append(run_update(fmt, "weyl", codes[sl].contiguous(), sc, x[sl].contiguous(),
                                    dt[sl].contiguous(), A, B[sl].contiguous(),
                                    C[sl].contiguous(), D, dither_block=128, step=3,
                                    entry_base=k * half * H * P * N))
        assert np.array_equal(np.concatenate([p[0] for p in parts]), full[0])
        assert np.array_equal(np.concatenate([p[2] for p in parts]), full[2])


def test_deterministic(ssmq):
    from ._parity import run_update
    A, D = wl.layer_params("mamba2", 8, 128, 1)
    x, dt, B, C = wl.step_inputs(4, 8, 64, 128, 2, 2)
    codes, scale = wl.initial_state("e4m3", 4, 8, 64, 128, 3)
    a = run_update("e4m3", "sr", codes, scale, x, dt, A, B, C, D, step=4)
    b = run_update("e4m3", "sr", codes, scale, x, dt, A, B, C, D, step=4)
    assert all(np.array_equal(u, v) for u, v in zip(a, b))


@pytest.mark.parametrize("rule", ["rtn", "sr", "weyl"])
def test_small_mamba1_workload_64_steps(ssmq, rule):
    """Mamba-1, batch 1, d_inner 1536, d_state 16, fp16: 64 teacher-forced steps."""
    import paper_2609_39185_amd as m
    w = wl.WORKLOADS["m1_small"]
    A, D = wl.layer_params("mamba1", w.nheads, w.dstate, 100)
    codes, _ = wl.initial_state("fp16", w.batch, w.nheads, 1, w.dstate, 101)
    st = codes.to(DEV)
    Ad, Dd = A.to(DEV), D.to(DEV)
    bar = Bar("fp16", f"m1_small {rule}, 64 steps")
    for t in range(1, w.steps + 1):
        x, dt, B, C = wl.step_inputs(w.batch, w.nheads, 1, w.dstate, 1, 1000 + t)
        before = wl.to_numpy_codes("fp16", st)
        y = torch.empty(x.shape, dtype=torch.float32, device=DEV)
        m.state_update(st, None, x.to(DEV), dt.to(DEV), Ad, B.to(DEV), C.to(DEV), Dd, y,
                       rule=rule, fmt="fp16", dither_block=16, step=t)
        torch.cuda.synchronize()
        r_codes, _, r_y, r_h = oracle.state_update("fp16", rule, before, None, x.numpy(),
                                                   dt.numpy(), A.numpy(), B.numpy(), C.numpy(),
                                                   D.numpy(), step=t, block=16)
        bar.codes(wl.to_numpy_codes("fp16", st), r_codes)
        bar.y(y.cpu().numpy(), r_y, y_magnitude(C.numpy(), r_h, D.numpy(), x.numpy(), w.nheads))
    bar.check()


@pytest.mark.parametrize("rule", ["rtn", "sr", "weyl"])
@pytest.mark.parametrize("fmt,group", [("e4m3", 0), ("bf16", None), ("int8", 128)])
def test_head_shape_64_steps(ssmq, fmt, group, rule):
    """Mamba-2 heads of 64 x 128 (E4M3 with one scale per head, bf16, INT8 with blocks
    of 128): 64 teacher-forced steps, each checked against the oracle from the state
    and scales the GPU holds (so a one-off difference cannot compound), with the
    scales evolving from step to step (E4M3: the per-head clamp taken or skipped as
    they fall)."""
    import paper_2609_39185_amd as m
    b, H, P, N, G = 2, 8, 64, 128, 2
    A, D = wl.layer_params("mamba2", H, N, 120)
    codes, scale = wl.initial_state(fmt, b, H, P, N, 121, group=group or 0)
    st = codes.to(DEV)
    sc = None if scale is None else scale.to(DEV)
    Ad, Dd = A.to(DEV), D.to(DEV)
    q = {} if group is None else {"scale_group": group}
    bar = Bar(fmt, f"{fmt} heads {rule}, 64 steps")
    for t in range(1, 65):
        x, dt, B, C = wl.step_inputs(b, H, P, N, G, 1200 + t)
        before = wl.to_numpy_codes(fmt, st)
        s_before = None if sc is None else sc.cpu().numpy()
        y = torch.empty((b, H, P), dtype=torch.float32, device=DEV)
        m.state_update(st, sc, x.to(DEV), dt.to(DEV), Ad, B.to(DEV), C.to(DEV), Dd, y,
                       rule=rule, fmt=fmt, dither_block=128, step=t, layer=3, **q)
        torch.cuda.synchronize()
        r_codes, r_scale, r_y, r_h = oracle.state_update(
            fmt, rule, before, s_before, x.numpy(), dt.numpy(), A.numpy(), B.numpy(),
            C.numpy(), D.numpy(), step=t, layer=3, block=128, group=group or 0)
        bar.codes(wl.to_numpy_codes(fmt, st), r_codes)
        if sc is not None:
            bar.scales(sc.cpu().numpy(), r_scale)
        bar.y(y.cpu().numpy(), r_y, y_magnitude(C.numpy(), r_h, D.numpy(), x.numpy(), H // G))
    bar.check()


def _prop1_prediction(rule, f, T, seed, layer, block, n):
    """Proposition 1 (Section 3) for a = 1 and a constant write of f grid steps:
    the accumulated error after T writes is -(N - T(1 - f)) steps, with N the
    number of writes whose threshold u_t satisfies u_t < 1 - f (the writes that
    round down). RTN is the rule with u = 1/2 (no ties occur here). Thresholds
    come from the oracle's generator."""
    count = np.zeros(n, np.int64)
    for t in range(1, T + 1):
        if rule == "rtn":
            u = np.full(n, 0.5)
        else:
            u = oracle.thresholds(rule, seed, layer, t, 0, n, block) / TWO24
        count += u < 1 - f
    return -(count - T * (1 - f))


@pytest.mark.parametrize("rule", ["rtn", "sr", "weyl", "philox"])
def test_proposition1_through_the_kernel(ssmq, rule):
    """fp16 Mamba-1 rows, A = 0 (a = exp(0) = 1) and a constant write w = f s per
    column: the GPU's stored state after T steps is h_0 + T w + e_T with e_T of
    Proposition 1, exactly, for every rule."""
    import paper_2609_39185_amd as m
    n, T = 64, 300
    f_num = np.arange(1, n + 1) * 127
    s = 2.0 ** -10                      # fp16 step in [1, 2)
    f = f_num / 8192
    w = (f * s).astype(np.float32)
    st = torch.full((1, 1, 1, n), 0x3C00, dtype=torch.int16, device=DEV)  # 1.0
    one = torch.ones((1, 1, 1), device=DEV)
    A = torch.zeros((1, n), device=DEV)
    B = torch.from_numpy(w).reshape(1, 1, n).to(DEV)
    C = torch.zeros((1, 1, n), device=DEV)
    y = torch.empty((1, 1, 1), device=DEV)
    say(f"case proposition 1 fp16 {rule}: {n} entries, {T} steps")
    for t in range(1, T + 1):
        m.state_update(st, None, one, torch.ones((1, 1), device=DEV), A, B, C, None, y,
                       rule=rule, fmt="fp16", dither_block=16, seed=3, layer=1, step=t)
    torch.cuda.synchronize()
    h = oracle.decode("fp16", wl.to_numpy_codes("fp16", st).ravel())
    e_T = (h - (1.0 + T * w.astype(np.float64))) / s
    want = _prop1_prediction(rule, f, T, 3, 1, 16, n)
    assert np.array_equal(e_T, want), (rule, np.nonzero(e_T != want)[0][:8])
    if rule == "rtn":  # Corollary 1 (a): below half a step every write is erased
        assert np.all(want == np.where(f < 0.5, -T * f, T * (1 - f)))


@pytest.mark.parametrize("rule", ["rtn", "sr", "weyl", "philox"])
def test_proposition1_through_the_kernel_e4m3_head(ssmq, rule):
    """E4M3 with one scale per 64 x 128 head (the slab kernel the bench times).
    Entry (0, 0) holds 448 and receives no write, so every step's scale is
    448 / 448 = 1 exactly and every product is exact. Columns n >= 1 start at 1.0
    and receive w = f/8, f = 3n / 8192 of the E4M3 step 1/8 in [1, 2), for T = 48
    steps. An entry's stored value after t steps is 1 + N_up(t)/8 (N_up: the writes
    that rounded up), so it stays in that binade, where Proposition 1 holds with one
    fixed step, exactly while N_up(T) <= 7; those entries (all but a few SR draws)
    follow Proposition 1 exactly, and column 0 stays where it started."""
    import paper_2609_39185_amd as m
    P, N, T = 64, 128, 48
    f = 3.0 * np.arange(N) / 8192
    codes = torch.full((1, 1, P, N), 0x38, dtype=torch.uint8)   # 1.0
    codes[0, 0, 0, 0] = 0x7E                                      # 448
    st = codes.to(DEV)
    sc = torch.ones(1, device=DEV)
    x = torch.ones((1, 1, P), device=DEV)
    dt = torch.ones((1, 1), device=DEV)
    A = torch.zeros(1, device=DEV)
    B = torch.from_numpy((f / 8).astype(np.float32)).reshape(1, 1, N).to(DEV)
    C = torch.zeros((1, 1, N), device=DEV)
    y = torch.empty((1, 1, P), device=DEV)
    say(f"case proposition 1 e4m3 head {rule}: {P * N} entries, {T} steps")
    for t in range(1, T + 1):
        m.state_update(st, sc, x, dt, A, B, C, None, y, rule=rule, fmt="e4m3", dither_block=128,
                       seed=5, layer=2, step=t)
    torch.cuda.synchronize()
    assert sc.item() == 1.0
    h = oracle.decode("e4m3", wl.to_numpy_codes("e4m3", st).ravel()).reshape(P, N)
    assert h[0, 0] == 448.0 and np.all(h[1:, 0] == 1.0)
    e_T = ((h - (1.0 + T * f / 8)) * 8)[:, 1:].ravel()
    ff = np.tile(f[1:], P)
    want = _prop1_prediction(rule, np.tile(f, P), T, 5, 2, 128, P * N).reshape(P, N)[:, 1:].ravel()
    n_up = np.rint(want + T * ff).astype(np.int64)       # N_up(T) = e_T + T f
    inside = n_up <= 7
    say(f"  {int(inside.sum())} of {inside.size} entries stay in [1, 2)")
    assert inside.mean() > 0.99
    assert np.array_equal(e_T[inside], want[inside]), (rule, np.nonzero(e_T[inside] != want[inside])[0][:8])
    if rule == "rtn":
        assert np.all(want == -T * ff)


# --------------------------------------------------------------------------
# full-size workloads, sampled tiles against the oracle
# --------------------------------------------------------------------------
def _full_size_sampled(ssmq, name, fmt, rule, n_tiles=24, group=None):
    """One full-size layer in the launch configuration the bench times; sampled head
    tiles against the oracle at the stated bar, summed over the tiles.
    group: entries per scale (0 = one per head; None = the workload's own)."""
    import paper_2609_39185_amd as m
    w = wl.WORKLOADS[name]
    b, H, P, N, G = w.batch, w.nheads, w.headdim, w.dstate, w.ngroups
    grp = wl.scale_group_of(w, fmt) if group is None else group
    per_tile = (P * N) // (grp or P * N) if fmt in oracle.SCALED else 0
    say(f"case full size {name} {fmt} {rule} group {grp}: {w.entries_per_layer} entries")
    A, D = wl.layer_params(w.family, H, N, 500, device=DEV)
    x, dt, B, C = wl.step_inputs(b, H, P, N, G, 501, device=DEV)
    codes, scale = wl.initial_state(fmt, b, H, P, N, 502, group=grp, device=DEV)
    before = codes.clone()
    sbefore = None if scale is None else scale.clone()
    y = torch.empty((b, H, P), dtype=torch.float32, device=DEV)
    m.state_update(codes, scale, x, dt, A, B, C, D, y, rule=rule, fmt=fmt,
                   dither_block=w.dither_block, scale_group=grp, step=777, layer=5)
    torch.cuda.synchronize()
    rng = np.random.default_rng(0)
    tiles = rng.choice(b * H, size=n_tiles, replace=False)
    tiles[0], tiles[-1] = 0, b * H - 1
    hpg = H // G
    bar = Bar(fmt, f"full size {name} {fmt} {rule}, {n_tiles} sampled tiles")
    for tile in tiles:
        bb, hh = divmod(int(tile), H)
        gg = hh // hpg
        cs = lambda t: t.detach().cpu()
        sl = slice(tile * per_tile, (tile + 1) * per_tile) if per_tile else None
        r_codes, r_scale, r_y, r_h = oracle.state_update(
            fmt, rule, wl.to_numpy_codes(fmt, cs(before[bb:bb + 1, hh:hh + 1])),
            None if sbefore is None else cs(sbefore[sl]).numpy(),
            cs(x[bb:bb + 1, hh:hh + 1]).numpy(), cs(dt[bb:bb + 1, hh:hh + 1]).numpy(),
            cs(A[hh:hh + 1]).numpy(), cs(B[bb:bb + 1, gg:gg + 1]).numpy(),
            cs(C[bb:bb + 1, gg:gg + 1]).numpy(), cs(D[hh:hh + 1]).numpy(),
            step=777, layer=5, block=w.dither_block, group=grp, entry_base=int(tile) * P * N)
        bar.codes(wl.to_numpy_codes(fmt, cs(codes[bb:bb + 1, hh:hh + 1])), r_codes)
        if scale is not None:
            bar.scales(cs(scale[sl]).numpy(), r_scale)
        Ch = cs(C[bb, gg]).numpy().astype(np.float64)
        mag = np.abs(Ch[None, :] * r_h[0, 0]).sum(-1) + abs(float(D[hh]) * cs(x[bb, hh]).numpy())
        bar.y(cs(y[bb, hh]).numpy(), r_y[0, 0], mag)
    bar.check()


BENCH_VARIANTS = [(f, r) for f in ("bf16", "e4m3", "int8") for r in ("weyl", "sr", "rtn", "philox")]
BENCH_VARIANTS += [("int4", r) for r in ("weyl", "sr", "rtn")]


@pytest.mark.parametrize("fmt,rule", BENCH_VARIANTS)
def test_full_size_hybrid_stack_layer(ssmq, fmt, rule):
    """Every format and rule the bench reports, at the bench's layer shape."""
    _full_size_sampled(ssmq, "hybrid_m2_stack", fmt, rule)


@pytest.mark.parametrize("fmt,rule,group", [("e4m3", "weyl", 128), ("e4m3", "rtn", 16),
                                            ("e4m3", "sr", 256), ("int8", "weyl", 16),
                                            ("int8", "weyl", 0), ("int4", "rtn", 0),
                                            ("int4", "sr", 16)])
def test_full_size_hybrid_layer_other_groups(ssmq, fmt, rule, group):
    """The scale groups timed beside the bench's own (bench.py --variants fmt/group:rule)."""
    _full_size_sampled(ssmq, "hybrid_m2_stack", fmt, rule, group=group)


def test_full_size_fp8_decode(ssmq):
    _full_size_sampled(ssmq, "m2_b64_fp8", "e4m3", "sr")


def test_full_size_ssd_decode(ssmq):
    _full_size_sampled(ssmq, "m2_ssd_b8", "bf16", "weyl")


# --------------------------------------------------------------------------
# errors surface as exceptions, before any work is queued
# --------------------------------------------------------------------------
@pytest.mark.parametrize("fmt", ["bf16", "e4m3", "int4"])
def test_empty_inputs_are_no_ops(ssmq, fmt):
    """Empty torch tensors (data pointer 0) through every entry point: each call
    returns without error and launches nothing."""
    H, P, N = 4, 64, 128
    per = 2 if fmt == "int4" else 1
    st = torch.empty((0, H, P, N // per), dtype=wl.CODE_TORCH_DTYPE[fmt], device=DEV)
    sc = torch.empty((0,), device=DEV) if fmt != "bf16" else None
    x, y = torch.empty((0, H, P), device=DEV), torch.empty((0, H, P), device=DEV)
    dt, BC = torch.empty((0, H), device=DEV), torch.empty((0, 2, N), device=DEV)
    A, D = torch.zeros(H, device=DEV), torch.zeros(H, device=DEV)
    ssmq.state_update(st, sc, x, dt, A, BC, BC, D, y, rule="weyl", fmt=fmt)
    ssmq.state_update(st, sc, x, dt, A, BC, BC, D, y, rule="sr", fmt=fmt, dt_softplus=True)
    ssmq.requantize(torch.empty(0, device=DEV), st.view(-1), sc, rule="weyl", fmt=fmt,
                    scale_group=16)
    ssmq.dither_fill(torch.empty(0, dtype=torch.int32, device=DEV), rule="weyl")
    cs = torch.empty((0, 8, 4), device=DEV)
    ssmq.conv1d_update(cs, torch.empty((0, 8), device=DEV), torch.zeros((8, 4), device=DEV),
                       None, torch.empty((0, 8), device=DEV))
    e = torch.empty((0,), dtype=torch.float64, device=DEV)
    ssmq.replay(torch.empty(0, device=DEV), torch.empty((0, 0), device=DEV),
                torch.empty((0, 0), device=DEV), e, rule="weyl", fmt=fmt,
                scale_group=0 if fmt == "bf16" else 16)
    torch.cuda.synchronize()


def test_errors(ssmq):
    import paper_2609_39185_amd as m
    st = torch.zeros((1, 4, 64, 128), dtype=torch.int16, device=DEV)
    x = torch.zeros((1, 4, 64), device=DEV)
    dt = torch.zeros((1, 4), device=DEV)
    A = torch.zeros(4, device=DEV)
    B = torch.zeros((1, 3, 128), device=DEV)
    y = torch.zeros((1, 4, 64), device=DEV)
    with pytest.raises(m.SsmqError) as e:
        m.state_update(st, None, x, dt, A, B, B, None, y, rule="weyl", fmt="bf16")
    assert e.value.status == 1
    with pytest.raises(m.SsmqError) as e:
        m.state_update(st, None, x, dt, A, B[:, :2], B[:, :2], None, y, rule="weyl", fmt="bf16",
                       dither_block=24)
    assert e.value.status == 1
    with pytest.raises(ValueError):
        m.state_update(st.cpu(), None, x, dt, A, B, B, None, y, rule="weyl", fmt="bf16")


# --------------------------------------------------------------------------
# E4M3 with one scale per head: the saturating clamp, and when it may be skipped
# --------------------------------------------------------------------------
def _scale_with_overshoot(over):
    """An old scale s0 for which a head whose maximum is the code 448 gets, after
    h = 448 s0 and the new scale s = fl32(h / 448), r = fl32(1 / s), a scaled
    maximum q = fl32(h r) of 448 + `over` fp32 ulps (over <= 0: at most 448)."""
    rng = np.random.default_rng(11)
    for _ in range(200000):
        s0 = np.float32(rng.uniform(1, 2) * 2.0 ** int(rng.integers(-12, 12)))
        m = np.float32(np.float32(448) * s0)
        s = np.float32(m / np.float32(448))
        q = np.float32(m * np.float32(np.float32(1) / s))
        if int(q.view(np.uint32)) - 0x43E00000 == over:
            return s0
    raise AssertionError(f"no scale found with overshoot {over}")


@pytest.mark.parametrize("rule", ["weyl", "sr"])
@pytest.mark.parametrize("over", [1, 0, -1])
def test_e4m3_head_scale_overshoot_saturates(ssmq, rule, over):
    """dt = 0 keeps h = 448 s0 at one entry and 0 elsewhere. When the scaled maximum
    passes 448 its threshold is chosen (from the oracle's generator) so that an
    unsaturated stochastic conversion would carry into the NaN code; the stored
    code must be 448 (0x7E), as the oracle's clamp gives, and every code and the
    scale must equal the oracle's. Without overshoot the clamp is skipped."""
    import paper_2609_39185_amd as m
    P, N = 64, 128
    s0 = _scale_with_overshoot(over)
    need = (1 << 24) - 16 * max(over, 1)  # carry past 448: over + (U >> 4) >= 2^20
    entry = step = None
    for t in range(1, 40000):
        U = oracle.thresholds(rule, 0, 2, t, 0, P * N, 128)
        hit = np.nonzero(U >= need)[0]
        if hit.size:
            entry, step = int(hit[0]), t
            break
    assert entry is not None
    say(f"case e4m3 {rule} overshoot {over}: entry {entry} step {step} s0 {float(s0)!r}")
    codes = torch.zeros((1, 1, P, N), dtype=torch.uint8)
    codes.view(-1)[entry] = 0x7E
    scale = torch.tensor([s0], dtype=torch.float32)
    x = torch.zeros((1, 1, P))
    dt = torch.zeros((1, 1))
    A = torch.tensor([-1.5])
    B = torch.randn((1, 1, N), generator=torch.Generator().manual_seed(3))
    C = torch.randn((1, 1, N), generator=torch.Generator().manual_seed(4))
    st, sc = codes.to(DEV), scale.to(DEV)
    y = torch.empty((1, 1, P), device=DEV)
    m.state_update(st, sc, x.to(DEV), dt.to(DEV), A.to(DEV), B.to(DEV), C.to(DEV), None, y,
                   rule=rule, fmt="e4m3", dither_block=128, layer=2, step=step)
    torch.cuda.synchronize()
    r_codes, r_scale, _, _ = oracle.state_update(
        "e4m3", rule, codes.numpy(), scale.numpy(), x.numpy(), dt.numpy(), A.numpy(), B.numpy(),
        C.numpy(), np.zeros(1, np.float32), layer=2, step=step, block=128)
    got = st.cpu().numpy()
    assert r_codes.ravel()[entry] == 0x7E and np.count_nonzero(r_codes) == 1
    assert np.array_equal(got, r_codes), (got.ravel()[entry], r_codes.ravel()[entry])
    assert np.array_equal(sc.cpu().numpy(), r_scale)


@pytest.mark.parametrize("fmt,rule,batch", [("bf16", "weyl", 2304), ("e4m3", "sr", 4608)])
def test_state_beyond_4gib(ssmq, fmt, rule, batch):
    """One call on a state past 2^31 entries and 4 GiB of codes (64-bit byte offsets
    and flat indices): hybrid-shaped heads at a large batch, sampled tiles up to the
    last one against the oracle."""
    import paper_2609_39185_amd as m
    H, P, N, G = 128, 64, 128, 8
    n = batch * H * P * N
    assert n > 2 ** 31 and n * ssmq.CODE_BYTES[fmt] > 2 ** 32
    say(f"case large state {fmt} {rule}: batch {batch}, {n} entries")
    A, D = wl.layer_params("mamba2", H, N, 600, device=DEV)
    x, dt, B, C = wl.step_inputs(batch, H, P, N, G, 601, device=DEV)
    codes = torch.empty((batch, H, P, N), dtype=wl.CODE_TORCH_DTYPE[fmt], device=DEV)
    scale = torch.empty(batch * H, device=DEV) if fmt == "e4m3" else None
    for b0 in range(0, batch, 256):  # fill in slices to bound the temporaries
        c, s = wl.initial_state(fmt, min(256, batch - b0), H, P, N, 602 + b0, device=DEV)
        codes[b0:b0 + c.shape[0]].copy_(c)
        if scale is not None:
            scale[b0 * H:(b0 + c.shape[0]) * H].copy_(s)
        del c, s
    tiles = [0, 12345, batch * H // 2 + 7, batch * H - 2, batch * H - 1]
    before = {t: codes.view(-1, P, N)[t].cpu().clone() for t in tiles}
    sbefore = None if scale is None else scale.cpu().clone()
    y = torch.empty((batch, H, P), device=DEV)
    m.state_update(codes, scale, x, dt, A, B, C, D, y, rule=rule, fmt=fmt, dither_block=128,
                   step=31, layer=4)
    torch.cuda.synchronize()
    hpg = H // G
    bar = Bar(fmt, f"state past 4 GiB, {len(tiles)} sampled tiles")
    for t in tiles:
        bb, hh = divmod(t, H)
        gg = hh // hpg
        cs = lambda v: v.detach().cpu()
        r_codes, r_scale, r_y, r_h = oracle.state_update(
            fmt, rule, wl.to_numpy_codes(fmt, before[t].view(1, 1, P, N)),
            None if sbefore is None else sbefore[t:t + 1].numpy(),
            cs(x[bb:bb + 1, hh:hh + 1]).numpy(), cs(dt[bb:bb + 1, hh:hh + 1]).numpy(),
            cs(A[hh:hh + 1]).numpy(), cs(B[bb:bb + 1, gg:gg + 1]).numpy(),
            cs(C[bb:bb + 1, gg:gg + 1]).numpy(), cs(D[hh:hh + 1]).numpy(),
            step=31, layer=4, block=128, entry_base=t * P * N)
        bar.codes(wl.to_numpy_codes(fmt, cs(codes.view(-1, P, N)[t]).view(1, 1, P, N)), r_codes)
        if scale is not None:
            bar.scales(cs(scale[t:t + 1]).numpy(), r_scale)
        Ch = cs(C[bb, gg]).numpy().astype(np.float64)
        mag = np.abs(Ch[None, :] * r_h[0, 0]).sum(-1) + abs(float(D[hh]) * cs(x[bb, hh]).numpy())
        bar.y(cs(y[bb, hh]).numpy(), r_y[0, 0], mag)
    bar.check()


@pytest.mark.parametrize("fmt,rule,group", [("bf16", "weyl", 0), ("int8", "sr", 128),
                                            ("e4m3", "philox", 0)])
def test_step_counter_wraps_and_resume_is_exact(ssmq, fmt, rule, group):
    """Steps 2^32 - 2, 2^32 - 1, 0, 1 (the counter is taken mod 2^32) match the
    oracle step by step, and saving the state to the host after two steps and
    restoring it resumes bit for bit: the codes (and scales) plus the step counter
    are the whole state."""
    import paper_2609_39185_amd as m
    b, H, P, N, G = 2, 4, 64, 128, 2
    A, D = wl.layer_params("mamba2", H, N, 70)
    codes, scale = wl.initial_state(fmt, b, H, P, N, 71, group=group)
    steps = [2 ** 32 - 2, 2 ** 32 - 1, 0, 1]
    inputs = [wl.step_inputs(b, H, P, N, G, 72 + k) for k in range(4)]

    def run(st, sc, ks):
        for k in ks:
            x, dt, B, C = (v.to(DEV) for v in inputs[k])
            y = torch.empty((b, H, P), device=DEV)
            m.state_update(st, sc, x, dt, A.to(DEV), B, C, D.to(DEV), y, rule=rule, fmt=fmt,
                           dither_block=128, scale_group=group, step=steps[k], layer=6)
        torch.cuda.synchronize()

    st = codes.to(DEV)
    sc = None if scale is None else scale.to(DEV)
    ref_c, ref_s = wl.to_numpy_codes(fmt, codes), None if scale is None else scale.numpy()
    bar = Bar(fmt, "steps 2^32 - 2 .. 1")
    for k in range(4):
        run(st, sc, [k])
        x, dt, B, C = (v.numpy() for v in inputs[k])
        want = oracle.state_update(fmt, rule, ref_c, ref_s, x, dt, A.numpy(), B, C, D.numpy(),
                                   step=steps[k], layer=6, block=128, group=group)
        got = wl.to_numpy_codes(fmt, st)
        bar.codes(got, want[0])
        if sc is not None:
            bar.scales(sc.cpu().numpy(), want[1])
        ref_c, ref_s = got, None if sc is None else sc.cpu().numpy()  # teacher-forced
    bar.check()
    # resume: two steps, a round trip through host memory, two more == four straight
    st2 = codes.to(DEV)
    sc2 = None if scale is None else scale.to(DEV)
    run(st2, sc2, [0, 1])
    saved = (st2.cpu(), None if sc2 is None else sc2.cpu())
    st3 = saved[0].to(DEV)
    sc3 = None if saved[1] is None else saved[1].to(DEV)
    run(st3, sc3, [2, 3])
    assert torch.equal(st3.cpu(), st.cpu())
    if sc is not None:
        assert torch.equal(sc3.cpu(), sc.cpu())


def test_full_size_m1_long_layer(ssmq):
    """One layer of the long-horizon Mamba-1 workload (batch 16, d_inner 5120, N 16,
    fp16, dither block 16) in the row kernel the study uses: sampled channels of
    every sequence against the oracle."""
    import paper_2609_39185_amd as m
    w = wl.WORKLOADS["m1_long"]
    b, d, N = w.batch, w.nheads, w.dstate
    A, D = wl.layer_params("mamba1", d, N, 800, device=DEV)
    x, dt, B, C = wl.step_inputs(b, d, 1, N, 1, 801, device=DEV)
    codes, _ = wl.initial_state("fp16", b, d, 1, N, 802, device=DEV)
    before = codes.cpu().clone()
    y = torch.empty((b, d, 1), device=DEV)
    say(f"case full size m1_long layer: {b * d * N} entries")
    for rule in ("weyl", "sr"):
        bar = Bar("fp16", f"m1_long layer {rule}, sampled channels")
        st = codes.clone()
        m.state_update(st, None, x, dt, A, B, C, D, y, rule=rule, fmt="fp16", dither_block=16,
                       step=1234, layer=17)
        torch.cuda.synchronize()
        chans = np.array([0, 1, 777, 2560, d - 1])
        for bb in (0, b - 1):
            sl = slice(int(chans.min()), int(chans.max()) + 1)
            cs = lambda v: v.detach().cpu()
            r_codes, _, r_y, r_h = oracle.state_update(
                "fp16", rule, wl.to_numpy_codes("fp16", before[bb:bb + 1, sl]), None,
                cs(x[bb:bb + 1, sl]).numpy(), cs(dt[bb:bb + 1, sl]).numpy(), cs(A[sl]).numpy(),
                cs(B[bb:bb + 1]).numpy(), cs(C[bb:bb + 1]).numpy(), cs(D[sl]).numpy(),
                step=1234, layer=17, block=16, entry_base=(bb * d + sl.start) * N)
            bar.codes(wl.to_numpy_codes("fp16", cs(st[bb:bb + 1, sl])), r_codes)
            bar.y(cs(y[bb:bb + 1, sl]).numpy(), r_y,
                  y_magnitude(cs(C[bb:bb + 1]).numpy(), r_h, cs(D[sl]).numpy(),
                              cs(x[bb:bb + 1, sl]).numpy(), sl.stop - sl.start))
        bar.check()
