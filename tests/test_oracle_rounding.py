"""Pins of the oracle's formats and rounding (CPU only).

What fixes the expected values here, independently of the oracle's code:
  - exact rational evaluation of eq. (dither), Q_u(x) = s floor(x/s + u), on the
    grid of the local exponent (Section 2; Appendix B "Formats");
  - torch's own casts for round-to-nearest (Appendix B "Formats": the RTN
    simulation matches the native casts bit for bit);
  - the format definitions (torch's float8_e4m3fn / numpy float16 decoders).
"""
import math
from fractions import Fraction

import numpy as np
import pytest
import torch

# (mantissa bits, smallest normal exponent, largest finite value)
SPEC = {
    "fp16": (10, -14, Fraction(65504)),
    "bf16": (7, -126, Fraction(2 ** 8 - 1, 2 ** 7) * Fraction(2) ** 127),
    "e4m3": (3, -6, Fraction(448)),
}
TWO24 = 1 << 24


def _floor_log2(q: Fraction) -> int:
    q = abs(q)
    e = q.numerator.bit_length() - q.denominator.bit_length()
    if Fraction(2) ** e > q:
        e -= 1
    return e


def _local_step(fmt, x: Fraction) -> Fraction:
    M, emin, _ = SPEC[fmt]
    e = max(_floor_log2(x), emin) if x != 0 else emin
    return Fraction(2) ** (e - M)


def eq_dither(fmt, xf: float, U: int):
    """Eq. (dither) in exact rational arithmetic; returns a Fraction or +-inf."""
    M, emin, vmax = SPEC[fmt]
    x = Fraction(xf)
    if fmt == "e4m3":
        x = max(-vmax, min(vmax, x))
    s = _local_step(fmt, x)
    v = s * math.floor(x / s + Fraction(U, TWO24))
    if abs(v) > vmax:
        return math.copysign(math.inf, v)
    return v


def nearest_even(fmt, xf: float):
    M, emin, vmax = SPEC[fmt]
    x = Fraction(xf)
    if fmt == "e4m3":
        x = max(-vmax, min(vmax, x))
    s = _local_step(fmt, x)
    k = math.floor(x / s)
    r = x / s - k
    if r > Fraction(1, 2) or (r == Fraction(1, 2) and k % 2 == 1):
        k += 1
    v = k * s
    if abs(v) > vmax:
        return math.copysign(math.inf, v)
    return v


def _random_floats(rng, n, emin, emax):
    """fp32 values with log-uniform magnitudes and random signs and mantissas."""
    e = rng.integers(emin, emax + 1, n)
    m = rng.integers(0, 1 << 23, n)
    sign = rng.integers(0, 2, n)
    bits = (sign.astype(np.uint64) << 31) | (np.clip(e + 127, 1, 254).astype(np.uint64) << 23) | m.astype(np.uint64)
    return bits.astype(np.uint32).view(np.float32)


RANGES = {"fp16": (-40, 16), "bf16": (-140, 127), "e4m3": (-26, 9)}


def _boundary_cases(fmt, rng, n):
    """x placed exactly on, and one fp32 step either side of, the point hi - u*s."""
    xs, us = [], []
    M, emin, vmax = SPEC[fmt]
    lo_e, hi_e = RANGES[fmt]
    for _ in range(n):
        U = int(rng.integers(0, TWO24))
        e = int(rng.integers(lo_e, min(hi_e, 8) + 1))
        sign = -1 if rng.integers(0, 2) else 1
        step = Fraction(2) ** (max(e, emin) - M)
        k = int(rng.integers(0, 1 << M)) if e >= emin else 0
        base = (Fraction(2) ** e if e >= emin else 0) + k * step
        hi = base + step
        point = hi - Fraction(U, TWO24) * step
        p = float(point) * sign
        p32 = np.float32(p)
        for v in (np.nextafter(p32, np.float32(-np.inf)), p32, np.nextafter(p32, np.float32(np.inf))):
            xs.append(v)
            us.append(U)
    return np.array(xs, np.float32), np.array(us, np.uint32)


@pytest.mark.parametrize("fmt", ["fp16", "bf16", "e4m3"])
def test_dither_rule_is_eq_dither_exactly(orc, fmt):
    """Every SR/Weyl rounding equals s*floor(x/s+u) on the local grid (brute force)."""
    rng = np.random.default_rng(1234 + len(fmt))
    lo_e, hi_e = RANGES[fmt]
    x = _random_floats(rng, 6000, lo_e, hi_e)
    U = rng.integers(0, TWO24, x.size).astype(np.uint32)
    # extreme thresholds and special values
    specials = np.array([0.0, -0.0, 1.0, -1.0, 1e-30, -1e-30, 3e-45, -3e-45], np.float32)
    x = np.concatenate([x, specials, specials])
    U = np.concatenate([U, np.zeros(8, np.uint32), np.full(8, TWO24 - 1, np.uint32)])
    bx, bU = _boundary_cases(fmt, rng, 1500)
    x = np.concatenate([x, bx])
    U = np.concatenate([U, bU])
    codes = orc.round_values(fmt, "weyl", x, U)
    got = orc.decode(fmt, codes)
    bad = 0
    for xi, ui, gi, ci in zip(x, U, got, codes):
        want = eq_dither(fmt, float(xi), int(ui))
        if isinstance(want, float):
            ok = gi == want
        else:
            ok = Fraction(float(gi)) == want
            if want == 0:  # a zero result keeps the sign of x
                sign_bit = 15 if fmt != "e4m3" else 7
                ok = ok and ((int(ci) >> sign_bit) & 1) == int(np.signbit(xi))
        bad += not ok
    assert bad == 0


@pytest.mark.parametrize("fmt", ["fp16", "bf16", "e4m3"])
def test_rtn_is_nearest_even_exactly(orc, fmt):
    """Random values, and exact midpoints between neighbouring values of the format
    (ties: the reference rounds them to the even step count)."""
    rng = np.random.default_rng(99 + len(fmt))
    lo_e, hi_e = RANGES[fmt]
    x = _random_floats(rng, 6000, lo_e, hi_e)
    vals, _ = orc.grid(fmt)
    vals = vals[np.isfinite(vals)]
    k = rng.integers(0, vals.size - 1, 500)
    mids = ((vals[k] + vals[k + 1]) / 2).astype(np.float32)
    assert np.array_equal(mids.astype(np.float64), (vals[k] + vals[k + 1]) / 2)  # exact in fp32
    x = np.concatenate([x, mids])
    codes = orc.round_values(fmt, "rtn", x)
    got = orc.decode(fmt, codes)
    for xi, gi in zip(x, got):
        want = nearest_even(fmt, float(xi))
        assert (gi == want) if isinstance(want, float) else (Fraction(float(gi)) == want)


TORCH_DT = {"fp16": torch.float16, "bf16": torch.bfloat16, "e4m3": torch.float8_e4m3fn}
VIEW_DT = {"fp16": torch.int16, "bf16": torch.int16, "e4m3": torch.uint8}


@pytest.mark.parametrize("fmt", ["fp16", "bf16", "e4m3"])
def test_rtn_matches_native_casts(orc, fmt):
    """RTN == torch's cast bit for bit on 2e5 values over >= 34 binades (+ exact ties)."""
    rng = np.random.default_rng(7)
    lo_e, hi_e = {"fp16": (-30, 15), "bf16": (-130, 120), "e4m3": (-14, 8)}[fmt]
    assert hi_e - lo_e >= 22
    x = _random_floats(rng, 200_000, lo_e, hi_e)
    if fmt == "e4m3":
        x = x[np.abs(x) < 464.0]  # torch's cast does not saturate above 464
    # exact ties between neighbours: 1 + half a step, and a subnormal midpoint
    ties = {"fp16": [1 + 2 ** -11, 1 + 3 * 2 ** -11, 2 ** -25, 3 * 2 ** -25],
            "bf16": [1 + 2 ** -8, 1 + 3 * 2 ** -8, 2 ** -134],
            "e4m3": [1 + 2 ** -4, 1 + 3 * 2 ** -4, 2 ** -10, 3 * 2 ** -10]}[fmt]
    t = np.array(ties, np.float32)
    x = np.concatenate([x, t, -t]).astype(np.float32)
    want = torch.from_numpy(x).to(TORCH_DT[fmt]).view(VIEW_DT[fmt]).numpy()
    want = want.view(np.uint16 if fmt != "e4m3" else np.uint8).astype(np.uint32)
    got = orc.round_values(fmt, "rtn", x)
    assert np.array_equal(got, want)


def test_e4m3_value_set(orc):
    vals, codes = orc.grid("e4m3")
    assert len(vals) == 253            # 256 codes - 2 NaN - duplicate zero
    assert vals.max() == 448.0 and vals.min() == -448.0
    pos = vals[vals > 0]
    assert pos.min() == 2.0 ** -9      # smallest subnormal
    assert 2.0 ** -6 in pos            # smallest normal
    assert np.all(np.diff(pos[pos < 2.0 ** -6]) == 2.0 ** -9)
    all_codes = np.arange(256, dtype=np.uint8)
    ref = torch.from_numpy(all_codes).view(torch.float8_e4m3fn).float().numpy().astype(np.float64)
    mine = orc.decode("e4m3", all_codes)
    nan = np.isnan(ref)
    assert set(np.nonzero(nan)[0]) == {0x7F, 0xFF}
    assert np.array_equal(np.isnan(mine), nan)
    assert np.array_equal(mine[~nan], ref[~nan])


@pytest.mark.parametrize("fmt", ["fp16", "bf16"])
def test_16bit_value_sets(orc, fmt):
    all_codes = np.arange(65536, dtype=np.uint16)
    if fmt == "fp16":
        ref = all_codes.view(np.float16).astype(np.float64)
    else:
        ref = torch.from_numpy(all_codes.view(np.int16)).view(torch.bfloat16).double().numpy()
    mine = orc.decode(fmt, all_codes)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(mine), nan)
    assert np.array_equal(mine[~nan], ref[~nan])
    vals, _ = orc.grid(fmt)
    assert np.all(np.diff(vals) > 0)


@pytest.mark.parametrize("fmt", ["fp16", "bf16"])
def test_overflow_goes_to_infinity(orc, fmt):
    big = {"fp16": [65519.0, 65520.0, 70000.0, 1e30], "bf16": [3.3e38, 3.4e38]}[fmt]
    x = np.array(big + [-b for b in big], np.float32)
    rtn = orc.decode(fmt, orc.round_values(fmt, "rtn", x))
    want = torch.from_numpy(x).to(TORCH_DT[fmt]).double().numpy()
    assert np.array_equal(rtn, want)
    # beyond the largest finite value the outer neighbour is infinity: a threshold
    # of 1 - 2^-24 rounds positive values up to it, a threshold of 0 takes
    # negative values down to it
    U = np.where(x > 0, TWO24 - 1, 0).astype(np.uint32)
    d = orc.decode(fmt, orc.round_values(fmt, "weyl", x, U))
    vmax = float(SPEC[fmt][2])
    assert np.all(np.isinf(d[np.abs(x) > vmax]))


def test_e4m3_saturates(orc):
    x = np.array([448.0, 449.0, 463.0, 465.0, 1e6, np.inf, -500.0, -np.inf], np.float32)
    for rule in ("rtn", "weyl", "sr"):
        U = np.full(x.size, TWO24 - 1, np.uint32)
        d = orc.decode("e4m3", orc.round_values("e4m3", rule, x, U))
        assert np.array_equal(d, np.sign(x) * 448.0)


@pytest.mark.parametrize("fmt", ["fp16", "bf16", "e4m3"])
def test_nan_gives_nan(orc, fmt):
    x = np.array([np.nan, -np.nan], np.float32)
    d = orc.decode(fmt, orc.round_values(fmt, "weyl", x, np.array([5, 6], np.uint32)))
    assert np.all(np.isnan(d))


def test_code_rank_is_value_order(orc):
    vals, codes = orc.grid("e4m3")
    ranks = orc.code_rank("e4m3", codes)
    assert np.array_equal(ranks, np.arange(len(vals)))
    assert orc.code_rank("e4m3", [0x80])[0] == orc.code_rank("e4m3", [0x00])[0]


def test_requantize_e4m3_scale_and_codes(orc):
    """Per-group scale s = fl32(max|h| / 448); RTN codes equal torch's cast of fl32(h * fl32(1/s))."""
    rng = np.random.default_rng(5)
    group = 128
    h = (rng.standard_normal(64 * group) * np.exp(rng.uniform(-8, 4, 64 * group))).astype(np.float32)
    h[:group] = 0.0                       # an all-zero group
    h[group:2 * group] *= np.float32(1e-39)  # a group whose scale would be subnormal
    codes, scale = orc.requantize("e4m3", "rtn", h, group=group)
    hg = h.reshape(-1, group)
    m = np.max(np.abs(hg), axis=1).astype(np.float32)
    s = (m / np.float32(448.0)).astype(np.float32)
    s[s < np.finfo(np.float32).tiny] = 0.0
    assert np.array_equal(scale, s)
    assert np.all(codes[:2 * group] & 0x7F == 0)
    live = s > 0
    r = (np.float32(1.0) / s[live]).astype(np.float32)
    q = (hg[live] * r[:, None]).astype(np.float32)
    assert np.all(np.abs(q) < 464)
    want = torch.from_numpy(q).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(codes.reshape(-1, group)[live], want)
