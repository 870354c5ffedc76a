"""Pins of the oracle's threshold generators (CPU only).

Expected values the paper prints are read from tests/golden/ (each file names
its passage): the Weyl time sequence (Section 1), Observation "Phase precision"'s
stream counts for a float32 phase, the separation d of the R2 and Knuth offsets
(Appendix B "Offset near-aliasing"), the LD_256 column of Table "Dither
sequences" and the hash-SR unit-test moments (Appendix B "Decode regime"). The
rest rests on mathematics: the decimal constants times 2^32 (Appendix B
"Dithers"), the golden increment and Knuth's constant 2654435761 (Section 6.4
"Three silent pitfalls"), the closed form of the fractional parts of t alpha,
the correlation 1 - 6 d (1 - d) of two rotated streams, the Philox4x32-10
known answers of its authors, and the MurmurHash3 known answers, which pin the
fmix32 finalizer of the hash SR.
"""
from decimal import Decimal, getcontext

import numpy as np
import pytest

from oracle import discrepancy as dsc

from ._golden import records, table

TWO24 = 1 << 24
TWO32 = 1 << 32


def test_weyl_constants_from_the_paper(orc):
    k = orc.weyl_constants()
    # "the above constants times 2^32", read as rounding to nearest
    for name, dec in (("A", "0.7548776662"), ("B", "0.5698402910"), ("L", "0.1234567"),
                      ("S", "0.3141592")):
        exact = Decimal(dec) * TWO32
        assert k[name] == int(exact.to_integral_value(rounding="ROUND_HALF_EVEN")), name
    getcontext().prec = 60
    alpha = (Decimal(5).sqrt() - 1) / 2          # golden-ratio increment phi - 1
    assert k["PHI"] == 2654435769 == int((alpha * TWO32).to_integral_value())
    assert k["PHI"] - 8 == 2654435761            # Knuth's multiplicative-hash constant


@pytest.mark.parametrize("entry", [0, 1, 17, 123456789, 2 ** 33 + 5])
def test_weyl_time_sequence(orc, entry):
    """Per entry the thresholds advance by alpha = phi - 1: 0.618, 0.236, 0.854 ..."""
    U = np.array([orc.thresholds("weyl", 3, 7, t, entry, 1, 16)[0] for t in range(4)], np.int64)
    steps = ((U[1:] - U[0]) % TWO24) / TWO24
    printed = records("weyl_time_sequence.txt")
    assert [int(r[0]) for r in printed] == [1, 2, 3]
    assert np.allclose(steps, [float(r[1]) for r in printed], atol=5e-4)   # three decimals
    getcontext().prec = 40
    alpha = (Decimal(5).sqrt() - 1) / 2
    exact = [float((t * alpha) % 1) for t in (1, 2, 3)]
    assert np.allclose(steps, exact, atol=2 ** -24 * 2)  # 24-bit thresholds of a 32-bit phase


def test_weyl_float_form_agrees_for_small_indices(orc):
    """Hardware form == {o_rc + t alpha} of the float form while r, t are small."""
    alpha = (5 ** 0.5 - 1) / 2
    rng = np.random.default_rng(0)
    for _ in range(300):
        block = int(rng.choice([16, 128]))
        i = int(rng.integers(0, 5000))
        layer, seed, t = int(rng.integers(0, 64)), int(rng.integers(0, 4)), int(rng.integers(0, 5000))
        r, c = divmod(i, block)
        o = (0.7548776662 * (r + 1) + 0.5698402910 * (c + 1) + 0.1234567 * layer
             + 0.3141592 * seed) % 1.0
        u_float = (o + (t * alpha) % 1.0) % 1.0
        u_int = orc.thresholds("weyl", seed, layer, t, i, 1, block)[0] / TWO24
        d = abs(u_int - u_float)
        assert min(d, 1 - d) < 2e-6


def test_r2_offsets_separation(orc):
    printed = table("offset_separation.txt")
    k = orc.weyl_constants()
    beta, gamma, alpha = k["A"] / TWO32, k["B"] / TWO32, k["PHI"] / TWO32
    d = dsc.separation(beta, gamma, alpha)
    assert abs(d - printed["r2"][0]) <= 0.5e-4   # printed to four decimals
    knuth = 2654435761 / TWO32
    assert dsc.separation(knuth, knuth, alpha) <= printed["knuth"][0] + 8 / TWO32  # exact aliasing


def test_rotated_streams_correlate_as_one_minus_6d(orc):
    """Two entries whose offsets differ by dr beta + dc gamma, compared l steps apart,
    are rotations by delta = {dr beta + dc gamma + l alpha}: over time their
    thresholds correlate as 1 - 6 delta (1 - delta)."""
    k = orc.weyl_constants()
    beta, gamma, alpha = k["A"] / TWO32, k["B"] / TWO32, k["PHI"] / TWO32
    block, r0, c0, T = 16, 5, 6, 6000
    U = np.stack([orc.thresholds("weyl", 0, 0, t, 0, block * 10, block) for t in range(T + 20)])
    U = U.astype(np.float64) / TWO24
    for dr, dc, lag in ((1, 0, 0), (0, 1, 0), (1, 2, 3), (-2, 1, 5), (2, -2, 16), (1, 1, 0)):
        i1, i2 = r0 * block + c0, (r0 + dr) * block + (c0 + dc)
        a, b = U[:T, i1], U[lag:T + lag, i2]
        delta = (dr * beta + dc * gamma + lag * alpha) % 1.0
        corr = np.corrcoef(a, b)[0, 1]
        assert abs(corr - (1 - 6 * delta * (1 - delta))) < 4e-3, (dr, dc, lag, corr, delta)


def test_knuth_offsets_alias_with_time(orc):
    """Observation 1: with o_i = i H the next entry gets this entry's next threshold."""
    H, PHI = 2654435761, orc.weyl_constants()["PHI"]
    i = np.arange(0, 4000, dtype=np.uint64)[:, None]
    t = np.arange(0, 200, dtype=np.uint64)[None, :]
    knuth = lambda ii, tt: (((ii * H + tt * PHI) % TWO32) >> 8)
    frac = np.mean(knuth(i + 1, t) == knuth(i, t + 1))
    assert abs(frac - (1 - 8 / 256)) < 0.005     # coincide except where a carry crosses
    # the oracle's offsets do not alias
    U = np.stack([orc.thresholds("weyl", 0, 0, int(tt), 0, 1001, 128) for tt in range(0, 51)])
    assert np.mean(U[:-1, 1:] == U[1:, :-1]) < 0.01


def test_float32_phase_collapses_streams(orc):
    """Observation 2: a float32 phase leaves at most 2^(p-1-k) streams; the integer one keeps all."""
    alpha32 = np.float32((5 ** 0.5 - 1) / 2)
    offsets = (np.arange(1 << 16, dtype=np.float64) / (1 << 16)).astype(np.float32)
    printed = [(int(t), int(n)) for t, n in records("float32_phase_streams.txt")]
    assert len(printed) == 3
    for t, expect in printed:
        phase = np.float32(np.float32(t) * alpha32)
        s = (offsets + phase).astype(np.float32)
        frac = (s - np.floor(s)).astype(np.float32)
        assert len(np.unique(frac)) == expect
    n = 1 << 14
    at0 = orc.thresholds("weyl", 0, 0, 0, 0, n, 16)
    late = orc.thresholds("weyl", 0, 0, 32767, 0, n, 16)
    assert len(np.unique(late)) == len(np.unique(at0)) >= n - 4


def _windows_weyl_oracle(orc, rng, count, W=256):
    wins = []
    for _ in range(count):
        i = int(rng.integers(0, 1 << 30))
        t0 = int(rng.integers(0, 1 << 20))
        wins.append(np.array([orc.thresholds("weyl", 0, 0, t0 + t, i, 1, 16)[0]
                              for t in range(1, W + 1)]) / TWO24)
    return wins


def test_ld256_table(orc):
    """LD_256 of Table "Dither sequences" (64 random phases; paper values +-12%)."""
    rng = np.random.default_rng(2026)
    printed = {k: v[0] for k, v in table("dither_sequences_ld256.txt").items()}

    def ld_float(alpha, windows=64):
        return dsc.local_discrepancy([dsc.weyl_float(alpha, rng.random(), int(rng.integers(0, 1 << 20)),
                                                     256) for _ in range(windows)])

    phi = (1 + 5 ** 0.5) / 2
    increments = {
        "weyl:sqrt2-1": 2 ** 0.5 - 1,
        "weyl:1/(2+phi)": 1 / (2 + phi),
        "weyl:phi-1": phi - 1,
        "weyl:e-2": np.e - 2,
        "weyl:1/4+2^-12": 0.25 + 2 ** -12,
        "weyl:1/3+2^-12": 1 / 3 + 2 ** -12,
        "weyl:1/2+2^-12": 0.5 + 2 ** -12,
    }
    assert set(increments) | {"sr", "weyl:per-entry-uniform[0.2,0.8]"} == set(printed)
    for name, alpha in increments.items():
        assert abs(ld_float(alpha) / printed[name] - 1) < 0.12, name
    # one increment per entry, drawn from U[0.2, 0.8]: the mean is dominated by the
    # increments near simple fractions, so it takes many windows to settle
    per_entry = dsc.local_discrepancy(
        [dsc.weyl_float(rng.uniform(0.2, 0.8), rng.random(), int(rng.integers(0, 1 << 20)), 256)
         for _ in range(4000)])
    assert abs(per_entry / printed["weyl:per-entry-uniform[0.2,0.8]"] - 1) < 0.15
    # the oracle's integer Weyl thresholds of one entry over time
    ld_int = dsc.local_discrepancy(_windows_weyl_oracle(orc, rng, 64))
    assert abs(ld_int / printed["weyl:phi-1"] - 1) < 0.12
    # SR: the oracle's hash over 256 steps of random entries
    wins = []
    for _ in range(200):
        i = int(rng.integers(0, 1 << 30))
        t0 = int(rng.integers(0, 1 << 20))
        wins.append(np.array([orc.thresholds("sr", 0, 0, t0 + t, i, 1, 16)[0]
                              for t in range(1, 257)]) / TWO24)
    assert abs(dsc.local_discrepancy(wins) / printed["sr"] - 1) < 0.08


def _moments(u):
    u = np.asarray(u, np.float64)
    c = u - u.mean()
    lag1 = np.dot(c[1:], c[:-1]) / np.dot(c, c)
    return u.mean(), u.var(), lag1


def test_sr_hash_moments(orc):
    """Hash-SR unit test: the moments of U(0, 1), as the paper's printed ones are."""
    printed = {k: v[0] for k, v in table("sr_hash_moments.txt").items()}
    # the printed moments are those of U(0, 1) up to sampling error
    assert abs(printed["mean"] - 0.5) < 1e-3 and abs(printed["variance"] - 1 / 12) < 1e-3
    assert abs(printed["lag1"]) < 1e-3
    n = 1 << 20
    over_entries = orc.thresholds("sr", 0, 0, 5, 0, n, 16) / TWO24
    m, v, r = _moments(over_entries)
    se = 1 / np.sqrt(12 * n)
    assert abs(m - 0.5) < 5 * se and abs(v - 1 / 12) < 5e-4 and abs(r) < 5 / np.sqrt(n)
    assert abs(m - printed["mean"]) < 1e-3 and abs(v - printed["variance"]) < 1e-3
    T = 1 << 15
    over_time = np.array([orc.thresholds("sr", 1, 3, t, 777, 1, 16)[0] for t in range(T)]) / TWO24
    m, v, r = _moments(over_time)
    assert abs(m - 0.5) < 5 / np.sqrt(12 * T) and abs(v - 1 / 12) < 2e-3 and abs(r) < 5 / np.sqrt(T)


def test_sr_keys_differ_by_seed_layer_step(orc):
    base = orc.thresholds("sr", 0, 0, 0, 0, 4096, 16)
    for args in ((1, 0, 0), (0, 1, 0), (0, 0, 1)):
        other = orc.thresholds("sr", *args, 0, 4096, 16)
        assert np.mean(base == other) < 0.01
    # a step's thresholds over entries are a bijection of the entry index (no repeats)
    assert len(np.unique(orc.thresholds("sr", 0, 0, 9, 0, 1 << 16, 16))) > (1 << 16) - 200


# MurmurHash3_x86_32 (Appleby, SMHasher) ends in the 32-bit finalizer fmix32 that
# the hash SR uses. Its published known answers, (bytes, seed) -> hash, pin the
# oracle's finalizer: the body and tail below are the hash's published
# definition, and every value passes through the oracle's fmix32 at the end.
MURMUR3_KAT = [
    (b"", 0, 0x00000000), (b"", 1, 0x514E28B7), (b"", 0xFFFFFFFF, 0x81F16F39),
    (b"\xff\xff\xff\xff", 0, 0x76293B50), (b"!Ce\x87", 0, 0xF55B516B),
    (b"!Ce\x87", 0x5082EDEE, 0x2362F9DE), (b"!Ce", 0, 0x7E4A8634), (b"!C", 0, 0xA0F7B07A),
    (b"!", 0, 0x72661CF4), (b"\0\0\0\0", 0, 0x2362F9DE), (b"\0\0\0", 0, 0x85F0B427),
    (b"\0\0", 0, 0x30F4C306), (b"\0", 0, 0x514E28B7), (b"aaaa", 0x9747B28C, 0x5A97808A),
    (b"Hello, world!", 0x9747B28C, 0x24884CBA),
    (b"The quick brown fox jumps over the lazy dog", 0x9747B28C, 0x2FA826CD),
]


def _murmur3_x86_32(data: bytes, seed: int, fmix) -> int:
    m32 = 0xFFFFFFFF

    def rotl(x, r):
        return ((x << r) | (x >> (32 - r))) & m32

    def scramble(k):
        return (rotl((k * 0xCC9E2D51) & m32, 15) * 0x1B873593) & m32

    h = seed & m32
    whole = len(data) // 4
    for i in range(whole):
        h ^= scramble(int.from_bytes(data[4 * i:4 * i + 4], "little"))
        h = (rotl(h, 13) * 5 + 0xE6546B64) & m32
    tail = data[4 * whole:]
    if tail:
        h ^= scramble(int.from_bytes(tail, "little"))
    return fmix(h ^ len(data))


@pytest.mark.parametrize("data,seed,want", MURMUR3_KAT)
def test_fmix32_through_murmur3_known_answers(orc, data, seed, want):
    assert _murmur3_x86_32(data, seed, orc.fmix32) == want


def test_sr_threshold_is_the_top_24_bits_of_fmix32(orc):
    """Hash SR (Appendix B "Decode regime"): u = fmix32(i 0x9E3779B1 + key) truncated
    to 24 bits, the key a per-(seed, layer, step) value; with the finalizer pinned
    above, the entry term is checked here: consecutive entries' pre-images differ by
    the paper's entry multiplier."""
    for x in (0, 1, 0x80000000, 0xDEADBEEF, 0xFFFFFFFF):
        assert _fmix32_inverse(orc.fmix32(x)) == x
    seed, layer, t, base = 3, 11, 12345, 2 ** 33 + 5
    got = orc.thresholds("sr", seed, layer, t, base, 8, 16)
    # a threshold keeps 24 of the hash's 32 bits: each entry's pre-image is one of
    # 256 values, and some choice for entry 0 must continue through all eight
    # entries in steps of 0x9E3779B1 (a chance fit has probability about 2^-160)
    pre = [{_fmix32_inverse((int(g) << 8) | lo) for lo in range(256)} for g in got]
    assert any(all(((p0 + k * 0x9E3779B1) & 0xFFFFFFFF) in pre[k] for k in range(1, 8))
               for p0 in pre[0])


def _fmix32_inverse(h: int) -> int:
    """Inverse of the MurmurHash3 finalizer (each xor-shift and odd multiply undone)."""
    m32 = 0xFFFFFFFF

    def unxorshift(x, s):
        y = x
        for _ in range(32 // s + 1):
            y = x ^ (y >> s)
        return y & m32

    h = unxorshift(h, 16)
    h = (h * pow(0xC2B2AE35, -1, 1 << 32)) & m32
    h = unxorshift(h, 13)
    h = (h * pow(0x85EBCA6B, -1, 1 << 32)) & m32
    return unxorshift(h, 16)


def test_rtn_nominal_threshold(orc):
    assert np.all(orc.thresholds("rtn", 5, 5, 5, 0, 64, 16) == 1 << 23)


# --------------------------------------------------------------------------
# Philox4x32-10 SR (the generator behind the paper's SR, Appendix B "Dithers")
# --------------------------------------------------------------------------
# Known-answer vectors of Philox4x32-10 published with the Random123 library
# (Salmon et al., SC 2011): (counter, key) -> output.
PHILOX_KAT = [
    ((0, 0, 0, 0), (0, 0), (0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8)),
    ((0xFFFFFFFF,) * 4, (0xFFFFFFFF,) * 2, (0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD)),
    ((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0),
     (0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1)),
]


@pytest.mark.parametrize("ctr,key,want", PHILOX_KAT)
def test_philox_known_answers(orc, ctr, key, want):
    assert tuple(orc.philox4x32_10(ctr, key)) == want


def test_philox_threshold_mapping(orc):
    """Entry i, step t: word i mod 4 of Philox(counter (i/4 lo, i/4 hi, t, 0), key (seed, layer))."""
    seed, layer, t = 7, 3, 41
    base = 2 ** 34 + 8
    got = orc.thresholds("philox", seed, layer, t, base, 12, 16)
    for k in range(12):
        i = base + k
        q = i >> 2
        words = orc.philox4x32_10((q & 0xFFFFFFFF, q >> 32, t, 0), (seed, layer))
        assert got[k] == words[i & 3] >> 8


def test_philox_moments_and_keys(orc):
    n = 1 << 18
    u = orc.thresholds("philox", 0, 0, 5, 0, n, 16) / TWO24
    m, v, r = _moments(u)
    assert abs(m - 0.5) < 5 / np.sqrt(12 * n) and abs(v - 1 / 12) < 1e-3 and abs(r) < 5 / np.sqrt(n)
    T = 1 << 13
    over_time = np.array([orc.thresholds("philox", 1, 3, t, 777, 1, 16)[0] for t in range(T)]) / TWO24
    m, v, r = _moments(over_time)
    assert abs(m - 0.5) < 5 / np.sqrt(12 * T) and abs(v - 1 / 12) < 4e-3 and abs(r) < 5 / np.sqrt(T)
    base = orc.thresholds("philox", 0, 0, 0, 0, 4096, 16)
    for args in ((1, 0, 0), (0, 1, 0), (0, 0, 1)):
        assert np.mean(base == orc.thresholds("philox", *args, 0, 4096, 16)) < 0.01
