"""Mutation tests of the oracle's pins (CPU only).

Each case builds a copy of the C oracle with one plausible mistake planted (a
strict comparison at a rounding point, ties to odd, a lost saturation, nibbles
swapped, a Weyl coefficient or phase off, a hash or Philox constant changed, a
term dropped from the step) and runs the pins named for it against that copy:
every one of them must fail. The scaled-format step has its own cases in
tests/test_oracle_scaled_step.py.
"""
import pytest

import oracle

from . import test_oracle_decode_ops as t_dec
from . import test_oracle_int as t_int
from . import test_oracle_replay as t_rep
from . import test_oracle_rounding as t_round
from . import test_oracle_step as t_step
from . import test_oracle_thresholds as t_thr
from ._mutants import build_mutant

MUTANTS = {
    "dither: strict comparison at the rounding point": (
        [("pick = (x >= hi - u * (hi - lo)) ? k + 1 : k;",
          "pick = (x > hi - u * (hi - lo)) ? k + 1 : k;")],
        [lambda o: t_round.test_dither_rule_is_eq_dither_exactly(o, "bf16"),
         lambda o: t_round.test_dither_rule_is_eq_dither_exactly(o, "e4m3")]),
    "RTN: ties to the odd code": (
        [("else pick = ((g->code[k] & 1u) == 0) ? k : k + 1;",
          "else pick = ((g->code[k] & 1u) == 0) ? k + 1 : k;")],
        [lambda o: t_round.test_rtn_is_nearest_even_exactly(o, "fp16"),
         lambda o: t_round.test_rtn_is_nearest_even_exactly(o, "e4m3"),
         lambda o: t_round.test_rtn_matches_native_casts(o, "bf16")]),
    "E4M3: no saturation at 448": (
        [("if (x > g->max_finite) x = g->max_finite;", "if (0) x = g->max_finite;")],
        [t_round.test_e4m3_saturates]),
    "INT: strict comparison at the rounding point": (
        [("return (x >= hi - u) ? (int32_t)hi : (int32_t)lo;",
          "return (x > hi - u) ? (int32_t)hi : (int32_t)lo;")],
        [lambda o: t_int.test_dither_rule_is_eq_dither_exactly(o, "int8")]),
    "INT RTN: ties rounded down": (
        [("if (x < mid) return (int32_t)lo;", "if (x <= mid) return (int32_t)lo;")],
        [lambda o: t_int.test_rtn_is_round_half_even(o, "int4")]),
    "INT4: entry order within a byte swapped": (
        [("const int sh = 4 * (int)(k % 2);", "const int sh = 4 * (int)(1 - k % 2);")],
        [t_int.test_int4_packs_two_entries_per_byte]),
    "Weyl: position offset from c instead of c + 1": (
        [("W_B * (uint32_t)(c + 1u)", "W_B * (uint32_t)c")],
        [t_thr.test_weyl_float_form_agrees_for_small_indices]),
    "Weyl: phase one step ahead": (
        [("W_PHI * t;", "W_PHI * (t + 1u);")],
        [t_thr.test_weyl_float_form_agrees_for_small_indices]),
    "Weyl: position coefficient mistyped": (
        [("W_B = from_unit(0.5698402910);", "W_B = from_unit(0.5698402901);")],
        [t_thr.test_weyl_constants_from_the_paper]),
    "Weyl: threshold of 23 bits": (
        [("if (rule == ORC_WEYL) return weyl_acc(i, block, layer, seed, t) >> 8;",
          "if (rule == ORC_WEYL) return weyl_acc(i, block, layer, seed, t) >> 9;")],
        [lambda o: t_thr.test_weyl_time_sequence(o, 0)]),
    "hash SR: finalizer shift 15 for 13": (
        [("h ^= h >> 13;", "h ^= h >> 15;")],
        [lambda o: t_thr.test_fmix32_through_murmur3_known_answers(o, *t_thr.MURMUR3_KAT[14])]),
    "hash SR: Knuth's entry multiplier": (
        [("fmix32((uint32_t)i * 0x9E3779B1u + sr_key(seed, layer, t)) >> 8",
          "fmix32((uint32_t)i * 0x9E3779B9u + sr_key(seed, layer, t)) >> 8")],
        [t_thr.test_sr_threshold_is_the_top_24_bits_of_fmix32]),
    "Philox: nine rounds": (
        [("for (int r = 0; r < 10; ++r) {", "for (int r = 0; r < 9; ++r) {")],
        [lambda o: t_thr.test_philox_known_answers(o, *t_thr.PHILOX_KAT[0])]),
    "Philox: key increment mistyped": (
        [("k1 += 0xBB67AE85u;", "k1 += 0xBB67AE86u;")],
        [lambda o: t_thr.test_philox_known_answers(o, *t_thr.PHILOX_KAT[2])]),
    "Philox: words taken in reverse order": (
        [("return out[i & 3u] >> 8;", "return out[3u - (i & 3u)] >> 8;")],
        [t_thr.test_philox_threshold_mapping]),
    "scale: maximum over qmax + 1": (
        [("float s = m / qmax;", "float s = m / (qmax + 1.0f);")],
        [t_round.test_requantize_e4m3_scale_and_codes,
         lambda o: t_int.test_requantize_block_scale(o, "int8", "rtn")]),
    "step: write without the step size": (
        [("const float w = dx * Bg[n];", "const float w = xv * Bg[n];")],
        [lambda o: t_step.test_fp32_step_is_the_recurrence(o, "mamba2", (2, 6, 8, 32, 2))]),
    "step: skip term dropped from y": (
        [("y[row] = acc + (double)Dv * (double)xv;", "y[row] = acc;")],
        [lambda o: t_step.test_fp32_step_is_the_recurrence(o, "mamba1", (3, 40, 1, 16, 1))]),
    "step: every head reads group 0's B": (
        [("const float *Bg = B + (b * ngroups + g) * dstate;",
          "const float *Bg = B + (b * ngroups) * dstate;")],
        [lambda o: t_step.test_fp32_step_is_the_recurrence(o, "mamba2", (2, 6, 8, 32, 2))]),
    "E4M3: exponent bias 8": (
        [("{8, 4, 3, 7, 0},", "{8, 4, 3, 8, 0},")],
        [t_round.test_e4m3_value_set]),
    "fp16: subnormals one binade low": (
        [("v = ldexp((double)m, 1 - d->bias - d->mbits);", "v = ldexp((double)m, -d->bias - d->mbits);")],
        [lambda o: t_round.test_16bit_value_sets(o, "fp16"), t_round.test_e4m3_value_set]),
    "E4M3: 0x7E read as NaN": (
        [("e == emax_field && m == (1u << d->mbits) - 1u", "e == emax_field && m >= (1u << d->mbits) - 2u")],
        [t_round.test_e4m3_value_set]),
    "softplus: threshold applied below 20 as well": (
        [("if (v > 20.0f) return v;", "if (v > 0.0f) return v;")],
        [t_dec.test_softplus_dt_and_gate]),
    "gate: silu with the wrong sign": (
        [("static double silu(double z) { return z / (1.0 + exp(-z)); }",
          "static double silu(double z) { return z / (1.0 + exp(z)); }")],
        [t_dec.test_softplus_dt_and_gate, t_dec.test_conv1d_update]),
    "conv1d: new input at the front of the window": (
        [("s[width - 1] = x[b * channels + c];", "s[0] = x[b * channels + c];")],
        [t_dec.test_conv1d_update]),
    "replay: reference driven by the stored state": (
        [("href[i] = fmaf(at, href[i], wt);", "href[i] = fmaf(at, hq[i], wt);")],
        [lambda o: t_rep.test_proposition1_count_through_the_replay(o, "weyl"),
         lambda o: t_rep.test_proposition1_count_through_the_replay(o, "sr")]),
    "replay: step counter not advanced": (
        [("step0 + (uint32_t)t, entry_base", "step0, entry_base")],
        [lambda o: t_rep.test_replay_follows_the_fused_step(o, "fp16", "weyl")]),
}


@pytest.mark.parametrize("mutant", sorted(MUTANTS))
def test_pins_reject_planted_mistakes(tmp_path, mutant):
    edits, pins = MUTANTS[mutant]
    so = build_mutant(str(tmp_path), edits)
    with oracle.using_library(so):
        for i, pin in enumerate(pins):
            with pytest.raises(AssertionError):
                pin(oracle)
