"""Planted-mistake tests for the oracle's pins (CPU only).

Each mutant is a copy of the oracle source with one plausible mistake (a
dropped term, a wrong sign, index or constant, a transposed operand). It is
compiled with gcc into a temporary library and the pin suite is run against
it: at least one pin must fail, otherwise the pins do not cover that part of
the oracle. The mistakes are planted in the oracle only, on the CPU.
"""
import os
import subprocess

import pytest

import oracle
from tests import oracle_pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "vcheck_oracle.c")

# (name, exact snippet of the oracle, replacement)
MUTANTS = [
    ("gate_rtol_on_cand", "rtol[p] * fabs(r)", "rtol[p] * fabs(c)"),
    ("gate_strict_lt", "finite && d <= t", "finite && d < t"),
    ("gate_drop_equality", "(c == r) || (finite", "(finite"),
    ("gate_equal_nan_or", "equal_nan[p] && c_nan && r_nan", "equal_nan[p] && (c_nan || r_nan)"),
    ("gate_drop_atol", "const double t = atol[p] + rtol[p] * fabs(r);",
     "const double t = rtol[p] * fabs(r);"),
    ("decode_f16_subnormal_scale", "ldexp((double)frac, -24)", "ldexp((double)frac, -25)"),
    ("decode_f16_bias", "ldexp((double)(1024 + frac), expo - 25)",
     "ldexp((double)(1024 + frac), expo - 24)"),
    ("decode_f16_inf_nan_swap", "frac ? NAN : INFINITY", "frac ? INFINITY : NAN"),
    ("decode_bf16_shift", "(uint32_t)h << 16", "(uint32_t)h << 15"),
    ("classify_inf_as_nan", "st->inf_cand += c_inf;", "st->inf_cand += c_nan;"),
    ("argmax_abs_last_tie", "d > st->max_abs", "d >= st->max_abs"),
    ("argmax_rel_last_tie", "q > st->max_rel", "q >= st->max_rel"),
    ("argmax_abs_no_init", "st->argmax_abs < 0 || d > st->max_abs", "d > st->max_abs"),
    ("rel_signed_ref", "d / fabs(r)", "d / r"),
    ("rel_undef_inverted", "} else if (c != 0.0) {", "} else if (c == 0.0) {"),
    ("sum_rel_adds_abs", "st->sum_rel += q;", "st->sum_rel += d;"),
    ("finite_ignores_inf", "const int finite = !c_nan && !c_inf && !r_nan && !r_inf;",
     "const int finite = !c_nan && !r_nan;"),
    ("tile_transposed", "(row / tile_h) * tiles_c + col / tile_w",
     "(col / tile_w) * tiles_r + row / tile_h"),
    ("tile_all_pairs", "      if (p != primary) continue;\n", "      if (0) continue;\n"),
    ("first_k_off_by_one", "first_k[n_found++] = i;", "first_k[n_found++] = i + 1;"),
    ("zero_bits_only", "integ->zero_cand += decode_one(dtype, cand, i) == 0.0;",
     "integ->zero_cand += bc == 0;"),
    ("eqfirst_by_value", "integ->eqfirst_cand += bc == first_cand;",
     "integ->eqfirst_cand += decode_one(dtype, cand, i) == decode_one(dtype, cand, 0);"),
    ("fp16rep_mask", "(w & 0x1fffu) == 0", "(w & 0x0fffu) == 0"),
    ("fp16rep_subnormal_grid", "double s = a * 0x1p24;", "double s = a * 0x1p23;"),
    ("fp16rep_upper_bound", "a <= 65504.0", "a <= 65536.0"),
    ("bf16rep_mask", "(w & 0xffffu) == 0", "(w & 0xff00u) == 0"),
    ("all_zero_ignores_ref", "integ->zero_cand == un && n >= 1 && integ->zero_ref < un",
     "integ->zero_cand == un && n >= 1"),
    ("constant_allows_zero", "integ->eqfirst_cand == un && n >= 2 && integ->zero_cand < un &&",
     "integ->eqfirst_cand == un && n >= 2 &&"),
    ("copy_ignores_ref", "(eq_cand >> j & 1u) && !(eq_ref >> j & 1u)", "(eq_cand >> j & 1u)"),
    ("copy_eligibility_dtype", "input_dtype[j] == dtype && input_numel[j] == n",
     "input_numel[j] == n"),
    ("lowprec_fp16_not_suppressed", "integ->fp16rep_cand == un && integ->bf16rep_cand < un &&",
     "integ->fp16rep_cand == un &&"),
    ("suite_ignores_flags", "if (ok && (!flags || flags[c] == 0)) certified += 1;",
     "if (ok) certified += 1;"),
    ("suite_ignores_status", "const int ok = status[c] >= 0 &&", "const int ok ="),
    ("tstats_argmin_last_tie", "v < out->min", "v <= out->min"),
    ("np_ratio_last_tie", "q > out->max_ratio", "q >= out->max_ratio"),
    ("hash_no_index", "orc_splitmix_finalize(w ^ ((uint64_t)i * 0x9E3779B97F4A7C15ull))",
     "orc_splitmix_finalize(w)"),
    ("hash_shift", "  z ^= z >> 27;\n", "  z ^= z >> 28;\n"),
    ("hash_word_big_endian", "<< (8 * b);", "<< (56 - 8 * b);"),
    ("hash_tail_dropped", "8 * i < nbytes; ++i", "8 * i + 8 <= nbytes; ++i"),
    ("hash_no_dtype", "^ ((uint64_t)dtype << 56)", "^ 0"),
    ("np_fail_ge", "const int fail = d > t;", "const int fail = d >= t;"),
    ("np_round_ties_up", "(frac == 0.5 && fmod(kr, 2.0) != 0.0)", "(frac == 0.5)"),
    ("np_key_unsigned", "return (h & 0x8000u) ? -mag : mag;", "return h;"),
    ("np_ratio_bin_off", "const int b = p - 1 > ORC_RATIO_BINS - 1 ? ORC_RATIO_BINS - 1 : p - 1;",
     "const int b = p > ORC_RATIO_BINS - 1 ? ORC_RATIO_BINS - 1 : p;"),
    ("tstats_zero_in_hist", "if (v != 0.0) out->hist[hist_bin(v)]++;", "out->hist[hist_bin(v)]++;"),
    ("tstats_bin_off_by_one", "const int b = (p - 1) - ORC_HIST_EMIN + 1;",
     "const int b = p - ORC_HIST_EMIN + 1;"),
    ("tstats_inf_in_sums", "    if (isinf(v)) {\n      out->inf++;\n      continue;\n    }",
     "    if (isinf(v)) {\n      out->inf++;\n    }"),
    ("tstats_sum_sq_abs", "out->sum_sq += v * v;", "out->sum_sq += fabs(v);"),
]


def _run_pins(lib):
    failed = []
    for pin in oracle_pins.PINS:
        try:
            pin(lib)
        except Exception as exc:  # noqa: BLE001 - any failure means the pin caught it
            failed.append("%s: %s" % (pin.__name__, type(exc).__name__))
            break
    return failed


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, name, old, new):
    src = open(SRC).read()
    assert src.count(old) == 1, "mutation site for %s must occur exactly once" % name
    mut_src = tmp_path / ("mut_%s.c" % name)
    mut_src.write_text(src.replace(old, new))
    hdr = os.path.join(os.path.dirname(SRC), "vcheck_oracle.h")
    (tmp_path / "vcheck_oracle.h").write_text(open(hdr).read())
    so = tmp_path / ("libmut_%s.so" % name)
    subprocess.run(["gcc", *oracle.GCC_FLAGS, "-o", str(so), str(mut_src), "-lm"], check=True)
    lib = oracle.load(str(so))
    assert _run_pins(lib), "no pin detects mutant %s" % name
