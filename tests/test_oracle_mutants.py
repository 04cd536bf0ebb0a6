"""Planted mistakes in the oracle must each fail at least one pin (no GPU).

Each mutation edits the oracle's C source text, builds it into a temporary
library and runs the pins against it.  Every mutation stays in bounds.
"""
import os

import pytest

import pins
from oracle import build as obuild
from oracle.oracle import Oracle

MUTATIONS = [
    ("drop_hiA_loB", "a_hi * b_hi + a_hi * b_lo + a_lo * b_hi", "a_hi * b_hi + a_lo * b_hi"),
    ("drop_hiA_hiB", "a_hi * b_hi + a_hi * b_lo + a_lo * b_hi", "a_hi * b_lo + a_lo * b_hi"),
    ("transposed_B_index", "double b_hi = bhk[j], b_lo = blk[j];",
     "double b_hi = bh[(j % K) * N + (k % N)], b_lo = bl[(j % K) * N + (k % N)];"),
    ("drop_loA_hiB", "a_hi * b_hi + a_hi * b_lo + a_lo * b_hi", "a_hi * b_hi + a_hi * b_lo"),
    ("sign_loA_hiB", "a_hi * b_hi + a_hi * b_lo + a_lo * b_hi", "a_hi * b_hi + a_hi * b_lo - a_lo * b_hi"),
    ("keep_loA_loB", "a_hi * b_hi + a_hi * b_lo + a_lo * b_hi",
     "a_hi * b_hi + a_hi * b_lo + a_lo * b_hi + a_lo * b_lo"),
    ("lo_uses_hi_of_B", "double b_hi = bhk[j], b_lo = blk[j];", "double b_hi = bhk[j], b_lo = bhk[j];"),
    ("reversed_k_of_A", "double a_hi = ah[k], a_lo = al[k];",
     "double a_hi = ah[K - 1 - k], a_lo = al[K - 1 - k];"),
    ("truncate_not_round", "if (dropped > 0x8000u || (dropped == 0x8000u && (kept & 1u)))", "if (0)"),
    ("ties_away", "if (dropped > 0x8000u || (dropped == 0x8000u && (kept & 1u)))", "if (dropped >= 0x8000u)"),
    ("ties_to_odd", "(dropped == 0x8000u && (kept & 1u))", "(dropped == 0x8000u && !(kept & 1u))"),
    ("lo_zero_for_nonfinite_hi", "float r = x - hf;", "float r = isfinite(hf) ? x - hf : 0.0f;"),
    ("lo_is_residual_truncated", "*lo = oracle_bf16_rne(r);", "*lo = (uint16_t)(bits_of(r) >> 16);"),
    ("nan_not_quiet", "return (uint16_t)(((u >> 16) & 0x8000u) | 0x7fc0u);", "return (uint16_t)(u >> 16);"),
    ("alpha_ignored", "c[j] = (float)((double)alpha * s[j]);", "c[j] = (float)s[j];"),
    ("alpha_after_round", "c[j] = (float)((double)alpha * s[j]);", "c[j] = alpha * (float)s[j];"),
    ("row_subset_ignored", "int64_t i = rows ? rows[r] : r;\n                for (int64_t k = 0; k < K; ++k) {\n                    uint16_t h, l;\n                    split_one(",
     "int64_t i = r < M ? r : M - 1;\n                for (int64_t k = 0; k < K; ++k) {\n                    uint16_t h, l;\n                    split_one("),
    ("float_accumulator", "s[j] += a_hi * b_hi + a_hi * b_lo + a_lo * b_hi;",
     "s[j] = (float)(s[j] + (a_hi * b_hi + a_hi * b_lo + a_lo * b_hi));"),
    # FP16 forms and INT16 scores
    ("f16_ties_away", "double q = rint(ldexp(a, 10 - E));", "double q = round(ldexp(a, 10 - E));"),
    ("f16_overflow_at_max", "if (a >= 65520.0) return", "if (a > 65504.0) return"),
    ("f16_flush_subnormals", "double q = rint(a * 0x1p24);", "double q = 0.0;"),
    ("f16_lo_not_shifted", "double r = ((double)x - oracle_f16_value(h)) * 1024.0;",
     "double r = ((double)x - oracle_f16_value(h));"),
    ("f16_lo_shift_2048", "double r = ((double)x - oracle_f16_value(h)) * 1024.0;",
     "double r = ((double)x - oracle_f16_value(h)) * 2048.0;"),
    ("exponent_off_by_one", "while (ldexp(maxabs, e + 1) <= 65504.0) ++e;",
     "while (ldexp(maxabs, e + 1) < 65504.0) ++e;"),
    ("exponent_one_too_high", "    return e;\n}", "    return e + 1;\n}"),
    ("weights_unscaled", "return oracle_f16_rne(ldexp((double)w, e));",
     "return oracle_f16_rne((double)w);"),
    ("full_drops_residual", "if (products == 2)", "if (products == 3)"),
    ("full_residual_2^-11", "ldexp(s_hi + ldexp(s_lo, -10), -e)", "ldexp(s_hi + ldexp(s_lo, -11), -e)"),
    ("output_scale_sign", "ldexp(s_hi + ldexp(s_lo, -10), -e)", "ldexp(s_hi + ldexp(s_lo, -10), e)"),
    ("full_residual_subtracted", "ldexp(s_hi + ldexp(s_lo, -10), -e)",
     "ldexp(s_hi - ldexp(s_lo, -10), -e)"),
    ("quant_ties_away", "q[i] = (int16_t)rint(t);", "q[i] = (int16_t)round(t);"),
    ("quant_2^15", "(32767.0 * (double)x[i]) / (double)m", "(32768.0 * (double)x[i]) / (double)m"),
    ("quant_truncates", "q[i] = (int16_t)rint(t);", "q[i] = (int16_t)t;"),
    ("quant_fp32_decision", "(32767.0 * (double)x[i]) / (double)m", "x[i] * (32767.0f / m)"),
    ("quant_fp32_quotient", "(32767.0 * (double)x[i]) / (double)m", "(float)(32767.0f * x[i] / m)"),
    ("unpack_lo_unshifted", "*lo = oracle_f16_rne(((double)q - oracle_f16_value(h)) * 1024.0);",
     "*lo = oracle_f16_rne(((double)q - oracle_f16_value(h)));"),
    ("scores_drop_lolo", "+ ql[k] * bh[k] + ql[k] * bl[k];", "+ ql[k] * bh[k];"),
    ("scores_drop_hilo", "s += qh[k] * bh[k] + qh[k] * bl[k] +", "s += qh[k] * bh[k] +"),
    ("f16w_row_subset_ignored", "int64_t i = rows ? rows[r] : r;\n                for (int64_t k = 0; k < K; ++k) {\n                    uint16_t h, l;\n                    split_f16_one(",
     "int64_t i = r < M ? r : M - 1;\n                for (int64_t k = 0; k < K; ++k) {\n                    uint16_t h, l;\n                    split_f16_one("),
    ("scores_row_subset_ignored", "int64_t i = rows ? rows[r] : r;\n                for (int64_t k = 0; k < K; ++k) {\n                    uint16_t h, l;\n                    oracle_unpack_i16(Q",
     "int64_t i = r < M ? r : M - 1;\n                for (int64_t k = 0; k < K; ++k) {\n                    uint16_t h, l;\n                    oracle_unpack_i16(Q"),
    ("scores_no_alpha", "return (double)alpha * (double)maxQ", "return (double)maxQ"),
    ("scores_factor_fp32",
     "return (double)alpha * (double)maxQ * (double)maxK / (32767.0 * 32767.0);",
     "return (double)(((maxQ / 32767.0f) * (maxK / 32767.0f)) * alpha);"),
]


@pytest.fixture(scope="module")
def source():
    with open(obuild.SOURCE) as f:
        return f.read()


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_mutant_is_caught(tmp_path, source, name, old, new):
    assert source.count(old) == 1, "mutation %s no longer applies" % name
    lib = obuild.build_from_source(source.replace(old, new), str(tmp_path / ("lib_%s.so" % name)),
                                     werror=False)
    orc = Oracle(lib)
    failures = []
    for pin in pins.SMALL_PINS:
        try:
            pin(orc)
        except Exception as e:  # an assertion, or arithmetic a planted mistake broke
            failures.append((pin.__name__, str(e)[:100]))
    assert failures, "mutation %s passed every pin" % name
