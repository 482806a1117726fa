"""Mutation tests for the oracle's pins (CPU only).

Each case copies sj_oracle.c, plants one plausible mistake (a dropped term, a
wrong sign or index, a strict instead of an inclusive test, a decoding slip,
a float accumulator ...), builds the copy into a temporary library and runs
every pin against it.  The pins are only worth something if each planted
mistake makes at least one of them fail.
"""
import ctypes
import os
import shutil

import pytest

import oracle
from oracle.oracle import _SRC, build, load
from pins import PINS

IP_LINE = "        s += elem(dtype, P, i * d + k) * elem(dtype, Q, j * d + k);"
L2_LINE = "        double t = elem(dtype, P, i * d + k) - elem(dtype, Q, j * d + k);"

MUTANTS = {
    "ip_strict": [("(score >= thr) : (score <= thr)", "(score > thr) : (score <= thr)")],
    "l2_strict": [("(score >= thr) : (score <= thr)", "(score >= thr) : (score < thr)")],
    "ip_drops_last_term": [("    for (int64_t k = 0; k < d; ++k)\n" + IP_LINE,
                            "    for (int64_t k = 0; k + 1 < d; ++k)\n" + IP_LINE)],
    "ip_wrong_q_index": [(IP_LINE, IP_LINE.replace("j * d + k", "j * d + (d - 1 - k)"))],
    "ip_uses_p_twice": [(IP_LINE, IP_LINE.replace("elem(dtype, Q, j", "elem(dtype, P, i"))],
    "l2_wrong_sign": [(L2_LINE, L2_LINE.replace(") - elem", ") + elem"))],
    "l2_abs_not_square": [("        s += t * t;", "        s += fabs(t);")],
    "l2_drops_first_term": [("        double t = elem", "        if (k == 0) continue;\n"
                             "        double t = elem")],
    "float_accumulator": [("    double s = 0.0;\n    for (int64_t k = 0; k < d; ++k)\n" + IP_LINE,
                           "    float s = 0.0f;\n    for (int64_t k = 0; k < d; ++k)\n" + IP_LINE)],
    "f16_subnormal_scale": [("ldexp((double)f, -24)", "ldexp((double)f, -25)")],
    "f16_exponent_bias": [("ldexp((double)(1024 + f), e - 25)", "ldexp((double)(1024 + f), e - 24)")],
    "f16_no_hidden_bit": [("ldexp((double)(1024 + f), e - 25)", "ldexp((double)(f), e - 25)")],
    "bf16_exponent_bias": [("ldexp((double)(128 + f), e - 134)", "ldexp((double)(128 + f), e - 133)")],
    "bf16_short_fraction": [("int f = h & 0x7f;", "int f = h & 0x3f;")],
    "bf16_drops_sign": [("    int sign = (h >> 15) & 1;\n    int e = (h >> 7)",
                         "    int sign = 0;\n    int e = (h >> 7)")],
    "i8_read_unsigned": [("(double)((const int8_t *)X)[idx]", "(double)((const uint8_t *)X)[idx]")],
    "pairs_swapped": [("out_pairs[2 * total] = (uint32_t)i;\n"
                       "                out_pairs[2 * total + 1] = ro[r].pairs[t];",
                       "out_pairs[2 * total + 1] = (uint32_t)i;\n"
                       "                out_pairs[2 * total] = ro[r].pairs[t];")],
    "skips_last_q_row": [("for (int64_t j = 0; j < n_q; ++j) {", "for (int64_t j = 0; j + 1 < n_q; ++j) {")],
    "skips_last_p_row": [("    for (int64_t r = 0; r < n_rows; ++r) {\n        int64_t i = rows ? rows[r] : r;\n"
                          "        row_out *o",
                          "    for (int64_t r = 0; r < n_rows - 1; ++r) {\n"
                          "        int64_t i = rows ? rows[r] : r;\n        row_out *o")],
    # LSH-bucketed join
    "lsh_sign_strict": [("v = z >= 0.0 ? 1 : 0;", "v = z > 0.0 ? 1 : 0;")],
    "lsh_truncates_quotient": [("(int64_t)floor((z + (double)B[f]) / (double)w)",
                                "(int64_t)((z + (double)B[f]) / (double)w)")],
    "lsh_drops_offset": [("floor((z + (double)B[f]) / (double)w)", "floor(z / (double)w)")],
    "lsh_key_order_reversed": [("<< (beta * u)", "<< (beta * (k - 1 - u))")],
    "lsh_a_transposed": [("(double)A[f * d + m]", "(double)A[m * (L * k) + f]")],
    "lsh_skips_last_table": [("for (int64_t t = 0; t < L && !collide; ++t)",
                              "for (int64_t t = 0; t + 1 < L && !collide; ++t)")],
    "lsh_no_exact_test": [("if (matches(metric, sc, thr) &&\n                    push_u32(&ro[i]",
                           "if (push_u32(&ro[i]")],
    # Section 4's front ends: rounding to binary16 / bfloat16, normalisation,
    # Hamming distance
    "round_ties_away": [("if (diff > 0.5 || (diff == 0.5 && fmod(f, 2.0) != 0.0))",
                         "if (diff >= 0.5)")],
    "round_truncates": [("        f += 1.0;\n    return f;", "        f += 0.0;\n    return f;")],
    "f16_round_subnormal_spacing": [("round_half_even_scaled(a, -24)",
                                     "round_half_even_scaled(a, -25)")],
    "bf16_round_precision": [("round_half_even_scaled(a, e - 7)",
                              "round_half_even_scaled(a, e - 8)")],
    "f16_round_no_infinity": [("    if (e > 15)\n        return sign | 0x7c00;", "")],
    "normalize_no_sqrt": [("double norm = sqrt(s);", "double norm = s;")],
    "normalize_drops_last_square": [("        for (int64_t k = 0; k < d; ++k) {\n"
                                     "            double x = elem(dtype, X, i * d + k);",
                                     "        for (int64_t k = 0; k + 1 < d; ++k) {\n"
                                     "            double x = elem(dtype, X, i * d + k);")],
    "hamming_skips_last_bit": [("    for (int64_t m = 0; m < d; ++m)\n        h += bit_at",
                                "    for (int64_t m = 0; m + 1 < d; ++m)\n        h += bit_at")],
    "hamming_strict": [("(double)or_hamming(P, i, Q, j, d) <= r", "(double)or_hamming(P, i, Q, j, d) < r")],
    "hamming_bit_order": [("return (X[row * stride + m / 8] >> (m % 8)) & 1;",
                           "return (X[row * stride + m / 8] >> (7 - m % 8)) & 1;")],
}


SLOW_PINS = {"decode_bf16_exhaustive", "real_scores_within_summation_bound",
             "hypercube_ip_counts", "lsh_sign_collision_probability",
             "lsh_quantised_collision_probability"}


@pytest.fixture(scope="module")
def mutant_dir(tmp_path_factory):
    return tmp_path_factory.mktemp("oracle_mutants")


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, mutant_dir):
    src = open(_SRC).read()
    for old, new in MUTANTS[name]:
        assert old in src, f"mutation site for {name} not found in sj_oracle.c"
        src = src.replace(old, new)
    d = mutant_dir / name
    d.mkdir()
    c = d / "sj_oracle.c"
    c.write_text(src)
    so = build(force=True, src=str(c), out=str(d / "libmut.so"))
    lib = load(so)
    caught = None
    # cheap pins first; one failing pin is enough
    order = sorted(PINS, key=lambda n: (n in SLOW_PINS, n))
    for pin_name in order:
        try:
            PINS[pin_name](lib)
        except Exception as e:  # a crash of the mutant counts as caught too
            caught = (pin_name, type(e).__name__)
            break
    assert caught, f"no pin catches the planted mistake {name!r}"
