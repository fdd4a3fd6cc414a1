"""Planted mistakes in a copy of the oracle must each fail some pin.

The real oracle source is patched in a temporary directory (never in the
tree), rebuilt with the same flags, and the whole pin battery is run against
it; a mutant that passes every pin would mean the pins cannot see that kind
of mistake.
"""
import os

import pytest

import oracle
from tests import pin_battery

MUTANTS = {
    "drop_last_k": ("for (int64_t k = 0; k < K; ++k)", "for (int64_t k = 0; k < K - 1; ++k)"),
    "w_transposed": ("bf16_bits_to_double(W[j * K + k])",
                     "bf16_bits_to_double(W[(k % N) * K + (j % K)])"),
    "x_wrong_row": ("bf16_bits_to_double(X[i * K + k])",
                    "bf16_bits_to_double(X[((i + 1) % M) * K + k])"),
    "residual_sign": ("acc += bf16_bits_to_double(R[i * N + j]);",
                      "acc -= bf16_bits_to_double(R[i * N + j]);"),
    "residual_transposed": ("acc += bf16_bits_to_double(R[i * N + j]);",
                            "acc += bf16_bits_to_double(R[(j % M) * N + (i % N)]);"),
    "float_accumulator": ("double acc = 0.0;", "float acc = 0.0f;"),
    "round_ties_away": ("rint(a / spacing)", "floor(a / spacing + 0.5)"),
    "round_truncate": ("rint(a / spacing)", "trunc(a / spacing)"),
    "round_no_subnormal_clamp": ("if (exp2 < -126) exp2 = -126;", "if (exp2 < -1022) exp2 = -1022;"),
    "ex_bias_dropped": ("        d += bf16_bits_to_double(bias[j]);", "        d += 0.0;"),
    "ex_ldx_ignored": ("bf16_bits_to_double(X[i * ldx + k])", "bf16_bits_to_double(X[i * K + k])"),
    "ex_ldw_ignored": ("bf16_bits_to_double(W[j * ldw + k])", "bf16_bits_to_double(W[j * K + k])"),
    "ex_alpha_on_c": ("d += beta * bf16_bits_to_double(C[i * ldc + j]);",
                      "d += alpha * beta * bf16_bits_to_double(C[i * ldc + j]);"),
    "ex_beta_zero_reads_c": ("if (C && beta != 0.0)", "if (C)"),
    "ex_alpha_dropped": ("double d = alpha * s;", "double d = s;"),
    "glu_silu_dropped": ("return silu(g) * u;", "return g * u;"),
    "glu_sigmoid_sign": ("return z / (1.0 + exp(-z));", "return z / (1.0 + exp(z));"),
    "glu_sigmoid_only": ("return z / (1.0 + exp(-z));", "return 1.0 / (1.0 + exp(-z));"),
    "glu_gate_up_swapped": ("return silu(g) * u;", "return silu(u) * g;"),
    "glu_gate_reads_up": ("g += x * bf16_bits_to_double(Wg[j * K + k]);",
                          "g += x * bf16_bits_to_double(Wu[j * K + k]);"),
    "glu_up_k_shifted": ("u += x * bf16_bits_to_double(Wu[j * K + k]);",
                         "u += x * bf16_bits_to_double(Wu[j * K + (k + 1) % K]);"),
    "glu_float_gate": ("    double g = 0.0;\n", "    float g = 0.0f;\n"),
    "glu_exp_base_2": ("return z / (1.0 + exp(-z));", "return z / (1.0 + exp2(-z));"),
    "i8_int16_accumulator": ("    int64_t acc = 0;\n    for (int64_t k = 0; k < K; ++k)\n        acc += (int64_t)x[k]",
                             "    int16_t acc = 0;\n    for (int64_t k = 0; k < K; ++k)\n        acc += (int64_t)x[k]"),
    "i8_unsigned_weights": ("acc += (int64_t)x[k] * (int64_t)w[k];", "acc += (int64_t)x[k] * (int64_t)(uint8_t)w[k];"),
    "i8_row_scale_by_col": ("double y = (double)sx[i] * (double)sw[j]", "double y = (double)sx[j % (i + 1)] * (double)sw[j]"),
    "i8_col_scale_dropped": ("double y = (double)sx[i] * (double)sw[j]", "double y = (double)sx[i]"),
    "i8_residual_dropped": ("    if (R)\n        y += bf16_bits_to_double(R[i * N + j]);", "    (void)R;"),
    "i8_glu_up_scale_from_gate": ("double u = (double)sx[i] * (double)swu[j]", "double u = (double)sx[i] * (double)swg[j]"),
    "i8_glu_float_gate": ("    double g = (double)sx[i] * (double)swg[j]", "    float g = (double)sx[i] * (double)swg[j]"),
    "f8_exponent_bias_8": ("v = ldexp((double)(8 + m), e - 10);", "v = ldexp((double)(8 + m), e - 11);"),
    "f8_subnormals_as_normals": ("v = ldexp((double)m, -9);", "v = ldexp((double)(8 + m), -10);"),
    "f8_sign_ignored": ("    return sign ? -v : v;\n}\n\nstatic double dot_f8", "    (void)sign;\n    return v;\n}\n\nstatic double dot_f8"),
    "f8_no_nan": ("    if (e == 15 && m == 7)\n        v = NAN;", "    if (0)\n        v = NAN;"),
    "f8_mantissa_dropped_bit": ("int m = b & 7;", "int m = b & 6;"),
    "grp_counts_ignored": ("            if (i >= group_rows(counts, e, Mpad)) continue;\n", "            (void)0;\n"),
    "grp_weight_stride": ("element(i, j, N, K, X + e * Mpad * K, W + e * N * K, NULL);",
                          "element(i, j, N, K, X + e * Mpad * K, W + (e / 2) * N * K, NULL);"),
    "grp_x_stride": ("element(i, j, N, K, X + e * Mpad * K, W + e * N * K, NULL);",
                     "element(i, j, N, K, X + e * K, W + e * N * K, NULL);"),
    "grp_swiglu_up_from_gate": ("element_swiglu(i, j, K, X + e * Mpad * K, Wg + e * N * K, Wu + e * N * K);",
                                "element_swiglu(i, j, K, X + e * Mpad * K, Wg + e * N * K, Wg + e * N * K);"),
    "grp_negative_counts_unclamped": ("return c < 0 ? 0 : (c > Mpad ? Mpad : c);",
                                      "return c < 0 ? Mpad : (c > Mpad ? Mpad : c);"),
}


def _patched_source(src, old, new, tmp_path):
    assert src.count(old) >= 1, f"mutation target {old!r} no longer in the oracle"
    text = src.replace(old, new)
    if "(i + 1) % M" in new or "(j % M)" in new:
        # these mutants need M in scope inside element(); pass it through
        text = text.replace("static double element(int64_t i, int64_t j, int64_t N, int64_t K,",
                            "static int64_t M_;\nstatic double element(int64_t i, int64_t j, int64_t N, int64_t K,")
        text = text.replace("% M)", "% M_)")
        text = text.replace("    if (M < 0 || N < 0 || K < 0) return -1;\n",
                            "    if (M < 0 || N < 0 || K < 0) return -1;\n    M_ = M;\n")
        text = text.replace("    if (M < 0 || N < 0 || K < 0 || n < 0) return -1;\n",
                            "    if (M < 0 || N < 0 || K < 0 || n < 0) return -1;\n    M_ = M;\n")
    path = tmp_path / "mutant.c"
    path.write_text(text)
    return str(path)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    with open(oracle.SOURCE) as f:
        src = f.read()
    old, new = MUTANTS[name]
    path = _patched_source(src, old, new, tmp_path)
    lib = oracle.build(path, str(tmp_path / "libmutant.so"))
    orc = oracle.Oracle(lib)
    failed = []
    for pin in pin_battery.ALL_PINS:
        try:
            pin(orc)
        except AssertionError:
            failed.append(pin.__name__)
    assert failed, f"planted mistake {name} passed every pin"
