"""The oracle's pins reject planted mistakes.

Each case below plants one plausible mistake in a copy of ``oracle/oracle.c``
(a wrong rounding rule, a dropped or wrong term, a flipped sign, a wrong index,
a transposed operand, a lost carry, a changed order), builds it, routes the
oracle module through it and runs the pins named for it: at least one of them
must fail.  A pin that passes a planted mistake would not be pinning anything.
The mistakes are planted on the CPU only.
"""
import os

import pytest

import oracle as O
import test_oracle_depths as DP
import test_oracle_gemm as G
import test_oracle_split as SP

SRC = os.path.join(os.path.dirname(O.__file__), "oracle.c")

# name -> (text in oracle.c, replacement, pins that must catch it)
MUTATIONS = {
    "bf16_ties_away_from_zero": (
        "return ((lo >> 16) & 1u) ? (uint16_t)(hi >> 16) : (uint16_t)(lo >> 16);",
        "return (uint16_t)(hi >> 16);",
        [SP.test_bf16_rne_f32_definition_samples]),
    "fp32_residual_sign_flipped": (
        "res = res - orc_bf16_value(h);",
        "res = orc_bf16_value(h) - res;",
        [SP.test_split_f32_residual_shrinks_by_u_bf16, G.test_sgemm_identity_reconstructs_input]),
    "fp64_to_bf16_double_rounding": (
        "double r = nearbyint(az / spacing) * spacing;",
        "double r = nearbyint((double)(float)az / spacing) * spacing;",
        [lambda: SP.test_bf16_rne_f64_against_fractions(1)]),
    "ceil_log2_off_at_powers_of_two": (
        "return (f == 0.5) ? e - 1 : e;",
        "return e;",
        [SP.test_split_f64_adversarial, SP.test_split_f64_bf16_exact_matrix_has_one_slice,
         lambda: SP.test_split_f64_exact_properties(O.SPLIT_SYM, "uniform")]),
    "projection_constant_literal_by_default": (
        "ldexp(0.75, vr + 45)",
        "ldexp(1.0, vr + 45)",
        [lambda: SP.test_split_f64_exact_properties(O.SPLIT_SYM, "uniform"),
         lambda: G.test_table_accuracy_fp64_columns(256)]),
    "fp64_residual_sign_flipped": (
        "W[i] = a - (double)orc_bf16_value(h);",
        "W[i] = a + (double)orc_bf16_value(h);",
        [lambda: SP.test_split_f64_exact_properties(O.SPLIT_SYM, "normal")]),
    "zero_residual_not_detected": (
        "if (m == 0.0 || !isfinite(m)) { zero_from = lev; break; }",
        "if (!isfinite(m)) { zero_from = lev; break; }",
        [SP.test_split_f64_zero_and_single_nonzero, SP.test_split_f64_bf16_exact_matrix_has_one_slice]),
    "dgemm_drops_last_product_of_each_diagonal": (
        "for (int i = 0; i <= l; ++i) {\n                int j = l - i;",
        "for (int i = 0; i < l; ++i) {\n                int j = l - i;",
        [lambda: G.test_dgemm_integers_give_exact_product(10),
         lambda: G.test_dgemm_identity_sums_retained_slices(6)]),
    "dgemm_extra_diagonal": (
        "for (int l = 0; l < d; ++l) {               /* diagonal l = i + j */",
        "for (int l = 0; l <= d && l < 6; ++l) {     /* diagonal l = i + j */",
        [lambda: G.test_dgemm_identity_sums_retained_slices(6),
         lambda: G.test_table_accuracy_fp64_columns(256)]),
    "dgemm_selection_drops_sixth_slice": (
        "if (i > 5 || j > 5) continue;       /* six slices per operand */",
        "if (i > 4 || j > 4) continue;       /* six slices per operand */",
        [lambda: DP.test_structured_operands_closed_form(7)]),
    "dgemm_selection_inclusive_bound": (
        "for (int l = 0; l < d; ++l) {               /* diagonal l = i + j */",
        "for (int l = 0; l <= d; ++l) {              /* diagonal l = i + j */",
        [lambda: DP.test_structured_operands_closed_form(6)]),
    "dgemm_product_count_map_shifted": (
        "if (i + j < d) ++n;",
        "if (i + j <= d) ++n;",
        [lambda: DP.test_structured_operands_closed_form(1), lambda: DP.test_other_product_counts_rejected(2)]),
    "dgemm_order_inside_diagonal_reversed": (
        "for (int i = 0; i <= l; ++i) {\n                int j = l - i;",
        "for (int i = l; i >= 0; --i) {\n                int j = l - i;",
        [lambda: G.test_dgemm_definition_bruteforce_order_sensitive(21)]),
    "dgemm_slice_index_transposed": (
        "const uint16_t *Ai = Av + (size_t)i * M * K + (size_t)m * K;\n                const uint16_t *Bj = Bv + (size_t)j * K * N + n;",
        "const uint16_t *Ai = Av + (size_t)j * M * K + (size_t)m * K;\n                const uint16_t *Bj = Bv + (size_t)i * K * N + n;",
        [lambda: G.test_dgemm_definition_bruteforce_order_sensitive(21)]),
    "dgemm_accumulates_in_fp32": (
        "c = c + (double)p32;                /* widen exactly, add in FP64 */",
        "c = (double)((float)c + p32);",
        [lambda: G.test_dgemm_integers_give_exact_product(21),
         lambda: G.test_table_accuracy_fp64_columns(256)]),
    "dgemm_whole_k_panel": (
        "double c = 0.0;                                 /* FP64 output accumulator */",
        "double c = 0.0; kc = K > 0 ? K : 1;             /* FP64 output accumulator */",
        [lambda: G.test_dgemm_definition_bruteforce(21, (2, 3, 520))]),
    "sgemm_wrong_cross_product": (
        "{{1, 1}, {1, 0}, {2, 0}, {0, 0}, {0, 1}, {0, 2}}",
        "{{2, 1}, {1, 0}, {2, 0}, {0, 0}, {0, 1}, {0, 2}}",
        [G.test_sgemm_cross_products_integers]),
    "sgemm_reuse_order_changed": (
        "{{1, 1}, {1, 0}, {2, 0}, {0, 0}, {0, 1}, {0, 2}}",
        "{{0, 0}, {1, 0}, {2, 0}, {1, 1}, {0, 1}, {0, 2}}",
        [lambda: G.test_sgemm_definition_bruteforce((2, 3, 300))]),
    "sgemm_b_index_transposed": (
        "for (i64 k = p0; k < p1; ++k) xacc_add_product(&x, Ai[k], Bj[(size_t)k * N]);\n            t = t + xacc_round_f32(&x);",
        "for (i64 k = p0; k < p1; ++k) xacc_add_product(&x, Ai[k], Bj[(size_t)k]);\n            t = t + xacc_round_f32(&x);",
        [G.test_sgemm_identity_reconstructs_input]),
    "panel_rounding_ties_away": (
        "if (guard && (sticky || (kept & 1u))) kept += 1;",
        "if (guard) kept += 1;",
        [G.test_dot_bf16_f32_ties_to_even]),
    "exact_accumulator_loses_carry": (
        "c = c1 | c2;",
        "c = c1;",
        [G.test_dot_bf16_f32_correct_rounding_wide_range]),
    "inexact_panel_never_flagged": (
        "    if (!isfinite(f)) return 0;\n    xacc d = *a;",
        "    return 1;\n    xacc d = *a;",
        [G.test_dgemm_inexact_panel_flag_long_panel,
         lambda: G.test_dgemm_inexact_flag_matches_definition(-45, 21)]),
    "double_double_drops_product_error": (
        "c += pe + te;",
        "c += te;",
        [G.test_dd_reference_error_bound]),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_reject_planted_mistake(name, tmp_path):
    old, new, pins = MUTATIONS[name]
    with open(SRC) as f:
        text = f.read()
    assert text.count(old) >= 1, f"mutation site not found: {old[:50]}"
    src = tmp_path / "oracle_mutant.c"
    src.write_text(text.replace(old, new, 1))
    so = O.compile_source(str(src), str(tmp_path / "liboracle_mutant.so"))
    failures = []
    with O.using_library(so):
        for pin in pins:
            try:
                pin()
            except AssertionError as e:
                failures.append(repr(e)[:120])
    assert failures, f"no pin rejected the planted mistake '{name}'"
