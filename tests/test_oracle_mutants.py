"""Strength of the oracle's pins: copies of the oracle with one planted
mistake each (built on the CPU, never used anywhere else) must each fail at
least one pin.  The real oracle source is read, not modified."""
import os
import subprocess

import pytest

from oracle import build_oracle
from oracle import oracle as O
import oracle_pins as P
import oracle_pins_fused as PF
import oracle_pins_acc16 as PA

# (name, text in oracle_gba.c, replacement) -- each a plausible slip.
MUTANTS = [
    ("sign_of_product", "acc[j] = acc[j] + a * brow[j];", "acc[j] = acc[j] - a * brow[j];"),
    ("dropped_bias", "(J->biasd ? J->biasd[j] : 0.0)", "0.0"),
    ("relu_before_bias", "double pre = acc[j] + (J->biasd ? J->biasd[j] : 0.0);\n"
     "        o[j] = (J->act == OR_ACT_RELU) ? (pre > 0.0 ? pre : 0.0) : pre;",
     "double r = (J->act == OR_ACT_RELU) ? (acc[j] > 0.0 ? acc[j] : 0.0) : acc[j];\n"
     "        o[j] = r + (J->biasd ? J->biasd[j] : 0.0);"),
    ("a_transposed", "J->layout_a == OR_ROW ? J->A[i * J->lda + k]",
     "J->layout_a == OR_COL ? J->A[i * J->lda + k]"),
    ("b_transposed", "layout_b == OR_ROW ? B[k * ldb + j]", "layout_b == OR_COL ? B[k * ldb + j]"),
    ("last_k_dropped", "for (int64_t k = 0; k < J->K; ++k) {", "for (int64_t k = 0; k + 1 < J->K; ++k) {"),
    ("first_k_dropped", "for (int64_t k = 0; k < J->K; ++k) {", "for (int64_t k = 1; k < J->K; ++k) {"),
    ("exponent_bias", "expo - 25", "expo - 24"),
    ("subnormal_scale", "ldexp((double)frac, -24)", "ldexp((double)frac, -25)"),
    ("implicit_bit", "(double)(1024 + frac)", "(double)(frac)"),
    ("relu_leaky", "(pre > 0.0 ? pre : 0.0)", "(pre > 0.0 ? pre : 0.01 * pre)"),
    ("relu_clamps_small", "(pre > 0.0 ? pre : 0.0)", "(pre > 0.5 ? pre : 0.0)"),
    ("relu_inverted", "J->act == OR_ACT_RELU", "J->act == OR_ACT_NONE"),
    ("lda_ignored", "J->A[i * J->lda + k] : J->A[k * J->lda + i]",
     "J->A[i * J->K + k] : J->A[k * J->M + i]"),
    ("ldb_ignored", "B[k * ldb + j] : B[j * ldb + k]", "B[k * N + j] : B[j * K + k]"),
    ("bias_index_by_row", "J->biasd ? J->biasd[j] : 0.0", "J->biasd ? J->biasd[i % J->N] : 0.0"),
    ("b_row_index", "const double *brow = J->Bd + k * J->N;",
     "const double *brow = J->Bd + (J->K - 1 - k) * J->N;"),
]

# Slips in the wider-idiom oracle (prologue, second product, bias kinds and
# signs, Sigmoid/Tanh); none of them reads outside the operands.
MUTANTS += [
    ("prologue_abs", "v = v > 0.0 ? v : 0.0;", "v = v > 0.0 ? v : -v;"),
    ("prologue_ignored", "if (pro_relu)\n        v = v > 0.0 ? v : 0.0;", "if (0)\n        v = v > 0.0 ? v : 0.0;"),
    ("prologue_negative_part", "v = v > 0.0 ? v : 0.0;", "v = v < 0.0 ? v : 0.0;"),
    ("second_sign_flipped", "c[j] - r[j]", "c[j] + r[j]"),
    ("second_always_added", "J->second > 0 ? c[j] + r[j]", "J->second != 0 ? c[j] + r[j]"),
    ("second_last_k_dropped", "J->Qd, J->K2, i, r)", "J->Qd, J->K2 - 1, i, r)"),
    ("second_uses_lda", "product_row(J, J->P, J->ldp,", "product_row(J, J->P, J->lda,"),
    ("full_bias_ignores_ld", "J->bias[i * J->ldbias + j]", "J->bias[i * J->N + j]"),
    ("full_bias_row_zero", "J->bias[i * J->ldbias + j]", "J->bias[j]"),
    ("bias_sign_ignored", "pre = J->bias_sign > 0 ? z + b : z - b;", "pre = z + b;"),
    ("sigmoid_sign", "1.0 / (1.0 + exp(-x))", "1.0 / (1.0 + exp(x))"),
    ("sigmoid_scale", "1.0 / (1.0 + exp(-x))", "1.0 / (1.0 + exp(-2.0 * x))"),
    ("tanh_half_argument", "return tanh(x);", "return tanh(0.5 * x);"),
    ("tanh_as_sigmoid", "case OR_ACT_TANH: return tanh(x);", "case OR_ACT_TANH: return 1.0 / (1.0 + exp(-x));"),
    ("fused_relu_leaky", "case OR_ACT_RELU: return x > 0.0 ? x : 0.0;", "case OR_ACT_RELU: return x > 0.0 ? x : 0.01 * x;"),
    ("fused_first_k_dropped", "for (int64_t k = 0; k < K; ++k) {\n        double x", "for (int64_t k = 1; k < K; ++k) {\n        double x"),
    ("fused_q_rows_reversed", "d[k * N + j] = oracle_f16_to_f64", "d[(K - 1 - k) * N + j] = oracle_f16_to_f64"),
    ("fused_a_k_reversed", "left_elem(J->layout_a, X, ldx, i, k, J->pro_relu)",
     "left_elem(J->layout_a, X, ldx, i, K - 1 - k, J->pro_relu)"),
]

# Slips in the binary16 rounding and the fp16-accumulation reading.
MUTANTS += [
    ("round_truncates", "double r = rint(ldexp(ax, -q));", "double r = trunc(ldexp(ax, -q));"),
    ("round_half_up", "double r = rint(ldexp(ax, -q));", "double r = floor(ldexp(ax, -q) + 0.5);"),
    ("round_no_subnormal_floor", "    if (q < -24)\n        q = -24;\n", "    if (q < -30)\n        q = -30;\n"),
    ("round_quantum_off_by_one", "int q = e - 11;", "int q = e - 10;"),
    ("round_overflow_threshold", "if (ax >= 65520.0)", "if (ax > 65520.0)"),
    ("acc16_group_16", "if (k % 32 == 31 || k == K - 1)", "if (k % 16 == 15 || k == K - 1)"),
    ("acc16_group_misaligned", "if (k % 32 == 31 || k == K - 1)", "if (k % 32 == 0 || k == K - 1)"),
    ("acc16_no_tail_rounding", "if (k % 32 == 31 || k == K - 1)", "if (k % 32 == 31)"),
    ("acc16_round_only_at_end", "if (k % 32 == 31 || k == K - 1)", "if (k == K - 1)"),
    ("acc16_second_not_subtracted", "J->second > 0 ? 1.0 : -1.0);", "1.0);"),
    # Listing 5's two accumulators instead of the one running sum: P.Q
    # accumulated (and rounded) on its own, then added in binary64
    ("acc16_two_accumulators",
     "product_row_acc16(J, J->P, J->ldp, J->Qd, J->K2, i, c, J->second > 0 ? 1.0 : -1.0);",
     "{ product_row_acc16(J, J->P, J->ldp, J->Qd, J->K2, i, r, J->second > 0 ? 1.0 : -1.0);\n"
     "                  for (int64_t j = 0; j < J->N; ++j) c[j] = c[j] + r[j]; }"),
]

ALL_PINS = P.PINS + PF.PINS + PA.PINS


def _build_mutant(tmp_path, name, old, new):
    src = open(build_oracle.SRC).read()
    assert src.count(old) >= 1, f"mutation anchor for {name} not found"
    mutated = src.replace(old, new, 1)
    c = tmp_path / f"mut_{name}.c"
    so = tmp_path / f"libmut_{name}.so"
    c.write_text(mutated)
    subprocess.run(["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fPIC", "-shared", "-w",
                    "-o", str(so), str(c), "-lm", "-lpthread"], check=True)
    return O.load_library(str(so))


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, name, old, new):
    lib = _build_mutant(tmp_path, name, old, new)
    failed = []
    for pin in ALL_PINS:
        try:
            pin(lib)
        except (AssertionError, ValueError):
            failed.append(pin.__name__)
    assert failed, f"mutant {name} passed every pin"


def test_unmutated_copy_passes(tmp_path):
    lib = _build_mutant(tmp_path, "none", "#include <math.h>", "#include <math.h>")
    for pin in ALL_PINS:
        pin(lib)
