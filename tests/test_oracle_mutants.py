"""Plant plausible mistakes in copies of the oracle (on the CPU) and check that the pins catch
every one: a dropped term, a wrong sign or index, a transposed operand, a wrong unit."""
from __future__ import annotations

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "oracle.c")

MUTANTS = {
    "wrong_operand": ("s += x * y;", "s += x * x;"),
    "transposed_a": ("(int64_t)row + (int64_t)p * d->lda", "(int64_t)p + (int64_t)row * d->lda"),
    "transposed_b": ("(int64_t)p + (int64_t)col * d->ldb", "(int64_t)col + (int64_t)p * d->ldb"),
    "a_trans_read_plain": ("(int64_t)row * d->lda + p", "(int64_t)row + (int64_t)p * d->lda"),
    "b_trans_read_plain": ("(int64_t)p * d->ldb + col", "(int64_t)p + (int64_t)col * d->ldb"),
    "dropped_k_term": ("for (int32_t p = 0; p < d->k; ++p)", "for (int32_t p = 1; p < d->k; ++p)"),
    "dropped_pair": ("for (int64_t i = 0; i < count; ++i) {\n        for (int32_t p",
                     "for (int64_t i = 1; i < count; ++i) {\n        for (int32_t p"),
    "stride_recurrence": ("if (i > 0) {", "if (i > 1) {"),
    "offset_in_bytes": ("out_a[i] = (const char*)a + offs_a[i] * es;",
                        "out_a[i] = (const char*)a + offs_a[i];"),
    "beta_dropped": ("v = d->beta * oracle_widen(c, ci, d->c_type) + s;",
                     "v = oracle_widen(c, ci, d->c_type) + s;"),
    "beta_zero_reads_c": ("if (d->beta != 0.0) v =", "if (1) v ="),
    "bias_by_column": ("v += (double)bias[row];", "v += (double)bias[col % d->m];"),
    "relu_sign": ("v = v > 0.0 ? v : 0.0;", "v = v < 0.0 ? v : 0.0;"),
    "gelu_sign": ("(1.0 + tanh(", "(1.0 - tanh("),
    "gelu_cubic": ("(1.0 + tanh(c * (x + 0.044715 * x * x * x)))",
                   "(1.0 + tanh(c * (x + 0.044715 * x * x)))"),
    "rne_ties_up": ("rest > 0x8000u ||", "rest >= 0x8000u ||"),
    "grid_swapped": ("co = gi_m * grid->c_step_m + gi_n * grid->c_step_n;",
                     "co = gi_n * grid->c_step_m + gi_m * grid->c_step_n;"),
    "explicit_b_offset": ("bo = b_off ? b_off[g] : 0;", "bo = a_off ? a_off[g] : 0;"),
    "csr_bounds": ("const int64_t lo = begin[g], hi = begin[g + 1];",
                   "const int64_t lo = begin[g], hi = begin[g + 1] - (g > 0);"),
    "reduce_square_dropped": ("ax2 = fold(op, ax2, x * x);", "ax2 = fold(op, ax2, x);"),
    "reduce_direction": ("const int32_t row = by_cols ? o : t;", "const int32_t row = by_cols ? t : o;"),
    "reduce_min_init": ("ax = (op == ORACLE_RED_MUL) ? 1.0 : (op == ORACLE_RED_SUM ? 0.0 : x);",
                        "ax = (op == ORACLE_RED_MUL) ? 1.0 : 0.0;"),
}

# Transform TPP mutants, caught by the transform pins.
TRANSFORM_MUTANTS = {
    "transpose_output_index": ("move_entry(out, (int64_t)c + (int64_t)r * ld_out, in,",
                               "move_entry(out, (int64_t)r + (int64_t)c * ld_out, in,"),
    "vnni_planar_not_interleaved": ("const int64_t oi = (int64_t)g * ld_out + (int64_t)r * alpha + a;",
                                    "const int64_t oi = (int64_t)g * ld_out + (int64_t)a * m + r;"),
    "vnni_group_of_column": ("const int32_t c = g * alpha + a;", "const int32_t c = a * alpha + g;"),
    "vnni_no_zero_fill": ("          if (c < n)\n            move_entry(out, oi, in, (int64_t)r + (int64_t)c * ld_in, es);\n          else\n            zero_entry(out, oi, es);",
                          "          if (c < n)\n            move_entry(out, oi, in, (int64_t)r + (int64_t)c * ld_in, es);"),
    "vnni_t_input_group": ("(int64_t)(c / alpha) * ld_in + (int64_t)r * alpha + c % alpha",
                           "(int64_t)(c % alpha) * ld_in + (int64_t)r * alpha + c / alpha"),
    "vnni_t_row_of_group": ("const int32_t r = g * alpha + a;", "const int32_t r = g + a * alpha;"),
    "vnni_t_pad_not_zero": ("          if (r < m)\n            move_entry(out, oi, in, (int64_t)(c / alpha) * ld_in",
                            "          if (r < m || 1)\n            move_entry(out, oi, in, (int64_t)(c / alpha) * ld_in"),
}

# Back-propagation mutants (inverse activations, saved pre-activation, batched loops), caught by
# the backward pins.
BACKWARD_MUTANTS = {
    "gelu_grad_dropped_term": (" + 0.5 * x * (1.0 - t * t) * c * (1.0 + 3.0 * 0.044715 * x * x);",
                               ";"),
    "gelu_grad_cubic_factor": ("(1.0 + 3.0 * 0.044715 * x * x)", "(1.0 + 0.044715 * x * x)"),
    "relu_inv_at_zero": ("v = z > 0.0 ? v : 0.0;", "v = z >= 0.0 ? v : 0.0;"),
    "gelu_inv_at_output": ("v = v * oracle_gelu_tanh_grad(oracle_widen(aux, ci, d->c_type));",
                           "v = v * oracle_gelu_tanh_grad(v);"),
    "preact_saved_after_act": (
        "if (d->flags & ORACLE_EPI_SAVE_PREACT) store_rounded(aux, ci, d->c_type, v);\n"
        "      if (d->flags & ORACLE_EPI_RELU) v = v > 0.0 ? v : 0.0;",
        "if (d->flags & ORACLE_EPI_RELU) v = v > 0.0 ? v : 0.0;\n"
        "      if (d->flags & ORACLE_EPI_SAVE_PREACT) store_rounded(aux, ci, d->c_type, v);"),
    "transform_batch_stride_bytes": ("(const char*)in + g * in_stride * es,",
                                     "(const char*)in + g * in_stride,"),
    "reduce_batch_out_packed": ("out_x ? out_x + g * out_stride : NULL", "out_x ? out_x + g * m : NULL"),
}

# Embedding gather-reduce mutants, caught by the embedding pins.
EMBEDDING_MUTANTS = {
    "emb_first_index_dropped": ("for (int64_t j = begin[b]; j < begin[b + 1]; ++j)\n        s +=",
                                "for (int64_t j = begin[b] + 1; j < begin[b + 1]; ++j)\n        s +="),
    "emb_row_stride": ("s += oracle_widen(W, idx[j] * ldw + e, w_type);",
                       "s += oracle_widen(W, idx[j] * E + e, w_type);"),
    "emb_out_stride": ("store_rounded(out, b * ldo + e, out_type, s);",
                       "store_rounded(out, b * E + e, out_type, s);"),
    "emb_index_as_position": ("s += oracle_widen(W, idx[j] * ldw + e, w_type);",
                              "s += oracle_widen(W, j * ldw + e, w_type);"),
}

# Matrix-equation mutants (Alg. 3, Alg. 4, the tree's value), caught by the equation pins.
EQUATION_MUTANTS = {
    "eq_binary_no_increment": ("v = l == rr ? l + 1 : (l > rr ? l : rr);", "v = l > rr ? l : rr;"),
    "eq_unary_over_leaf": ("v = nodes[x->child[0]].arity == ORACLE_EQ_LEAF ? 1 : c;", "v = c;"),
    "eq_plan_min_first": ("(best < 0 || score[x->child[c]] > score[x->child[best]])",
                          "(best < 0 || score[x->child[c]] < score[x->child[best]])"),
    "eq_keeps_right_tmp": ("if (nodes[x->child[0]].arity != ORACLE_EQ_LEAF) {\n    keep = 0;",
                           "if (0) {\n    keep = 0;"),
    "eq_reserve_skips_zero": ("for (int32_t i = 0; i < 64; ++i)\n    if (!p->used[i])",
                              "for (int32_t i = 1; i < 64; ++i)\n    if (!p->used[i])"),
    "eq_bcast_col_as_row": ("else if (L->bcast == ORACLE_BC_COL) at = row;",
                            "else if (L->bcast == ORACLE_BC_COL) at = col;"),
    "eq_div_swapped": ("case ORACLE_EQ_DIV: return a / b;", "case ORACLE_EQ_DIV: return b / a;"),
}


@pytest.fixture(scope="module")
def source():
    with open(SRC) as f:
        return f.read()


def _caught(old, new, pins, source, tmp_path, name):
    assert source.count(old) == 1, f"mutation site for {name} not unique"
    mutated = source.replace(old, new)
    src = tmp_path / "oracle.c"
    src.write_text(mutated)
    (tmp_path / "oracle.h").write_text(open(os.path.join(ROOT, "oracle", "oracle.h")).read())
    so = tmp_path / "liboracle_mutant.so"
    subprocess.run(["gcc", "-O1", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-o", str(so),
                    str(src), "-lm"], check=True)
    env = dict(os.environ, ORACLE_LIB_OVERRIDE=str(so), OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", pins)],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"no pin caught mutant {name}:\n{r.stdout[-2000:]}"


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_mistake(name, source, tmp_path):
    old, new = MUTANTS[name]
    _caught(old, new, "test_oracle_pins.py", source, tmp_path, name)


@pytest.mark.parametrize("name", sorted(TRANSFORM_MUTANTS))
def test_transform_pins_catch_planted_mistake(name, source, tmp_path):
    old, new = TRANSFORM_MUTANTS[name]
    _caught(old, new, "test_oracle_transform_pins.py", source, tmp_path, name)


@pytest.mark.parametrize("name", sorted(BACKWARD_MUTANTS))
def test_backward_pins_catch_planted_mistake(name, source, tmp_path):
    old, new = BACKWARD_MUTANTS[name]
    _caught(old, new, "test_oracle_backward_pins.py", source, tmp_path, name)


@pytest.mark.parametrize("name", sorted(EMBEDDING_MUTANTS))
def test_embedding_pins_catch_planted_mistake(name, source, tmp_path):
    old, new = EMBEDDING_MUTANTS[name]
    _caught(old, new, "test_oracle_embedding_pins.py", source, tmp_path, name)


@pytest.mark.parametrize("name", sorted(EQUATION_MUTANTS))
def test_equation_pins_catch_planted_mistake(name, source, tmp_path):
    old, new = EQUATION_MUTANTS[name]
    _caught(old, new, "test_oracle_equation_pins.py", source, tmp_path, name)
