"""Plant plausible mistakes in the oracle (on the CPU) and check that the pins catch each.

Every mutant is the oracle's C source with one edit (a dropped term, a wrong
sign, index or operand), compiled into a temporary library.  The pin tests of
the other oracle test files are then run against the mutant; at least one of
them must fail."""
import ctypes
import os
import subprocess

import pytest

import oracle
from tests import test_oracle_attn as A
from tests import test_oracle_decode_step as DS
from tests import test_oracle_index as I
from tests import test_oracle_kd as KD
from tests import test_oracle_project as PJ
from tests import test_oracle_topk as T

SRC = os.path.join(os.path.dirname(oracle.__file__), "clsa_oracle.c")

PINS = [
    I.test_matches_blas_float64, I.test_exact_on_small_integers,
    I.test_unit_vector_probe_reads_the_right_component, I.test_paged_equals_contiguous,
    I.test_causal_prefix,
    lambda o: T.test_exhaustive_subsets_tiny(o, 9), T.test_matches_numpy_stable_argsort,
    T.test_signed_zero_is_a_tie, T.test_k_at_least_len_selects_all_and_pads,
    T.test_causal_rows_only_see_their_prefix,
    A.test_matches_masked_sdpa, A.test_lse_matches_scipy, A.test_single_token_returns_its_value_row,
    A.test_gqa_head_mapping, A.test_empty_set,
    lambda o: DS.test_step_matches_library_composition(o, 100),
    PJ.test_matches_numpy_float64, PJ.test_exact_on_small_integers, PJ.test_unit_vector_probe,
    PJ.test_destination_rows,
    KD.test_target_is_a_mean_of_scipy_softmaxes, KD.test_target_rows_sum_to_one,
    KD.test_kl_of_the_indexer_distribution_with_itself_is_zero,
    KD.test_loss_matches_scipy_relative_entropy, KD.test_gradient_matches_central_differences,
    KD.test_rows_without_keys_do_not_count,
]

MUTANTS = {
    "target_not_averaged": ("a[j] /= (double)n_layers * (double)Hq;", "a[j] /= (double)n_layers;"),
    "target_unscaled_logits": ("z[j] = s->softmax_scale * acc;", "z[j] = acc;"),
    "kd_gradient_sign": ("const double g = (exp(sc[j] - lse) - p[j]) / (double)n_rows;",
                         "const double g = (p[j] - exp(sc[j] - lse)) / (double)n_rows;"),
    "kd_loss_not_normalised": ("*loss = n_rows > 0 ? total / (double)n_rows : 0.0;",
                               "*loss = total;"),
    "kd_dk_uses_keys": ("dk[e] += g * oracle_bf16_to_double(qr[e]);",
                        "dk[e] += g * oracle_bf16_to_double(kr[e]);"),
    "projection_weight_transposed": ("oracle_bf16_to_double(w[(size_t)c * d_model + i]);",
                                     "oracle_bf16_to_double(w[(size_t)i * n_out + c]);"),
    "projection_drops_last_term": ("for (int i = 0; i < d_model; i++)\n                acc +=",
                                   "for (int i = 0; i < d_model - 1; i++)\n                acc +="),
    "destination_ignores_page_table": ("(int64_t)token_row(s, page_table, b, p, 1);",
                                       "(int64_t)((size_t)b * (size_t)s->max_len + (size_t)p);"),
    "drop_first_index_component": ("for (int i = 0; i < d_idx; i++)", "for (int i = 1; i < d_idx; i++)"),
    "index_key_off_by_one_token": ("token_row(s, a->page_table, b, j, (size_t)d_idx)",
                                   "token_row(s, a->page_table, b, (j + 1) % s->max_len, (size_t)d_idx)"),
    "select_lowest_scores": ("if (a->s > b->s) return -1;\n    if (a->s < b->s) return 1;",
                             "if (a->s < b->s) return -1;\n    if (a->s > b->s) return 1;"),
    "ties_to_highest_index": ("return (a->j > b->j) - (a->j < b->j);",
                              "return (a->j < b->j) - (a->j > b->j);"),
    "unsorted_output": ("qsort(out, (size_t)m, sizeof *out, by_int);", ""),
    "zero_padding": ("out[i] = -1;", "out[i] = 0;"),
    "causal_exclusive": ("int lim = q_pos[(size_t)b * s->n_q + t] + 1;",
                         "int lim = q_pos[(size_t)b * s->n_q + t];"),
    "gqa_modulo_mapping": ("const int g = h / group;", "const int g = h % Hkv;"),
    "no_softmax_scale": ("z[i] = s->softmax_scale * acc;", "z[i] = acc;"),
    "keys_read_from_values": ("const uint16_t *kr = a->k_cache + token_row(s, a->page_table, b, S[i]",
                              "const uint16_t *kr = a->v_cache + token_row(s, a->page_table, b, S[i]"),
    "unnormalised_weights": ("const double w = exp(z[i] - zmax) / denom;",
                             "const double w = exp(z[i] - zmax);"),
    "lse_without_max": ("lse[r * Hq + h] = zmax + log(denom);", "lse[r * Hq + h] = log(denom);"),
    "page_offset_wrong_stride": ("((size_t)page * (size_t)s->page_size + (size_t)(j % s->page_size))",
                                 "((size_t)page * (size_t)s->page_size + (size_t)(j / s->page_size))"),
}


def _build_mutant(tmp_path, name, find, repl):
    src = open(SRC).read()
    assert src.count(find) >= 1, f"mutation {name} does not apply"
    msrc = tmp_path / f"{name}.c"
    msrc.write_text(src.replace(find, repl))
    (tmp_path / "clsa_oracle.h").write_text(open(SRC.replace(".c", ".h")).read())
    lib = tmp_path / f"lib{name}.so"
    subprocess.run(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-pthread", "-o", str(lib), str(msrc), "-lm"],
                   check=True)
    return str(lib)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(tmp_path, name):
    find, repl = MUTANTS[name]
    path = _build_mutant(tmp_path, name, find, repl)
    saved_lib, saved_path = oracle._lib, oracle._LIB
    oracle._lib = None
    oracle._LIB = path
    try:
        oracle._load()
        caught = []
        for pin in PINS:
            try:
                pin(oracle)
            except AssertionError as e:
                caught.append(getattr(pin, "__name__", "lambda"))
            except Exception as e:        # a crash in the mutant also counts as caught
                caught.append(f"{getattr(pin, '__name__', 'lambda')}:{type(e).__name__}")
        assert caught, f"no pin caught mutant {name}"
    finally:
        oracle._lib, oracle._LIB = saved_lib, saved_path
