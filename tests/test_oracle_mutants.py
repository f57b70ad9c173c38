"""Planted mistakes in the oracle must be caught by the pins.

Each mutant is a copy of oracle.c with one plausible slip (a flipped
comparison, swapped children, a dropped term, a wrong index). It is compiled
into a temporary library on the CPU and must fail at least one pin.
"""
import os

import pytest

import oracle
import pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "oracle.c")

MUTANTS = {
    "ties_go_left": ("if (x[f] < J->threshold[base + v])", "if (x[f] <= J->threshold[base + v])"),
    "children_swapped": ("      v = J->left[base + v];\n    else\n      v = J->right[base + v];",
                         "      v = J->right[base + v];\n    else\n      v = J->left[base + v];"),
    "nan_goes_left": ("if (x[f] < J->threshold[base + v])", "if (!(x[f] >= J->threshold[base + v]))"),
    "mean_not_divided": ("if (J->aggregation == ORACLE_AGG_MEAN) s /= (double)J->n_trees;", ""),
    "class_ignored": ("int32_t c = J->tree_class ? J->tree_class[t] : 0;", "int32_t c = 0;"),
    "leaf_vector_index": ("J->leaf_value[node * J->leaf_dim + k]", "J->leaf_value[node + k]"),
    "sigmoid_sign": ("out[k] = 1.0 / (1.0 + exp(-raw[k]))", "out[k] = 1.0 / (1.0 + exp(raw[k]))"),
    "softmax_no_normalise": ("for (int32_t k = 0; k < K; ++k) out[k] /= z;", ""),
    "base_score_dropped": ("if (J->base_score) s += (double)J->base_score[k];", ""),
    "last_tree_skipped": ("for (int32_t t = 0; t < J->n_trees; ++t) {\n      int64_t leaf",
                          "for (int32_t t = 0; t < J->n_trees - 1; ++t) {\n      int64_t leaf"),
    "feature_off_by_one": ("if (x[f] < J->threshold", "if (x[f == 0 ? 0 : f - 1] < J->threshold"),
    "default_left_ignored": ("if (J->default_left && isnan(x[f]))", "if (0)"),
    "default_left_inverted": ("J->default_left[node] ? J->left[node] : J->right[node]",
                              "J->default_left[node] ? J->right[node] : J->left[node]"),
    "category_set_inverted": ("v = in_set ? J->left[node] : J->right[node];",
                              "v = in_set ? J->right[node] : J->left[node];"),
    "category_rounded": ("const int64_t c = (int64_t)x[f]; /* integer part */",
                         "const int64_t c = (int64_t)(x[f] + 0.5f);"),
    "category_negative_as_zero": ("if (x[f] >= 0.0f && (double)x[f] < 32.0 * (double)words) {",
                                  "if (x[f] > -1.0f && (double)x[f] < 32.0 * (double)words) {"),
    "category_bit_order": ("(J->cat_bits[J->cat_offset[node] + c / 32] >> (c % 32))",
                           "(J->cat_bits[J->cat_offset[node] + c / 32] >> (31 - c % 32))"),
    "category_wraps": ("if (x[f] >= 0.0f && (double)x[f] < 32.0 * (double)words) {\n        const int64_t c = (int64_t)x[f]; /* integer part */",
                       "if (x[f] >= 0.0f && x[f] < 1e9f) {\n        const int64_t c = ((int64_t)x[f]) % (32 * words);"),
    "category_ignored": ("else if (J->cat_offset && J->cat_offset[node + 1] > J->cat_offset[node]) {",
                         "else if (0) {"),
    "category_nan_default_ignored": ("    if (J->default_left && isnan(x[f]))\n      v = J->default_left[node]",
                                     "    if (J->default_left && isnan(x[f]) && !(J->cat_offset && J->cat_offset[node + 1] > J->cat_offset[node]))\n      v = J->default_left[node]"),
}

PINS = [pins.pin_golden, pins.pin_brute_force, pins.pin_gemm_closed_form, pins.pin_closed_forms,
        pins.pin_sklearn, pins.pin_categorical]


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert old in src, f"mutation anchor for {name} not found"
    mut_c = tmp_path / "oracle_mut.c"
    mut_c.write_text(src.replace(old, new, 1))
    so = tmp_path / "liboracle_mut.so"
    import subprocess
    subprocess.run(["gcc", "-O2", "-std=c99", "-D_POSIX_C_SOURCE=200809L", "-shared", "-fPIC",
                    "-o", str(so), str(mut_c), "-lpthread", "-lm"], check=True)
    lib = oracle.load(str(so))
    failures = 0
    for pin in PINS:
        try:
            pin(lib)
        except (AssertionError, ValueError):
            failures += 1
    assert failures > 0, f"no pin caught mutant {name}"
