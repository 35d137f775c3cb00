"""The pins constrain the oracle: plant one plausible mistake at a time in a
copy of the oracle's C source (on the CPU), rebuild it, and check that the
pin suite fails.  Equivalent mutants for this method's inputs (for example
dropping |.| from the L1 norm while every y_i >= 0) are not listed."""
import os
import shutil
import tempfile

import pytest

import oracle
import test_oracle_pins as pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "gpic_oracle.c")

# name -> (original text, mutated text); the original must occur in the
# source, and every occurrence is replaced
MUTATIONS = {
    "gaussian_width_missing_factor_2": ("2.0 * sigma * sigma", "sigma * sigma"),
    "gaussian_sign": ("return exp(-dist2 / two_sigma2);", "return exp(dist2 / two_sigma2);"),
    "distance_sum_not_difference": ("(double)xi[c] - (double)xj[c]",
                                    "(double)xi[c] + (double)xj[c]"),
    "diagonal_not_zero": ("    if (i == j)\n        return 0.0;\n", ""),
    "start_vector_uniform": ("v0[i] = degree[i] / total;", "v0[i] = 1.0 / (double)n;"),
    "product_with_transposed_W": ("y += op->W[i * op->n + j] * v[j];",
                                  "y += op->W[j * op->n + i] * v[j];"),
    "csr_gathers_own_entry": ("y += op->w[p] * v[op->col[p]];", "y += op->w[p] * v[i];"),
    "onthefly_column_degree": ("y += (gauss_affinity(op->X, op->d, i, j, two_sigma2) / di) * v[j];",
                               "y += (gauss_affinity(op->X, op->d, i, j, two_sigma2) / op->degree[j]) * v[j];"),
    "statistic_without_previous_velocity": ("const double change = fabs(vel - delta[i]);",
                                            "const double change = fabs(vel);"),
    "velocity_not_carried": ("            delta[i] = vel;\n", ""),
    "strict_stop_test": ("if (mode == 1 && s <= eps)", "if (mode == 1 && s < eps)"),
    "iterations_off_by_one": ("done = t + 1;", "done = t;"),
    "segment_size_off_by_one": ("double m = (double)(i - j + 1);", "double m = (double)(i - j + 2);"),
    "cosine_without_shift": ("return 0.5 * (1.0 + dot / (sqrt(ni) * sqrt(nj)));",
                             "return dot / (sqrt(ni) * sqrt(nj));"),
    "cosine_norm_not_square_rooted": ("return 0.5 * (1.0 + dot / (sqrt(ni) * sqrt(nj)));",
                                      "return 0.5 * (1.0 + dot / (ni * nj));"),
    "knn_ties_to_larger_index": ("if (m == k && !(dj < bd[k - 1]))", "if (m == k && dj > bd[k - 1])"),
    "knn_directed_only": ("                e[(2 * i) * (int64_t)k + 2 * t + 1].row = bj[t];\n                e[(2 * i) * (int64_t)k + 2 * t + 1].col = i;\n",
                          "                e[(2 * i) * (int64_t)k + 2 * t + 1].row = i;\n                e[(2 * i) * (int64_t)k + 2 * t + 1].col = bj[t];\n"),
    "dc_left_bound_too_tight": ("dc_layer(P, run_start, prev, cur, opt, lo, mid - 1, olo, opt[mid]);",
                                "dc_layer(P, run_start, prev, cur, opt, lo, mid - 1, olo, opt[mid] - 1);"),
}


def _pin_suite(orc):
    """Run every pin; return the names that failed."""
    failed = []
    calls = [
        ("affinity_scipy", lambda: pins.test_affinity_matches_scipy_distance(orc)),
        ("affinity_closed", lambda: pins.test_affinity_closed_form_two_points(orc)),
        ("affinity_invariant", lambda: pins.test_affinity_symmetric_and_invariant(orc)),
        ("cosine_scipy", lambda: pins.test_cosine_affinity_matches_scipy_distance(orc)),
        ("cosine_closed", lambda: pins.test_cosine_affinity_closed_form_and_invariance(orc)),
        ("brute_gauss", lambda: pins.test_brute_force_fifty_digits(orc, 8, 2, "gauss")),
        ("knn_ckdtree", lambda: pins.test_knn_graph_matches_ckdtree(orc)),
        ("knn_ties", lambda: pins.test_knn_graph_ties_and_structure(orc)),
        ("knn_rows", lambda: pins.test_knn_rows_matches_ckdtree(orc)),
        ("brute_cosine", lambda: pins.test_brute_force_fifty_digits(orc, 7, 3, "cosine")),
        ("row_sums_v0", lambda: pins.test_rows_of_W_sum_to_one_and_v0(orc)),
        ("zero_degree", lambda: pins.test_zero_degree_row_is_counted(orc)),
        ("two_points", lambda: pins.test_two_points_give_swap_matrix(orc)),
        ("trace2", lambda: pins.test_hand_worked_traces(orc, "two_node_trace")),
        ("trace3", lambda: pins.test_hand_worked_traces(orc, "three_node_path_trace")),
        ("uniform", lambda: pins.test_uniform_vector_is_fixed_point(orc)),
        ("less_or_equal", lambda: pins.test_stop_test_is_less_or_equal(orc)),
        ("const_blocks", lambda: pins.test_constant_blocks_are_fixed_points(orc)),
        ("block_diag", lambda: pins.test_block_diagonal_components_never_mix(orc)),
        ("closed_form", lambda: pins.test_closed_form_eigendecomposition(orc)),
        ("one_update", lambda: pins.test_single_update_and_zero_updates(orc)),
        ("csr_dense", lambda: pins.test_csr_full_pattern_equals_dense(orc)),
        ("csr_scipy", lambda: pins.test_csr_sparse_matches_scipy(orc)),
        ("onthefly", lambda: pins.test_onthefly_equals_dense(orc)),
        ("km_exhaustive", lambda: pins.test_kmeans_exact_against_all_labellings(orc, 0)),
        ("km_special", lambda: pins.test_kmeans_special_cases(orc)),
        ("km_dc", lambda: pins.test_kmeans_dc_equals_plain(orc, 1)),
    ]
    for name, fn in calls:
        try:
            fn()
        except Exception:
            failed.append(name)
    return failed


@pytest.fixture(scope="module")
def workdir():
    d = tempfile.mkdtemp(prefix="oracle_mut_")
    yield d
    shutil.rmtree(d, ignore_errors=True)


def test_unmutated_copy_passes(workdir):
    out = oracle.compile_source(SRC, os.path.join(workdir, "orig.so"))
    with oracle.use_library(out):
        assert _pin_suite(oracle) == []


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(workdir, name):
    old, new = MUTATIONS[name]
    text = open(SRC).read()
    assert old in text, f"mutation {name} no longer matches the source"
    src = os.path.join(workdir, f"{name}.c")
    with open(src, "w") as f:
        f.write(text.replace(old, new))
    lib = oracle.compile_source(src, os.path.join(workdir, f"{name}.so"))
    with oracle.use_library(lib):
        failed = _pin_suite(oracle)
    assert failed, f"no pin caught mutation {name}"
