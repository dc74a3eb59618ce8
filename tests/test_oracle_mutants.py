"""Plant plausible mistakes in a copy of the oracle source and check that the
oracle's pins (tests/test_oracle.py for the Lloyd iteration,
tests/test_oracle_init.py for the initial centres, tests/test_oracle_diameter.py
for the diameter and the centre of gravity, tests/test_oracle_l1.py for the L1
assignment) catch every one of them.

Each mutant is a textual edit of oracle/kmeans_oracle.c compiled into a
temporary library; the pin suite then runs against it in a subprocess (through
KMEANS_ORACLE_LIB) and must fail. Everything here runs on the CPU.
"""
import os
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTANTS = {
    "drop_last_feature": ("for (int32_t j = 0; j < M; ++j) {\n        double e",
                          "for (int32_t j = 0; j < M - 1; ++j) {\n        double e"),
    "drop_first_feature": ("for (int32_t j = 0; j < M; ++j) {\n        double e",
                           "for (int32_t j = 1; j < M; ++j) {\n        double e"),
    "wrong_sign": ("double e = (double)x[j] - (double)c[j];",
                   "double e = (double)x[j] + (double)c[j];"),
    "ties_to_highest_index": ("if (d < best) {", "if (d <= best) {"),
    "wrong_centre_stride": ("sqdist(x, C + (int64_t)k * M, M)",
                            "sqdist(x, C + (int64_t)k * (M > 1 ? M - 1 : 1), M)"),
    "transposed_object_index": ("const float *x = X + i * (int64_t)M;\n        double best",
                                "const float *x = X + (i % M) * (int64_t)M;\n        double best"),
    "empty_cluster_to_zero": ("centers[o] = prev[o];", "centers[o] = 0.0f;"),
    "sum_not_mean": ("centers[o] = (float)(S[o] / (double)cnt[k]);",
                     "centers[o] = (float)(S[o] / (double)(cnt[k] + 1));"),
    "skip_first_object_in_sum": ("int32_t l = labels[i];\n        if (l < 0 || l >= K) {",
                                 "int32_t l = labels[i];\n        if (i == 0) continue;\n        if (l < 0 || l >= K) {"),
    "compare_from_first_iteration": ("t >= 2 && congruent", "t >= 1 && congruent"),
    "never_stop": ("if (stop) break;", "if (0 && stop) break;"),
    "fp32_difference": ("double e = (double)x[j] - (double)c[j];\n        double sq = e * e;",
                        "float e = x[j] - c[j];\n        double sq = e * e;"),
    "count_off_by_one": ("cnt[l] += 1;", "cnt[l] += (i > 0);"),
}

# mistakes in the diameter and the centre of gravity of the whole set, caught by
# tests/test_oracle_diameter.py
DIAM_MUTANTS = {
    "diam_ties_to_last_pair": ("if (!have || d > best) {", "if (!have || d >= best) {"),
    "diam_self_pairs": ("for (int64_t l = k + 1; l < n; ++l) {", "for (int64_t l = k; l < n; ++l) {"),
    "diam_drops_last_feature": ("double d = sqdist(X + k * (int64_t)M, X + l * (int64_t)M, M);",
                                "double d = sqdist(X + k * (int64_t)M, X + l * (int64_t)M, "
                                "M > 1 ? M - 1 : M);"),
    "diam_skips_last_object": ("for (int64_t l = k + 1; l < n; ++l) {",
                               "for (int64_t l = k + 1; l < n - 1; ++l) {"),
    "centroid_divides_by_n_minus_1": ("centroid[j] = (float)(s / (double)n);",
                                      "centroid[j] = (float)(s / (double)(n > 1 ? n - 1 : 1));"),
    "centroid_skips_first_object": ("for (int64_t i = 0; i < n; ++i)\n            s = s + (double)X",
                                    "for (int64_t i = 1; i < n; ++i)\n            s = s + (double)X"),
}

# mistakes in the L1 assignment, caught by tests/test_oracle_l1.py
L1_MUTANTS = {
    "l1_squares_instead_of_abs": ("sum = sum + fabs(diff);", "sum = sum + diff * diff;"),
    "l1_signed_difference": ("sum = sum + fabs(diff);", "sum = sum + diff;"),
    "l1_ties_to_highest_index": ("if (dk < nearest) {", "if (dk <= nearest) {"),
    "l1_drops_last_feature": ("for (int32_t f = 0; f < M; ++f) {\n        double diff",
                              "for (int32_t f = 0; f < (M > 1 ? M - 1 : M); ++f) {\n        double diff"),
    "l1_run_uses_l2": ("if (l1)\n            rc = oracle_assign_l1", "if (0)\n            rc = oracle_assign_l1"),
}

# mistakes in the initial-centre traversal, caught by tests/test_oracle_init.py
INIT_MUTANTS = {
    "init_ties_to_highest_index": ("nearest[i] > nearest[far]", "nearest[i] >= nearest[far]"),
    "init_chosen_not_excluded": ("if (chosen[i])\n                continue;",
                                 "if (0 && chosen[i])\n                continue;"),
    "init_newest_centre_only": ("if (d < nearest[i])\n                nearest[i] = d;",
                                "nearest[i] = d;"),
    "init_nearest_as_max": ("if (d < nearest[i])\n                nearest[i] = d;",
                            "if (nearest[i] == INFINITY || d > nearest[i])\n"
                            "                nearest[i] = d;"),
    "init_starts_at_last_object": ("idx[0] = 0;\n    chosen[0] = 1;",
                                   "idx[0] = (int32_t)(n - 1);\n    chosen[n - 1] = 1;"),
    "from_ties_to_highest_index": ("closest[obj] > closest[pick]", "closest[obj] >= closest[pick]"),
    "from_second_seed_ignored": ("if (m < S) {\n            idx[m] = seeds[m];",
                                 "if (m < 1) {\n            idx[m] = seeds[m];"),
    "from_taken_not_excluded": ("if (taken[obj])\n                    continue;",
                                "if (0 && taken[obj])\n                    continue;"),
    "init_drops_last_feature": ("double d = sqdist(X + i * (int64_t)M, c, M);",
                                "double d = sqdist(X + i * (int64_t)M, c, M > 1 ? M - 1 : M);"),
}


@pytest.fixture(scope="module")
def source():
    with open(oracle.SRC) as f:
        return f.read()


@pytest.mark.slow
@pytest.mark.parametrize("name", sorted(MUTANTS) + sorted(INIT_MUTANTS) + sorted(DIAM_MUTANTS)
                         + sorted(L1_MUTANTS))
def test_pins_catch_planted_mistake(name, source, tmp_path):
    for table, pins in ((MUTANTS, "test_oracle.py"), (INIT_MUTANTS, "test_oracle_init.py"),
                        (DIAM_MUTANTS, "test_oracle_diameter.py"),
                        (L1_MUTANTS, "test_oracle_l1.py")):
        if name in table:
            old, new = table[name]
            break
    assert source.count(old) == 1, f"mutant {name} does not apply"
    src = tmp_path / "mutant.c"
    src.write_text(source.replace(old, new))
    lib = tmp_path / "libmutant.so"
    subprocess.check_call(["gcc", *oracle.CFLAGS, "-o", str(lib), str(src), "-lm"])
    env = dict(os.environ, KMEANS_ORACLE_LIB=str(lib))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        "-m", "not slow", os.path.join(ROOT, "tests", pins)],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"mutant {name} survived the oracle pins:\n{r.stdout[-2000:]}"
