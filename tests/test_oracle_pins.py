"""CPU tests: the oracle against what the paper and the mathematics fix.

Parity of the HIP path is judged against the oracle, so the oracle is pinned
first, by checks that do not re-use its own formula (tests/oracle_pins.py),
and by a mutation check: each plausible slip planted in a copy of oracle.c
(wrong sign, dropped square, dropped term, transposed stride, wrong
tie-break, lost block offset, wrong second best, dropped feature, the
rank-2/rank-3 slips of the two-best oracle, the value slips of the
real-valued oracle, and the window, pass, quotient and support slips of the update)
must make at least one pin fail.
"""
import os
import subprocess

import pytest

import oracle
import oracle_pins as P


@pytest.mark.parametrize("check", P.ALL_CHECKS, ids=lambda f: f.__name__)
def test_oracle_pin(check):
    check(oracle.load())


def test_exact_integer_full_tiny_workload():
    # all 10,000 rows of the tiny 16x16 workload: exact indices and distances
    P.check_exact_integer_tiny(oracle.load())


MUTANTS = [
    ("sign", "const double diff = x[v] - (double)wrow[k];", "const double diff = x[v] + (double)wrow[k];"),
    ("dropped_square", "D[k] += diff * diff;", "D[k] += diff;"),
    ("input_ignored", "        x[v] = 1.0;\n", "        (void)v;\n"),
    ("transposed_stride", "const float *wrow = W + v * ldw;\n        for (int64_t k = 0; k < B; ++k) {\n            const double diff",
     "const float *wrow = W + v;\n        for (int64_t k = 0; k < B; ++k) {\n            const double diff"),
    ("tie_highest_index", "if (D[k] < D[best]) best = k;", "if (D[k] <= D[best]) best = k;"),
    ("block_offset_lost", "bmu[s] = (int32_t)(i0 + best);", "bmu[s] = (int32_t)best;"),
    ("second_best_includes_best", "if (k != best && D[k] < second)", "if (D[k] < second)"),
    ("last_feature_dropped",
     "for (int64_t v = 0; v < V; ++v) {\n        const float *wrow = W + v * ldw;\n        for (int64_t k = 0; k < B; ++k) {\n            const double diff",
     "for (int64_t v = 0; v < V - 1; ++v) {\n        const float *wrow = W + v * ldw;\n        for (int64_t k = 0; k < B; ++k) {\n            const double diff"),
    ("norm_not_squared", "norms[k] += w * w;", "norms[k] += w;"),
    ("x_off_by_one", "x[v] = 1.0;", "x[v < V - 1 ? v + 1 : v] = 1.0;"),
    ("rank2_tie_highest_index", "} else if (r2 < 0 || D[k] < D[r2]) {", "} else if (r2 < 0 || D[k] <= D[r2]) {"),
    ("rank2_not_demoted", "                r3 = r2;\n                r2 = r1;\n                r1 = k;",
     "                r3 = r2;\n                r1 = k;"),
    ("rank2_block_offset_lost", "bmu2[s] = r2 < 0 ? -1 : (int32_t)(i0 + r2);", "bmu2[s] = r2 < 0 ? -1 : (int32_t)r2;"),
    ("rank3_ignored", "} else if (r3 < 0 || D[k] < D[r3]) {", "} else if (r3 < 0) {"),
    ("sf_value_ignored", "x[v] = (double)values[p];", "x[v] = 1.0;"),
    ("sf_value_squared", "x[v] = (double)values[p];", "x[v] = (double)values[p] * (double)values[p];"),
    ("box_window_off_by_one", "if (i - r - 1 >= 0) s -= line[(i - r - 1) * stride];",
     "if (i - r >= 0) s -= line[(i - r) * stride];"),
    ("zero_den_filled", "W_out[v * M + i] = W_in[v * M + i];", "W_out[v * M + i] = 0.0f;"),
    ("support_ignored", "if (sup[i] > 0 && den[i] > 0.0f) {", "if (den[i] > 0.0f) {"),
    ("support_radius_r", "occupied_support(cnt, E, 3 * radius, sup)", "occupied_support(cnt, E, radius, sup)"),
    ("two_row_passes", "for (int pass = 0; pass < 3; ++pass) box_pass(f + row * E, E, 1, r, tmp);",
     "for (int pass = 0; pass < 2; ++pass) box_pass(f + row * E, E, 1, r, tmp);"),
    ("columns_skipped", "for (int pass = 0; pass < 3; ++pass) box_pass(f + col, E, E, r, tmp);",
     "for (int pass = 0; pass < 0; ++pass) box_pass(f + col, E, E, r, tmp);"),
    ("den_not_blurred", "    blur_field(den, E, radius, tmp);\n", "\n"),
    ("sf_rank2_tie_highest_index", "} else if (q2 < 0 || D[k] < D[q2]) {", "} else if (q2 < 0 || D[k] <= D[q2]) {"),
]


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, name, old, new):
    src = open(os.path.join(os.path.dirname(oracle.__file__), "oracle.c")).read()
    assert src.count(old) == 1, f"mutation site for {name} not found exactly once"
    mutated = tmp_path / "oracle_mut.c"
    mutated.write_text(src.replace(old, new))
    # the header sits next to the original source
    inc = os.path.dirname(oracle.__file__)
    so = tmp_path / "liboracle_mut.so"
    subprocess.run(["gcc", *oracle.CFLAGS, f"-I{inc}", str(mutated), "-o", str(so), "-lm"], check=True)
    lib = oracle.load(str(so))
    failures = []
    for check in P.ALL_CHECKS:
        try:
            check(lib)
        except (AssertionError, ValueError):
            failures.append(check.__name__)
    assert failures, f"mutant {name} passed every pin"
