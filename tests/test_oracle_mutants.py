"""Planted mistakes in copies of the oracle must each fail at least one pin.

Each mutant rewrites one spot of ``oracle/kmeans_oracle.c`` (a dropped term, a
wrong sign, a wrong index, a wrong tie-break, a wrong empty-cluster rule, ...),
is compiled into a temporary folder, and the fast pin battery runs against it.
"""
import os

import pytest

import oracle_pins as P
from oracle import Oracle
from oracle import build as obuild

MUTANTS = {
    "dropped_last_dim": ("const double t = x[j] - c[j];",
                         "const double t = (j + 1 < D) ? x[j] - c[j] : 0.0;"),
    "sign_flip": ("const double t = x[j] - c[j];", "const double t = x[j] + c[j];"),
    "abs_not_square": ("d += t * t;", "d += fabs(t);"),
    "tie_to_highest": ("if (arg < 0 || d < best) {", "if (arg < 0 || d <= best) {"),
    "nonfinite_centroid_used": ("if (!usable[k]) continue;", "(void)usable[k];"),
    "nonfinite_point_assigned": ("const int point_ok = all_finite(x, D);", "const int point_ok = 1;"),
    "unassigned_in_objective": ("if (idx[b * N + i] >= 0) J += min_dist[b * N + i];",
                                "J += min_dist[b * N + i];"),
    "invalid_idx_ends_instance": ("if (k < 0 || k >= K) continue;", "if (k < 0 || k >= K) break;"),
    "index_off_by_one": ("arg = k;", "arg = k ? k - 1 : 0;"),
    "no_runner_up": ("} else if (d < second) {", "} else if (0) {"),
    "empty_cluster_zeroed": (": prev[j];", ": 0.0;"),
    "divide_by_n_plus_1": ("S[k * D + j] / (double)n[k]", "S[k * D + j] / (double)(n[k] + 1)"),
    "singletons_kept": ("n[k] > 0 ?", "n[k] > 1 ?"),
    "transposed_read": ("S[k * D + j] += widen_one(X, dtype, row * D + j);",
                        "S[k * D + j] += widen_one(X, dtype, (row * D + j) % D * N + row % N);"),
    "f16_bias": ("v = ldexp((double)(1024 + m), e - 25);", "v = ldexp((double)(1024 + m), e - 24);"),
    "f16_subnormal": ("v = ldexp((double)m, -24);", "v = ldexp((double)m, -25);"),
    "bf16_shift": ("uint32_t u = (uint32_t)h << 16;", "uint32_t u = ((uint32_t)h << 16) | 1u;"),
    "objective_drops_first": ("J += min_dist[b * N + i];", "J += (i > 0) ? min_dist[b * N + i] : 0.0;"),
    "count_double": ("n[k] += 1;", "n[k] += (k == 0) ? 2 : 1;"),
    "instance_stride": ("const double* Cb = C + b * K * D;", "const double* Cb = C;"),
}


# planted mistakes in the KNN search, each caught by the KNN pins
KNN_MUTANTS = {
    "knn_tie_to_later": ("while (pos > 0 && e < ld[pos - 1]) {", "while (pos > 0 && e <= ld[pos - 1]) {"),
    "knn_sign_flip": ("const double t = q[l] - r[l];", "const double t = q[l] + r[l];"),
    "knn_keeps_k_only": ("int64_t n = 0;  /* entries in the list, at most k + 1 */",
                         "int64_t n = 1;  /* entries in the list, at most k + 1 */"),
    "knn_next_is_kth": ("if (next_dist) next_dist[row] = n > k ? ld[k] : INFINITY;",
                        "if (next_dist) next_dist[row] = n > k ? ld[k - 1] : INFINITY;"),
    "knn_instance_stride": ("rw[j] = widen_one(R, dtype, b * N * D + j);", "rw[j] = widen_one(R, dtype, j);"),
    "knn_drops_last_dim": ("for (int64_t l = 0; l < D; ++l) {\n                        const double t",
                           "for (int64_t l = 0; l + 1 < D; ++l) {\n                        const double t"),
}


@pytest.fixture(scope="module")
def src():
    with open(obuild.SRC) as f:
        return f.read()


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, src, tmp_path):
    old, new = MUTANTS[name]
    assert src.count(old) == 1, f"mutation site for {name} not unique"
    path = tmp_path / "mutant.c"
    path.write_text(src.replace(old, new))
    lib = obuild.build(str(path), str(tmp_path / f"lib_{name}.so"))
    o = Oracle(lib)
    for pin in P.FAST_PINS:
        try:
            pin(o)
        except Exception:  # an AssertionError, or an error the mistake provoked
            return
    pytest.fail(f"mutant {name} passed every pin")


@pytest.mark.parametrize("name", sorted(KNN_MUTANTS))
def test_knn_mutant_is_caught(name, src, tmp_path):
    old, new = KNN_MUTANTS[name]
    assert src.count(old) == 1, f"mutation site for {name} not unique"
    path = tmp_path / "mutant.c"
    path.write_text(src.replace(old, new))
    lib = obuild.build(str(path), str(tmp_path / f"lib_{name}.so"))
    o = Oracle(lib)
    for pin in P.KNN_PINS:
        try:
            pin(o)
        except Exception:
            return
    pytest.fail(f"mutant {name} passed every KNN pin")
