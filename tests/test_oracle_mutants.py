"""Each plausible single mistake planted in the oracle must fail the pins.

The mutants are built on the CPU from a patched copy of oracle/ga_oracle.c
and the pin suites (test_oracle_merge.py, test_oracle_pins.py) are run
against each in a subprocess.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "ga_oracle.c")

MUTANTS = {
    "tie_goes_to_highest_index": ("if (s < best) {", "if (s <= best) {"),
    "distance_drops_centre_norm": ("return fma(-2.0, dot, nrm);", "return fma(-2.0, dot, 0.0);"),
    "distance_wrong_sign": ("return fma(-2.0, dot, nrm);", "return fma(2.0, dot, nrm);"),
    "dot_skips_last_coordinate": ("for (int c = 0; c < d; ++c) dot = fma(k[c], r[c], dot);",
                                  "for (int c = 0; c < d - 1; ++c) dot = fma(k[c], r[c], dot);"),
    "init_not_strided": ("int64_t src = ((int64_t)j * n) / N;", "int64_t src = (int64_t)j;"),
    "representative_not_rounded": ("R[(size_t)j * d + c] = round_dt(C[(size_t)j * d + c], dtype);",
                                   "R[(size_t)j * d + c] = (double)C[(size_t)j * d + c];"),
    "centroid_divides_by_count_plus_one": ("/ (double)count[j]);", "/ (double)(count[j] + 1));"),
    "empty_group_reset_to_zero": ("if (count[j] == 0) continue; /* empty group keeps its centroid */",
                                  "if (count[j] == 0) { for (int c = 0; c < d; ++c) C[(size_t)j * d + c] = 0.0f; continue; }"),
    "aggregate_shifts_group": ("int j = belong[u * (int64_t)n + i];", "int j = (belong[u * (int64_t)n + i] + 1) % N;"),
    "scores_unscaled": ("p[j] = scale * dot;", "p[j] = dot;"),
    "scores_transposed_operand": ("dot += q[c] * R[(size_t)j * d + c];", "dot += q[c] * R[(size_t)c * N + j];"),
    "denominator_without_count": ("s += (double)cnt[j] * e;", "s += e;"),
    "numerator_counts_twice": ("o[c] += e * vs[(size_t)j * d + c];", "o[c] += cnt[j] * e * vs[(size_t)j * d + c];"),
    "attend_ignores_representative_rounding": ("R[x] = round_dt(centroid[u * (int64_t)N * d + x], dtype);",
                                               "R[x] = (double)centroid[u * (int64_t)N * d + x];"),
    # merge plan (adaptive group count)
    "merge_rule_symmetric_threshold": ("dij + rj <= 0.5 * t", "dij + rj <= t"),
    "merge_threshold_without_factor_two": ("log_eps / (2.0 * rprime)", "log_eps / rprime"),
    "merge_query_norm_unscaled": ("fabs(scale) * sqrt(qmax2)", "sqrt(qmax2)"),
    "merge_radius_of_last_member": ("if (r2 > rad2[g]) rad2[g] = r2;", "rad2[g] = r2;"),
    "merge_partner_searched_in_both_halves": ("for (int i = 0; i < half; ++i) {", "for (int i = 0; i < N; ++i) {"),
    "merge_empty_groups_take_part": ("if (cnt[i] <= 0) continue;\n", "\n"),
}
PIN_FILES = ("test_oracle_merge.py", "test_oracle_pins.py")


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_fails_the_pins(name, tmp_path):
    sys.path.insert(0, ROOT)
    import oracle

    old, new = MUTANTS[name]
    text = open(SRC).read()
    assert text.count(old) == 1, f"mutation site not unique for {name}"
    src = tmp_path / "mutant.c"
    src.write_text(text.replace(old, new))
    lib = oracle.build(force=True, src=str(src), out=str(tmp_path / "libmutant.so"))
    env = dict(os.environ, GA_ORACLE_LIB=lib, OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        *(os.path.join(ROOT, "tests", f) for f in PIN_FILES)],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"mutant {name} passed every pin:\n{r.stdout[-2000:]}"
