"""The oracle pins must catch plausible mistakes in the oracle.

Each case plants one mistake in a copy of ``oracle/sparrow_oracle.c`` (on the
CPU, in a temporary directory), builds it, and runs the pin suite against the
broken build in a child process; the suite has to fail.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE = os.path.join(ROOT, "oracle")
SOURCES = ("sparrow_oracle.c", "acceptance_oracle.c", "selector_oracle.c")

MUTANTS = {
    "topk_ties_to_higher_index": ("return (a->p > b->p) - (a->p < b->p);",
                                  "return (a->p < b->p) - (a->p > b->p);"),
    "score_min_instead_of_max": ("s32 += lo > hi ? lo : hi;", "s32 += lo < hi ? lo : hi;"),
    "score_max_row_is_min_row": ("const uint16_t *mx = mn + D;", "const uint16_t *mx = mn;"),
    "attention_drops_scale": ("z[n_tok] = scale * dot;", "z[n_tok] = dot;"),
    "attention_reads_past_length": (
        "                int64_t t_end = L - p * ps < ps ? L - p * ps : ps;\n"
        "                for (int64_t t = 0; t < t_end; ++t) {\n"
        "                    const uint16_t *kt",
        "                int64_t t_end = L - p * ps < ps ? L - p * ps + 1 : ps;\n"
        "                for (int64_t t = 0; t < t_end; ++t) {\n"
        "                    const uint16_t *kt"),
    "attention_values_from_keys": (
        "const uint16_t *vt = v_cache + ", "const uint16_t *vt = k_cache + "),
    "meta_skips_last_token": ("for (int64_t t = 1; t < t_end; ++t) {\n                        uint16_t v",
                              "for (int64_t t = 1; t < t_end - 1; ++t) {\n                        uint16_t v"),
    "meta_ignores_signed_zero_order": ("if (a == b && (a_bits & 0x8000u) && !(b_bits & 0x8000u))",
                                       "if (0)"),
    "budget_floor_instead_of_ceil": ("(n * (int64_t)frac_num[bin] + frac_den - 1) / frac_den",
                                     "(n * (int64_t)frac_num[bin]) / frac_den"),
    "budget_bin_off_by_one": ("int64_t bin = (int64_t)(L - 1) / bin_tokens;",
                              "int64_t bin = (int64_t)L / bin_tokens;"),
    "budget_no_page_clamp": ("    if (k > n)\n        k = n;\n    return (int32_t)k;",
                             "    return (int32_t)k;"),
    "select_pads_with_zero": ("row[i] = -1;", "row[i] = 0;"),
    "append_to_next_slot": ("int64_t pos = L - 1;", "int64_t pos = L;"),
    "append_skips_meta_rebuild": ("        int32_t first = (int32_t)pos;\n        oracle_page_meta(",
                                  "        int32_t first = (int32_t)L;\n        oracle_page_meta("),
}


# Mistakes in the acceptance-rate oracle: (file, old, new), pinned by test_oracle_acceptance.py.
ACCEPTANCE_MUTANTS = {
    "acceptance_max_instead_of_min": (
        "- Q);\n            a += p < q ? p : q;", "- Q);\n            a += p > q ? p : q;"),
    "acceptance_lse_without_log_sum": ("    return m + log(s);", "    return m;"),
    "acceptance_ignores_temperature": (
        "    for (int32_t x = 0; x < V; ++x)\n        s += exp(tau * logit_value(row, dtype, x) - m);",
        "    for (int32_t x = 0; x < V; ++x)\n        s += exp(logit_value(row, dtype, x) - m);"),
    "percentile_nearest_rank": ("quantile[b] = x_lo + (h - (double)lo) * (x_hi - x_lo);",
                                "quantile[b] = x_lo;"),
    "tail_bin_not_clamped": ("            if (bin > n_bins - 1)\n                bin = n_bins - 1;",
                             "            if (bin > n_bins)\n                bin = n_bins - 1;"),
}
# Mistakes in the selector-variant oracle, pinned by test_oracle_selector.py.
SELECTOR_MUTANTS = {
    "mean_divides_by_page_size": ("s32 += bf16f(qj[i]) * (sm[i] / (float)valid);",
                                  "s32 += bf16f(qj[i]) * (sm[i] / (float)ps);"),
    "mean64_divides_by_page_size": (
        "s64 += (double)bf16f(qj[i]) * ((double)sm[i] / (double)valid);",
        "s64 += (double)bf16f(qj[i]) * ((double)sm[i] / (double)ps);"),
    "key_sums_skip_last_token": ("for (int64_t t = 0; t < valid; ++t)\n                        s +=",
                                 "for (int64_t t = 0; t < valid - 1; ++t)\n                        s +="),
    "forced_ignores_local_pages": ("r[p].forced = (p < sink || p >= n - local) ? 0 : 1;",
                                   "r[p].forced = (p < sink) ? 0 : 1;"),
    "forced_ties_to_higher_index": ("return (a->p > b->p) - (a->p < b->p);",
                                    "return (a->p < b->p) - (a->p > b->p);"),
}
CASES = [(n, "sparrow_oracle.c", o, w, "test_oracle.py") for n, (o, w) in MUTANTS.items()] + \
        [(n, "acceptance_oracle.c", o, w, "test_oracle_acceptance.py")
         for n, (o, w) in ACCEPTANCE_MUTANTS.items()] + \
        [(n, "selector_oracle.c", o, w, "test_oracle_selector.py")
         for n, (o, w) in SELECTOR_MUTANTS.items()]


@pytest.mark.parametrize("name,fname,old,new,pins", sorted(CASES), ids=[c[0] for c in sorted(CASES)])
def test_pins_catch_planted_mistake(name, fname, old, new, pins, tmp_path):
    srcs = []
    for f in SOURCES:
        text = open(os.path.join(ORACLE, f)).read()
        if f == fname:
            assert text.count(old) == 1, f"mutation site for {name} not found exactly once"
            text = text.replace(old, new)
        (tmp_path / f).write_text(text)
        srcs.append(str(tmp_path / f))
    lib = tmp_path / "liboracle_mutant.so"
    subprocess.check_call(["gcc", "-O2", "-std=c99", "-fPIC", "-fopenmp", "-ffp-contract=off",
                           "-shared", "-o", str(lib)] + srcs + ["-lm"])
    env = dict(os.environ, SPARROW_ORACLE_LIB=str(lib), OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", pins)],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"pins did not catch mutant {name}:\n{r.stdout[-2000:]}"
