"""The oracle's pins must catch plausible mistakes.

Each case plants one mistake (a dropped term, an off-by-one, a wrong sign,
index or operand order) in a temporary copy of the oracle's C source, builds
it, and runs the oracle pin tests against that build in a subprocess: at
least one pin must fail. Everything runs on the CPU.
"""
import os
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ALLOC = "tests/test_oracle_alloc.py"
SCORES = "tests/test_oracle_scores.py"
SELDEC = "tests/test_oracle_select_decode.py"
VARIANTS = "tests/test_oracle_alloc_variants.py"
IPT = "tests/test_oracle_ipt.py"
WINDOW = "tests/test_oracle_window.py"
APPEND = "tests/test_oracle_decode_append.py"

MUTANTS = {
    "lse_not_causal": ("int64_t last = win0 + i; /* causal: keys 0..last that the cache holds */",
                       "int64_t last = C - 1 + 0 * i;", SCORES),
    "append_skips_new": ("int64_t n = (r1 > r0 ? r1 - r0 : 0) + n_new;", "int64_t n = (r1 > r0 ? r1 - r0 : 0);", APPEND),
    "append_wrong_head": ("const double* kn = knew + ((int64_t)b * Hkv + h) * cap * d;",
                          "const double* kn = knew + ((int64_t)b * Hkv) * cap * d;", APPEND),
    "append_value_offset": ("const double* vr = e < nc ? vc + (r0 + e) * d : vn + (e - nc) * d;",
                            "const double* vr = e < nc ? vc + (r0 + e) * d : vn + (e - nc + 1) * d;", APPEND),
    "lse_window_unclamped": ("    if (last > C - 1) last = C - 1;\n", "", WINDOW),
    "select_scored_range": ("if (n_scored < 0 || s < 0 || C - W > n_scored ||", "if (n_scored < 0 || s < 0 || C - W > n_scored + 1 ||",
                            WINDOW),
    "lse_off_by_one": ("for (int64_t j = 0; j <= last; ++j) z +=", "for (int64_t j = 0; j < last; ++j) z +=", SCORES),
    "colsum_no_group_mean": ("colsum[c] = acc / (double)G;", "colsum[c] = acc;", SCORES),
    "colsum_lse_sign": ("acc += exp(scale * orc_dot(q_win + r * d, kj, d) - lse[r]",
                        "acc += exp(scale * orc_dot(q_win + r * d, kj, d) + lse[r] - 2.0 * lse[r] * (i == 0)", SCORES),
    "colsum_no_scale": ("acc += exp(scale * orc_dot(q_win + r * d, kj, d)", "acc += exp(orc_dot(q_win + r * d, kj, d)", SCORES),
    "lse_wrong_group": ("int64_t h = q / G;\n    const double* qi", "int64_t h = q % Hkv;\n    const double* qi", SCORES),
    "pool_divisor": ("pooled[row * n + j] = s / (double)kp;", "pooled[row * n + j] = s / (double)(kp - 1);", SCORES),
    "pool_window": ("for (int64_t t = j - r; t <= j + r; ++t)", "for (int64_t t = j - r; t < j + r; ++t)", SCORES),
    "select_tie_high": ("return (a->j < b->j) ? -1 : (a->j > b->j);\n}\n\nstatic int orc_cmp_i32",
                        "return (a->j > b->j) ? -1 : (a->j < b->j);\n}\n\nstatic int orc_cmp_i32", SELDEC),
    "alloc_no_reserve": ("for (int64_t h = 0; h < n; ++h) x[h] = (sg[h] / sgsum) * (double)T;",
                         "for (int64_t h = 0; h < n; ++h) x[h] = (sg[h] / sgsum) * (double)(T + n);", ALLOC),
    "alloc_greedy_ascending": ("if (a->sigma > b->sigma) return -1;\n  if (a->sigma < b->sigma) return 1;\n  return (a->idx < b->idx) ? -1 : (a->idx > b->idx);\n}\n\nint orc_allocate",
                               "if (a->sigma < b->sigma) return -1;\n  if (a->sigma > b->sigma) return 1;\n  return (a->idx < b->idx) ? -1 : (a->idx > b->idx);\n}\n\nint orc_allocate", ALLOC),
    "alloc_round_smallest": ("if (a->frac > b->frac) return -1;\n  if (a->frac < b->frac) return 1;",
                             "if (a->frac < b->frac) return -1;\n  if (a->frac > b->frac) return 1;", ALLOC),
    "decode_no_normalise": ("for (int t = 0; t < d; ++t) o[t] += p * vc[r * d + t];\n    }\n    for (int t = 0; t < d; ++t) o[t] /= z;",
                            "for (int t = 0; t < d; ++t) o[t] += p * vc[r * d + t];\n    }\n", SELDEC),
    "append_no_normalise": ("for (int t = 0; t < d; ++t) o[t] += p * vr[t];\n    }\n    for (int t = 0; t < d; ++t) o[t] /= z;",
                            "for (int t = 0; t < d; ++t) o[t] += p * vr[t];\n    }\n", APPEND),
    "decode_wrong_group": ("int64_t b = bq / Hq, qh = bq % Hq, h = qh / G;\n    int64_t r0 = offsets[b * Hkv + h], r1 = offsets[b * Hkv + h + 1];\n    const double* qv",
                           "int64_t b = bq / Hq, qh = bq % Hq, h = qh % Hkv;\n    int64_t r0 = offsets[b * Hkv + h], r1 = offsets[b * Hkv + h + 1];\n    const double* qv",
                           SELDEC),
    "thr_at_mean": ("t[h] = sigma[h] < mean ? 0.0 : sigma[h];", "t[h] = sigma[h] <= mean ? 0.0 : sigma[h];", VARIANTS),
    "reverse_whole_budget": ("budgets[h] = s + W + (M - (budgets[h] - s - W));", "budgets[h] = s + W + (M - budgets[h]);",
                             VARIANTS),
    "mix_precedence": ("t[h] = (a + b) / 2.0;", "t[h] = a + b / 2.0;", VARIANTS),
    "binary_round_up": ("int64_t k = (int64_t)floor(f * (double)n);", "int64_t k = (int64_t)ceil(f * (double)n);",
                        VARIANTS),
    "binary_reverse_same_side": ("budgets[order[variant == 4 ? j : n - 1 - j].idx] = C;", "budgets[order[j].idx] = C;",
                                 VARIANTS),
    "ipt_max_as_min": ("out = (g == 0 || v > out) ? v : out;", "out = (g == 0 || v < out) ? v : out;", IPT),
    "ipt_mean_no_divide": ("colsum[c] = agg == 2 ? out / (double)G : out;", "colsum[c] = out;", IPT),
    "ipt_only_tie_high": ("if (qscore[h * G + g] > qscore[h * G + gstar]) gstar = g;",
                          "if (qscore[h * G + g] >= qscore[h * G + gstar]) gstar = g;", IPT),
    "ipt_unweighted": ("double v = qscore[q] * A;", "double v = A;", IPT),
    "ipt_no_lse": ("A += exp(scale * orc_dot(q_win + r * d, kj, d) - lse[r]);",
                   "A += exp(scale * orc_dot(q_win + r * d, kj, d));", IPT),
}


@pytest.mark.slow
@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name, tmp_path):
    old, new, pins = MUTANTS[name]
    src = open(oracle.SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not unique"
    mutated = tmp_path / "mutant.c"
    mutated.write_text(src.replace(old, new))
    lib = str(tmp_path / "libmutant.so")
    oracle.build(force=True, src=str(mutated), out=lib)
    env = dict(os.environ, SGDKV_ORACLE_LIB=lib, OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:randomly",
                        "--hypothesis-seed=0", pins], cwd=ROOT, env=env,
                       capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"mutant {name} survived the pins:\n{r.stdout[-2000:]}"
    assert "failed" in r.stdout or "error" in r.stdout.lower()
