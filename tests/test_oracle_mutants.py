"""The oracle's pins must catch plausible mistakes.

Each case plants one mistake in a copy of the oracle's C source (on the CPU,
in a temporary directory), builds it, and runs the pin suite against that
build in a subprocess: the suite must fail.  The mistakes are the ones a
reader checking the oracle against the paper would worry about: a dropped
or misindexed h, a sign error, the wrong tie rule, the wrong init divisor,
a missing clip, an off-by-one window, a nibble order swap, a missing fp32
rounding point, a wrong subnormal scale.
"""
import os
import subprocess
import sys
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parent.parent
SRC = ROOT / "oracle" / "hscale_oracle.c"

MUTANTS = {
    "drop_h": ("double hj = h ? h[j] : 1.0;", "double hj = 1.0;"),
    "sign_of_residual": ("double d = w[j] - q;", "double d = w[j] + q;"),
    "e2m1_ties_to_odd": ("(d == best_d && (i % 2) == 0)", "(d == best_d && (i % 2) == 1)"),
    "e4m3_ties_to_odd": ("(d == best_d && (c % 2) == 0)", "(d == best_d && (c % 2) == 1)"),
    "argmin_keeps_last": ("if (d == -down || e < best_e) {", "if (d == -down || e <= best_e) {"),
    "init_divides_by_4": ("double s_init = rn32(amax / 6.0);", "double s_init = rn32(amax / 4.0);"),
    "walk_clip_to_0": ("if (c < 1) c = 1;\n        if (c > ORACLE_M) c = ORACLE_M;\n        double e =",
                       "if (c < 0) c = 0;\n        if (c > ORACLE_M) c = ORACLE_M;\n        double e ="),
    "h_slice_misindexed": ("hh[j] = (double)h[i * 16 + j];\n            int c0v;",
                           "hh[j] = (double)h[(j * 16 + i) % n];\n            int c0v;"),
    "nibble_order_swapped": ("dst[k] = (uint8_t)(nib[2 * k] | (nib[2 * k + 1] << 4));",
                             "dst[k] = (uint8_t)(nib[2 * k + 1] | (nib[2 * k] << 4));"),
    "reciprocal_not_fp32": ("R[c] = (float)(1.0 / (double)S[c]);",
                            "R[c] = (float)(1.0 / ((double)s_g * oracle_e4m3_value(c)));"),
    "scaled_weight_exact_division": ("double x = rn32(fabs(w[j]) * (double)R);",
                                     "double x = fabs(w[j]) / (double)S;"),
    "window_off_by_one": ("for (int d = -down; d <= up; ++d, ++k) {", "for (int d = -down; d < up; ++d, ++k) {"),
    "hdiag_abs_not_square": ("h[j] += x * x;", "h[j] += fabs(x);"),
    "e4m3_subnormal_scale": ("if (e == 0) return (double)m / 8.0 * ldexp(1.0, -6);",
                             "if (e == 0) return (double)m / 8.0 * ldexp(1.0, -7);"),
    "4over6_tie_to_anchor_6": ("return loss[0] <= loss[1] ? code[0] : code[1];",
                               "return loss[0] < loss[1] ? code[0] : code[1];"),
    "4over6_anchor_3": ("static const double anchors[2] = {4.0, 6.0};",
                        "static const double anchors[2] = {3.0, 6.0};"),
    "given_init_unclipped": ("c0v = init_codes[r * G + i];\n                if (c0v < 1) c0v = 1;",
                             "c0v = init_codes[r * G + i];\n                if (c0v < 0) c0v = 1;"),
    "accumulate_overwrites": ("            h[j] += x * x;\n        }\n    }\n}\n\n/* Loads group",
                              "            h[j] = x * x;\n        }\n    }\n}\n\n/* Loads group"),
    "zero_drops_sign": ("if (nib) nib[j] = (uint8_t)((neg[j] << 3) | i);",
                        "if (nib) nib[j] = (uint8_t)(((neg[j] && i) << 3) | i);"),
    "delta_sign": ("delta[r * n + j] = (double)wf - v * (double)S[c];",
                   "delta[r * n + j] = (double)wf + v * (double)S[c];"),
    "delta_nibble_order": ("int nib = (j % 2 == 0) ? (byte & 15) : (byte >> 4);",
                           "int nib = (j % 2 == 0) ? (byte >> 4) : (byte & 15);"),
    "output_error_not_squared": ("row_err[r] += y * y;", "row_err[r] += fabs(y);"),
    "output_error_reversed_column": ("y += x[j] * delta[r * n + j];", "y += x[j] * delta[r * n + (n - 1 - j)];"),
    "output_error_overwrites": ("row_err[r] += y * y;", "row_err[r] = y * y;"),
    "summary_rel_wrong_denominator": ("sum_rel[k] += (e_init[g] - e_best[g]) / e_init[g];",
                                      "sum_rel[k] += (e_init[g] - e_best[g]) / e_best[g];"),
    "summary_rel_unguarded_zero_init": ("if (e_init[g] > 0.0) sum_rel[k] +=", "if (1) sum_rel[k] +="),
    "summary_rel_not_relative": ("sum_rel[k] += (e_init[g] - e_best[g]) / e_init[g];",
                                 "sum_rel[k] += (e_init[g] - e_best[g]);"),
    "summary_swaps_sums": ("sum_init[k] += e_init[g];\n        sum_best[k] += e_best[g];",
                           "sum_init[k] += e_best[g];\n        sum_best[k] += e_init[g];"),
    "stats_init_error_at_wrong_shift": ("if (d == 0 && e_init) *e_init = e;", "if (d == 1 && e_init) *e_init = e;"),
    "delta_code_off_by_one": ("int c = codes[r * G + j / 16];", "int c = codes[r * G + j / 16] + 1;"),
    "stats_shift_not_first_min": ("            best_c = c;\n            best_d = d;",
                                  "            best_c = c;\n            best_d = d - (d > 0);"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_mistake(name, tmp_path):
    before, after = MUTANTS[name]
    src = SRC.read_text()
    assert before in src, "mutation site moved; update the mutant"
    mutant = tmp_path / "mutant.c"
    mutant.write_text(src.replace(before, after, 1))
    lib = tmp_path / "liboracle_mutant.so"
    subprocess.run(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
                    "-o", str(lib), str(mutant), "-lm"], check=True)
    env = dict(os.environ, HSCALE_ORACLE_LIB=str(lib))
    r = subprocess.run([sys.executable, "-m", "pytest", str(ROOT / "tests" / "test_oracle_pins.py"),
                        str(ROOT / "tests" / "test_oracle_pins_init.py"),
                        str(ROOT / "tests" / "test_oracle_pins_diag.py"),
                        "-q", "-x", "-p", "no:cacheprovider"],
                       capture_output=True, text=True, env=env, cwd=str(ROOT), timeout=600)
    assert r.returncode != 0, f"mutant {name} survived the pins:\n{r.stdout[-2000:]}"
