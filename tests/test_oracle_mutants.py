"""Each plausible single mistake in the oracle must fail at least one pin.

A mutant is the oracle's C source with one edit, compiled to a temporary
library and checked in a child process (so a crash also counts as caught).
"""
import os
import subprocess
import sys

import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))

MUTANTS = [
    ("ties_away_from_zero", "double q = nearbyint(t);", "double q = round(t);"),
    ("floor_rounding", "double q = nearbyint(t);", "double q = floor(t);"),
    ("no_upper_clip", "if (q > (double)M) q = (double)M;", ""),
    ("levels_off_by_one", "return (1 << (bits - 1)) - 1;", "return (1 << (bits - 1));"),
    ("argmax_not_argmin", "(best < 0 || E[g] < E[best])", "(best < 0 || E[g] > E[best])"),
    ("ties_to_largest_scale", "(best < 0 || E[g] < E[best])", "(best < 0 || E[g] <= E[best])"),
    ("zero_scale_not_skipped", "if (g < 0) break;                               /* S3: no scale */",
     "if (g < 0) g = 0;"),
    ("residual_sign", "r[j] = r[j] - as * (double)q[j]; /* Eq. (7) */",
     "r[j] = r[j] + as * (double)q[j]; /* Eq. (7) */"),
    ("grid_missing_M", "a[g] = (float)((double)m * (double)c[g] / (double)M);",
     "a[g] = (float)((double)m * (double)c[g]);"),
    ("grid_descending", "c[g] = (float)((double)(g + 1) / (double)G);",
     "c[g] = (float)((double)(G - g) / (double)G);"),
    ("max_without_abs", "double v = fabs(r[j]);", "double v = r[j];"),
    ("no_minimum_one_point", "if (n >= 1 && Er <= tol * Ew) return 1;",
     "if (Er <= tol * Ew) return 1;"),
    ("strict_stop", "if (n >= 1 && Er <= tol * Ew) return 1;",
     "if (n >= 1 && Er < tol * Ew) return 1;"),
    ("stop_ignores_cap", "if (n >= P) return 1;", "if (n > P) return 1;"),
    ("err_before_update", "err[n - 1] = sum_sq(r, d);", "err[n - 1] = Er;"),
    ("codes_at_wrong_scale", "oracle_codes(r, d, as, M, q);", "oracle_codes(r, d, (double)a[0], M, q);"),
    ("x_transposed", "Xt[n * d + j] = X[j * N + n];", "Xt[n * d + j] = X[n * d + j];"),
    ("output_error_not_mean", "err[s] = se / (double)N;", "err[s] = se;"),
    ("reconstruct_drops_last_point", "for (int i = 0; i < counts[k]; ++i)\n                s = s +",
     "for (int i = 0; i + 1 < counts[k]; ++i)\n                s = s +"),
    ("verifier_accepts_any_scale", "if (E[go] <= (1.0 + 1e-6) * E[gbest]) ct++;", "if (1) ct++;"),
    ("verifier_skips_codes", "if (qo != qr) {", "if (0) {"),
    ("calib_error_not_mean", "return s / (double)N;", "return s;"),
    ("calib_strict_stop", "if (n >= 1 && e <= thr) return 1;", "if (n >= 1 && e < thr) return 1;"),
    ("calib_threshold_never_relative",
     "return cal->relative ? cal->eps * calib_error(w, d, cal->X, cal->N) : cal->eps;",
     "return cal->eps;"),
    ("calib_x_transposed", "y += v[j] * (double)X[j * N + t];", "y += v[j] * (double)X[t * d + j];"),
    ("calib_error_of_weights", "e = calib_error(r, d, cal->X, cal->N);          /* Eq. (12) */",
     "e = calib_error(w, d, cal->X, cal->N);          /* Eq. (12) */"),
    ("calib_no_fp32_allowance", "const double lam = 4.0 * 0x1p-24 * sqrt((double)d);",
     "const double lam = 0.0;"),
    ("calib_loose_fp32_allowance", "const double lam = 4.0 * 0x1p-24 * sqrt((double)d);",
     "const double lam = 0x1p-8 * sqrt((double)d);"),
    ("int_shift_truncates", "Y[k * N + t] = (int64_t)s >> p;",
     "Y[k * N + t] = (int64_t)s / ((int64_t)1 << p);"),
    ("int_scale_floor", "v = rint(ldexp((double)scales[k * P + i], p));",
     "v = floor(ldexp((double)scales[k * P + i], p));"),
    ("int_scale_ties_away", "v = rint(ldexp((double)scales[k * P + i], p));",
     "v = round(ldexp((double)scales[k * P + i], p));"),
    ("int_forward_all_points", "for (int i = 0; i < counts[k]; ++i) {\n                const int8_t *q",
     "for (int i = 0; i < P; ++i) {\n                const int8_t *q"),
    ("int_x_transposed", "(int64_t)X[t * d + j]", "(int64_t)X[j * N + t]"),
    ("int_scale_no_clamp", "if (v > lim) { v = lim; ++clamped; }", "if (v > lim) { ++clamped; }"),
    ("refit_abs_norm", "qq += (double)q[j] * (double)q[j];", "qq += fabs((double)q[j]);"),
    ("refit_residual_at_grid_scale", "            as = (double)a_pt;\n", "            (void)0;\n"),
    ("refit_verifier_any_scale",
     "if (!(ao == (float)aref || fabs(as - aref) <= 0x1p-23 * fabs(aref))) {", "if (0) {"),
    ("clip_argmax", "if (best < 0 || e[g] < e[best]) best = g;", "if (best < 0 || e[g] > e[best]) best = g;"),
    ("clip_ties_largest", "if (best < 0 || e[g] < e[best]) best = g;", "if (best < 0 || e[g] <= e[best]) best = g;"),
    ("clip_error_of_weights", "e[g] = calib_error(R, d, X, N);", "e[g] = calib_error(D, d, X, N);"),
    ("clip_wrong_levels", "oracle_candidate_scales(D, d, M, cc, clipG, a);",
     "oracle_candidate_scales(D, d, M + 1, cc, clipG, a);"),
    ("clip_verifier_any", "if (cl.e[go] <= cl.e[cbest] * (1.0 + 1e-5) + sg) ct++;", "if (1) ct++;"),
    ("gap_not_halved", "    return gap / 2.0;", "    return gap;"),
    ("gap_counts_zero_diff", "if (diff > 0.0 && (gap == 0.0 || diff < gap)) gap = diff;",
     "if (diff >= 0.0 && (gap == 0.0 || diff < gap)) gap = diff;"),
    ("paper_step_max", "    if (g > eta) g = eta;", "    if (g < eta) g = eta;"),
    ("paper_range_half", "*count = (int64_t)floor(2.0 * (double)M * sqrt(sum_sq(r, d)) / g);",
     "*count = (int64_t)floor((double)M * sqrt(sum_sq(r, d)) / g);"),
    ("paper_no_vertex", "                        cand[1] = gv;\n                        cand[2] = gv + 1;",
     "                        cand[1] = 0;\n                        cand[2] = 0;"),
    ("paper_two_point_bracket", "int64_t around[3] = {g0 - 1, g0, g0 + 1};",
     "int64_t around[3] = {g0, g0 + 1, g0 + 1};"),
    ("paper_ties_largest", "if (E < Eb || (E == Eb && h < best)) { Eb = E; best = h; }",
     "if (E <= Eb) { Eb = E; best = h; }"),
    ("asym_offset_max", "const float beta = (float)((mx + mn) / 2.0);   /* B2: the midpoint */",
     "const float beta = (float)mx;"),
    ("asym_stop_centred",
     "for (int64_t j = 0; j < d; ++j) r[j] = (double)w[j] - (double)beta;   /* B2 */",
     "for (int64_t j = 0; j < d; ++j) r[j] = (double)w[j] - (double)beta;\n        Ew = sum_sq(r, d);"),
    ("asym_recon_no_offset", "double s = offsets ? (double)offsets[k] : 0.0;", "double s = 0.0;"),
    ("asym_error_no_offset", "D[j] = (double)w[j] - (double)beta;", "D[j] = (double)w[j];"),
    ("calib_stop_ignores_cap", "if (n >= P || Er == 0.0) return 1;", "if (Er == 0.0) return 1;"),
    ("calib_no_minimum_one_point", "if (n >= 1 && e <= thr) return 1;", "if (e <= thr) return 1;"),
    ("gate_keeps_failing_naive", "if (cal ? eN <= thr : EN <= tol * Ew) {            /* Algorithm 2's test */",
     "if (1) {"),
    ("gate_naive_wrong_step", "oracle_candidate_scales(r, d, M, &one, 1, &aN);    /* a_N = fl32(m / M) */",
     "oracle_candidate_scales(r, d, M + 1, &one, 1, &aN);"),
    ("gate_continues_from_naive",
     "            memset(codes, 0, (size_t)d);                    /* discarded: Algorithm 1 from w */",
     "            memcpy(r, R, sizeof(double) * (size_t)d);\n            scales[0] = aN;\n"
     "            err[0] = EN;\n            n = 1;\n            e = eN;"),
    ("gate_verifier_accepts_any", "if (pass && !nearN) { st = 10; break; }", "if (0) { st = 10; break; }"),
]


@pytest.fixture(scope="module")
def source():
    with open(oracle.SRC) as f:
        return f.read()


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, source, name, old, new):
    assert source.count(old) == 1, f"mutation site of {name} not unique/present"
    src = tmp_path / f"{name}.c"
    src.write_text(source.replace(old, new))
    lib = oracle.build(force=True, src=str(src), out=str(tmp_path / f"{name}.so"))
    env = dict(os.environ, OMP_NUM_THREADS="2")
    p = subprocess.run([sys.executable, os.path.join(HERE, "oracle_mutant_driver.py"), lib],
                       capture_output=True, text=True, timeout=300, env=env)
    assert p.returncode != 0, f"mutant {name} passed every pin:\n{p.stdout}\n{p.stderr}"


def test_unmutated_oracle_passes_driver():
    env = dict(os.environ, OMP_NUM_THREADS="2")
    p = subprocess.run([sys.executable, os.path.join(HERE, "oracle_mutant_driver.py"),
                        oracle.build(force=False)], capture_output=True, text=True,
                       timeout=300, env=env)
    assert p.returncode == 0, p.stdout + p.stderr
