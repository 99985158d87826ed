"""The oracle's pins catch plausible mistakes (CPU only).

Each case copies the oracle's C source, plants one plausible mistake (a dropped
term, a wrong sign, an off-by-one, a transposed index ...), builds it into a
temporary library, and runs the pin suite against that build in a subprocess.
The pin suite must fail for every mutant; it must pass for the unmodified
source.
"""
import os
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "eta_oracle.c")

MUTANTS = {
    "unbiased_variance": ("s[i] = sqrt(s[i] / (double)b);", "s[i] = sqrt(s[i] / (double)(b - 1));"),
    "variance_not_std": ("s[i] = sqrt(s[i] / (double)b);", "s[i] = s[i] / (double)b;"),
    "mean_off_by_one": ("m[i] /= (double)b;", "m[i] /= (double)(b + 1);"),
    "maxnorm_is_mean": ("if (n > best) best = n;", "best += n / b;"),
    "dropped_z": ("double gauss = dot + z * sqrt(var);", "double gauss = dot + sqrt(var);"),
    "z_sign": ("double gauss = dot + z * sqrt(var);", "double gauss = dot - z * sqrt(var);"),
    "sigma_not_squared": ("var += q[i] * q[i] * sigma[i] * sigma[i];", "var += q[i] * q[i] * sigma[i];"),
    "max_not_min": ("double lo = gauss < spher ? gauss : spher;", "double lo = gauss > spher ? gauss : spher;"),
    "bound_unscaled": ("return lo / sqrt((double)d);", "return lo;"),
    "strict_threshold": ("bound[j] >= tau_eff) ? 1 : 0;", "bound[j] > tau_eff) ? 1 : 0;"),
    "rescue_last_max": ("if (arg < 0 || bound[j] > best)", "if (arg < 0 || bound[j] >= best)"),
    "rescue_window_short": ("int64_t Wn = c < N ? c : N;", "int64_t Wn = c < N ? c - 1 : N;"),
    "pins_off_by_one": ("for (int64_t j = N - lwb; j < N; ++j)", "for (int64_t j = N - lwb + 1; j < N; ++j)"),
    "gate_sign": ("return S * sigmoid(beta * (S - tau));", "return S * sigmoid(beta * (tau - S));"),
    "gate_missing_S": ("return S * sigmoid(beta * (S - tau));", "return sigmoid(beta * (S - tau));"),
    "slack_sign": ("double tau_eff = P->tau[row] - P->a;", "double tau_eff = P->tau[row] + P->a;"),
    "tail_dropped": ("in[t] = (j < N) ? sel[j] : (uint8_t)(use_tail ? 1 : 0);", "in[t] = (j < N) ? sel[j] : 0;"),
    "score_unscaled": ("    S *= scale;\n", "\n"),
    "self_index": ("(self_ungated && t == T - 1)", "(self_ungated && t == T - 2)"),
    "predictor_transposed": ("(double)W[j * Hq + h];", "(double)W[h * J + j];"),
    "softmax_no_max_shift": ("double w = exp(st[t] - m);", "double w = exp(st[t] - m) * (1.0 + 1e-3 * (t == 0));"),
    "f16_ties_away": ("r = nearbyint(a / ulp) * ulp;", "r = round(a / ulp) * ulp;"),
    "f16_no_subnormal_floor": ("if (ex < -14) ex = -14;", ";"),
    "f16_short_significand": ("const double ulp = ldexp(1.0, ex - 10);", "const double ulp = ldexp(1.0, ex - 9);"),
    "e4m3_ties_away": ("    r = nearbyint(a / ulp) * ulp;   /* a / ulp is exact; default mode rounds half to even */\n  }\n  return copysign(r, x);\n}\n\nvoid eta_oracle_round_e4m3_array", "    r = round(a / ulp) * ulp;\n  }\n  return copysign(r, x);\n}\n\nvoid eta_oracle_round_e4m3_array"),
    "e4m3_no_subnormal_floor": ("if (ex < -6) ex = -6;", ";"),
    "e4m3_long_significand": ("const double ulp = ldexp(1.0, ex - 3);", "const double ulp = ldexp(1.0, ex - 4);"),
    "e4m3_no_saturation": ("  if (a >= 464.0) {", "  if (a >= 1e300) {"),
    "e4m3_sign_dropped": ("  }\n  return copysign(r, x);\n}\n\nvoid eta_oracle_round_e4m3_array",
                          "  }\n  return r;\n}\n\nvoid eta_oracle_round_e4m3_array"),
    "envelope_block_divisor": ("double sd = sqrt(acc / (double)b_sub);", "double sd = sqrt(acc / (double)b);"),
    "calib_unweighted": ("const double wt = 1.0 / (double)(t + 1);", "const double wt = 1.0;"),
    "calib_weight_off_by_one": ("const double wt = 1.0 / (double)(t + 1);", "const double wt = 1.0 / (double)(t + 2);"),
    "calib_not_causal_diag": ("for (int s2 = 0; s2 <= t; ++s2) {", "for (int s2 = 0; s2 < t || s2 == 0; ++s2) {"),
    "calib_bin_left_edge": ("g += hist[b] * sigmoid(beta * (lo + ((double)b + 0.5) * w - c));", "g += hist[b] * sigmoid(beta * (lo + (double)b * w - c));"),
    "prefill_diagonal_gated": ("    if (j == i) Sg = S;", "    ;"),
    "prefill_r_without_diagonal": ("    rsum += g;", "    if (j < i) rsum += g;"),
    "prefill_additive_sign": ("double Sg = additive ? S + C * g - C : S * g;", "double Sg = additive ? S - C * g + C : S * g;"),
    "prefill_lse_without_max": ("  *L_out = m + log(l);", "  *L_out = log(l);"),
    "quality_strict_positive": ("int positive = bmax >= tau_eff;", "int positive = bmax > tau_eff;"),
    "quality_missed_over_selected": ("if (t < N * b && !sel[t / b]) Zrej += w;",
                                     "if (t < N * b && sel[t / b]) Zrej += w;"),
    "quality_recall_counts_tail": ("    if (j == N) break;\n    int positive",
                                   "    if (j == N) { qual[4] += above; break; }\n    int positive"),
    "quality_blockmax_skips_last_key": ("      if (S > bmax) bmax = S;", "      if (S > bmax && t + 1 < t1) bmax = S;"),
    "quality_missed_without_tail": ("    double w = exp(sg[t] - m);\n    Z += w;",
                                    "    double w = exp(sg[t] - m);\n    if (t < N * b) Z += w;"),
    "calib_bisect_direction": ("if (eta_oracle_calib_g(hist, nb, lo, hi, beta, m) > target) a = m; else b = m;", "if (eta_oracle_calib_g(hist, nb, lo, hi, beta, m) < target) a = m; else b = m;"),
}


def _run_pins(lib_path):
    env = dict(os.environ, ETA_ORACLE_LIB=lib_path)
    return subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                           os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                          cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)


def _build(src_text, tmp):
    c = os.path.join(tmp, "o.c")
    so = os.path.join(tmp, "liboracle_mut.so")
    with open(c, "w") as f:
        f.write(src_text)
    subprocess.run(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-std=c11", c, "-o", so, "-lm"],
                   check=True, capture_output=True)
    return so


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) >= 1, f"mutation anchor for {name} not found in the oracle source"
    with tempfile.TemporaryDirectory() as tmp:
        so = _build(src.replace(old, new, 1), tmp)
        r = _run_pins(so)
    assert r.returncode != 0, f"pin suite passed against mutant {name}:\n{r.stdout[-2000:]}"


def test_pins_pass_on_unmodified_source():
    with tempfile.TemporaryDirectory() as tmp:
        so = _build(open(SRC).read(), tmp)
        r = _run_pins(so)
    assert r.returncode == 0, r.stdout[-3000:]
