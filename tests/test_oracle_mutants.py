"""Planted mistakes in copies of the oracle must fail the pin suite.

Each mutant is a one-line slip in ``oracle/dsde_oracle.c`` (built on the CPU
into a temporary library); the pin tests are run against it in a child
process and must fail.  This shows the pins constrain every part of the
oracle, not only its happy path.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "dsde_oracle.c")

MUTANTS = {
    "kl_direction": ("if (p > 0.0) csum_add(&kls, p * (lp - lq));", "if (p > 0.0) csum_add(&kls, p * (lq - lp));"),
    "no_temperature_in_lse": ("csum_add(&S, exp(logit(base, dtype, V, row, v) / T - m));",
                              "csum_add(&S, exp(logit(base, dtype, V, row, v) - m));"),
    "residual_sign": ("w[v] = p - q > 0.0 ? p - q : 0.0;", "w[v] = q - p > 0.0 ? q - p : 0.0;"),
    "target_row_index": ("const int64_t trow0 = first + b;", "const int64_t trow0 = first;"),
    "bonus_row_index": ("tr = trow0 + SL;", "tr = trow0 + SL - 1;"),
    "acceptance_not_strict": ("if (u < thr) {", "if (u <= thr) {"),
    "cdf_not_strict": ("if (C > target_mass) {", "if (C >= target_mass) {"),
    "short_window_off_by_one": ("int32_t ns = n_short < count ? n_short : count;",
                                "int32_t ns = n_short + 1 < count ? n_short + 1 : count;"),
    "bessel_variance": ("*var = sv / sa;", "*var = sv / (sa - 1.0);"),
    "weights_reversed": ("double alpha = pow(delta, (double)(i - 1));\n    sa += alpha;",
                         "double alpha = pow(delta, (double)(n - i));\n    sa += alpha;"),
    "cdf_weights_rescaled": ("    csum_add(&Cs, w[v]);\n    C = csum_value(&Cs);", "    C += w[v] * (1.0 + 1e-9);"),
    "wvir_guard_always_added": ("*wvir = *var_s / (*var_l > 0.0 ? *var_l : eps);",
                                "*wvir = *var_s / (*var_l + eps);"),
    "window_not_shifted": ("sad += alpha * (newest_first[i - 1] - h1);", "sad += alpha * newest_first[i - 1];"),
    "scale_factor": ("*sf = exp(2.0 * mu_last) - 1.0;", "*sf = exp(mu_last) - 1.0;"),
    "cap_not_mean": ("double cap = n > 0 ? sum / (double)n : NAN;",
                     "double cap = n > 0 ? sum / (double)(n + 1) : NAN;"),
    "round_down": ("double r = floor(x + 0.5);", "double r = floor(x);"),
    "sl_hat_branch": ("if (pen <= 1.0) return (1.0 - pen) * (sl_max - sl_min) + sl_min;",
                      "if (pen <= 1.0) return (1.0 - pen) * sl_max + sl_min;"),
    "push_skipped": ("ring[head[b]] = mu;", "(void)0;"),
    "greedy_tie_takes_last": ("    if (z > m) {\n      m = z;\n      best = v;", "    if (z >= m) {\n      m = z;\n      best = v;"),
    "greedy_emits_next_row": ("tok[a] = (int32_t)row_argmax(J->target, J->dtype, V, trow0 + a);",
                              "tok[a] = (int32_t)row_argmax(J->target, J->dtype, V, trow0 + a + (a < SL));"),
    "entropy_sign": ("if (q > 0.0) csum_add(&h, -q * lq);", "if (q > 0.0) csum_add(&h, q * lq);"),
    "budget_off_by_one": ("int32_t room = budget[b] - 1 > 0 ? budget[b] - 1 : 0;",
                          "int32_t room = budget[b] > 0 ? budget[b] : 0;"),
    "greedy_kld_at_zero_scale": ("const double T = greedy ? 1.0 : (double)J->temperature[b];",
                                 "const double T = greedy ? 2.0 : (double)J->temperature[b];"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_mistake(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation site for {name} not found exactly once"
    mpath = tmp_path / "mutant.c"
    mpath.write_text(src.replace(old, new))
    lib = tmp_path / "libmutant.so"
    subprocess.run(["gcc", "-O2", "-std=c11", "-shared", "-fPIC", "-o", str(lib), str(mpath), "-lm",
                    "-lpthread"], check=True)
    env = dict(os.environ, DSDE_ORACLE_LIB=str(lib))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode != 0, f"mutant {name} survived the pin suite"
