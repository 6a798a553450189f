"""Planted mistakes in the oracle (on the CPU) must each fail a pin.

Each mutation rewrites one line of ``oracle/dart_oracle.c``, builds it into a
temporary library and runs the pins of ``test_oracle_pins.py`` against it
*excluding* the comparison with the pure-Python mini oracle, so what catches the
mistake is a closed form, an invariant, brute force, a library routine or the
finite differences, not the second implementation.
"""

import os
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTATIONS = {
    "entropy_in_bits": ("ksum_add(&h, -p * log_p)", "ksum_add(&h, -p * log_p / log(2.0))"),
    "entropy_sign": ("ksum_add(&h, -p * log_p)", "ksum_add(&h, p * log_p)"),
    "probability_unnormalised": ("const double p = e[v] / sum;", "const double p = e[v];"),
    "logp_vs_max_not_normaliser": ("logp[t] = (inv_temp * logit_at(z, dtype, ld, t, target[t]) - m) - log_s;",
                                   "logp[t] = (inv_temp * logit_at(z, dtype, ld, t, target[t]) - m);"),
    "target_gradient_sign": ("out[t * V + y] = inv_temp * g[t] * -expm1(logp[t]);",
                             "out[t * V + y] = inv_temp * g[t] * expm1(logp[t]);"),
    "step_mean_wrong_denominator": ("/ (double)(off[s + 1] - off[s]);",
                                    "/ (double)(off[s + 1] - off[s] + 1);"),
    "kept_count_floor": ("ceil(rho * (double)S - 1e-6)", "floor(rho * (double)S)"),
    "ties_to_higher_index": ("Hs32[o] == Hs32[s] && o < s", "Hs32[o] == Hs32[s] && o > s"),
    "selection_keeps_lowest": ("Hs32[o] > Hs32[s] ||", "Hs32[o] < Hs32[s] ||"),
    "ratio_inverted": ("exp(logp[t] - (double)lp_old[t])", "exp((double)lp_old[t] - logp[t])"),
    "tis_weight_dropped": ("                w = ratio_tis < C ? ratio_tis : C;",
                           "                w = 1.0;"),
    "tis_weight_uncapped": ("                w = ratio_tis < C ? ratio_tis : C;",
                            "                w = ratio_tis;"),
    "clip_bounds_swapped": ("if (rc < 1.0 - eps_low) rc = 1.0 - eps_low;",
                            "if (rc < 1.0 - eps_high) rc = 1.0 - eps_high;"),
    "loss_sign": ("const double lt = -M * om * (w * o - beta * klv);",
                  "const double lt = M * om * (w * o - beta * klv);"),
    "gradient_through_clip": ("const double d_obj = u <= c ? r * A * dlog : 0.0;",
                              "const double d_obj = r * A * dlog;"),
    "mean_over_all_tokens": ("        if (mask[s]) {\n            N += off[s + 1] - off[s];",
                             "        if (1) {\n            N += off[s + 1] - off[s];"),
    "dlogits_wrong_sign_softmax": ("out[t * V + v] = inv_temp * g[t] * (delta - p);",
                                   "out[t * V + v] = inv_temp * g[t] * (delta + p);"),
    "kl_k3_sign": ("return exp(delta) - delta - 1.0;", "return exp(delta) + delta - 1.0;"),
    "kl_k3_derivative": ("if (kl == KL_K3) return 1.0 - exp(delta);",
                         "if (kl == KL_K3) return exp(delta) - 1.0;"),
    "kl_inside_tis_weight": ("const double lt = -M * om * (w * o - beta * klv);",
                             "const double lt = -M * om * w * (o - beta * klv);"),
    "step_mean_weight": ("om = K > 0 ? 1.0 / ((double)K * (double)len) : 0.0;",
                         "om = K > 0 ? 1.0 / (double)K : 0.0;"),
    "token_mean_all_weight": ("if (agg == AGG_TOKEN_MEAN_ALL) om = 1.0 / (double)T;",
                              "if (agg == AGG_TOKEN_MEAN_ALL) om = 1.0 / (double)N;"),
    "geomean_derivative": ("dlog = ratio == RATIO_STEP_GEOMEAN ? 1.0 / (double)len : 1.0;",
                           "dlog = 1.0;"),
    "step_ratio_product_vs_mean": ("            if (ratio == RATIO_STEP_GEOMEAN) {\n                lr /= (double)len;",
                                   "            if (ratio == RATIO_STEP_PRODUCT) {\n                lr /= (double)len;"),
    "grpo_sample_variance": ("const double sd = count > 0 ? sqrt(ksum_value(&sq) / (double)count) : 0.0;",
                             "const double sd = count > 1 ? sqrt(ksum_value(&sq) / (double)(count - 1)) : 0.0;"),
    "grpo_weights_trajectories_not_steps": ("            for (int64_t s = traj_off[i]; s < traj_off[i + 1]; ++s) {\n                ksum_add(&sum, (double)reward[i]);",
                                            "            for (int64_t s = traj_off[i]; s < traj_off[i] + 1; ++s) {\n                ksum_add(&sum, (double)reward[i]);"),
    "grpo_no_centering": ("const double a = sd > 0.0 ? ((double)reward[i] - mean) / sd : 0.0;",
                          "const double a = sd > 0.0 ? (double)reward[i] / sd : 0.0;"),
    "temperature_not_in_gradient": ("out[t * V + v] = inv_temp * g[t] * (delta - p);",
                                    "out[t * V + v] = g[t] * (delta - p);"),
    "temperature_not_in_logp": ("logp[t] = (inv_temp * logit_at(z, dtype, ld, t, target[t]) - m) - log_s;",
                                "logp[t] = (logit_at(z, dtype, ld, t, target[t]) - m) - log_s;"),
    "dlogits_wrong_target": ("const double delta = v == target[t] ? 1.0 : 0.0;",
                             "const double delta = v == (target[t] + 1) % V ? 1.0 : 0.0;"),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(name, tmp_path):
    old, new = MUTATIONS[name]
    with open(oracle.SRC) as fh:
        src = fh.read()
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    mutated = tmp_path / "mutated.c"
    mutated.write_text(src.replace(old, new))
    lib = tmp_path / "liboracle_mut.so"
    oracle.build(src=str(mutated), out=str(lib))
    env = dict(os.environ, ORACLE_LIB=str(lib))
    proc = subprocess.run(
        [sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
         os.path.join(ROOT, "tests", "test_oracle_pins.py"),
         os.path.join(ROOT, "tests", "test_oracle_ext_pins.py"),
         os.path.join(ROOT, "tests", "test_oracle_grpo_pins.py"), "-k", "not mini"],
        cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert proc.returncode != 0, f"mutation {name} survived the pins:\n{proc.stdout[-2000:]}"
