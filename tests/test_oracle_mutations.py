"""The oracle pins catch plausible mistakes.

Each case plants one mistake in a copy of the oracle's C source (on the CPU),
builds it, and runs the pin suite against that build: the suite must fail.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "vp_oracle.c")

MUTANTS = {
    "tanh_sigmoid_swapped": ("a += (double)wh[l] * tanh(x) * sigmoid(y);",
                             "a += (double)wh[l] * sigmoid(x) * tanh(y);"),
    "gate_weight_dropped": ("a += (double)wh[l] * tanh(x) * sigmoid(y);",
                            "a += tanh(x) * sigmoid(y);"),
    "U_replaced_by_W": ("y += (double)Uh[l * c->d + k] * (double)q[k];",
                        "y += (double)Wh[l * c->d + k] * (double)q[k];"),
    "router_scale_dropped": ("t[j] = c->scale * dot;", "t[j] = dot;"),
    "saliency_not_max": ("if (r > smax) smax = r;", "smax += r / (double)N;"),
    "mean_wrong_count": ("mean[e] /= (double)N;", "mean[e] /= (double)(N - 1 > 0 ? N - 1 : 1);"),
    "attn_scale_dropped": ("l[j] = dot * c->scale;", "l[j] = dot;"),
    "attn_not_normalised": ("for (int e = 0; e < d; ++e) y[e] /= sum;", "(void)sum;"),
    "attn_wrong_head_keys": ("const float *k = c->K + (j * H + h) * (int64_t)d;\n            double dot = 0.0;\n            for (int e = 0; e < d; ++e) dot += (double)q[e]",
                             "const float *k = c->K + (j * H + (h + 1) % H) * (int64_t)d;\n            double dot = 0.0;\n            for (int e = 0; e < d; ++e) dot += (double)q[e]"),
    "concat_order_swapped": ("z[e] = (double)v[e];\n            z[d + e] = c->C[e];",
                             "z[d + e] = (double)v[e];\n            z[e] = c->C[e];"),
    "gate_sigmoid_dropped": ("y[e] = c->C[e] + sigmoid(g[e]) * dl[e];", "y[e] = c->C[e] + g[e] * dl[e];"),
    "context_residual_dropped": ("y[e] = c->C[e] + sigmoid(g[e]) * dl[e];", "y[e] = sigmoid(g[e]) * dl[e];"),
    "gelu_tanh_form": ("return 0.5 * x * (1.0 + erf(x / sqrt(2.0)));",
                       "return 0.5 * x * (1.0 + tanh(0.7978845608 * (x + 0.044715 * x * x * x)));"),
    "tau_high_exclusive": ("s >= (double)tau_high", "s > (double)tau_high"),
    "tau_low_exclusive": ("s <= (double)tau_low", "s < (double)tau_low"),
    "argmax_last_tie": ("if (lg[m] > lg[best]) best = m;", "if (lg[m] >= lg[best]) best = m;"),
    "logit_bias_dropped": ("logits[r] = acc + (double)br[r];", "logits[r] = acc;"),
    "binary_keeps_surr": ("else if (rule == 2 || s <= (double)tau_low)", "else if (s <= (double)tau_low)"),
    "binary_tie_to_full": ("modes[h] = full_l > mean_l ? OR_MODE_FULL : OR_MODE_MEAN;",
                           "modes[h] = full_l >= mean_l ? OR_MODE_FULL : OR_MODE_MEAN;"),
    "no_residual_keeps_correction": ("if (c->variant == 2) {", "if (c->variant == 99) {"),
    "identity_not_added": ("if (c->variant == 3) y[e] += z[e];", "if (c->variant == 3) y[e] += 0.0;"),
    "linattn_phi_no_shift": ("return x > 0.0 ? x + 1.0 : exp(x);", "return x > 0.0 ? x : exp(x);"),
    "linattn_not_normalised": ("for (int e = 0; e < d; ++e) y[e] = acc[e] / den;",
                               "for (int e = 0; e < d; ++e) y[e] = acc[e] / (double)c->N;"),
    # dense block around the layer (pins in test_oracle_block_pins.py)
    "ln_unbiased_variance": ("        var /= c->D;", "        var /= (c->D - 1);", "block"),
    "ln_eps_outside_sqrt": ("const double r = 1.0 / sqrt(var + c->eps);",
                            "const double r = 1.0 / (sqrt(var) + c->eps);", "block"),
    "ln_bias_dropped": ("* (double)c->g[k] + (double)c->b[k];", "* (double)c->g[k];", "block"),
    "rope_sign_flipped": ("t[j] = u * cos(a) - w * sin(a);", "t[j] = u * cos(a) + w * sin(a);",
                          "block"),
    "rope_adjacent_pairs": ("const double u = t[j], w = t[j + q];",
                            "const double u = t[2 * j], w = t[2 * j + 1];", "block"),
    "rope_halves_same_coordinate": ("const double coord = (double)c->pos[2 * i + half];",
                                    "const double coord = (double)c->pos[2 * i];", "block"),
    "rope_frequency_exponent": ("pow(c->base, -2.0 * j / (double)m)", "pow(c->base, -1.0 * j / (double)m)",
                                "block"),
    "block_gelu_tanh_form": ("X[i] = 0.5 * X[i] * (1.0 + erf(X[i] / sqrt(2.0)));",
                             "X[i] = 0.5 * X[i] * (1.0 + tanh(0.7978845608 * (X[i] + 0.044715 * X[i] * X[i] * X[i])));",
                             "block"),
    # distillation targets (pins in test_oracle_distill_pins.py)
    "colmax_key_stat": ("const double a = exp(qk_dot(c, q, k) - c->m[q]) / c->s[q];",
                        "const double a = exp(qk_dot(c, q, k) - c->m[k]) / c->s[k];", "distill"),
    "colmax_unnormalised": ("const double a = exp(qk_dot(c, q, k) - c->m[q]) / c->s[q];",
                            "const double a = exp(qk_dot(c, q, k) - c->m[q]);", "distill"),
    "colmax_scale_dropped": ("    return dot * c->scale;\n}", "    return dot;\n}", "distill"),
    "colmax_sum_not_max": ("            if (a > best) best = a;", "            best += a / (double)c->N;",
                           "distill"),
    # token merging (pins in test_oracle_tome_pins.py)
    "tome_metric_one_head": ("for (int h = 0; h < H; ++h) s += K[(i * H + h) * (int64_t)d + e];",
                             "for (int h = 0; h < 1; ++h) s += K[(i * H + h) * (int64_t)d + e];",
                             "tome"),
    "tome_metric_truncated": ("u += 0x7fffu + ((u >> 16) & 1u);", "u += 0u;", "tome"),
    "tome_stride_not_smallest": ("if ((S - 1) * (np - ndst) >= M) break;",
                                 "if ((S - 1) * (np - ndst) > M) break;", "tome"),
    "tome_view0_merged": ("(uint8_t)(v == 0 || k < 0 || k % g == 0)", "(uint8_t)(k < 0 || k % g == 0)",
                          "tome"),
    "tome_dot_not_cosine": ("dot / (na * c->dnorm[j]);", "dot / na;", "tome"),
    "tome_match_last_tie": ("if (best < 0 || cs > bs) {", "if (best < 0 || cs >= bs) {", "tome"),
    "tome_select_least_similar": ("if (a->score > b->score) return -1;\n    if (a->score < b->score) return 1;",
                                  "if (a->score > b->score) return 1;\n    if (a->score < b->score) return -1;",
                                  "tome"),
    "tome_select_tie_high_index": ("return a->tok < b->tok ? -1 : (a->tok > b->tok ? 1 : 0);",
                                   "return a->tok > b->tok ? -1 : (a->tok < b->tok ? 1 : 0);", "tome"),
    "tome_merge_sum_not_mean": ("Xm[r * F + f] /= (double)cnt[r];", "Xm[r * F + f] /= 1.0;", "tome"),
    "tome_rows_count_merged": ("if (into[t] < 0) row[t] = r++;", "row[t] = r++;", "tome"),
}
PIN_FILES = {"layer": "test_oracle_pins.py", "block": "test_oracle_block_pins.py",
             "distill": "test_oracle_distill_pins.py", "tome": "test_oracle_tome_pins.py"}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name, tmp_path):
    old, new = MUTANTS[name][:2]
    pins = PIN_FILES[MUTANTS[name][2] if len(MUTANTS[name]) > 2 else "layer"]
    src = open(SRC).read()
    assert src.count(old) == 1, "mutation anchor not found once: " + name
    msrc = tmp_path / "mutant.c"
    msrc.write_text(src.replace(old, new))
    lib = tmp_path / "libmutant.so"
    subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-std=c11", "-o", str(lib),
                           str(msrc), "-lm", "-lpthread"])
    env = dict(os.environ, VP_ORACLE_LIB=str(lib))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", pins)],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, "pins did not catch mutant %s:\n%s" % (name, r.stdout[-2000:])
