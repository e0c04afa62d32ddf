"""The oracle's pins must catch plausible mistakes.

Each case plants one mistake in a copy of oracle.c or head.py (a dropped term, a wrong
sign, a swapped index, a transposed operand, a wrong rounding), builds it into
a temporary directory and runs the pin file that should notice; the pins must
fail. Runs on the CPU only; the real oracle is never modified.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTATIONS = {
    "combine_sum_for_mul": ("gather", "? qrow[c] * rrow[c] : qrow[c] + rrow[c]",
                            "? qrow[c] + rrow[c] : qrow[c] + rrow[c]"),
    "pool_seeded_with_zero": ("gather", "acc[c] = started ? acc[c] + e : e;",
                              "acc[c] = (started ? acc[c] : 0.0f) + e;"),
    "rounding_ties_away": ("gather", "u = (u + 0x7fffu + keep_lsb) & 0xffff0000u;",
                           "u = (u + 0x8000u) & 0xffff0000u;"),
    "quotient_remainder_swapped": ("gather", "int64_t q = id / m;\n                int64_t r = id - q * m;\n"
                                   "                if (q >= rows_q) {\n                    ++bad;",
                                   "int64_t r = id / m;\n                int64_t q = id - r * m;\n"
                                   "                if (q >= rows_q) {\n                    ++bad;"),
    "temperature_inverted": ("dcn", "row[j] = q[i] * k[j] / tau;", "row[j] = q[i] * k[j] * tau;"),
    "softmax_over_queries": ("dcn", "row[j] = q[i] * k[j] / tau;", "row[j] = q[j] * k[i] / tau;"),
    "skip_dropped": ("dcn", "h[i] = beta * v[i] + alpha * oi;", "h[i] = alpha * oi;"),
    "up_projection_transposed": ("dcn", "for (int64_t i = 0; i < hr; ++i) s += U[c * hr + i] * h[i];",
                                 "for (int64_t i = 0; i < hr; ++i) s += U[(i * d + c) % (d * hr)] * h[i];"),
    "bias_dropped": ("dcn", "double s = bl[c];", "double s = 0.0;"),
    "residual_dropped": ("dcn", "xn[c] = x0[c] * s + xl[c];", "xn[c] = x0[c] * s;"),
    "multiplier_x_l_not_x0": ("dcn", "xn[c] = x0[c] * s + xl[c];", "xn[c] = xl[c] * s + xl[c];"),
    "bwd_x0_term_dropped": ("grad", "gx0[c] += g[c] * t[c];", "gx0[c] += 0.0;"),
    "bwd_score_sign": ("grad", "* (v[j] - o[i]);", "* (o[i] - v[j]);"),
    "bwd_key_temperature": ("grad", "dk[j] = s / tau;", "dk[j] = s;"),
    "bwd_value_skip_dropped": ("grad", "dv[j] = beta * dha[j] + s;", "dv[j] = s;"),
    "bwd_final_input_term_dropped": ("grad", "grad_x0[b * d + c] = gx0[c] + g[c];", "grad_x0[b * d + c] = gx0[c];"),
    "emb_product_rule_wrong_row": ("grad", "gq[c] += g[c] * (double)rrow[c];", "gq[c] += g[c] * (double)qrow[c];"),
    "quant_middle_weights_swapped": ("quant", "(mx * 128.0f + mn * 127.0f) / 255.0f", "(mx * 127.0f + mn * 128.0f) / 255.0f"),
    "quant_scale_over_256": ("quant", "(mx - mn) / 255.0f", "(mx - mn) / 256.0f"),
    "quant_truncating_round": ("quant", "q = rintf((row[c] - middle) / scale);", "q = truncf((row[c] - middle) / scale);"),
    "quant_ties_away": ("quant", "q = rintf((row[c] - middle) / scale);", "q = roundf((row[c] - middle) / scale);"),
    "quant_dequant_minus": ("quant", "fmaf((float)codes[i * D + c], params[2 * i + 1], params[2 * i])",
                            "fmaf((float)codes[i * D + c], -params[2 * i + 1], params[2 * i])"),
    "quant_dequant_two_roundings": ("quant", "fmaf((float)codes[i * D + c], params[2 * i + 1], params[2 * i])",
                                    "(float)codes[i * D + c] * params[2 * i + 1] + params[2 * i]"),
    "par_plain_grad_dropped": ("parallel", "for (int64_t i = 0; i < r; ++i) dP[i] = dh[i];",
                               "for (int64_t i = 0; i < r; ++i) dP[i] = 0.0;"),
    "par_attention_reads_plain_rows": ("parallel", "const double* Wa = par ? W + r * d : W;", "const double* Wa = W;"),
    "par_plain_branch_scaled_by_skip": ("parallel", "                h[i] = s;\n            }\n        }",
                                        "                h[i] = beta * s;\n            }\n        }"),
    "hash_shift_46": ("hash", "const int r = 47;", "const int r = 46;"),
    "hash_final_mix_dropped": ("hash", "    h ^= h >> r;\n    h *= m;\n    h ^= h >> r;\n    return h;",
                               "    h ^= h >> r;\n    h *= m;\n    return h;"),
    "hash_big_endian_blocks": ("hash", "for (int b = 7; b >= 0; --b) k = (k << 8) | p[8 * i + b];",
                               "for (int b = 0; b < 8; ++b) k = (k << 8) | p[8 * i + b];"),
    "hash_halves_swapped": ("hash", "const uint64_t half[2] = {hsh & 0xffffffffull, hsh >> 32};",
                            "const uint64_t half[2] = {hsh >> 32, hsh & 0xffffffffull};"),
    "hash_bwd_other_row": ("hash", "                            gq[c] += g[c] * (double)rrow[c];\n"
                           "                            gr[c] += g[c] * (double)qrow[c];\n                        } else {\n"
                           "                            gq[c] += g[c];\n                            gr[c] += g[c];\n"
                           "                        }\n                    }\n                }",
                           "                            gq[c] += g[c] * (double)qrow[c];\n"
                           "                            gr[c] += g[c] * (double)qrow[c];\n                        } else {\n"
                           "                            gq[c] += g[c];\n                            gr[c] += g[c];\n"
                           "                        }\n                    }\n                }"),
    "head_gate_derivative_missing_one_minus": ("head", "g_s = g_rho * rho * (1.0 - rho)", "g_s = g_rho * rho", "head.py"),
    "head_gate_input_gradient_dropped": ("head", "ga = ga + np.outer(g_s, Gl)", "ga = ga", "head.py"),
    "head_relu_gradient_ungated": ("head", "g_z = g_relu * (z > 0.0)", "g_z = ga * (z > 0.0)", "head.py"),
    "head_bias_gradient_before_mask": ("head", "gb[l] = g_z.sum(axis=0)", "gb[l] = g_relu.sum(axis=0)", "head.py"),
    "head_bucket_remainder_off_by_one": ("head", "v[here, i] = t[here] - step * k[here]",
                                         "v[here, i] = t[here] - step * (k[here] + 1)", "head.py"),
    "head_bucket_bound_inclusive": ("head", "k += (t32 > bound).astype(np.int64)",
                                    "k += (t32 >= bound).astype(np.int64)", "head.py"),
    "head_slope_ignores_embedding": ("head", "np.sum(np.maximum(e + w, 0.0) * v, axis=1)",
                                     "np.sum(np.maximum(w, 0.0) * v, axis=1)", "head.py"),
    "head_logit_gradient_next_bucket": ("head", "np.maximum(pre[rows, k], 0.0)",
                                        "np.maximum(pre[rows, np.minimum(k + 1, K - 1)], 0.0)", "head.py"),
    "head_logloss_sign": ("head", "return softplus(y_cal) - label * y_cal, sigmoid(y_cal) - label",
                          "return softplus(y_cal) - label * y_cal, label - sigmoid(y_cal)", "head.py"),
    "head_output_weight_gradient_uncalibrated": ("head", "g_wout = g_y @ aL", "g_wout = np.asarray(g_cal) @ aL",
                                                 "head.py"),
}
PIN_FILE = {"gather": "test_oracle_gather.py", "dcn": "test_oracle_dcn.py", "grad": "test_oracle_grad.py",
            "quant": "test_oracle_quant.py", "parallel": "test_oracle_parallel.py", "hash": "test_oracle_hash.py",
            "head": "test_oracle_head.py"}


@pytest.mark.parametrize("name", list(MUTATIONS))
def test_pins_catch_planted_mistake(name, tmp_path):
    which, old, new = MUTATIONS[name][:3]
    fname = MUTATIONS[name][3] if len(MUTATIONS[name]) > 3 else "oracle.c"
    src = open(os.path.join(ROOT, "oracle", fname)).read()
    assert src.count(old) >= 1, "mutation anchor not found: " + name
    for sub in ("oracle", "tests", "paper_2402_06859_amd"):
        shutil.copytree(os.path.join(ROOT, sub), tmp_path / sub,
                        ignore=shutil.ignore_patterns("*.so", "__pycache__", "_build*"))
    (tmp_path / "oracle" / fname).write_text(src.replace(old, new, 1))
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join("tests", PIN_FILE[which])], cwd=tmp_path, capture_output=True, text=True)
    assert r.returncode == 1, "planted mistake %r was not caught:\n%s" % (name, r.stdout[-2000:])
