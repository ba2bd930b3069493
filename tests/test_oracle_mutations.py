"""The pins must catch plausible mistakes in the oracle.

Each case plants one mistake in a copy of the oracle's C source (on the CPU,
in a temporary directory), builds it, and runs the pin suite against it: the
suite must fail.  The unmodified source must pass.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "flexmoe_oracle.c")

MUTANTS = {
    "silu_dropped": ("h[c] = g / (1.0 + exp(-(double)g)) * u;", "h[c] = g * u;"),
    "silu_sign": ("h[c] = g / (1.0 + exp(-(double)g)) * u;", "h[c] = g / (1.0 + exp((double)g)) * u;"),
    "tie_break_reversed": ("    return ia < ib;\n}", "    return ia > ib;\n}"),
    "norm_flag_inverted": ("if (norm_topk)", "if (!norm_topk)"),
    "down_transposed": ("acc += (acc_t)h[c] * (acc_t)elem(wd, dtype, wd_off + (size_t)n * ld_down + c);",
                        "acc += (acc_t)h[c] * (acc_t)elem(wd, dtype, wd_off + (size_t)c * d + n);"),
    "dispatch_unstable": ("int32_t p = offsets[e] + fill[e]++;",
                          "int32_t p = offsets[e + 1] - 1 - fill[e]++;"),
    "zero_expert_not_skipped": ("offsets[e] + (keep[e] > 0 ? counts[e] : 0)",
                                "offsets[e] + counts[e]"),
    "softmax_unshifted": ("w[(size_t)t * k + j] = exp((double)l[e] - m) / z;",
                          "w[(size_t)t * k + j] = exp((double)l[e]) / z;"),
    "reorder_down_unpermuted": ("((size_t)e * d + n) * I + pi[c]);", "((size_t)e * d + n) * I + c);"),
    "ratio_floor": ("double k = ceil(r * (double)I - 1e-9);", "double k = floor(r * (double)I + 1e-9);"),
    "shared_half_weight": ("yt[n] += s[n];", "yt[n] += 0.5 * s[n];"),
    "router_weight_dropped": ("yt[n] += wt * O[(size_t)p * d + n];", "yt[n] += O[(size_t)p * d + n];"),
    "grad_dsilu_term_dropped": ("dsilu = sg * (1.0 + g[c] * (1.0 - sg));", "dsilu = sg;"),
    "grad_router_weight_dropped": ("dO[n] = w[a] * y[xo + n];", "dO[n] = y[xo + n];"),
    "grad_down_uses_preactivation": ("g_down[wb + (size_t)n * I + c] += dO[n] * h;",
                                     "g_down[wb + (size_t)n * I + c] += dO[n] * silu;"),
    "grad_up_gets_gate_term": ("g_up[wb + (size_t)c * d + i] += du * xi;",
                               "g_up[wb + (size_t)c * d + i] += dg * xi;"),
    "saliency_down_not_squared": ("acc += td * td;", "acc += fabs(td);"),
    "saliency_gate_term_dropped": ("acc += tg * tg + tu * tu;", "acc += tu * tu;"),
    "dmask_only_kept_channels": ("dmask[(size_t)e * I + c] += dh * silu * u[c];",
                                 "if (c < kk) dmask[(size_t)e * I + c] += dh * silu * u[c];"),
    "router_grad_ignores_renorm": ("double g = norm_topk ? (dw[(size_t)t * k + j] - dwsum) / S : dw[(size_t)t * k + j];",
                                   "double g = dw[(size_t)t * k + j];"),
    "st_gradient_without_tau": ("double g_quality = z[kk] * (dz[kk] - zdz) / tau;",
                                "double g_quality = z[kk] * (dz[kk] - zdz);"),
    "entropy_gradient_sign": ("double g_ent = p[kk] > 0.0 ? -p[kk] * (log(p[kk]) + He) / E : 0.0;",
                              "double g_ent = p[kk] > 0.0 ? p[kk] * (log(p[kk]) + He) / E : 0.0;"),
    "cost_not_load_weighted": ("double q = (double)counts[e] / (double)assignments;", "double q = 1.0;"),
    "sample_tie_takes_last": ("if (a[k] + g[k] > a[best] + g[best])", "if (a[k] + g[k] >= a[best] + g[best])"),
    "shared_input_grad_dropped": ("                    dxt[i] += dg * elem(ws_gate, dtype, (size_t)c * d + i) +\n"
                                  "                              du * elem(ws_up, dtype, (size_t)c * d + i);",
                                  "                    dxt[i] += 0.0 * dg * elem(ws_gate, dtype, (size_t)c * d + i);"),
    "prefix_short_by_one": ("    for (int c = 0; c < kk; ++c) {\n        acc_t g = 0, u = 0;",
                            "    for (int c = 0; c < kk; ++c) {\n        if (c == kk - 1 && kk > 1) { h[c] = 0; continue; }\n        acc_t g = 0, u = 0;"),
}


def _run_pins(lib_path):
    # small pin cases: one OpenMP thread per run (parallel test workers would oversubscribe)
    env = dict(os.environ, FLEXMOE_ORACLE_LIB=lib_path, OMP_NUM_THREADS="1")
    return subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                           os.path.join(ROOT, "tests", "test_oracle_pins.py"),
                           os.path.join(ROOT, "tests", "test_saliency_pins.py"),
                           os.path.join(ROOT, "tests", "test_action_pins.py")],
                          cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)


def _build(src_text, tmp_path, name):
    c = tmp_path / (name + ".c")
    so = tmp_path / (name + ".so")
    c.write_text(src_text)
    subprocess.run(["gcc", "-O1", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-o", str(so),
                    str(c), "-lm"], check=True)
    return str(so)


def test_unmodified_oracle_passes(tmp_path):
    so = _build(open(SRC).read(), tmp_path, "clean")
    r = _run_pins(so)
    assert r.returncode == 0, r.stdout[-2000:]


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) >= 1, "mutation anchor not found: %s" % name
    so = _build(src.replace(old, new, 1), tmp_path, name)
    r = _run_pins(so)
    assert r.returncode != 0, "pins did not catch mutant %s" % name
