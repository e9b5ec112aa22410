"""Planted mistakes in the oracle must fail its pins.

Each case copies the oracle's C source, applies one plausible mistake (a wrong
sign, a dropped term, a transposed operand, a wrong tie-break ...), builds it
into a temporary library and runs the pin tests against that library in a
subprocess. Every mutant must make at least one pin fail. Nothing here touches
a GPU.
"""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "moe_oracle.c")

MUTANTS = {
    "sigmoid_sign": ("float z = -s;", "float z = s;"),
    "drop_ln2_lo": ("r = fmaf(-n, S_LN2_LO, r);", "r = r;"),
    "taylor_coeff": ("p = fmaf(p, r, c4);", "p = fmaf(p, r, c5);"),
    "upper_clamp_missing": ("if (z > 87.0f) z = 87.0f;", ";"),
    "bias_in_gate": ("gate[j] = sig[idx[j]] / den;",
                     "gate[j] = (sig[idx[j]] + (bias ? bias[idx[j]] : 0.0f)) / den;"),
    "gate_den_drops_first": ("float den = sig[idx[0]];", "float den = 0.0f;"),
    "tie_to_higher_index": ("key > best_key", "key >= best_key"),
    "logit_reversed_order": ("for (int i = 0; i < d; ++i) s = fmaf(x[i], w[i], s);",
                             "for (int i = d - 1; i >= 0; --i) s = fmaf(x[i], w[i], s);"),
    "logit_unfused": ("s = fmaf(x[i], w[i], s);", "s = x[i] * w[i] + s;"),
    "logit_wrong_index": ("s = fmaf(x[i], w[i], s);", "s = fmaf(x[i], w[d - 1 - i], s);"),
    "permute_unstable": ("for (size_t n = 0; n < n_slots; ++n) sorted_slots",
                         "for (size_t n = n_slots; n-- > 0;) sorted_slots"),
    "gelu_wrong_scale": ("erf(v * 0.70710678118654752440)", "erf(v)"),
    "w1_transposed": ("a += (double)w[i] * (double)x[i];",
                      "a += (double)w1[(size_t)i * h + k] * (double)x[i];"),
    "w2_transposed": ("o += (double)w[k] * hid[k];", "o += (double)w2[(size_t)k * d + c] * hid[k];"),
    "act_not_rounded": ("hid[k] = act_bf16 ? oracle_round_bf16(a) : a;", "hid[k] = a;"),
    "round_ties_away": ("double q = nearbyint(ldexp(m, 8));", "double q = round(ldexp(m, 8));"),
    "shared_dropped": ("y[c] += (double)lambda * o[c];", "y[c] += 0.0 * o[c];"),
    "combine_ignores_lambda": ("if (shared) acc += lambda * shared[(size_t)t * d + c];",
                               "if (shared) acc += shared[(size_t)t * d + c];"),
    "bias_sign_flipped": ("if (scaled > total) bias[e] = bias[e] - alpha;",
                          "if (scaled > total) bias[e] = bias[e] + alpha;"),
    "bias_sign_zero_moves": ("else if (scaled < total) bias[e] = bias[e] + alpha;",
                             "else bias[e] = bias[e] + alpha;"),
    "zscore_sample_deviation": ("var = var / (double)E;", "var = var / (double)(E - 1);"),
    "zscore_no_mean": ("double dev = (double)counts[e] - mu;", "double dev = (double)counts[e];"),
    "zscore_wrong_direction": ("bias[e] = (float)((double)bias[e] - step);",
                               "bias[e] = (float)((double)bias[e] + step);"),
    "silu_wrong_sign": ("return v / (1.0 + exp(-v));", "return v / (1.0 + exp(v));"),
    "swiglu_gate_up_swapped": ("a = oracle_silu(a) * up;", "a = oracle_silu(up) * a;"),
    "swiglu_up_reads_gate_rows": ("const float *wu = w1 + ((size_t)h + k) * d;", "const float *wu = w1 + (size_t)k * d;"),
    "swiglu_expert_stride": ("const size_t w1_rows = swiglu ? 2 * (size_t)h : (size_t)h;",
                             "const size_t w1_rows = (size_t)h;"),
    "gelu_grad_drops_density": ("+ v * exp(-0.5 * v * v) * 0.39894228040143267794", ""),
    "bwd_w2_not_transposed": ("acc += (double)w2[(size_t)c * h + k] * (double)g[c];",
                              "acc += (double)w2[(size_t)k * d + c] * (double)g[c];"),
    "bwd_dw2_uses_preactivation": ("act[(size_t)r * h + k] = act_bf16 ? oracle_round_bf16(a) : a;",
                                   "act[(size_t)r * h + k] = act_bf16 ? oracle_round_bf16(p) : p;"),
    "bwd_dp_not_rounded": ("dpre[(size_t)r * hr + k] = act_bf16 ? oracle_round_bf16(dp) : dp;",
                           "dpre[(size_t)r * hr + k] = dp;"),
    "bwd_swiglu_dq_wrong": ("dq = da[k] * oracle_silu(p);", "dq = da[k] * p;"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    before, after = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(before) >= 1, f"mutation site for {name} not found"
    mutated = src.replace(before, after)
    c_path = tmp_path / "mutant.c"
    so_path = tmp_path / "libmutant.so"
    c_path.write_text(mutated)
    sys.path.insert(0, ROOT)
    from oracle.oracle import CFLAGS

    subprocess.run(["gcc", *CFLAGS, "-w", str(c_path), "-o", str(so_path), "-lm"], check=True)
    env = dict(os.environ, MOE_ORACLE_LIB=str(so_path), OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode != 0, f"mutant {name} passed every pin:\n{r.stdout[-2000:]}"
