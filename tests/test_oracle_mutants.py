"""Mistakes planted in a copy of the oracle must each fail at least one pin.

Each mutant is a plausible slip (a dropped term, a wrong index or sign, a transposed head
mapping).  The copy is compiled on the CPU and the pin suite is run against it with the
VXO_LIB hook; the pins must catch every mutant.  The committed oracle is never modified.
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "vxo.c")

MUTANTS = {
    "mean_divides_by_page_size": ("mean[o] = s / n;", "mean[o] = s / ps;"),
    "quest_takes_min_of_pair": ("acc += (a > b ? a : b);", "acc += (a < b ? a : b);"),
    "quest_sums_heads": ("if (acc > s) s = acc;", "s = (s == -INFINITY ? 0 : s) + acc;"),
    "block_score_drops_head_mean": ("s = total / g;", "s = total;"),
    "gqa_heads_interleaved": ("const uint16_t *qr = q + ((int64_t)i * Hq + r) * Dqk;",
                              "const uint16_t *qr = q + ((int64_t)i * Hq + (r % g) * H + h) * Dqk;"),
    "ties_to_higher_index": ("return (x->j > y->j) - (x->j < y->j);", "return (x->j < y->j) - (x->j > y->j);"),
    "softmax_scale_dropped": ("z[t] = sm_scale * dot;", "z[t] = dot;"),
    "partial_page_read_whole": ("return n < ps ? n : ps;", "return ps;"),
    "local_window_off_by_one": ("if (j < n_sink || j >= P - n_local)", "if (j < n_sink || j > P - n_local)"),
    "aliased_v_wrong_stride": ("row_v[t_all] = v ? (((p * H) + h) * ps + t) * Dv : row_k[t_all];",
                               "row_v[t_all] = (((p * H) + h) * ps + t) * Dv;"),
    "score_uses_wrong_kv_head": ("const double *S = sa + (p * H + h) * D;",
                                 "const double *S = sa + (p * H + (H - 1 - h)) * D;"),
    "approx_stop_rule_inverted": ("(int64_t)c * 65536 >= (65536 - tau_q) * Kfree",
                                  "(int64_t)c * 65536 >= tau_q * Kfree"),
    "approx_stop_rule_strict": ("(int64_t)c * 65536 >= (65536 - tau_q) * Kfree",
                                "(int64_t)c * 65536 > (65536 - tau_q) * Kfree"),
    "approx_remap_reversed": ("(uint32_t)floor(((double)x - mn) * scale)",
                              "(uint32_t)floor((mx - (double)x) * scale)"),
    "approx_first_pass_seven_bits": ("int b = t0 >= 7 ? t0 - 7 : 0;", "int b = t0 >= 6 ? t0 - 6 : 0;"),
    "approx_stops_one_pass_late": ("{ early = 1; break; }",
                                   "{ early = 1; if (b >= 8) { b -= 8; M = 0xffffffffu << b; } break; }"),
    "approx_samples_on_exact_end": ("if (n == Kfree - c || b == 0) break;",
                                    "if (n == Kfree - c || b == 0) { early = 1; break; }"),
    "approx_sample_ascending_hash": ("bin[nb].v = early ? lowbias32(z ^ (uint32_t)kl[m].j) >> 24 : 0u;",
                                     "bin[nb].v = early ? 255u - (lowbias32(z ^ (uint32_t)kl[m].j) >> 24) : 0u;"),
    "approx_sample_in_page_order": ("bin[nb].v = early ? lowbias32(z ^ (uint32_t)kl[m].j) >> 24 : 0u;",
                                    "bin[nb].v = 0u;"),
    "approx_bin_ties_to_higher_page": ("return x->j < y->j ? -1 : (x->j > y->j);",
                                       "return x->j > y->j ? -1 : (x->j < y->j);"),
    "approx_sample_unit_of_wrong_layout": ("lowbias32(seed ^ lowbias32((uint32_t)(i * H + h)))",
                                           "lowbias32(seed ^ lowbias32((uint32_t)(h * batch + i)))"),
    "fp8_e4m3_bias_off_by_one": ("v = e ? ldexp(1.0 + m / 8.0, e - 7) : ldexp(m / 8.0, -6);",
                                 "v = e ? ldexp(1.0 + m / 8.0, e - 8) : ldexp(m / 8.0, -6);"),
    "fp8_e5m2_subnormal_exponent": ("ldexp(m / 4.0, -14)", "ldexp(m / 4.0, -15)"),
    "fp8_scale_product_unrounded": ("float x = scale * (float)fp8_code_value(c, fmt);",
                                    "double x = (double)scale * fp8_code_value(c, fmt);"),
    "v_dequantised_with_k_scale": ("const float vs = v ? v_scale : k_scale;", "const float vs = k_scale;"),
    "aliased_v_takes_the_v_scale": ("const float vs = v ? v_scale : k_scale;", "const float vs = v_scale;"),
    "summary_max_not_rounded_to_bf16": ("if (maxv) maxv[o] = to_bf16_rne(mx);", "if (maxv) maxv[o] = mx;"),
    "consensus_takes_max_over_heads": ("            if (acc < s) s = acc;", "            if (acc > s) s = acc;"),
    "pessimistic_takes_max_per_channel": ("acc += kind == VXO_ENVELOPE_LOWER ? (a < b ? a : b) : (a > b ? a : b);",
                                          "acc += (a > b ? a : b);"),
    "rectified_drops_relu": ("acc += a > 0.0 ? a : 0.0;", "acc += a;"),
    "append_slot_off_by_one": ("int j = t / ps, slot = t % ps;", "int j = t / ps, slot = (t + 1) % ps;"),
    "append_rows_of_wrong_head": ("(const char *)k_new + (((int64_t)i * H + h) * Dqk) * esz",
                                  "(const char *)k_new + (((int64_t)i * H + (H - 1 - h)) * Dqk) * esz"),
    "content_score_reads_rope_channels": ("int nch = kind == VXO_MEAN_DOT_CONTENT ? Dc : D;", "int nch = D;"),
    "conv_kernel_reversed": ("y[j] = w[0] * left + w[1] * x[j] + w[2] * right;",
                             "y[j] = w[2] * left + w[1] * x[j] + w[0] * right;"),
    "conv_replicate_padding": ("double left = j > 0 ? x[j - 1] : 0.0;", "double left = j > 0 ? x[j - 1] : x[j];"),
    "nsa_softmax_not_normalised": ("for (int j = 0; j < P; j++) prob[j] /= l;", ""),
    "nsa_logits_not_rounded_to_fp32": ("] = (double)(float)dot;", "] = dot;"),
    "nsa_logits_wrong_kv_head": ("const double *S = mean + (p * H + r / g) * D;",
                                 "const double *S = mean + (p * H + r % H) * D;"),
}


def _run_mutant(name, tmp):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, name
    d = os.path.join(tmp, name)
    os.makedirs(d, exist_ok=True)
    c = os.path.join(d, "vxo.c")
    open(c, "w").write(src.replace(old, new))
    import shutil
    shutil.copy(os.path.join(ROOT, "oracle", "vxo.h"), d)
    lib = os.path.join(d, "libvxo.so")
    subprocess.check_call(["gcc", "-O1", "-std=gnu11", "-fopenmp", "-fPIC", "-shared", "-o", lib, c, "-lm"])
    env = dict(os.environ, VXO_LIB=lib, OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    return name, r.returncode, r.stdout[-400:]


def test_every_mutant_fails_a_pin(tmp_path):
    with ThreadPoolExecutor(max_workers=4) as ex:
        results = list(ex.map(lambda n: _run_mutant(n, str(tmp_path)), sorted(MUTANTS)))
    survivors = [(n, out) for n, rc, out in results if rc == 0]
    assert not survivors, f"mutants not caught by any pin: {survivors}"
    for n, rc, out in results:
        assert rc == 1, (n, rc, out)     # 1 = tests failed (not a crash or collection error)
