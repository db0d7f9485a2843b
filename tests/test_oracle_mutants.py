"""Planted mistakes in the oracle (CPU).  Each mutant is a copy of
oracle/ecokv_oracle.c with one plausible error -- a dropped or wrong divisor,
a flipped sign, a wrong index range or domain, swapped weights, a transposed
operand, a broken tie rule -- built with gcc into a temporary library.  The
pins of test_oracle_pins.py run against it in a child process and must fail.
A mutant that passes every pin would be a mistake the pins cannot see.  The
oracle itself is untouched: the copies live in pytest's temporary directory.
"""
import os
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PINS = os.path.join(ROOT, "tests", "test_oracle_pins.py")

# (name, text in the source, replacement); each text occurs exactly once
MUTANTS = [
    # input decode: bf16 bit patterns are the upper half of a binary32
    ("bf16_decode_shift", "uint32_t u = (uint32_t)((const uint16_t *)base)[i] << 16;",
     "uint32_t u = (uint32_t)((const uint16_t *)base)[i] << 15;"),
    ("bf16_decode_low_half", "uint32_t u = (uint32_t)((const uint16_t *)base)[i] << 16;",
     "uint32_t u = (uint32_t)((const uint16_t *)base)[i];"),
    # window importance (Sec. 3, Sec. 5.2)
    ("logit_scale_dropped", "logit[i] = dot * inv_sqrt_d;", "logit[i] = dot;"),
    ("causal_row_short", "const int last = p->causal ? P + j : T - 1;", "const int last = p->causal ? P + j - 1 : T - 1;"),
    ("window_mean_over_rows_only", "a[i] /= (double)(G * w);", "a[i] /= (double)w;"),
    ("pool_divisor_count", "imp[i] = acc / (double)p->pool_kernel;", "imp[i] = acc / (double)(2 * half);"),
    ("pool_window_one_sided",
     "for (int t = -half; t <= half; ++t)\n            if (i + t >= 0 && i + t < P) acc += a[i + t];",
     "for (int t = -half; t < half; ++t)\n            if (i + t >= 0 && i + t < P) acc += a[i + t];"),
    ("value_norm_squared", "imp[i] *= sqrt(n2);", "imp[i] *= n2;"),
    # first-sweep results handed over by a prefill (Eq. (1), App. A.1, Sec. 3)
    ("prefill_logit_scale_dropped", "lg[i] = dot * inv_sqrt_d;", "lg[i] = dot;"),
    ("prefill_causal_row_short", "const int seen = causal ? P + j : T - 1;", "const int seen = causal ? P + j - 1 : T - 1;"),
    ("prefill_khat_unnormalised", "pre[D + d] += x / nrm;", "pre[D + d] += x;"),
    ("prefill_sum_not_shifted", "z += exp(lg[i] - m);", "z += exp(lg[i]);"),
    ("prefill_rows_transposed", "pre[2 * D + g * w + j] = m;", "pre[2 * D + j * G + g] = m;"),
    # anchors and geometry (Eq. (1), App. A.1)
    ("kbar_over_prefix_count", "        kbar[d] /= (double)T;\n        mu[d] /= (double)T;",
     "        kbar[d] /= (double)(T - 1);\n        mu[d] /= (double)T;"),
    ("mu_unnormalised", "mu[d] += ora_get(K, dtype, (size_t)i * D + d) / nrm;", "mu[d] += ora_get(K, dtype, (size_t)i * D + d);"),
    ("prefix_centroid_over_T", "            kbar[d] /= (double)P;", "            kbar[d] /= (double)T;"),
    ("cos_sign", "sC[i] = (1.0 - cosmu[i]) / 2.0;", "sC[i] = (1.0 + cosmu[i]) / 2.0;"),
    ("cos_not_normalised", "cosmu[i] = dot / fmax(sqrt(n2), 1e-12);", "cosmu[i] = dot;"),
    ("rC_plain_mu2", "const double rC = ((double)T * mu2 - 1.0) / ((double)T - 1.0);", "const double rC = mu2;"),
    ("dE_squared", "dE[i] = sqrt(s2);", "dE[i] = s2;"),
    ("dE_extrema_over_T", "for (int i = 1; i < P; ++i) {\n        if (dE[i] < dmin)",
     "for (int i = 1; i < T; ++i) {\n        if (dE[i] < dmin)"),
    ("sE_reversed", "sE[i] = (dE[i] - dmin) / (dmax - dmin + p->eps);", "sE[i] = (dmax - dE[i]) / (dmax - dmin + p->eps);"),
    ("winsor_upper_quantile", "hi = ora_quantile(dE, P, 1.0 - p->winsor_q);", "hi = ora_quantile(dE, P, 1.0 - 2.0 * p->winsor_q);"),
    ("mad_sign", "exp(-(dE[i] - med) / (p->mad_tau * mad + p->eps))", "exp((dE[i] - med) / (p->mad_tau * mad + p->eps))"),
    ("quantile_rank_n", "const double h = q * (double)(n - 1);", "const double h = q * (double)n;"),
    ("quantile_no_interpolation", "c[j] + (h - j) * (c[j + 1] - c[j])", "c[j]"),
    ("mad_deviation_signed", "sE[i] = fabs(dE[i] - med);", "sE[i] = dE[i] - med;"),
    # redundancy and weight (Eq. (4)-(6), App. D)
    ("DE_over_prefix", "    DE /= (double)T;", "    DE /= (double)P;"),
    ("rE_missing_complement", "double rE = 2.0 - 2.0 / (1.0 + exp(-DE / tau));", "double rE = 2.0 / (1.0 + exp(-DE / tau));"),
    ("tau_D", "const double tau = p->tau > 0.0 ? p->tau : sqrt((double)D);", "const double tau = p->tau > 0.0 ? p->tau : (double)D;"),
    ("rstd_variance", "const double Dstd = sqrt(ss / (double)T);", "const double Dstd = ss / (double)T;"),
    ("lambda_weights_swapped", "double lambda = p->beta * rE + (1.0 - p->beta) * rC;",
     "double lambda = p->beta * rC + (1.0 - p->beta) * rE;"),
    # composite and final score (Eq. (3), (7))
    ("alpha_swapped", "sdiv[i] = p->alpha * sE[i] + (1.0 - p->alpha) * sC[i];",
     "sdiv[i] = p->alpha * sC[i] + (1.0 - p->alpha) * sE[i];"),
    ("scale_dropped", "const double scale = imp_mean / (sbar_mean + p->eps);", "const double scale = 1.0;"),
    ("final_mix_swapped", "S[i] = lambda * stilde + (1.0 - lambda) * imp[i];", "S[i] = lambda * imp[i] + (1.0 - lambda) * stilde;"),
    ("sbar_not_normalised", "        const double sbar = (sdiv[i] - smin) / (smax - smin + p->eps);\n        const double stilde",
     "        const double sbar = sdiv[i];\n        const double stilde"),
    # selection, compaction, decode (Sec. 3, App. A.1)
    ("tie_larger_position_first", "return a->key < b->key ? -1 : (a->key > b->key ? 1 : 0);",
     "return a->key > b->key ? -1 : (a->key < b->key ? 1 : 0);"),
    ("window_shifted", "for (int j = 0; j < w; ++j) idx[k + j] = P + j;", "for (int j = 0; j < w; ++j) idx[k + j] = P + j - 1;"),
    ("head_budget_of_layer", "const int32_t b = budget[u / B];", "const int32_t b = budget[(u / B) / Hkv];"),
    ("head_budget_units_by_sequence", "const int n = ora_select_unit(S + lh * Ptot + (cu[s] - s * w), T, w, budget[lh], idx + start[u]);",
     "const int n = ora_select_unit(S + lh * Ptot + (cu[s] - s * w), T, w, budget[s % Hkv], idx + start[u]);"),
    ("flat_tie_position_major", "it[(int64_t)h * P + i].key = (int64_t)h * P + i;", "it[(int64_t)h * P + i].key = (int64_t)i * H + h;"),
    ("compact_V_from_K", "(const char *)V + (base + i) * row, row);", "(const char *)K + (base + i) * row, row);"),
    ("decode_scale_dropped", "x[j] = dot * inv_sqrt_d;", "x[j] = dot;"),
    ("decode_lse_without_max", "lse[r] = m + log(z);", "lse[r] = log(z);"),
    ("decode_gqa_interleaved", "const int h = q / G;", "const int h = q % Hkv;"),
]


def run_pins_against(src_text, tmp_path):
    """Build src_text into a temporary library and run the pins on it; returns the child's result."""
    c = tmp_path / "copy.c"
    c.write_text(src_text)
    so = tmp_path / "copy.so"
    subprocess.check_call(["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-fopenmp", "-o", str(so), str(c), "-lm"])
    code = (f"import sys; sys.path.insert(0, {ROOT!r}); import oracle; oracle.use_library({str(so)!r}); "
            f"import pytest; sys.exit(pytest.main(['-x', '-q', '-p', 'no:cacheprovider', {PINS!r}]))")
    return subprocess.run([sys.executable, "-c", code], cwd=ROOT, capture_output=True, text=True, timeout=600)


def test_unaltered_copy_passes_every_pin(tmp_path):
    # the control: the same route with the source unchanged passes, so a
    # mutant's failure comes from its mistake
    r = run_pins_against(open(oracle._SRC).read(), tmp_path)
    assert r.returncode == 0, r.stdout[-2000:]


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_fails_a_pin(name, old, new, tmp_path):
    src = open(oracle._SRC).read()
    assert src.count(old) == 1, f"{name}: the text to alter occurs {src.count(old)} times"
    r = run_pins_against(src.replace(old, new), tmp_path)
    # exit 1: tests ran and some failed (an import or collection error would be 2 or more)
    assert r.returncode == 1, f"mutant {name} passed every pin (exit {r.returncode}):\n{r.stdout[-2000:]}"
