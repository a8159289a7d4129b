"""Mutation check of the pins: each plausible mistake planted in a copy of
the oracle's source (built on the CPU into a temporary library) must make at
least one pin fail.  The real oracle is never modified."""
import os
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# (name, original text, planted mistake)
MUTANTS = [
    ("row_norm_dropped", "double s = dot / (fmax(mn, 1e-8) * fmax(qn, 1e-8));",
     "double s = dot / fmax(qn, 1e-8);"),
    ("question_norm_dropped", "double s = dot / (fmax(mn, 1e-8) * fmax(qn, 1e-8));",
     "double s = dot / fmax(mn, 1e-8);"),
    ("score_sign", "double s = dot / (fmax(mn, 1e-8) * fmax(qn, 1e-8));",
     "double s = -dot / (fmax(mn, 1e-8) * fmax(qn, 1e-8));"),
    ("tie_break_reversed", "return (x->j > y->j) - (x->j < y->j);",
     "return (x->j < y->j) - (x->j > y->j);"),
    ("no_document_order", "qsort(out, (size_t)k, sizeof(int32_t), by_value);",
     "(void)by_value;"),
    ("norm_of_query_in_row", "mm += m * m;", "mm += (double)q[d] * (double)q[d];"),
    ("select_key_element_order", "const double m = load_elem(sel_keys, keys_bf16, row + d);",
     "const double m = load_elem(sel_keys, keys_bf16, row + (d ^ 1));"),
    ("row_norms_row_stride", "const double x = load_elem(rows, is_bf16, (size_t)r * D + d);",
     "const double x = load_elem(rows, is_bf16, (size_t)r * (D / 2) + d);"),
    ("window_start_full_W", "long long s = alpha - W / 2;", "long long s = alpha - W;"),
    ("window_start_no_clamp_hi", "if (s > hi) s = hi;", "(void)hi;"),
    ("ring_slot_off_by_one", "int slot = (int)(((long long)c + t) % W);",
     "int slot = (int)(((long long)c + t + 1) % W);"),
    ("ring_count_not_advanced", "win_count[b] = c + T_new;", "win_count[b] = c;"),
    ("gqa_modulo_mapping", "const int kv = h / G;", "const int kv = h % Hkv;"),
    ("window_always_full", "(win_count[b] < W ? win_count[b] : W)", "W"),
    ("index_list_ignored", "int r = idx ? idx[(size_t)b * k + i] : i;", "int r = i;"),
    ("keys_from_values", "kb[i] = cme_k;", "kb[i] = cme_v;"),
    ("scale_dropped", "z[i] = scale * acc;", "z[i] = acc;"),
    ("no_max_subtraction", "z[i] = exp(z[i] - m);", "z[i] = exp(z[i]);"),
    ("no_normaliser", "o[d] = n > 0 ? acc / den : 0.0;", "o[d] = n > 0 ? acc : 0.0;"),
    ("value_element_index", "acc += z[i] * load_elem(vb[i], kv_is_bf16, row[i] + d);",
     "acc += z[i] * load_elem(vb[i], kv_is_bf16, row[i] + (Dh - 1 - d));"),
    ("window_row_stride", "row[k + s] = (((size_t)b * Hkv + kv) * W + (size_t)s) * Dh;",
     "row[k + s] = (((size_t)b * Hkv + kv) * W + (size_t)(valid - 1 - s) / 2) * Dh;"),
    ("bf16_widening", "uint32_t u = ((uint32_t)h) << 16;", "uint32_t u = ((uint32_t)h) << 15;"),
    ("locate_tie_to_later_row", "if (norms[(size_t)b * N + j] > norms[(size_t)b * N + best])",
     "if (norms[(size_t)b * N + j] >= norms[(size_t)b * N + best])"),
    ("locate_row_not_chunk", "int chunk = best / mems_per_chunk;", "int chunk = best;"),
    ("locate_chunk_modulo", "int chunk = best / mems_per_chunk;", "int chunk = best % mems_per_chunk;"),
    ("locate_all_rows", "if (nb > N) nb = N;", "nb = N;"),
    ("locate_no_midpoint", "alpha = ctx_len[b] / 2;", "alpha = 0;"),
    ("row_norm_squared", "norms_out[r] = sqrt(s);", "norms_out[r] = s;"),
    ("denoise_strict_threshold", "keep = max_cos[(size_t)b * n + i] >= tau;",
     "keep = max_cos[(size_t)b * n + i] > tau;"),
    ("denoise_neighbourhood_short", "for (int j = i + 1; j <= i + g && j < nb; ++j) {",
     "for (int j = i + 1; j < i + g && j < nb; ++j) {"),
    ("denoise_past_sequence_end", "for (int j = i + 1; j <= i + g && j < nb; ++j) {",
     "for (int j = i + 1; j <= i + g && j < n; ++j) {"),
    ("denoise_floor_off_by_one", "if (keep_min_every > 0 && i - last >= keep_min_every)",
     "if (keep_min_every > 0 && i - last > keep_min_every)"),
    ("denoise_floor_start", "int last = -1, count = 0;", "int last = 0, count = 0;"),
    ("denoise_upstream_norm", "double c = dot / (fmax(ni, 1e-8) * fmax(sqrt(nj), 1e-8));",
     "double c = dot / (fmax(ni, 1e-8) * fmax(ni, 1e-8));"),
    ("bridge_gelu_tanh_form", "return 0.5 * x * (1.0 + erf(x / sqrt(2.0)));",
     "return 0.5 * x * (1.0 + tanh(0.7978845608028654 * (x + 0.044715 * x * x * x)));"),
    ("bridge_no_hidden_bias", "double u = (double)b1[f];", "double u = 0.0;"),
    ("bridge_no_output_bias", "double acc = (double)b2[j];", "double acc = 0.0;"),
    ("bridge_w2_transposed", "acc += hidden[(size_t)r * F + f] * widen_bf16(w2[(size_t)j * F + f]);",
     "acc += hidden[(size_t)r * F + f] * widen_bf16(w2[((size_t)f * Hd + j) % ((size_t)Hd * F)]);"),
    ("bridge_unbiased_variance", "var /= Hd;", "var /= (Hd > 1 ? Hd - 1 : 1);"),
    ("bridge_eps_outside_sqrt", "double inv = 1.0 / sqrt(var + eps);", "double inv = 1.0 / (sqrt(var) + eps);"),
    ("bridge_cap_at_nu", "double c = (nrm > 0.0 && 2.0 * nu / nrm < 1.0) ? 2.0 * nu / nrm : 1.0;",
     "double c = (nrm > 0.0 && nu / nrm < 1.0) ? nu / nrm : 1.0;"),
    ("bridge_gamma_beta_swapped",
     "double m_hat = (double)gamma[j] * (y[j] - mean) * inv + (double)beta[j];",
     "double m_hat = (double)beta[j] * (y[j] - mean) * inv + (double)gamma[j];"),
    ("bridge_no_tanh", "y[j] = nu * tanh(m_hat);", "y[j] = nu * m_hat;"),
    ("denoise_chunk_first_token", "int v = c < nc ? kept_idx[(size_t)b * n + (size_t)c * chunk_tokens] : -1;",
     "int v = c < nc ? kept_idx[(size_t)b * n + (size_t)c] : -1;"),
]


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_kill_mutant(tmp_path, name, old, new):
    src = open(oracle.SOURCE).read()
    assert src.count(old) == 1, f"mutation site for {name} not unique"
    mutated = tmp_path / "mutant.c"
    mutated.write_text(src.replace(old, new))
    lib = oracle.compile_source(str(mutated), str(tmp_path / "libmutant.so"))
    r = subprocess.run([sys.executable, "-m", "tests.pins", lib], cwd=ROOT,
                       capture_output=True, text=True, timeout=300)
    assert r.returncode != 0, f"mutant {name} survived every pin:\n{r.stdout}{r.stderr}"
