"""Plant plausible mistakes in a copy of the oracle (on the CPU) and check that
the pins catch every one of them.  This is what makes the pins worth trusting:
a dropped term, a wrong sign, index or operand order anywhere in the oracle
fails at least one of them."""
import os
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "lodestar_oracle.c")

# (name, original text, replacement): each must occur exactly once in the source
MUTANTS = [
    ("overlap_counts_all_cached", "if (!in_set(s, h[j])) break;", "if (!in_set(s, h[j])) continue;"),
    ("overlap_off_by_one", "int32_t l = 0;\n    for (int64_t j = 0; j < n; ++j) {",
     "int32_t l = 1;\n    for (int64_t j = 1; j < n; ++j) {"),
    ("sets_not_deduplicated_wrongly", "if (u == 0 || k[u - 1] != k[t]) k[u++] = k[t];",
     "if (u == 0 || k[u - 1] != k[t]) k[u++] = k[t]; else break;"),
    ("hit_ratio_half_block", "int64_t hit_tokens = (int64_t)LSO_BLOCK_TOKENS * l;",
     "int64_t hit_tokens = (int64_t)(LSO_BLOCK_TOKENS / 2) * l;"),
    ("uncached_tokens_sign", "x[d_inst + 4] = (double)((int64_t)L - hit_tokens);",
     "x[d_inst + 4] = (double)(hit_tokens - (int64_t)L);"),
    ("columns_swapped", "x[d_inst + 0] = (double)L;\n    x[d_inst + 1] = (double)n;",
     "x[d_inst + 0] = (double)n;\n    x[d_inst + 1] = (double)L;"),
    ("f64_normalise_sign", "buf_a[k] = (x[k] - (double)mu[k]) * (double)inv_sigma[k];",
     "buf_a[k] = (x[k] + (double)mu[k]) * (double)inv_sigma[k];"),
    ("lowp_normalise_divides", "t = t * inv_sigma[k];\n        buf_a[k]", "t = t / inv_sigma[k];\n        buf_a[k]"),
    ("f64_drops_bias", "double acc = (double)net->b[l][j];\n            for (int k = 0; k < K; ++k) acc +=",
     "double acc = 0.0;\n            for (int k = 0; k < K; ++k) acc +="),
    ("lowp_drops_bias", "float acc = net->b[l][j];", "float acc = 0.0f;"),
    ("f64_transposed_weight", "acc += (double)net->W[l][(int64_t)j * K + k] * a[k];",
     "acc += (double)net->W[l][(int64_t)k * O + j] * a[k];"),
    ("lowp_skips_last_input", "for (int k = 0; k < K; ++k) {\n                acc = fmaf(",
     "for (int k = 0; k + 1 < K; ++k) {\n                acc = fmaf("),
    ("f64_no_relu", "for (int j = 0; j < O; ++j) z[j] = z[j] > 0.0 ? z[j] : 0.0;", ""),
    ("lowp_leaky_relu", "float h = z[j] > 0.0f ? z[j] : 0.0f;", "float h = z[j] > 0.0f ? z[j] : 0.01f * z[j];"),
    ("bf16_skips_weights", "q[net->W_off[l] + t] = lso_bf16_round(params[net->W_off[l] + t]);",
     "q[net->W_off[l] + t] = params[net->W_off[l] + t];"),
    ("bf16_ties_away", "double q = nearbyint((double)x * scale);", "double q = round((double)x * scale);"),
    ("bf16_truncates", "double q = nearbyint((double)x * scale);", "double q = trunc((double)x * scale);"),
    ("argmin_tie_highest", "    return ia < ib;\n}\n\nint32_t lso_argmin", "    return ia > ib;\n}\n\nint32_t lso_argmin"),
    ("argmin_nan_first", "if (isnan(b)) return 1;", "if (isnan(b)) return 0;"),
    ("argmin_is_argmax", "if (a < b) return 1;\n    if (a > b) return 0;", "if (a > b) return 1;\n    if (a < b) return 0;"),
    ("update_wrong_sign", "params[t] = (float)((double)params[t] - (double)lr * grad[t]);",
     "params[t] = (float)((double)params[t] + (double)lr * grad[t]);"),
    ("update_no_factor_two", "double g = 2.0 * err / (double)B;", "double g = err / (double)B;"),
    ("update_sum_not_mean", "double g = 2.0 * err / (double)B;", "double g = 2.0 * err;"),
    ("update_mask_ignored", "double dk = zp[k] > 0.0 ? s : 0.0;", "double dk = s;"),
    ("update_weight_grad_transposed", "for (int k = 0; k < K; ++k) gw[k] += dj * a[k];",
     "for (int k = 0; k < K; ++k) gw[k] += dj * a[(k + 1) % K];"),
    ("update_backprop_uses_row", "s += Wq[net.W_off[l] + (int64_t)j * K + k] * delta[j];",
     "s += Wq[net.W_off[l] + (int64_t)k * O + j] * delta[j];"),
    ("update_bf16_backprop_skips_unit", "for (int j = 0; j < O; ++j) f = fmaf(",
     "for (int j = 1; j < O; ++j) f = fmaf("),
    ("update_no_bias_grad", "grad[net.b_off[l] + j] += dj;", ""),
    ("update_bf16_delta_unrounded", "dnext[k] = bf ? (double)lso_bf16_round((float)dk) : dk;", "dnext[k] = dk;"),
    ("update_lowp_forward_unfused", "f = fmaf((float)Wq[net.W_off[l] + (int64_t)j * K + k], (float)a[k], f);",
     "f = f + (float)Wq[net.W_off[l] + (int64_t)j * K + k] * (float)a[k];"),
    ("update_lowp_inputs_in_double", "a0[k] = bf ? (double)lso_bf16_round(t) : (double)t;",
     "a0[k] = bf ? (double)lso_bf16_round(t) : ((double)xb[k] - (double)mu[k]) * (double)inv_sigma[k];"),
    ("update_loss_not_mean", "if (loss_out) *loss_out = loss / (double)B;", "if (loss_out) *loss_out = loss;"),
    ("mix_constant", "* 0xbf58476d1ce4e5b9ull", "* 0xbf58476d1ce4e5b8ull"),
    ("hrw_index_offset", "0x9e3779b97f4a7c15ull * (uint64_t)(i + 1)", "0x9e3779b97f4a7c15ull * (uint64_t)i"),
    ("hrw_lightest", "if (best < 0 || w > bw) { best = i; bw = w; }", "if (best < 0 || w < bw) { best = i; bw = w; }"),
    ("alg1_strict_overload", "if (!(c[i] <= limit)) continue;", "if (!(c[i] < limit)) continue;"),
    ("alg1_sample_std", "double sigma = sqrt(var / (double)N);",
     "double sigma = sqrt(var / (double)(N > 1 ? N - 1 : 1));"),
    ("alg1_count_desc", "(m[i] == m[b] && c[i] < c[b])", "(m[i] == m[b] && c[i] > c[b])"),
    ("alg1_no_imbalance_check", "if (cmax - cmin > theta) return argmin_count(N, c);", ""),
    ("alg2_ge_tau", "if ((double)m[b] > tau) return b;", "if ((double)m[b] >= tau) return b;"),
    ("cold_start_le", "if (pol->n_samples < pol->n_min) {", "if (pol->n_samples <= pol->n_min) {"),
    ("ood_open_bounds", "static int in_bounds(float v, float lo, float hi) { return lo <= v && v <= hi; }",
     "static int in_bounds(float v, float lo, float hi) { return lo < v && v < hi; }"),
    ("ood_ignores_instances", "for (int32_t i = 0; i < N; ++i) ood |= !inst_ok[i];", ""),
    ("explore_le", "(uint64_t)rnd[(int64_t)r * 3] < explore_thr", "(uint64_t)rnd[(int64_t)r * 3] <= explore_thr"),
    ("explore_wrong_word", "chosen = scale_u32(rnd[(int64_t)r * 3 + 1], N);",
     "chosen = scale_u32(rnd[(int64_t)r * 3 + 2], N);"),
    ("kfilter_ignores_benefit", "saturated && kl_max > pol->tau_ben", "saturated"),
    ("tiebreak_ignores_scope", "if (scope && s[i] <= lim) S[ns++] = i;", "if (s[i] <= lim) S[ns++] = i;"),
    ("tiebreak_strict", "if (scope && s[i] <= lim) S[ns++] = i;", "if (scope && s[i] < lim) S[ns++] = i;"),
    ("gcr_admits_ties", "if (!(dc > nnd[js])) continue;", "if (!(dc >= nnd[js])) continue;"),
    ("gcr_replaces_most_isolated", "if (nnd[k] < nnd[js]) js = k;", "if (nnd[k] > nnd[js]) js = k;"),
    ("gcr_stale_neighbours", "            if (nni[k] == slot) {\n                nn_of(emb, H, n, k, &nnd[k], &nni[k]);",
     "            if (0) {\n                nn_of(emb, H, n, k, &nnd[k], &nni[k]);"),
    ("fifo_head_not_advanced", "*fifo_head = (slot + 1) % fifo_cap;", "*fifo_head = slot;"),
    ("embed_abs_residual", "float res = t - y[k];", "float res = fabsf(t - y[k]);"),
    ("train_drops_partial_batch", "int32_t m = n - s < batch ? n - s : batch;",
     "int32_t m = batch;\n            if (n - s < batch) break;"),
    ("train_skips_replay", "int32_t n = fifo_count + rep_count;", "int32_t n = fifo_count;"),
    ("commit_keeps_oldest", "    const lso_entry* y = (const lso_entry*)b;\n    if (x->s != y->s) return x->s > y->s ? -1 : 1;\n    return 0;\n}\n\n/* in_off",
     "    const lso_entry* y = (const lso_entry*)b;\n    if (x->s != y->s) return x->s < y->s ? -1 : 1;\n    return 0;\n}\n\n/* in_off"),
    ("commit_block_keeps_first_stamp", "if (x->h != y->h) return x->h < y->h ? -1 : 1;\n    if (x->s != y->s) return x->s > y->s ? -1 : 1;",
     "if (x->h != y->h) return x->h < y->h ? -1 : 1;\n    if (x->s != y->s) return x->s < y->s ? -1 : 1;"),
    ("commit_head_first_eviction", "(uint64_t)(((uint32_t)1 << LSO_STAMP_K_BITS) - 1u - k);", "(uint64_t)k;"),
    ("commit_requests_reversed", "((uint64_t)r << LSO_STAMP_K_BITS)", "((uint64_t)(0xFFFFFFu - r) << LSO_STAMP_K_BITS)"),
    ("commit_capacity_off_by_one", "int64_t keep = u < capacity[i] ? u : capacity[i];",
     "int64_t keep = u < capacity[i] ? u : capacity[i] - 1;"),
    ("commit_no_dedup", "if (u == 0 || A[u - 1].h != A[t].h) A[u++] = A[t];", "A[u++] = A[t];"),
    ("commit_skips_first_request", "if (chosen[r] != i) continue;", "if (chosen[r] != i || r == 0) continue;"),
    ("dropout_keeps_below", "    return (u >> 11) < thr53;", "    return (u >> 11) >= thr53;"),
    ("dropout_no_scale", "                    else if (thr53) h = lowp ? (double)((float)h * scale_f) : h * scale_d;\n", ""),
    ("dropout_backward_unmasked", "if (lso_dropped(seed, step, l - 1, b, k, thr53)) dk = 0.0;", "if (0) dk = 0.0;"),
    ("dropout_backward_wrong_layer", "if (lso_dropped(seed, step, l - 1, b, k, thr53)) dk = 0.0;",
     "if (lso_dropped(seed, step, l, b, k, thr53)) dk = 0.0;"),
    ("dropout_row_ignored", "    uint64_t c = ((((step * 4u + (uint64_t)layer) << 24) | (uint64_t)row) << 10) | (uint64_t)unit;",
     "    uint64_t c = ((((step * 4u + (uint64_t)layer) << 24) | (uint64_t)0 * row) << 10) | (uint64_t)unit;"),
    ("dropout_round_same_step", "lr, p, seed,\n                                        step++, NULL, &loss);",
     "lr, p, seed,\n                                        step, NULL, &loss);"),
]

_RUNNER = r"""
import sys
sys.path[:0] = [{root!r}, {tests!r}]
import oracle
oracle.use_library({lib!r})
import oracle_pins
failed = []
for pin in oracle_pins.ALL_PINS:
    try:
        pin()
    except Exception as e:
        failed.append(pin.__name__)
print("FAILED:" + ",".join(failed))
"""


@pytest.mark.slow
@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_mutant(name, old, new, tmp_path):
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} must occur once"
    mutant_src = tmp_path / "mutant.c"
    mutant_src.write_text(src.replace(old, new))
    lib = str(tmp_path / "libmutant.so")
    oracle.compile_c(str(mutant_src), lib)
    code = _RUNNER.format(root=ROOT, tests=os.path.join(ROOT, "tests"), lib=lib)
    proc = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    if proc.returncode != 0:
        return                                  # the mutant crashed: caught
    line = [l for l in proc.stdout.splitlines() if l.startswith("FAILED:")][-1]
    assert line != "FAILED:", f"no pin caught mutant {name}"
