"""Plant plausible mistakes in a copy of the oracle and check the pins catch each.

Every mutant is a one-place text edit of oracle.c (a dropped term, a wrong
sign, a wrong or transposed index), compiled with gcc into a temporary
library.  The pin battery from pins.py must fail on every mutant; a mutant
that survives means the pins leave that part of the oracle unchecked.
"""
import os

import pytest

import oracle
import pins

MUTANTS = [
    # (name, original text, replacement, which battery)
    ("gqa_head_map", "const int32_t kh = h / r;", "const int32_t kh = h % Hkv;", "attn"),
    ("dropped_scale", "x[j] = sigma * dot;", "x[j] = dot;", "attn"),
    ("suffix_index", "(suffix_start[s] + (j - Lp)) * Hkv + kh) * (int64_t)D;\n                double dot",
     "(suffix_start[s] + j) * Hkv + kh) * (int64_t)D;\n                double dot", "attn"),
    ("prompt_of_candidate", "const int64_t p = s / G;", "const int64_t p = s % P;", "attn"),
    ("unnormalised_weights", "const double w = exp(x[j] - m) / Z;", "const double w = exp(x[j] - m);", "attn"),
    ("lse_drops_max", "lse[s * Hq + h] = m + log(Z);", "lse[s * Hq + h] = log(Z);", "attn"),
    ("prefix_of_first_prompt", "? k_prefix + ((prefix_start[p] + j)", "? k_prefix + ((prefix_start[0] + j)", "attn"),
    ("value_from_key_cache", "? v_prefix + ((prefix_start[p] + j)", "? k_prefix + ((prefix_start[p] + j)", "attn"),
    ("query_index_swapped", "const uint16_t *qv = q + (s * Hq + h) * (int64_t)D;",
     "const uint16_t *qv = q + ((int64_t)h * S + s) * (int64_t)D;", "attn"),
    ("max_not_subtracted", "Z += exp(x[j] - m);", "Z += exp(x[j]);", "attn"),
    ("logprob_sign", "if (t >= 0 && t < V) return z[t] - l;", "if (t >= 0 && t < V) return l - z[t];", "lp"),
    ("transposed_weight", "for (int32_t k = 0; k < H; ++k) dot += h[k] * bf16_to_f64(wr[k]);",
     "for (int32_t k = 0; k < H; ++k) dot += h[k] * bf16_to_f64(w_lm[(int64_t)k * V + v]);", "lp"),
    ("dropped_temperature", "z[v] = inv_T * dot;", "z[v] = dot;", "lp"),
    ("lse_missing_max", "return M + log(sum);", "return log(sum);", "lp"),
    ("masked_row_not_zero", "if (t == -1) return 0.0;", "if (t == -1) return -l;", "lp"),
    ("gather_off_by_one", "if (t >= 0 && t < V) return z[t] - l;", "if (t >= 0 && t < V) return z[t > 0 ? t - 1 : 0] - l;", "lp"),
    ("last_vocab_id_dropped", "for (int32_t v = 0; v < V; ++v) sum += exp(z[v] - M);",
     "for (int32_t v = 0; v < V - 1; ++v) sum += exp(z[v] - M);", "lp"),
    # group-relative advantages and the clipped surrogate
    ("adv_population_std", "sqrt(ss / (G - 1))", "sqrt(ss / G)", "grpo"),
    ("adv_not_centred", "(r[i] - mean) / sd : 0.0;", "r[i] / sd : 0.0;", "grpo"),
    ("adv_wrong_group_base", "const double *r = reward + p * G;", "const double *r = reward;", "grpo"),
    ("clip_upper_bound", "(rho > 1.0 + eps ? 1.0 + eps : rho)", "(rho > 1.0 + eps ? 1.0 - eps : rho)", "grpo"),
    ("max_not_min", "total += (u <= c ? u : c) * w;", "total += (u >= c ? u : c) * w;", "grpo"),
    ("surrogate_grad_sign", "grad[r] = u <= c ? -w * rho * adv[i] : 0.0;", "grad[r] = u <= c ? w * rho * adv[i] : 0.0;", "grpo"),
    ("grad_missing_ratio", "grad[r] = u <= c ? -w * rho * adv[i] : 0.0;", "grad[r] = u <= c ? -w * adv[i] : 0.0;", "grpo"),
    ("no_token_mean", "const double w = 1.0 / ((double)P * G * (double)count[i]);", "const double w = 1.0 / ((double)P * G);", "grpo"),
    ("ratio_inverted", "const double rho = exp(logp_new[r] - logp_old[r]);", "const double rho = exp(logp_old[r] - logp_new[r]);", "grpo"),
    # log-prob backward
    ("bwd_missing_temperature", "const double scale = grad_logprob[r] * inv_T;", "const double scale = grad_logprob[r];", "bwd"),
    ("bwd_target_row_dropped", "dh[k] = scale * (bf16_to_f64(wt[k]) + dh[k]);", "dh[k] = scale * dh[k];", "bwd"),
    ("bwd_unnormalised_p", "const double pv = exp(z[v] - l);", "const double pv = exp(z[v]);", "bwd"),
    ("bwd_wrong_target_row", "const uint16_t *wt = w_lm + (int64_t)t * H;", "const uint16_t *wt = w_lm + (int64_t)(V - 1 - t) * H;", "bwd"),
    ("bwd_masked_not_zero", "if (t == -1) {\n            for (int32_t k = 0; k < H; ++k) dh[k] = 0.0;",
     "if (t == -1) {\n            for (int32_t k = 0; k < H; ++k) dh[k] = 1.0;", "bwd"),
    # nucleus sampling
    ("rank_ascending", "if (x->y > y->y) return -1;\n    if (x->y < y->y) return 1;",
     "if (x->y > y->y) return 1;\n    if (x->y < y->y) return -1;", "samp"),
    ("ties_larger_id_first", "return (x->v > y->v) - (x->v < y->v);", "return (x->v < y->v) - (x->v > y->v);", "samp"),
    ("nucleus_drops_crossing_token", "in_n[rk[n].v] = 1;", "if (cum < top_p) in_n[rk[n].v] = 1;", "samp"),
    ("nucleus_not_renormalised", "const double target = uniform[r] * zn;", "const double target = uniform[r];", "samp"),
    ("cdf_in_rank_order", "for (int32_t v = 0; v < V; ++v) {\n            if (!in_n[v]) continue;",
     "for (int32_t i = 0; i < V; ++i) {\n            const int32_t v = rk[i].v;\n            if (!in_n[v]) continue;", "samp"),
    ("sampling_temperature_dropped", "const double lse = row_logits(H, V, h, w_lm, inv_T, y);",
     "const double lse = row_logits(H, V, h, w_lm, 1.0, y);", "samp"),
    ("interval_includes_own_mass", "if (v < t) below += pv;", "if (v <= t) below += pv;", "samp"),
    ("sample_logprob_unnormalised", "logprob[r] = y[t] - lse;", "logprob[r] = y[t];", "samp"),
    # extend (prefill) attention of a refinement turn
    ("ext_excludes_self", "const int64_t visible = n_pre + (n_suf - n_new + i) + 1;",
     "const int64_t visible = n_pre + (n_suf - n_new + i);", "ext"),
    ("ext_new_at_suffix_start", "const int64_t visible = n_pre + (n_suf - n_new + i) + 1;",
     "const int64_t visible = n_pre + i + 1;", "ext"),
    ("ext_not_causal", "const int64_t visible = n_pre + (n_suf - n_new + i) + 1;",
     "const int64_t visible = n_pre + n_suf;", "ext"),
    ("ext_query_rows_reversed", "const int64_t qrow = q_start[c] + i;",
     "const int64_t qrow = q_start[c] + (n_new - 1 - i);", "ext"),
    ("ext_head_map", "const int32_t kv_head = head / heads_per_kv;", "const int32_t kv_head = head % Hkv;", "ext"),
    ("ext_prompt_of_candidate", "const int64_t prompt = c / G;", "const int64_t prompt = c % P;", "ext"),
    ("ext_dropped_scale", "score[j] = (double)scale * qk;", "score[j] = qk;", "ext"),
    ("ext_lse_drops_max", "lse[qrow * Hq + head] = mx + log(zsum);", "lse[qrow * Hq + head] = log(zsum);", "ext"),
    ("ext_suffix_row_index", "k_suffix + ((suffix_start[c] + (j - n_pre))", "k_suffix + ((suffix_start[c] + j)", "ext"),
    ("ext_value_from_prefix_keys", "? v_prefix + ((prefix_start[prompt] + j)",
     "? k_prefix + ((prefix_start[prompt] + j)", "ext"),
    ("ext_unnormalised", "const double wj = exp(score[j] - mx) / zsum;", "const double wj = exp(score[j] - mx);", "ext"),
]


@pytest.fixture(scope="module")
def source():
    with open(oracle.SRC_PATH) as f:
        return f.read()


@pytest.mark.parametrize("name,old,new,battery", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, source, name, old, new, battery):
    assert source.count(old) == 1, f"mutation site for {name} must occur exactly once"
    src = tmp_path / f"oracle_{name}.c"
    src.write_text(source.replace(old, new))
    lib = oracle.compile_c(str(src), str(tmp_path / f"liboracle_{name}.so"))
    orc = oracle.Oracle(lib)
    battery_fns = {"attn": pins.ATTENTION_PINS, "lp": pins.LOGPROB_PINS, "grpo": pins.GRPO_PINS,
                   "bwd": pins.BACKWARD_PINS, "samp": pins.SAMPLING_PINS,
                   "ext": pins.EXTEND_PINS}[battery]
    caught = []
    for pin in battery_fns:
        try:
            pin(orc)
        except Exception:  # any failing pin catches the mutant
            caught.append(pin.__name__)
    assert caught, f"mutant {name} survived every pin"
