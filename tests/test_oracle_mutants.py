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
    ("logprob_sign", "logprob[r] = z[t] - l;", "logprob[r] = l - z[t];", "lp"),
    ("transposed_weight", "dot += bf16_to_f64(hr[k]) * bf16_to_f64(wr[k]);",
     "dot += bf16_to_f64(hr[k]) * bf16_to_f64(w_lm[(int64_t)k * V + v]);", "lp"),
    ("dropped_temperature", "z[v] = inv_T * dot;", "z[v] = dot;", "lp"),
    ("lse_missing_max", "const double l = M + log(sum);", "const double l = log(sum);", "lp"),
    ("masked_row_not_zero", "if (t == -1)\n            logprob[r] = 0.0;", "if (t == -1)\n            logprob[r] = -l;", "lp"),
    ("gather_off_by_one", "logprob[r] = z[t] - l;", "logprob[r] = z[t > 0 ? t - 1 : 0] - l;", "lp"),
    ("last_vocab_id_dropped", "for (int32_t v = 1; v < V; ++v) if (z[v] > M) M = z[v];\n        double sum = 0.0;\n        for (int32_t v = 0; v < V; ++v)",
     "for (int32_t v = 1; v < V; ++v) if (z[v] > M) M = z[v];\n        double sum = 0.0;\n        for (int32_t v = 0; v < V - 1; ++v)", "lp"),
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
    battery_fns = pins.ATTENTION_PINS if battery == "attn" else pins.LOGPROB_PINS
    caught = []
    for pin in battery_fns:
        try:
            pin(orc)
        except Exception:  # any failing pin catches the mutant
            caught.append(pin.__name__)
    assert caught, f"mutant {name} survived every pin"
