"""Planted mistakes in the CPU oracle must be caught by the pin battery.

Each mutant is a copy of oracle_attn.c with one plausible mistake (a wrong
head mapping, a dropped term, a wrong sign/offset/index, a wrong log base),
compiled on the CPU into a temporary library.  The pins that the real
oracle passes must fail for every one of them.  All mutants keep every
memory access inside its buffer.
"""
import os

import pytest

import pins
from oracle import oracle as orc

SRC = os.path.join(os.path.dirname(orc.__file__), "oracle_attn.c")

# name -> (original text, mutated text, expected occurrences)
MUTANTS = {
    "gqa_interleaved_heads": ("int g = hq / G;\n        int i = job->rows",
                              "int g = hq % job->Hkv;\n        int i = job->rows", 1),
    "scale_dropped": ("s_buf[j] = scale * dot;", "s_buf[j] = dot;", 1),
    "not_normalised": ("double p = s_buf[j] / l;", "double p = s_buf[j];", 1),
    "lse_log2": ("*lse_out = m + log(l);", "*lse_out = m + log2(l);", 1),
    "lse_without_max": ("*lse_out = m + log(l);", "*lse_out = log(l);", 1),
    "weights_without_max": ("s_buf[j] = exp(s_buf[j] - m);", "s_buf[j] = exp(s_buf[j]);", 1),
    "top_left_causal": ("int off = L - job->Sq;", "int off = 0;", 1),
    "causal_strict_diagonal": ("if (last + 1 < n_valid) n_valid = last + 1;",
                               "if (last < n_valid) n_valid = last;", 2),
    "value_head_zero": ("const uint16_t *v_head = job->v + ((size_t)b * job->Hkv + g)",
                        "const uint16_t *v_head = job->v + ((size_t)b * job->Hkv + 0)", 1),
    "query_element_zero": ("dot += bf16_bits_to_double(q_row[d]) *\n                   bf16_bits_to_double(k_head[(size_t)j * D + d]);",
                           "dot += bf16_bits_to_double(q_row[0]) *\n                   bf16_bits_to_double(k_head[(size_t)j * D + d]);", 1),
    "negative_length_not_clamped_to_zero": ("if (len < 0) return 0;", "if (len < 0) return 1;", 1),
    "bf16_widening_shift": ("((uint32_t)bits) << 16;", "((uint32_t)bits) << 15;", 1),
    "row_subset_ignored": ("int i = job->rows ? job->rows[it] : (int)r;", "int i = (int)r;", 1),
    "combine_weight_by_max": ("double w = exp(ls[s] - L);", "double w = exp(ls[s] - M);", 1),
    "combine_lse_without_max": ("double L = M + log(sum);", "double L = log(sum);", 1),
    "paged_table_row_stride": ("block_table[(size_t)b * max_pages + j / page_size]",
                               "block_table[(size_t)b + j / page_size]", 1),
    "paged_row_reversed": ("(size_t)(j % page_size);", "(size_t)(page_size - 1 - j % page_size);", 1),
    "paged_head_ignored": ("return ((size_t)page * Hkv + g) * page_size",
                           "return ((size_t)page * Hkv + 0) * page_size", 1),
    "varlen_causal_top_left": ("if (causal && i + Skv - Sq + 1 < n_valid) n_valid = i + Skv - Sq + 1;",
                               "if (causal && i + 1 < n_valid) n_valid = i + 1;", 1),
    "varlen_lse_token_major": ("lse_row = lse + (size_t)hq * total_q + (q0 + i);",
                               "lse_row = lse + (size_t)(q0 + i) * Hq + hq;", 1),
    "bwd_delta_dropped": ("const double ds = p[j] * (dp[j] - delta);",
                          "const double ds = p[j] * (dp[j]);", 1),
    "bwd_dk_without_scale": ("dk[kv0 + (size_t)j * D + d] += scale * ds *",
                             "dk[kv0 + (size_t)j * D + d] += ds *", 1),
    "bwd_dv_from_ds": ("dv[kv0 + (size_t)j * D + d] += p[j] *",
                       "dv[kv0 + (size_t)j * D + d] += ds *", 1),
    "bwd_dq_from_values": ("dq[qi + d] += scale * ds * bf16_bits_to_double(k[kv0",
                           "dq[qi + d] += scale * ds * bf16_bits_to_double(v[kv0", 1),
    "mla_rope_not_in_scores": ("for (int d = 0; d < Dk; ++d)\n                    dot +=",
                               "for (int d = 0; d < Dc; ++d)\n                    dot +=", 1),
    "mla_value_past_rope": ("o_row[e] += p * bf16_bits_to_double(cache[(size_t)j * Dk + e]);",
                            "o_row[e] += p * bf16_bits_to_double(cache[(size_t)j * Dk + Dr + e]);", 1),
    "mla_cache_of_batch_zero": ("const uint16_t *cache = ckv + (size_t)b * Smax * Dk;",
                                "const uint16_t *cache = ckv;", 1),
    "mla_scale_dropped": ("s[j] = scale * dot;\n                if (s[j] > m) m = s[j];\n            }\n"
                          "            double l = 0.0;\n            for (int j = 0; j < L; ++j) { s[j] = exp",
                          "s[j] = dot;\n                if (s[j] > m) m = s[j];\n            }\n"
                          "            double l = 0.0;\n            for (int j = 0; j < L; ++j) { s[j] = exp", 1),
    "probs_scale_dropped": ("s[j] = scale * dot;\n                }\n                double m = s[0];",
                            "s[j] = dot;\n                }\n                double m = s[0];", 1),
    "probs_gqa_interleaved_heads": ("int g = hq / G;\n                int L = clamp_len(",
                                    "int g = hq % Hkv;\n                int L = clamp_len(", 1),
    "ragged_paged_causal_top_left": ("if (causal && i + L - Sq + 1 < n_valid) n_valid = i + L - Sq + 1;",
                                     "if (causal && i + 1 < n_valid) n_valid = i + 1;", 1),
    "ragged_paged_value_head_zero": ("page_size, Hkv, g, j);\n                    const double p = s[j] / l;",
                                     "page_size, Hkv, 0, j);\n                    const double p = s[j] / l;", 1),
    "ragged_paged_last_key_dropped": ("int n_valid = L;\n                if (causal && i + L - Sq",
                                      "int n_valid = L > 1 ? L - 1 : L;\n                if (causal && i + L - Sq", 1),
    "ragged_paged_lse_token_major": ("double *lse_row = &lse[(size_t)hq * total_q + q0 + i];",
                                     "double *lse_row = &lse[(size_t)(q0 + i) * Hq + hq];", 1),
    "varlen_key_start_ignored": ("const uint16_t *k_row = k + ((size_t)(k0 + j) * Hkv + g) * D;",
                                 "const uint16_t *k_row = k + ((size_t)(j) * Hkv + g) * D;", 1),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    old, new, count = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == count, f"mutation site for {name} not found as expected"
    mut_src = tmp_path / f"oracle_{name}.c"
    mut_src.write_text(src.replace(old, new))
    lib_path = orc.build(str(mut_src), str(tmp_path / f"liboracle_{name}.so"))
    lib = orc.load(lib_path)
    caught = []
    for pin in pins.ALL_PINS:
        try:
            pin(lib)
        except AssertionError as exc:
            caught.append(f"{pin.__name__}: {exc}")
            break
    assert caught, f"mutant {name} passed every pin"
