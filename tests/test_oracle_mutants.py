"""Planted mistakes: each mutant of oracle.c (compiled on the CPU into a
temporary library) must fail at least one pin of tests/test_oracle.py.
This shows the pins constrain every part of the oracle, not just its shape."""
import contextlib
import os
import subprocess
import tempfile

import pytest

import oracle
import test_oracle as pins
import test_oracle_prefill as prefill_pins
import test_oracle_rope as rope_pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "oracle.c")

# (name, original text, mutated text)
MUTANTS = [
    ("drop_scale", "w[t] = dot * scale;", "w[t] = dot;"),
    ("scale_by_D", "1.0 / sqrt((double)D)", "1.0 / (double)D"),
    ("no_max_shift", "w[t] = exp(w[t] - s_max);", "w[t] = exp(w[t]);"),
    ("no_normalisation", "o[d] /= Z;", "o[d] /= 1.0;"),
    ("swap_k_and_v", "q + ((size_t)b * h + i) * D, Kc + row, Vc + row, L",
     "q + ((size_t)b * h + i) * D, Vc + row, Kc + row, L"),
    ("drop_last_token", "long L = seq_lens[b];", "long L = seq_lens[b] - 1;"),
    ("interleaved_q_groups", "int j = (i - 1) / heads_per_kv + 1;", "int j = (i - 1) % g + 1;"),
    ("interleaved_layer_groups", "int k = (n - 1) / layers_per_group + 1;",
     "int k = (n - 1) % m + 1;"),
    ("top_layer_owns", "(k - 1) * layers_per_group; /* bottom layer */",
     "k * layers_per_group - 1;"),
    ("append_swaps_k_v", "size_t src = ((size_t)b * n_kv + kv) * D;\n      memcpy(Kc + dst, k_new + src",
     "size_t src = ((size_t)b * n_kv + kv) * D;\n      memcpy(Kc + dst, v_new + src"),
    ("attend_before_append",
     "    oracle_append(n, B, n_kv, S, D, owner_of, Kc, Vc, k_new, v_new, ctx);\n"
     "    oracle_decode_attention(n, B, h, n_kv, S, D, kv_of, q_all + (size_t)n * B * h * D, Kc, Vc,\n"
     "                            lens_scratch, out_all + (size_t)n * B * h * D);",
     "    oracle_decode_attention(n, B, h, n_kv, S, D, kv_of, q_all + (size_t)n * B * h * D, Kc, Vc,\n"
     "                            lens_scratch, out_all + (size_t)n * B * h * D);\n"
     "    oracle_append(n, B, n_kv, S, D, owner_of, Kc, Vc, k_new, v_new, ctx);"),
    ("value_row_of_first_token", "o[d] += w[t] * bf16_value(V[t * ld + d]);",
     "o[d] += w[t] * bf16_value(V[d]);"),
    # rotary embedding
    ("rope_sign", "y[j] = x[j] * c - x[j + half] * s;", "y[j] = x[j] * c + x[j + half] * s;"),
    ("rope_frequency", "const double theta = pos * pow(base, -2.0 * j / rd);",
     "const double theta = pos * pow(base, -1.0 * j / rd);"),
    ("rope_interleaved_pairs", "b = bf16_value(x[j + half]);", "b = bf16_value(x[j ^ 1]);"),
    ("rope_rounding_truncates", "nearbyint(m * 256.0)", "trunc(m * 256.0)"),
    ("rope_step_key_position", "oracle_rope(k_new + off, D, rd, base, ctx[b], k_rot + off);",
     "oracle_rope(k_new + off, D, rd, base, ctx[b] + 1, k_rot + off);"),
    # prefill
    ("prefill_excludes_itself", "long L = (long)ctx[b] + t + 1;", "long L = (long)ctx[b] + t;"),
    ("prefill_sees_next_token", "long L = (long)ctx[b] + t + 1;", "long L = (long)ctx[b] + t + 2;"),
    ("prefill_ignores_new_tokens", "long L = (long)ctx[b] + t + 1;", "long L = (long)ctx[b] + 1;"),
    ("prefill_swap_k_and_v", "oracle_attend_one(q + qo, Kc + row, Vc + row,",
     "oracle_attend_one(q + qo, Vc + row, Kc + row,"),
    ("prefill_append_swaps_k_v",
     "size_t src = (((size_t)b * T + t) * n_kv + kv) * D;\n        memcpy(Kc + dst, k_new + src",
     "size_t src = (((size_t)b * T + t) * n_kv + kv) * D;\n        memcpy(Kc + dst, v_new + src"),
    ("prefill_slot_shifted", "long slot = (long)ctx[b] + t;", "long slot = (long)ctx[b] + t + 1;"),
    ("prefill_rows_token_major", "size_t src = (((size_t)b * T + t) * n_kv + kv) * D;",
     "size_t src = (((size_t)t * B + b) * n_kv + kv) * D;"),
    ("prefill_query_of_first_token", "size_t qo = (((size_t)b * T + t) * h + i) * D;\n"
     "        oracle_attend_one(q + qo,",
     "size_t qo = (((size_t)b * T + t) * h + i) * D;\n"
     "        oracle_attend_one(q + qo - (size_t)t * h * D,"),
]


def _pin_calls():
    calls = []
    for row in pins._read_table("table2_variants.txt"):
        calls.append(("table2 " + row[0], lambda r=row: pins.test_map_matches_table2_head_counts(r)))
    calls.append(("map special cases", pins.test_map_special_cases))
    for lmg in [(2, 4, 2, 4), (2, 4, 2, 1), (4, 4, 2, 2), (3, 6, 1, 3)]:
        calls.append((f"brute force {lmg}",
                      lambda a=lmg: pins.test_decode_attention_matches_brute_force(a)))
    calls += [
        ("sdpa mha", pins.test_identity_map_matches_torch_sdpa_fp64),
        ("sdpa gqa", pins.test_gqa_matches_torch_sdpa_with_repeated_kv),
        ("two tokens", pins.test_two_tokens_closed_form),
        ("L=1", pins.test_single_position_returns_v_exactly),
        ("identical keys", pins.test_identical_keys_give_mean_of_values),
        ("sum to one", pins.test_weights_sum_to_one_and_are_nonnegative),
        ("needle", lambda: pins.test_needle_dominates_and_large_scores_stay_finite(31)),
        ("append", pins.test_append_writes_only_owned_slots),
        ("mlkv2 ctx0", pins.test_step_mlkv2_empty_context_outputs_owner_values),
        ("non-owner sees new token", pins.test_step_non_owner_layer_sees_token_appended_this_step),
        ("bf16 rounding", rope_pins.test_bf16_rounding_is_nearest_ties_to_even),
        ("rope identity", rope_pins.test_position_zero_and_zero_channels_are_identity),
        ("rope closed form", rope_pins.test_closed_form_of_a_four_channel_rotation),
        ("rope lengths", rope_pins.test_pairs_keep_their_length),
        ("rope relative position", rope_pins.test_scores_depend_only_on_the_position_difference),
        ("rope bf16", rope_pins.test_bf16_rope_is_the_rounded_double_rotation),
        ("rope step", rope_pins.test_step_with_rope_is_the_step_on_rotated_inputs),
        ("prefill T=1", prefill_pins.test_one_new_token_is_the_decode_step),
        ("prefill = decode steps",
         lambda: prefill_pins.test_prompt_equals_decode_steps_one_token_at_a_time((4, 6, 2, 2))),
        ("prefill sdpa", prefill_pins.test_matches_torch_sdpa_with_a_causal_mask),
        ("prefill causal", prefill_pins.test_later_tokens_do_not_change_earlier_outputs),
        ("prefill two tokens", prefill_pins.test_two_new_tokens_closed_form),
        ("prefill rows", prefill_pins.test_owners_write_the_new_rows_at_consecutive_slots),
    ]
    return calls


@contextlib.contextmanager
def _mutant_library(src_text):
    with tempfile.TemporaryDirectory() as d:
        c = os.path.join(d, "mutant.c")
        so = os.path.join(d, "libmutant.so")
        with open(c, "w") as f:
            f.write(src_text)
        subprocess.check_call(["gcc", "-O1", "-fopenmp", "-fPIC", "-shared", "-std=c11", c,
                               "-o", so, "-lm"])
        saved_lib, saved_path = oracle._lib, oracle._LIB
        oracle._lib, oracle._LIB = None, so
        try:
            oracle._load()
            yield
        finally:
            oracle._lib, oracle._LIB = saved_lib, saved_path


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_is_caught(name, old, new):
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    caught = []
    with _mutant_library(src.replace(old, new)):
        for label, call in _pin_calls():
            try:
                call()
            except (AssertionError, ValueError, IndexError):
                caught.append(label)
    assert caught, f"no pin caught the planted mistake {name}"


def test_unmutated_oracle_passes_every_pin():
    for label, call in _pin_calls():
        call()
