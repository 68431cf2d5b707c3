"""Plants plausible mistakes in a temporary copy of the oracle's C source and
checks that the pin suite (test_oracle_pins.py) rejects every one of them.

Each mutant is compiled to a scratch library under pytest's tmp_path and run in
a child process, so a mutant that crashes counts as detected without taking the
test runner down.  The committed oracle is never modified.
"""
import multiprocessing as mp
import os
import subprocess

import pytest

import oracle

SRC = os.path.join(os.path.dirname(oracle.__file__), "kva_oracle.c")

# (name, original text, replacement)
MUTANTS = [
    ("no_max_subtraction",
     [("s[t] = exp(s[t] - m);", "s[t] = exp(s[t]);"), ("*lse = m + log(l);", "*lse = log(l);")]),
    ("wrong_sign_in_exp", [("s[t] = exp(s[t] - m);", "s[t] = exp(m - s[t]);")]),
    ("kv_head_modulo", [("const int g = h / group;", "const int g = h % Hkv;")]),
    ("kv_layout_transposed",
     [("size_t row = ((size_t)b * (size_t)Lmax + (size_t)t) * (size_t)Hkv + (size_t)g;",
       "size_t row = ((size_t)b * (size_t)Hkv + (size_t)g) * (size_t)Lmax + (size_t)t;")]),
    ("missing_scale", [("s[t] = scale * dot;", "s[t] = dot;")]),
    ("lse_without_log", [("*lse = m + log(l);", "*lse = m + l;")]),
    ("page_slot_off_by_one", [("(size_t)(t % page_size)", "(size_t)((t + 1) % page_size)")]),
    ("page_index_from_slot",
     [("block_table[(size_t)b * max_pages + t / page_size];\n                size_t row",
       "block_table[(size_t)b * max_pages + (t / page_size + 1) % (lens[b] / page_size + 1)];\n                size_t row")]),
    ("drops_first_value",
     [("for (int t = 0; t < L; ++t) acc += s[t] * bf16_to_f64(vrow[t][d]);",
       "for (int t = 1; t < L; ++t) acc += s[t] * bf16_to_f64(vrow[t][d]);")]),
    ("values_read_from_keys", [("vr[t] = v + row * (size_t)D;", "vr[t] = k + row * (size_t)D;")]),
    ("query_of_kv_head",
     [("attend_one(q + ((size_t)b * Hq + h) * D, kr, vr, lens[b], D, scale,\n                       out + ((size_t)b * Hq + h) * D, &l_out, s);\n            if (lse) lse[(size_t)b * Hq + h] = l_out;\n        }\n    }\n    free(s); free(kr); free(vr);\n    return KVO_OK;\n}\n\n/*\n * Paged",
       "attend_one(q + ((size_t)b * Hq + g) * D, kr, vr, lens[b], D, scale,\n                       out + ((size_t)b * Hq + h) * D, &l_out, s);\n            if (lse) lse[(size_t)b * Hq + h] = l_out;\n        }\n    }\n    free(s); free(kr); free(vr);\n    return KVO_OK;\n}\n\n/*\n * Paged")]),
    ("combine_min_not_max", [("if (li > M) M = li;", "if (li < M || M == -INFINITY) M = li;")]),
    ("combine_unshifted_weights",
     [("wsum += exp(li - M);", "wsum += exp(li);")]),
    ("combine_drops_last_part",
     [("for (int i = 0; i < S; ++i) {\n                double li = lse_parts[(size_t)i * BH + bh];\n                if (li == -INFINITY) continue;\n                acc +=",
       "for (int i = 0; i < S - 1; ++i) {\n                double li = lse_parts[(size_t)i * BH + bh];\n                if (li == -INFINITY) continue;\n                acc +=")]),
]


# mistakes in the new-token preparation (RMS normalisation, rotary, placement)
APPEND_MUTANTS = [
    ("rms_sum_not_mean", [("sqrt(ss / (double)D + eps)", "sqrt(ss + eps)")]),
    ("rms_eps_outside_sqrt", [("sqrt(ss / (double)D + eps)", "(sqrt(ss / (double)D) + eps)")]),
    ("gain_reversed", [("tmp[d] * r * (double)w[d]", "tmp[d] * r * (double)w[D - 1 - d]")]),
    ("rotary_sign_flipped", [("y[i] = tmp[i] * c - tmp[i + half] * s;",
                              "y[i] = tmp[i] * c + tmp[i + half] * s;")]),
    ("rotary_wrong_partner", [("y[i] = tmp[i] * c - tmp[i + half] * s;",
                               "y[i] = tmp[i] * c - tmp[(i + half + 1) % D] * s;")]),
    ("rotary_exponent_without_two", [("pow(theta, -2.0 * (double)i / (double)D)",
                                      "pow(theta, -(double)i / (double)D)")]),
    ("rotary_position_plus_one", [("const double a = (double)pos * pow",
                                   "const double a = (double)(pos + 1) * pow")]),
    ("append_slot_off_by_one", [("row = (int64_t)page * page_size + pos % page_size;",
                                 "row = (int64_t)page * page_size + (pos + 1) % page_size;")]),
    ("append_page_of_previous_token",
     [("block_table[(size_t)b * max_pages + pos / page_size];\n                if (page >= 0",
       "block_table[(size_t)b * max_pages + (pos > 0 ? pos - 1 : 0) / page_size];\n                if (page >= 0")]),
    ("append_ignores_bad_page", [("if (page >= 0 && (int64_t)page < num_pages)", "if (1)")]),
    ("new_lens_always_grows", [("new_lens[b] = row >= 0 ? pos + 1 : pos;", "new_lens[b] = pos + 1;")]),
]


# mistakes in the fp8 cache path (format decode, scales, addressing)
FP8_MUTANTS = [
    ("fp8_exponent_bias_off_by_one", [("ldexp((double)(8 + m), e - 10)", "ldexp((double)(8 + m), e - 11)")]),
    ("fp8_subnormal_step", [("ldexp((double)m, -9)", "ldexp((double)m, -10)")]),
    ("fp8_no_nan_code", [("if (e == 15 && m == 7) return NAN;", "if (0) return NAN;")]),
    ("fp8_sign_ignored", [("return sign ? -v : v;", "return v;")]),
    ("fp8_key_scale_from_values",
     [("(k_scale * fp8_e4m3_to_f64(krow[t][d]))", "(v_scale * fp8_e4m3_to_f64(krow[t][d]))")]),
    ("fp8_value_scale_dropped",
     [("acc += s[t] * (v_scale * fp8_e4m3_to_f64(vrow[t][d]));",
       "acc += s[t] * fp8_e4m3_to_f64(vrow[t][d]);")]),
    ("fp8_paged_slot_off_by_one",
     [("row = ((size_t)page * (size_t)page_size + (size_t)(t % page_size)) *\n                              (size_t)Hkv",
       "row = ((size_t)page * (size_t)page_size + (size_t)((t + 1) % page_size)) *\n                              (size_t)Hkv")]),
]


# mistakes in chunked prefill (positions, query packing, the causal mask)
PREFILL_MUTANTS = [
    ("prefill_position_off_by_one", [("const int pos = lens[b] - nb + i;",
                                      "const int pos = lens[b] - nb + i - 1;")]),
    ("prefill_position_from_chunk_start", [("const int pos = lens[b] - nb + i;",
                                            "const int pos = i;")]),
    ("prefill_query_row_ignores_offset", [("const size_t row_q = (size_t)q_start[b] + (size_t)i;",
                                           "const size_t row_q = (size_t)i;")]),
    ("prefill_no_causal_mask", [("const int Lq = pos >= 0 ? pos + 1 : 0;",
                                 "const int Lq = lens[b];")]),
]


def _prefill_pins():
    import test_oracle_prefill as T
    return [
        T.test_one_token_chunk_is_decode_attention,
        lambda: T.test_every_token_is_decode_over_its_causal_prefix(16),
        T.test_whole_prompt_matches_torch_causal_sdpa,
        T.test_chunk_after_context_matches_masked_sdpa,
        T.test_empty_chunks_and_tokens_before_position_zero,
    ]


def _fp8_pins():
    import test_oracle_fp8 as T
    return [
        T.test_every_code_matches_torch_float8_e4m3fn,
        T.test_unit_scales_equal_the_bf16_oracle_bitwise,
        T.test_scales_fold_into_scores_and_outputs,
        T.test_nan_codes_past_the_length_are_never_read,
        T.test_paged_equals_numpy_gather_of_contiguous,
    ]


def _append_pins():
    import test_oracle_append as T
    return [
        T.test_rms_of_a_constant_row,
        T.test_rms_is_scale_invariant_without_eps,
        T.test_rms_gain_applies_per_dim,
        T.test_rms_of_zero_row_is_zero_and_no_gain_means_no_normalisation,
        T.test_rotary_at_position_zero_is_identity,
        lambda: T.test_rotary_pairs_dim_i_with_dim_i_plus_half(3),
        lambda: T.test_rotary_frequencies_are_theta_to_minus_2i_over_d(5),
        T.test_rotation_preserves_pair_norms,
        T.test_rotary_scores_depend_on_relative_position_only,
        T.test_values_pass_through_unchanged,
        T.test_append_row_is_what_attention_reads_as_position_L,
        T.test_append_skips_full_caches_and_bad_pages,
        T.test_append_contiguous_rows,
    ]


def _pins():
    import test_oracle_pins as T
    pins = [
        T.test_single_position_returns_that_value_row_exactly,
        lambda: T.test_uniform_weights_give_mean_of_values("zero_query"),
        lambda: T.test_uniform_weights_give_mean_of_values("zero_scale"),
        lambda: T.test_dominant_score_returns_that_row(17),
        T.test_empty_sequence_gives_zero_and_minus_inf,
        T.test_two_positions_logistic_weights,
        T.test_position_permutation_invariance,
        T.test_paged_equals_numpy_gather_of_contiguous,
        lambda: T.test_physical_page_remap_invariance(16),
        T.test_gqa_mapping_consecutive_heads_share_a_kv_head,
        T.test_key_shift_invariance_with_huge_scores,
        T.test_matches_torch_sdpa_ragged_batch,
        lambda: T.test_matches_mpmath_50_digits(8, 1.0),
        lambda: T.test_matches_mpmath_50_digits(7, 128.0),
        lambda: T.test_combine_of_disjoint_parts_equals_whole([0, 16, 17, 299, 300]),
        T.test_combine_identities,
        T.test_combine_with_huge_lse_spread_is_stable,
    ]
    return pins


def _child(lib_path, q, group="attn"):
    import ctypes
    import sys
    sys.path.insert(0, os.path.dirname(__file__))
    oracle._lib = None
    real = oracle._LIB
    oracle._LIB = lib_path
    oracle._SRC = lib_path                  # mtime check: never rebuild from the real source
    try:
        oracle._load()
    finally:
        oracle._LIB = real
    caught = 0
    pins = {"append": _append_pins, "fp8": _fp8_pins, "prefill": _prefill_pins}.get(group, _pins)()
    for pin in pins:
        try:
            pin()
        except Exception:
            caught += 1
    q.put(caught)


@pytest.mark.parametrize("name,edits,group",
                         [(n, e, "attn") for n, e in MUTANTS] +
                         [(n, e, "append") for n, e in APPEND_MUTANTS] +
                         [(n, e, "fp8") for n, e in FP8_MUTANTS] +
                         [(n, e, "prefill") for n, e in PREFILL_MUTANTS],
                         ids=[m[0] for m in MUTANTS] + [m[0] for m in APPEND_MUTANTS] +
                         [m[0] for m in FP8_MUTANTS] + [m[0] for m in PREFILL_MUTANTS])
def test_pins_reject_planted_mistake(name, edits, group, tmp_path):
    src = open(SRC).read()
    for old, new in edits:
        assert old in src, f"mutation anchor for {name} not found"
        src = src.replace(old, new)
    c = tmp_path / f"{name}.c"
    so = tmp_path / f"{name}.so"
    c.write_text(src)
    subprocess.run(["gcc", "-O2", "-std=c99", "-ffp-contract=off", "-fPIC", "-shared", "-o",
                    str(so), str(c), "-lm"], check=True)
    # children fork from a clean server process: forking this test process after
    # torch has started its thread pools can deadlock the child
    ctx = mp.get_context("forkserver")
    q = ctx.Queue()
    p = ctx.Process(target=_child, args=(str(so), q, group))
    p.start()
    p.join(300)
    if p.is_alive():
        p.kill()
        pytest.fail(f"mutant {name} hung")
    if p.exitcode != 0:
        return                                  # crashed: detected
    caught = q.get(timeout=5)
    assert caught >= 1, f"no pin rejects the planted mistake {name}"
