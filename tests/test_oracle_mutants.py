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


def _child(lib_path, q):
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
    for pin in _pins():
        try:
            pin()
        except Exception:
            caught += 1
    q.put(caught)


@pytest.mark.parametrize("name,edits", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_reject_planted_mistake(name, edits, tmp_path):
    src = open(SRC).read()
    for old, new in edits:
        assert old in src, f"mutation anchor for {name} not found"
        src = src.replace(old, new)
    c = tmp_path / f"{name}.c"
    so = tmp_path / f"{name}.so"
    c.write_text(src)
    subprocess.run(["gcc", "-O2", "-std=c99", "-ffp-contract=off", "-fPIC", "-shared", "-o",
                    str(so), str(c), "-lm"], check=True)
    ctx = mp.get_context("fork")
    q = ctx.Queue()
    p = ctx.Process(target=_child, args=(str(so), q))
    p.start()
    p.join(300)
    if p.is_alive():
        p.kill()
        pytest.fail(f"mutant {name} hung")
    if p.exitcode != 0:
        return                                  # crashed: detected
    caught = q.get(timeout=5)
    assert caught >= 1, f"no pin rejects the planted mistake {name}"
