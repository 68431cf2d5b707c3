"""The seeded input generator: determinism, ranges, page tables, poison, and
consistency of the five rollout-shaped configs with the shapes the paper
prints for its RL runs (tests/golden/rollout_shapes.json)."""
import json
import os

import numpy as np
import pytest

import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "rollout_shapes.json")


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.0 + 2**-8, 1.0 + 3 * 2**-8, -2.5, 1.0 + 2**-9], np.float32)
    got = W.bits_to_f32(W.bf16_bits(x))
    assert list(got) == [1.0, 1.0, 1.0 + 2**-6, -2.5, 1.0]   # ties to even, else nearest


def test_generator_is_deterministic_and_thread_independent():
    ss = np.random.SeedSequence([1, 2, 3])
    a = W.normal_bf16(ss, 20000, 2, 128, threads=1)
    b = W.normal_bf16(np.random.SeedSequence([1, 2, 3]), 20000, 2, 128, threads=4)
    assert np.array_equal(a, b)
    x = W.bits_to_f32(a).astype(np.float64)
    rms = np.sqrt(np.mean(x * x, axis=-1))
    assert np.all(np.abs(rms - 1.0) < 1e-2)


@pytest.mark.parametrize("k", [1, 2])
def test_contig_configs(k):
    w = W.make_config(k)
    assert w.layout == "contig" and w.Hq == 32 and w.Hkv == 8 and w.D == 128
    lo, hi = {1: (256, 256), 2: (1024, 4096)}[k]
    assert np.all((w.seq_lens >= lo) & (w.seq_lens <= hi))
    for b in range(w.B):
        L = int(w.seq_lens[b])
        assert np.all(w.k[b, L:] == W.BF16_NAN) and np.all(w.v[b, L:] == W.BF16_NAN)
        assert not np.any(w.k[b, :L] == W.BF16_NAN)


def test_config_lengths_ranges():
    l3 = W.config_lengths(3); l4 = W.config_lengths(4); l5 = W.config_lengths(5)
    assert l3.shape == (64,) and l3.min() >= 512 and l3.max() <= 8192
    assert l4.shape == (256,) and l4.min() >= 256 and l4.max() <= 16384
    assert 2000 < np.median(l4) < 4000 and np.sum(l4 > 8192) >= 5
    assert l5.shape == (128,) and l5.min() >= 2048 + 256 and l5.max() <= 2048 + 8192
    assert np.array_equal(l3, W.config_lengths(3))


def test_paged_table_is_a_valid_shuffled_allocation():
    lens = [1, 16, 17, 100, 0, 250]
    w = W.make_paged(lens, page_size=16, Hq=8, Hkv=2, key=(5,))
    used = []
    for b, L in enumerate(lens):
        n = (L + 15) // 16
        assert np.all(w.block_table[b, :n] >= 0) and np.all(w.block_table[b, n:] == -1)
        used.extend(w.block_table[b, :n].tolist())
        if L % 16:
            tail = w.k[w.block_table[b, n - 1], L % 16:]
            assert np.all(tail == W.BF16_NAN)
    assert len(set(used)) == len(used)                       # no page used twice
    spare = sorted(set(range(w.num_pages)) - set(used))
    assert len(spare) >= 1 and np.all(w.k[spare] == W.BF16_NAN)
    assert used != sorted(used)                              # shuffled


def test_shared_prefix_pages_are_shared_within_a_group():
    lens = [40, 50, 64, 33, 70, 80]
    w = W.make_paged(lens, page_size=16, Hq=8, Hkv=2, key=(6,), shared_prefix=(3, 32))
    for grp in (0, 3):
        assert np.array_equal(w.block_table[grp, :2], w.block_table[grp + 1, :2])
        assert np.array_equal(w.block_table[grp, :2], w.block_table[grp + 2, :2])
        assert w.block_table[grp, 2] != w.block_table[grp + 1, 2]
    assert not np.array_equal(w.block_table[0, :2], w.block_table[3, :2])
    assert w.kv_bytes_unique() < w.kv_bytes_logical()


def test_configs_follow_the_papers_rollout_shapes():
    g = json.load(open(GOLDEN))
    tri, hip = g["triton_rl"], g["hip_rl"]
    G = tri["group_size"]
    # config 3: 8 prompts x G samples, lengths up to the HIP RL sequence length
    assert len(W.config_lengths(3)) == 8 * G and W.config_lengths(3).max() <= hip["sequence_length"]
    # config 4: lengths clipped at the Triton RL sequence length
    assert W.config_lengths(4).max() <= tri["sequence_length"]
    # config 5: 16 prompts x G samples sharing each prompt's prefix
    assert len(W.config_lengths(5)) == 16 * G
    assert W.config_lengths(5).max() <= tri["sequence_length"]
