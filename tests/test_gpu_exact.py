"""Bit-exact GPU properties: single positions, dominant scores, page-table
indexing (gather hook), poison, page remap, determinism and GQA head mapping."""
import numpy as np
import pytest

import workloads as W
from kva_testlib import DeviceWorkload, assert_parity, bits_f64, dev, run_gpu, run_oracle

pytestmark = pytest.mark.gpu


def test_single_position_returns_value_row_bit_exact():
    print("[exact] L=1", flush=True)
    for layout in ("contig", "paged"):
        w = (W.make_contig([1] * 5, 8, key=(600,)) if layout == "contig"
             else W.make_paged([1] * 5, key=(600,)))
        out, _ = run_gpu(DeviceWorkload(w))
        for b in range(w.B):
            for h in range(w.Hq):
                if layout == "contig":
                    row = w.v[b, 0, h // 4]
                else:
                    row = w.v[w.block_table[b, 0], 0, h // 4]
                assert np.array_equal(out[b, h].astype(np.float64), bits_f64(row)), (layout, b, h)


PROBE_POSITIONS = [0, 1, 15, 16, 17, 31, 32, 255, 256, 4095, 4096, 4097, 8191, 8192, 12000, 16383]


@pytest.mark.parametrize("layout", ["contig", "paged"])
def test_dominant_score_returns_that_row_bit_exact(layout):
    """Sequence b holds a key aligned with the query of KV head g = b % 8 whose
    score is ~2900 natural-log units above the rest, at position t*_b; the four
    query heads of g must return V[t*_b] bit for bit, whichever wave or split
    the position falls in."""
    print(f"[exact] dominant probes {layout}", flush=True)
    L = 16384
    n = len(PROBE_POSITIONS)
    w = (W.make_contig([L] * n, L, key=(601,)) if layout == "contig"
         else W.make_paged([L] * n, key=(601,)))
    for b, ts in enumerate(PROBE_POSITIONS):
        g = b % 8
        u = w.q[b, 4 * g].copy()
        w.q[b, 4 * g:4 * g + 4] = u
        big = W.bf16_bits(W.bits_to_f32(u) * np.float32(256.0))
        if layout == "contig":
            w.k[b, ts, g] = big
        else:
            w.k[w.block_table[b, ts // 16], ts % 16, g] = big
    out, _ = run_gpu(DeviceWorkload(w))
    for b, ts in enumerate(PROBE_POSITIONS):
        g = b % 8
        row = w.v[b, ts, g] if layout == "contig" else w.v[w.block_table[b, ts // 16], ts % 16, g]
        for h in range(4 * g, 4 * g + 4):
            assert np.array_equal(out[b, h].astype(np.float64), bits_f64(row)), (b, ts, h)
    ref, _ = run_oracle(w)
    assert_parity(out, ref, tag="dominant probes")


@pytest.mark.parametrize("k", [3, 4, 5])
def test_gather_hook_is_bit_exact(k):
    """kva_debug_gather_paged (same page-address code as the attention kernels)
    against a numpy fancy-index gather of the pool, on the paged configs."""
    import torch
    import paper_2609_12471_amd as kva
    print(f"[exact] gather config {k}", flush=True)
    w = W.make_config(k)
    pool = dev(w.k)
    bt_all = w.block_table
    step = 16
    for b0 in range(0, w.B, step):
        b1 = min(w.B, b0 + step)
        lens = w.seq_lens[b0:b1]
        Lcap = int(lens.max()) + 3
        dst = torch.full((b1 - b0, Lcap, w.Hkv, w.D), 0x1234, dtype=torch.int16, device="cuda")
        kva.kva_debug_gather_paged(pool, dev(bt_all[b0:b1]), dev(lens), dst)
        got = dst.cpu().numpy().view(np.uint16)
        for i, L in enumerate(lens):
            t = np.arange(L)
            exp = w.k[bt_all[b0 + i, t // 16], t % 16]
            assert np.array_equal(got[i, :L], exp), (k, b0 + i)
            assert np.all(got[i, L:] == 0)


def test_gather_small_pages_and_bad_ids():
    import torch
    import paper_2609_12471_amd as kva
    for P in (1, 4, 64):
        w = W.make_paged([1, 5, 64, 130], page_size=P, Hq=8, Hkv=2, key=(602, P))
        Lcap = 140
        dst = torch.zeros((w.B, Lcap, w.Hkv, w.D), dtype=torch.int16, device="cuda")
        kva.kva_debug_gather_paged(dev(w.k), dev(w.block_table), dev(w.seq_lens), dst)
        got = dst.cpu().numpy().view(np.uint16)
        for b, L in enumerate(w.seq_lens):
            t = np.arange(L)
            assert np.array_equal(got[b, :L], w.k[w.block_table[b, t // P], t % P])
    # ids outside [0, num_pages) read page 0 instead of faulting
    w = W.make_paged([32], page_size=16, Hq=8, Hkv=2, key=(603,))
    bt = w.block_table.copy()
    bt[0, 0] = -7
    bt[0, 1] = w.num_pages + 100
    dst = torch.zeros((1, 32, 2, 128), dtype=torch.int16, device="cuda")
    kva.kva_debug_gather_paged(dev(w.k), dev(bt), dev(w.seq_lens), dst)
    got = dst.cpu().numpy().view(np.uint16)
    assert np.array_equal(got[0, :16], w.k[0]) and np.array_equal(got[0, 16:], w.k[0])


@pytest.mark.parametrize("layout", ["contig", "paged"])
def test_poison_never_reaches_the_output(layout):
    """NaN in rows past each length, page tails and spare pages: the output is
    bitwise equal to the run whose unused memory holds zeros."""
    print(f"[exact] poison {layout}", flush=True)
    lens = [1, 15, 17, 33, 250, 1001, 3000]
    mk = (lambda p: W.make_contig(lens, 3008, key=(604,), poison=p)) if layout == "contig" else \
         (lambda p: W.make_paged(lens, key=(604,), poison=p))
    a, b = mk(True), mk(False)
    out_a, lse_a = run_gpu(DeviceWorkload(a))
    out_b, lse_b = run_gpu(DeviceWorkload(b))
    assert np.all(np.isfinite(out_a))
    assert np.array_equal(out_a, out_b) and np.array_equal(lse_a, lse_b)


def test_physical_page_remap_is_bitwise_invariant():
    print("[exact] remap", flush=True)
    w = W.make_config(3)
    out, lse = run_gpu(DeviceWorkload(w))
    rng = np.random.default_rng(605)
    perm = rng.permutation(w.num_pages)
    k2 = np.empty_like(w.k); v2 = np.empty_like(w.v)
    k2[perm] = w.k; v2[perm] = w.v
    w.block_table = np.where(w.block_table >= 0, perm[np.maximum(w.block_table, 0)], -1).astype(np.int32)
    w.k, w.v = k2, v2
    out2, lse2 = run_gpu(DeviceWorkload(w))
    assert np.array_equal(out, out2) and np.array_equal(lse, lse2)


def test_repeated_calls_are_bitwise_identical():
    print("[exact] determinism", flush=True)
    w = W.make_config(2)
    dw = DeviceWorkload(w)
    out1, lse1 = run_gpu(dw)
    out2, lse2 = run_gpu(dw)
    assert np.array_equal(out1, out2) and np.array_equal(lse1, lse2)


def test_gqa_mapping_exact_zeros():
    """V nonzero only on KV head g*: query heads outside 4g*..4g*+3 are exactly 0."""
    w = W.make_paged([100, 1000], key=(606,))
    gs = 3
    live = w.v != W.BF16_NAN
    for g in range(8):
        if g != gs:
            w.v[:, :, g][live[:, :, g]] = 0
    out, _ = run_gpu(DeviceWorkload(w))
    for h in range(32):
        if h // 4 == gs:
            assert np.all(np.abs(out[:, h]).max(axis=-1) > 0)
        else:
            assert np.all(out[:, h] == 0.0)


def test_huge_scores_stay_finite_and_match():
    """Keys shifted by a common vector so scores reach ~1e3 (exp would overflow
    without the running maximum): finite, and equal to the oracle."""
    print("[exact] huge scores", flush=True)
    rng = np.random.default_rng(607)
    lens = [40, 300, 2000]
    w = W.make_contig(lens, 2000, key=(607,), poison=False)
    qi = rng.integers(0, 4, size=(3, 32, 128)).astype(np.float32)
    w.q[:] = W.bf16_bits(qi)
    base = rng.integers(-3, 4, size=w.k.shape).astype(np.float32)
    w.k[:] = W.bf16_bits(base + np.float32(64.0))
    out, lse = run_gpu(DeviceWorkload(w))
    ref, rlse = run_oracle(w)
    assert np.all(np.isfinite(out)) and np.min(rlse) > 700
    # scores of ~1e3 carry fp32 rounding of ~1e-4 in absolute terms, which the
    # softmax turns into relative weight errors of the same size: gate only
    assert_parity(out, ref, tag="huge scores", diag=False)
    np.testing.assert_allclose(lse, rlse, rtol=2e-6, atol=0)
