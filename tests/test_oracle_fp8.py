"""Pins of the oracle's fp8 (OCP E4M3, e4m3fn) cache path.

* the value of every code against torch's float8_e4m3fn (a library routine);
* with unit scales, fp8 attention equals the bf16 oracle on the same values
  (every e4m3fn value is exactly a bf16 value), bitwise;
* the two scales enter where they must: k_scale folds into the score scale and
  v_scale multiplies the output (an identity of the definition);
* NaN codes past a sequence's length are never read; paged equals a numpy
  gather of the contiguous layout."""
import numpy as np
import pytest

import oracle
import workloads as W


def test_every_code_matches_torch_float8_e4m3fn():
    import torch
    ref = torch.arange(256, dtype=torch.int32).to(torch.uint8).view(torch.float8_e4m3fn)
    ref = ref.to(torch.float64).numpy()
    got = oracle.fp8_table()
    assert np.array_equal(got, ref, equal_nan=True)
    # a few values by hand: 1.0, largest finite, smallest subnormal, smallest normal, NaN
    assert got[0x38] == 1.0 and got[0x7E] == 448.0 and got[0xFE] == -448.0
    assert got[0x01] == 2.0 ** -9 and got[0x08] == 2.0 ** -6
    assert np.isnan(got[0x7F]) and np.isnan(got[0xFF])


def _fp8_case(lens, Lmax, key, **kw):
    w = W.make_contig(lens, Lmax, key=key, **kw)
    return w, W.to_fp8_codes(w.k, W.FP8_K_SCALE), W.to_fp8_codes(w.v, W.FP8_V_SCALE)


def _bf16_of_codes(codes):
    """bf16 bits of the fp8 values (exact: e4m3fn values have 4 significant bits)."""
    vals = oracle.fp8_table()[codes].astype(np.float32)
    return W.bf16_bits(vals)


def test_unit_scales_equal_the_bf16_oracle_bitwise():
    lens = np.array([1, 17, 300, 0, 1000], np.int32)
    w, k8, v8 = _fp8_case(lens, 1000, (5100,))
    out8, lse8 = oracle.decode_attn_fp8(w.q, k8, v8, lens, w.scale, 1.0, 1.0)
    kb, vb = _bf16_of_codes(k8), _bf16_of_codes(v8)
    out, lse = oracle.decode_attn(w.q, kb, vb, lens, w.scale)
    assert np.array_equal(out8, out)
    assert np.array_equal(lse8, lse)


def test_scales_fold_into_scores_and_outputs():
    lens = np.array([5, 64, 777], np.int32)
    w, k8, v8 = _fp8_case(lens, 777, (5200,))
    a, c = 0.0371, 2.6
    out, lse = oracle.decode_attn_fp8(w.q, k8, v8, lens, w.scale, a, c)
    out1, lse1 = oracle.decode_attn_fp8(w.q, k8, v8, lens, w.scale * a, 1.0, 1.0)
    np.testing.assert_allclose(out, c * out1, rtol=1e-12, atol=1e-12 * np.abs(out).max())
    np.testing.assert_allclose(lse, lse1, rtol=1e-12, atol=1e-15)
    # and they are not interchangeable
    outs, _ = oracle.decode_attn_fp8(w.q, k8, v8, lens, w.scale, c, a)
    assert np.max(np.abs(outs - out)) > 1e-3


def test_nan_codes_past_the_length_are_never_read():
    lens = np.array([3, 100, 64], np.int32)
    w, k8, v8 = _fp8_case(lens, 128, (5300,))          # rows past L hold NaN codes
    assert np.isnan(oracle.fp8_table()[k8[0, 3:]]).all()
    out, lse = oracle.decode_attn_fp8(w.q, k8, v8, lens, w.scale, W.FP8_K_SCALE, W.FP8_V_SCALE)
    assert np.isfinite(out).all() and np.isfinite(lse).all()


def test_paged_equals_numpy_gather_of_contiguous():
    lens = np.array([40, 0, 333, 16, 95], np.int32)
    wp = W.quantize_fp8(W.make_paged(lens, page_size=16, key=(5400,)))
    P = wp.page_size
    Lmax = int(lens.max())
    kc = np.zeros((len(lens), Lmax, wp.Hkv, wp.D), np.uint8)
    vc = np.zeros_like(kc)
    for b, L in enumerate(lens):
        t = np.arange(L)
        kc[b, :L] = wp.k[wp.block_table[b, t // P], t % P]
        vc[b, :L] = wp.v[wp.block_table[b, t // P], t % P]
    ks, vs = wp.meta["k_scale"], wp.meta["v_scale"]
    outp, lsep = oracle.decode_attn_fp8(wp.q, wp.k, wp.v, lens, wp.scale, ks, vs,
                                        block_table=wp.block_table)
    outc, lsec = oracle.decode_attn_fp8(wp.q, kc, vc, lens, wp.scale, ks, vs)
    assert np.array_equal(outp, outc) and np.array_equal(lsep, lsec)


def test_quantised_cache_is_close_to_the_bf16_one():
    """Sanity of the generator (not of the oracle): e4m3 keeps ~4 significant
    bits, so attention over the fp8 cache stays within a few percent."""
    lens = np.array([512, 2048], np.int32)
    w, k8, v8 = _fp8_case(lens, 2048, (5500,))
    out8, _ = oracle.decode_attn_fp8(w.q, k8, v8, lens, w.scale, W.FP8_K_SCALE, W.FP8_V_SCALE)
    out, _ = oracle.decode_attn(w.q, w.k, w.v, lens, w.scale)
    rel = np.linalg.norm(out8 - out) / np.linalg.norm(out)
    assert rel < 0.08, rel
