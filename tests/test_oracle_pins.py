"""Pins for the fp64 oracle: closed forms, invariants, reductions to library
routines and 50-digit brute force.  None of these re-types the oracle's own
formula in binary64; each is chosen so that a plausible slip in the oracle (a
dropped max-subtraction, a wrong sign, a wrong head or position index, a
transposed operand, a missing scale or log) fails at least one of them.
"""
import math

import mpmath
import numpy as np
import pytest
import torch

import oracle
import workloads as W

D = 128


def f64(bits):
    return W.bits_to_f32(bits).astype(np.float64)


def small_contig(lens, Lmax, Hq=8, Hkv=2, key=(77,), scale=W.SCALE, poison=True):
    return W.make_contig(lens, Lmax, Hq=Hq, Hkv=Hkv, D=D, key=key, scale=scale, poison=poison)


def run(w, scale=None):
    s = w.scale if scale is None else scale
    if w.layout == "contig":
        return oracle.decode_attn(w.q, w.k, w.v, w.seq_lens, s)
    return oracle.decode_attn_paged(w.q, w.k, w.v, w.block_table, w.seq_lens, s)


# ---------------------------------------------------------------- closed forms

def test_single_position_returns_that_value_row_exactly():
    w = small_contig([1, 1, 1], 4, Hq=8, Hkv=2)
    out, lse = run(w)
    grp = w.Hq // w.Hkv
    for b in range(w.B):
        for h in range(w.Hq):
            assert np.array_equal(out[b, h], f64(w.v[b, 0, h // grp]))
    assert np.all(np.isfinite(lse))


@pytest.mark.parametrize("how", ["zero_query", "zero_scale"])
def test_uniform_weights_give_mean_of_values(how):
    lens = [1, 5, 33, 64]
    w = small_contig(lens, 64, Hq=8, Hkv=2, key=(78,))
    scale = w.scale
    if how == "zero_query":
        w.q[:] = 0
    else:
        scale = 0.0
    out, lse = run(w, scale)
    grp = w.Hq // w.Hkv
    for b, L in enumerate(lens):
        for h in range(w.Hq):
            ref = np.mean(f64(w.v[b, :L, h // grp]), axis=0, dtype=np.float64)
            np.testing.assert_allclose(out[b, h], ref, rtol=0, atol=1e-15)
            assert lse[b, h] == pytest.approx(math.log(L), abs=1e-14)


@pytest.mark.parametrize("tstar", [0, 15, 16, 17, 100, 255])
def test_dominant_score_returns_that_row(tstar):
    L = 256
    w = small_contig([L], L, Hq=4, Hkv=1, key=(79,))
    u = w.q[0, 0].copy()
    w.q[0, :] = u                                    # all four heads query with u
    # 64 * u is exact in bf16 (exponent shift); its score is ~64 * 128 * scale
    w.k[0, tstar, 0] = W.bf16_bits(W.bits_to_f32(u) * np.float32(64.0))
    out, lse = run(w)
    for h in range(4):
        np.testing.assert_allclose(out[0, h], f64(w.v[0, tstar, 0]), rtol=0, atol=1e-15)
    # the log-sum-exp is dominated by the same score
    s_star = w.scale * float(np.dot(f64(u), f64(w.k[0, tstar, 0])))
    assert lse[0, 0] == pytest.approx(s_star, rel=1e-12)


def test_empty_sequence_gives_zero_and_minus_inf():
    w = small_contig([0, 3], 4, key=(80,))
    out, lse = run(w)
    assert np.all(out[0] == 0.0) and np.all(np.isneginf(lse[0]))
    assert np.all(np.isfinite(out[1])) and np.all(np.isfinite(lse[1]))


def test_two_positions_logistic_weights():
    """With two keys the softmax weight of key 0 is the logistic of s0 - s1."""
    w = small_contig([2], 2, Hq=1, Hkv=1, key=(81,))
    out, _ = run(w)
    q = f64(w.q[0, 0]); k0 = f64(w.k[0, 0, 0]); k1 = f64(w.k[0, 1, 0])
    v0 = f64(w.v[0, 0, 0]); v1 = f64(w.v[0, 1, 0])
    delta = w.scale * (float(np.dot(q, k0)) - float(np.dot(q, k1)))
    p0 = 1.0 / (1.0 + math.exp(-delta))
    np.testing.assert_allclose(out[0, 0], p0 * v0 + (1.0 - p0) * v1, rtol=0, atol=1e-14)


# ---------------------------------------------------------------- invariants

def test_position_permutation_invariance():
    lens = [37, 200]
    w = small_contig(lens, 200, key=(82,))
    out, lse = run(w)
    rng = np.random.default_rng(5)
    w2 = small_contig(lens, 200, key=(82,))
    for b, L in enumerate(lens):
        p = rng.permutation(L)
        w2.k[b, :L] = w.k[b, p]
        w2.v[b, :L] = w.v[b, p]
    out2, lse2 = run(w2)
    np.testing.assert_allclose(out2, out, rtol=0, atol=1e-13)
    np.testing.assert_allclose(lse2, lse, rtol=1e-13, atol=0)


def test_paged_equals_numpy_gather_of_contiguous():
    lens = [1, 16, 17, 300, 0, 31]
    w = W.make_paged(lens, page_size=16, Hq=8, Hkv=2, key=(83,))
    out_p, lse_p = run(w)
    Lmax = max(lens)
    k = np.zeros((w.B, Lmax, w.Hkv, D), np.uint16)
    v = np.zeros_like(k)
    for b, L in enumerate(lens):
        t = np.arange(L)
        rows_page = w.block_table[b, t // 16]
        k[b, :L] = w.k[rows_page, t % 16]
        v[b, :L] = w.v[rows_page, t % 16]
    out_c, lse_c = oracle.decode_attn(w.q, k, v, w.seq_lens, w.scale)
    assert np.array_equal(out_p, out_c) and np.array_equal(lse_p, lse_c)


@pytest.mark.parametrize("page_size", [1, 4, 16, 64])
def test_physical_page_remap_invariance(page_size):
    lens = [5, 64, 129, 250]
    w = W.make_paged(lens, page_size=page_size, Hq=8, Hkv=2, key=(84, page_size))
    out, lse = run(w)
    rng = np.random.default_rng(6)
    perm = rng.permutation(w.num_pages)              # new id of old page i is perm[i]
    k2 = np.empty_like(w.k); v2 = np.empty_like(w.v)
    k2[perm] = w.k; v2[perm] = w.v
    bt2 = np.where(w.block_table >= 0, perm[np.maximum(w.block_table, 0)], -1).astype(np.int32)
    out2, lse2 = oracle.decode_attn_paged(w.q, k2, v2, bt2, w.seq_lens, w.scale)
    assert np.array_equal(out, out2) and np.array_equal(lse, lse2)


def test_gqa_mapping_consecutive_heads_share_a_kv_head():
    Hq, Hkv = 32, 8
    w = small_contig([50, 9], 64, Hq=Hq, Hkv=Hkv, key=(85,))
    gstar = 5
    for g in range(Hkv):
        if g != gstar:
            w.v[:, :, g] = 0
    out, _ = run(w)
    grp = Hq // Hkv
    for h in range(Hq):
        if h // grp == gstar:
            assert np.all(np.abs(out[:, h]).max(axis=-1) > 0)
        else:
            assert np.all(out[:, h] == 0.0)
    # heads of g* never read other KV heads: poisoning them leaves g* unchanged
    w2 = small_contig([50, 9], 64, Hq=Hq, Hkv=Hkv, key=(85,))
    w2.v[:] = w.v
    for g in range(Hkv):
        if g != gstar:
            w2.k[:, :, g] = W.BF16_NAN
            w2.v[:, :, g] = W.BF16_NAN
    out2, _ = run(w2)
    sl = slice(gstar * grp, (gstar + 1) * grp)
    assert np.array_equal(out2[:, sl], out[:, sl])


def test_key_shift_invariance_with_huge_scores():
    """Adding the same vector u to every key shifts each head's scores by the
    constant scale*q.u, which the softmax ignores.  With |scale*q.u| ~ 1e3 an
    implementation without max-subtraction overflows; the output must not move
    and lse must shift by exactly that constant (up to rounding)."""
    L = 40
    rng = np.random.default_rng(7)
    w = small_contig([L], L, Hq=4, Hkv=1, key=(86,), poison=False)
    # keys built as small integers so K and K+u are exact in bf16 and binary64
    base = rng.integers(-3, 4, size=(L, D)).astype(np.float32)
    u = np.full(D, 64.0, np.float32)
    qi = rng.integers(0, 4, size=(4, D)).astype(np.float32)
    qi[2:] *= -1                                     # two heads shift up, two down
    w.q[0] = W.bf16_bits(qi)
    w.k[0, :, 0] = W.bf16_bits(base)
    out, lse = run(w)
    w.k[0, :, 0] = W.bf16_bits(base + u)
    out2, lse2 = run(w)
    qf = f64(w.q[0])
    shift = w.scale * (qf @ u.astype(np.float64))
    assert np.all(np.isfinite(out2)) and np.min(np.abs(shift)) > 750
    np.testing.assert_allclose(out2[0], out[0], rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse2[0], lse[0] + shift, rtol=1e-12, atol=1e-9)


# ---------------------------------------------------------------- library routines and brute force

def _sdpa_reference(w):
    """torch's scaled_dot_product_attention in float64 with enable_gqa, plus a
    logsumexp of the masked scores, on the gathered rows."""
    B, Hq, Hkv = w.B, w.Hq, w.Hkv
    Lmax = w.k.shape[1]
    q = torch.from_numpy(f64(w.q)).reshape(B, Hq, 1, D)
    valid = np.arange(Lmax)[None, :] < w.seq_lens[:, None]
    kf = np.where(valid[:, :, None, None], f64(w.k), 0.0)
    vf = np.where(valid[:, :, None, None], f64(w.v), 0.0)
    k = torch.from_numpy(kf).permute(0, 2, 1, 3).contiguous()
    v = torch.from_numpy(vf).permute(0, 2, 1, 3).contiguous()
    mask = torch.from_numpy(valid).reshape(B, 1, 1, Lmax)
    out = torch.nn.functional.scaled_dot_product_attention(
        q, k, v, attn_mask=mask, scale=w.scale, enable_gqa=True)
    kk = k.repeat_interleave(Hq // Hkv, dim=1)
    scores = (q @ kk.transpose(-1, -2)) * w.scale
    scores = scores.masked_fill(~mask, float("-inf"))
    lse = torch.logsumexp(scores, dim=-1)
    return out.reshape(B, Hq, D).numpy(), lse.reshape(B, Hq).numpy()


def test_matches_torch_sdpa_on_config_1():
    w = W.make_config(1)
    out, lse = run(w)
    ref, rlse = _sdpa_reference(w)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-13)
    np.testing.assert_allclose(lse, rlse, rtol=1e-13, atol=0)


def test_matches_torch_sdpa_ragged_batch():
    lens = [1, 2, 15, 16, 17, 100, 333, 512]
    w = small_contig(lens, 512, Hq=32, Hkv=8, key=(87,))
    out, lse = run(w)
    ref, rlse = _sdpa_reference(w)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-13)
    np.testing.assert_allclose(lse, rlse, rtol=1e-13, atol=0)


def _mp_reference(q, K, V, scale):
    mpmath.mp.dps = 50
    s = [mpmath.mpf(scale) * mpmath.fsum(mpmath.mpf(a) * mpmath.mpf(b) for a, b in zip(q, k))
         for k in K]
    m = max(s)
    w = [mpmath.exp(x - m) for x in s]
    l = mpmath.fsum(w)
    out = [mpmath.fsum(wi * mpmath.mpf(vi[d]) for wi, vi in zip(w, V)) / l for d in range(len(q))]
    return [float(o) for o in out], float(m + mpmath.log(l))


@pytest.mark.parametrize("L,qmul", [(1, 1.0), (3, 1.0), (8, 1.0), (5, 32.0), (7, 128.0)])
def test_matches_mpmath_50_digits(L, qmul):
    """Tiny inputs against 50-digit arithmetic.  qmul scales q by a power of two
    (exact in bf16) so that scores reach several hundred; exp of such scores
    overflows binary64 unless the maximum is subtracted first."""
    w = small_contig([L], 8, Hq=4, Hkv=2, key=(88, L))
    w.q[:] = W.bf16_bits(W.bits_to_f32(w.q) * np.float32(qmul))
    out, lse = run(w)
    assert np.all(np.isfinite(out))
    for h in range(4):
        g = h // 2
        ref, rlse = _mp_reference(f64(w.q[0, h]), f64(w.k[0, :L, g]), f64(w.v[0, :L, g]), w.scale)
        np.testing.assert_allclose(out[0, h], ref, rtol=0, atol=1e-13)
        assert lse[0, h] == pytest.approx(rlse, rel=1e-13)


# ---------------------------------------------------------------- split / combine

@pytest.mark.parametrize("cuts", [[0, 300], [0, 1, 300], [0, 0, 150, 150, 300], [0, 16, 17, 299, 300]])
def test_combine_of_disjoint_parts_equals_whole(cuts):
    L = 300
    w = small_contig([L], L, Hq=8, Hkv=2, key=(89,))
    whole, wlse = run(w)
    parts, plse = [], []
    for a, b in zip(cuts[:-1], cuts[1:]):
        part = small_contig([b - a], L, Hq=8, Hkv=2, key=(89,))
        part.k[0, :b - a] = w.k[0, a:b]
        part.v[0, :b - a] = w.v[0, a:b]
        o, l = run(part)
        parts.append(o); plse.append(l)
    out, lse = oracle.combine(np.stack(parts), np.stack(plse))
    np.testing.assert_allclose(out, whole, rtol=0, atol=1e-13)
    np.testing.assert_allclose(lse, wlse, rtol=1e-13, atol=0)


def test_combine_identities():
    rng = np.random.default_rng(9)
    o = rng.standard_normal((1, 3, 4, D))
    l = rng.standard_normal((1, 3, 4))
    out, lse = oracle.combine(o, l)
    assert np.array_equal(out, o[0]) and np.array_equal(lse, l[0])
    out2, lse2 = oracle.combine(np.concatenate([o, o]), np.concatenate([l, l]))
    np.testing.assert_allclose(out2, o[0], rtol=0, atol=1e-15)
    np.testing.assert_allclose(lse2, l[0] + math.log(2.0), rtol=0, atol=1e-14)
    empty = np.full((2, 3, 4), -np.inf)
    out3, lse3 = oracle.combine(np.zeros((2, 3, 4, D)), empty)
    assert np.all(out3 == 0.0) and np.all(np.isneginf(lse3))


def test_combine_with_huge_lse_spread_is_stable():
    """Parts whose log-sum-exps differ by ~1600 must merge without overflow:
    the largest part dominates exactly and the merged lse equals it."""
    rng = np.random.default_rng(10)
    o = rng.standard_normal((3, 1, 2, D))
    l = np.array([[[800.0, -3.0]], [[-800.0, -3.0]], [[5.0, -3.0]]])
    out, lse = oracle.combine(o, l)
    np.testing.assert_allclose(out[0, 0], o[0, 0, 0], rtol=0, atol=1e-15)
    assert lse[0, 0] == 800.0
    np.testing.assert_allclose(out[0, 1], o[:, 0, 1].mean(axis=0), rtol=0, atol=1e-15)
    assert lse[0, 1] == pytest.approx(-3.0 + math.log(3.0), abs=1e-14)


# ---------------------------------------------------------------- argument checking

def test_oracle_rejects_out_of_range_lengths_and_pages():
    w = small_contig([3], 4, key=(90,))
    with pytest.raises(ValueError):
        oracle.decode_attn(w.q, w.k, w.v, np.array([5], np.int32), w.scale)
    p = W.make_paged([20], page_size=16, Hq=8, Hkv=2, key=(91,))
    bt = p.block_table.copy(); bt[0, 1] = p.num_pages
    with pytest.raises(ValueError):
        oracle.decode_attn_paged(p.q, p.k, p.v, bt, p.seq_lens, p.scale)
