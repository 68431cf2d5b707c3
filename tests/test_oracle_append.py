"""Pins of the oracle's new-token preparation (RMS normalisation of q and k,
rotary position embedding, placement of the new k/v row in the cache).

Each test fixes the oracle against something other than itself: closed forms
(constant rows, one-hot vectors, frequencies made exact by a power-of-two
theta), invariants (scale invariance of RMS normalisation, rotation preserves
pair norms, attention scores depend on relative position only) and a cross-pin
through the attention oracle (the row the append writes is the row attention
reads as position L)."""
import numpy as np
import pytest

import oracle
import workloads as W

D = 128
HALF = D // 2


def bf(x):
    """float values that bf16 represents exactly -> bf16 bits."""
    f = np.ascontiguousarray(np.asarray(x, np.float32))
    u = f.view(np.uint32)
    assert np.all((u & 0xFFFF) == 0), "value not exactly representable in bf16"
    return (u >> 16).astype(np.uint16)


def rand_rows(seed, n, heads):
    return W.normal_bf16(np.random.SeedSequence([4242, seed]), n, heads, D)


def run_q(x_bits, w=None, *, eps=1e-6, theta=-1.0, pos=0):
    """The oracle on one query row (B = 1, Hq = Hkv = 1, contiguous)."""
    q = np.ascontiguousarray(x_bits.reshape(1, 1, D))
    z = np.zeros((1, 1, D), np.uint16)
    qo, _, _, _, _ = oracle.append(q, z, z, w, None, np.array([pos], np.int32), Lmax=pos + 1,
                                   eps=eps, theta=theta)
    return qo[0, 0]


# ------------------------------------------------------------------ RMS normalisation

def test_rms_of_a_constant_row():
    x = bf(np.full(D, 0.5))
    ones = np.ones(D, np.float32)
    # mean of squares 0.25; with eps 0.75 the divisor is exactly 1
    assert np.array_equal(run_q(x, ones, eps=0.75), np.full(D, 0.5))
    # eps 0: x / |x|
    assert np.array_equal(run_q(x, ones, eps=0.0), np.ones(D))


def test_rms_is_scale_invariant_without_eps():
    x = rand_rows(1, 1, 1)[0, 0]
    ones = np.ones(D, np.float32)
    x4 = bf(W.bits_to_f32(x) * 4.0)
    assert np.array_equal(run_q(x, ones, eps=0.0), run_q(x4, ones, eps=0.0))


def test_rms_gain_applies_per_dim():
    x = rand_rows(2, 1, 1)[0, 0]
    full = run_q(x, np.ones(D, np.float32))
    for j in (0, 37, 64, 127):
        w = np.zeros(D, np.float32)
        w[j] = 1.0
        y = run_q(x, w)
        assert y[j] == full[j]
        assert np.count_nonzero(y) == (1 if full[j] != 0 else 0)
    y2 = run_q(x, np.full(D, 2.0, np.float32))
    assert np.array_equal(y2, 2.0 * full)


def test_rms_of_zero_row_is_zero_and_no_gain_means_no_normalisation():
    z = np.zeros(D, np.uint16)
    assert np.array_equal(run_q(z, np.ones(D, np.float32), eps=1e-6), np.zeros(D))
    x = rand_rows(3, 1, 1)[0, 0]
    assert np.array_equal(run_q(x, None), W.bits_to_f32(x).astype(np.float64))


# ------------------------------------------------------------------ rotary embedding

def test_rotary_at_position_zero_is_identity():
    x = rand_rows(4, 1, 1)[0, 0]
    w = np.ones(D, np.float32)
    assert np.array_equal(run_q(x, w, theta=1e6, pos=0), run_q(x, w, theta=-1.0, pos=0))


@pytest.mark.parametrize("pos", [1, 3, 1000])
def test_rotary_pairs_dim_i_with_dim_i_plus_half(pos):
    e0 = np.zeros(D, np.float32)
    e0[0] = 1.0
    y = run_q(bf(e0), None, theta=1e6, pos=pos)
    # frequency of pair 0 is theta^0 = 1: angle = pos
    assert y[0] == pytest.approx(np.cos(pos), abs=1e-15)
    assert y[HALF] == pytest.approx(np.sin(pos), abs=1e-15)
    assert np.count_nonzero(np.delete(y, [0, HALF])) == 0
    e64 = np.zeros(D, np.float32)
    e64[HALF] = 1.0
    y = run_q(bf(e64), None, theta=1e6, pos=pos)
    assert y[HALF] == pytest.approx(np.cos(pos), abs=1e-15)
    assert y[0] == pytest.approx(-np.sin(pos), abs=1e-15)


@pytest.mark.parametrize("i", [1, 2, 5, 10, 31, 63])
def test_rotary_frequencies_are_theta_to_minus_2i_over_d(i):
    # theta = 2^64 makes the frequency of pair i exactly 2^-i; position
    # 3 * 2^i then turns pair i by exactly 3 radians
    ei = np.zeros(D, np.float32)
    ei[i] = 1.0
    pos = 3 * (1 << i) if i <= 20 else 3 << 20
    angle = pos * 2.0 ** -i
    y = run_q(bf(ei), None, theta=2.0 ** 64, pos=pos)
    assert y[i] == pytest.approx(np.cos(angle), abs=1e-12)
    assert y[i + HALF] == pytest.approx(np.sin(angle), abs=1e-12)


def test_rotation_preserves_pair_norms():
    x = rand_rows(5, 1, 1)[0, 0]
    xf = W.bits_to_f32(x).astype(np.float64)
    for pos in (7, 4095, 16383):
        y = run_q(x, None, theta=1e6, pos=pos)
        np.testing.assert_allclose(y[:HALF] ** 2 + y[HALF:] ** 2, xf[:HALF] ** 2 + xf[HALF:] ** 2,
                                   rtol=1e-13, atol=1e-300)


def test_rotary_scores_depend_on_relative_position_only():
    q = rand_rows(6, 4, 1)
    k = rand_rows(7, 4, 1)
    w = np.ones(D, np.float32)
    # the same (q, k) at positions (p, p') and (p + s, p' + s)
    pos_q = np.array([100, 100 + 37, 5000, 5000 + 37], np.int32)
    pos_k = np.array([90, 90 + 37, 4000, 4000 + 37], np.int32)
    qq = np.ascontiguousarray(np.repeat(q[:1], 4, axis=0))
    kk = np.ascontiguousarray(np.repeat(k[:1], 4, axis=0))
    qo, _, _, _, _ = oracle.append(qq, kk, kk, w, w, pos_q, Lmax=1 << 20)
    _, ko, _, _, _ = oracle.append(qq, kk, kk, w, w, pos_k, Lmax=1 << 20)
    s = np.einsum("bd,bd->b", qo[:, 0], ko[:, 0])
    assert s[0] == pytest.approx(s[1], rel=1e-11)
    assert s[2] == pytest.approx(s[3], rel=1e-11)
    assert abs(s[0] - s[2]) > 1e-3          # but they do depend on it


def test_values_pass_through_unchanged():
    q = rand_rows(8, 3, 4)
    k = rand_rows(9, 3, 2)
    v = rand_rows(10, 3, 2)
    w = np.ones(D, np.float32)
    _, _, vo, _, _ = oracle.append(q, k, v, w, w, np.array([1, 2, 3], np.int32), Lmax=8)
    assert np.array_equal(vo, W.bits_to_f32(v).astype(np.float64))


# ------------------------------------------------------------------ placement in the cache

def test_append_row_is_what_attention_reads_as_position_L():
    """Write the new k/v rows where the oracle says, then ask the attention
    oracle (paging pinned independently) for position L: with a query that
    makes position L's key dominant, attention returns the appended value."""
    lens = np.array([37, 0, 16, 100, 63], np.int32)
    B, Hkv, P = len(lens), 2, 16
    w = W.make_paged(lens + 1, page_size=P, Hq=2, Hkv=Hkv, key=(4300,), poison=False)
    bt, kp, vp = w.block_table, w.k.copy(), w.v.copy()
    q_new = rand_rows(11, B, 2)
    k_new = rand_rows(12, B, Hkv)
    v_new = rand_rows(13, B, Hkv)
    _, _, _, dest, new_lens = oracle.append(q_new, k_new, v_new, None, None, lens,
                                            block_table=bt, page_size=P, num_pages=w.num_pages,
                                            theta=-1.0)
    assert np.array_equal(new_lens, lens + 1)
    kflat = kp.reshape(-1, Hkv, D)
    vflat = vp.reshape(-1, Hkv, D)
    big = bf(np.full(D, 8.0))
    q_old = rand_rows(18, B, 2)
    before, _ = oracle.decode_attn_paged(q_old, kp, vp, bt, lens, 1.0)
    for b in range(B):
        assert dest[b] >= 0
        kflat[dest[b]] = big                      # the key every query will prefer
        vflat[dest[b]] = v_new[b]
    # query = the same large vector: position L scores 8*8*128*scale above any
    # unit-RMS key, so its weight is 1 to binary64 precision
    q = np.ascontiguousarray(np.broadcast_to(big, (B, 2, D)))
    out, _ = oracle.decode_attn_paged(q, kp, vp, bt, new_lens, 1.0)
    for b in range(B):
        np.testing.assert_array_equal(out[b, 0], W.bits_to_f32(v_new[b, 0]))
        np.testing.assert_array_equal(out[b, 1], W.bits_to_f32(v_new[b, 1]))
    # and no earlier position moved: attention over the first L positions is unchanged
    after, _ = oracle.decode_attn_paged(q_old, kp, vp, bt, lens, 1.0)
    np.testing.assert_array_equal(after, before)


def test_append_skips_full_caches_and_bad_pages():
    lens = np.array([32, 31, 5, 40], np.int32)
    P = 16
    bt = np.array([[3, 4], [5, 6], [-1, 7], [8, 9]], np.int32)   # cap = 32
    q = rand_rows(14, 4, 1)
    k = rand_rows(15, 4, 1)
    _, _, _, dest, new_lens = oracle.append(q, k, k, None, None, lens, block_table=bt,
                                            page_size=P, num_pages=10)
    # b0: full; b1: page 6 slot 15; b2: page id -1 -> nothing; b3: clamped to 32, full
    assert list(dest) == [-1, 6 * 16 + 15, -1, -1]
    assert list(new_lens) == [32, 32, 5, 32]
    _, _, _, dest, _ = oracle.append(q, k, k, None, None, lens, block_table=bt, page_size=P,
                                     num_pages=6)
    assert list(dest) == [-1, -1, -1, -1]          # page 6 is outside a 6-page pool


def test_append_contiguous_rows():
    lens = np.array([0, 7, 8, 9], np.int32)
    q = rand_rows(16, 4, 1)
    k = rand_rows(17, 4, 1)
    _, _, _, dest, new_lens = oracle.append(q, k, k, None, None, lens, Lmax=8)
    assert list(dest) == [0, 8 + 7, -1, -1]
    assert list(new_lens) == [1, 8, 8, 8]


# ------------------------------------------------------------------ rounding to bf16

def test_round_bf16_ties_to_even_and_exact_values():
    one = 1.0
    ulp = 2.0 ** -7
    x = np.array([one, one + ulp / 2, one + 3 * ulp / 2, one + ulp / 2 + 2.0 ** -30,
                  -one - ulp / 2, 0.0, -0.0, 2.0 ** -133, 3.0 * 2.0 ** -134, 65280.0], np.float64)
    got = W.bits_to_f32(oracle.round_bf16(x)).astype(np.float64)
    want = [one, one, one + 2 * ulp, one + ulp, -one, 0.0, 0.0, 2.0 ** -133, 2.0 ** -132, 65280.0]
    assert list(got) == want
    assert oracle.round_bf16(np.array([-0.0]))[0] == 0x8000


def test_round_bf16_matches_the_float32_path_on_float32_values():
    # for values that are floats, rounding float32 -> bf16 (nearest even) is
    # the same single rounding
    rng = np.random.default_rng(5)
    f = (rng.standard_normal(100000) * np.exp(rng.uniform(-20, 20, 100000))).astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    ref = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    assert np.array_equal(oracle.round_bf16(f.astype(np.float64)), ref)
