"""The new-token step on the GPU (kva_append_paged / kva_append) against the
fp64 oracle.

Values: every bf16 output must be one of the two bf16 neighbours of the exact
value (|gpu - exact| <= ulp/2 of bf16 plus 1e-5 of the row's largest value for
fp32 rounding before the final rounding), and at least 99.9 % must equal the
oracle's nearest-even rounding.  Placement is index work and is checked
bitwise: the new rows land exactly where the oracle says, and every other byte
of the cache is unchanged.  An end-to-end case runs attention over the
appended caches on both sides."""
import dataclasses

import numpy as np
import pytest

import oracle
import workloads as W
from kva_testlib import assert_parity, dev, torch

pytestmark = pytest.mark.gpu

EPS = 1e-6
THETA = 1e6


def bf16_ulp(x):
    ax = np.abs(x)
    e = np.floor(np.log2(np.where(ax > 0, ax, 1.0)))
    return np.where(ax > 0, 2.0 ** (e - 7), 2.0 ** -133)


def check_values(gpu_bits, exact, tag):
    got = W.bits_to_f32(gpu_bits).astype(np.float64)
    rowmax = np.max(np.abs(exact), axis=-1, keepdims=True)
    tol = 0.5 * bf16_ulp(exact) + 1e-5 * rowmax
    err = np.abs(got - exact)
    bad = err > tol
    assert not bad.any(), f"{tag}: {int(bad.sum())} values off, worst {float((err - tol).max()):.3e}"
    same = np.mean(gpu_bits == oracle.round_bf16(exact))
    assert same >= 0.999, f"{tag}: only {same:.5f} equal to the nearest-even rounding"


def inputs(B, Hq, Hkv, seed, *, gains=True):
    rng = np.random.default_rng(seed)
    # projections with arbitrary per-head scales (the normalisation removes them)
    def rows(n):
        x = W.bits_to_f32(W.normal_bf16(np.random.SeedSequence([seed, n]), B, n, 128))
        return W.bf16_bits(x * rng.uniform(0.05, 20.0, size=(B, n, 1)).astype(np.float32))
    q, k, v = rows(Hq), rows(Hkv), rows(Hkv)
    qw = (1.0 + 0.1 * rng.standard_normal(128)).astype(np.float32) if gains else None
    kw = (1.0 + 0.1 * rng.standard_normal(128)).astype(np.float32) if gains else None
    return q, k, v, qw, kw


def run_paged(w, lens, q, k, v, qw, kw, *, theta=THETA, in_place=False):
    import paper_2609_12471_amd as kva
    t = torch()
    kp, vp, bt = dev(w.k), dev(w.v), dev(w.block_table)
    qi = dev(q)
    qo = qi if in_place else t.empty_like(qi)
    sl = dev(lens)
    nl = sl if in_place else t.empty_like(sl)
    kva.kva_append_paged(qi, dev(k), dev(v), qo, kp, vp, bt, sl, nl,
                         q_norm_w=None if qw is None else dev(qw),
                         k_norm_w=None if kw is None else dev(kw), eps=EPS, rope_theta=theta)
    t.cuda.synchronize()
    return (qo.cpu().numpy().view(np.uint16), kp.cpu().numpy().view(np.uint16),
            vp.cpu().numpy().view(np.uint16), nl.cpu().numpy())


def check_paged(w, lens, q, k, v, qw, kw, tag, *, theta=THETA, in_place=False):
    print(f"[append] {tag}: B={len(lens)} P={w.page_size} Hq={q.shape[1]} Hkv={k.shape[1]}",
          flush=True)
    qo, kp, vp, nl = run_paged(w, lens, q, k, v, qw, kw, theta=theta, in_place=in_place)
    rq, rk, rv, dest, rnl = oracle.append(q, k, v, qw, kw, lens, block_table=w.block_table,
                                          page_size=w.page_size, num_pages=w.num_pages,
                                          eps=EPS, theta=theta)
    assert np.array_equal(nl, rnl), tag
    check_values(qo, rq, tag + " q")
    Hkv = k.shape[1]
    kf = kp.reshape(-1, Hkv, 128)
    vf = vp.reshape(-1, Hkv, 128)
    k0 = w.k.reshape(-1, Hkv, 128)
    v0 = w.v.reshape(-1, Hkv, 128)
    wrote = dest >= 0
    if wrote.any():
        check_values(kf[dest[wrote]], rk[wrote], tag + " k")
        assert np.array_equal(vf[dest[wrote]], v[wrote]), tag + " v rows"
    keep = np.ones(kf.shape[0], bool)
    keep[dest[wrote]] = False
    assert np.array_equal(kf[keep], k0[keep]), tag + ": k pool changed outside the new rows"
    assert np.array_equal(vf[keep], v0[keep]), tag + ": v pool changed outside the new rows"
    return dest


def paged_case(lens, P, Hq, Hkv, key, *, room=True):
    lens = np.asarray(lens, np.int32)
    # pages for L + 1 tokens, so position L exists (unless room is False)
    w = W.make_paged(lens + 1 if room else lens, page_size=P, Hq=Hq, Hkv=Hkv, key=key)
    return w, lens


def test_append_c3_shapes():
    lens = W.config_lengths(3)
    w, lens = paged_case(lens, 16, 32, 8, (8100,))
    q, k, v, qw, kw = inputs(len(lens), 32, 8, 1)
    dest = check_paged(w, lens, q, k, v, qw, kw, "c3 lengths")
    assert np.all(dest >= 0)


@pytest.mark.parametrize("P,Hq,Hkv", [(1, 32, 8), (4, 32, 8), (16, 8, 8), (16, 16, 8),
                                      (64, 64, 8), (1024, 32, 8), (16, 4, 1)])
def test_append_page_sizes_and_head_groups(P, Hq, Hkv):
    lens = [0, 1, P - 1 if P > 1 else 0, P, 3 * P + 5, 700, 1500]
    w, lens = paged_case(lens, P, Hq, Hkv, (8200, P, Hq))
    q, k, v, qw, kw = inputs(len(lens), Hq, Hkv, 2 + P)
    check_paged(w, lens, q, k, v, qw, kw, f"P={P} Hq={Hq} Hkv={Hkv}")


def test_append_full_caches_and_bad_pages_write_nothing():
    lens = np.array([64, 63, 20, 5, 40], np.int32)
    w = W.make_paged(np.array([64, 64, 64, 64, 64], np.int32), page_size=16, key=(8300,))
    bt = w.block_table.copy()
    bt[2, 1] = -1                      # position 20 of sequence 2: no page
    bt[3, 0] = w.num_pages + 7         # position 5 of sequence 3: outside the pool
    w = dataclasses.replace(w, block_table=bt)
    q, k, v, qw, kw = inputs(5, 32, 8, 3)
    dest = check_paged(w, lens, q, k, v, qw, kw, "full / bad pages")
    assert list(dest >= 0) == [False, True, False, False, True]


def test_append_without_gains_or_rotation():
    lens = [100, 2000, 4095]
    w, lens = paged_case(lens, 16, 32, 8, (8400,))
    q, k, v, _, _ = inputs(3, 32, 8, 4, gains=False)
    check_paged(w, lens, q, k, v, None, None, "no gains", theta=THETA)
    q, k, v, qw, kw = inputs(3, 32, 8, 5)
    check_paged(w, lens, q, k, v, qw, kw, "no rotation", theta=0.0)


def test_append_in_place_q_and_lengths():
    lens = [10, 300, 8191]
    w, lens = paged_case(lens, 16, 32, 8, (8500,))
    q, k, v, qw, kw = inputs(3, 32, 8, 6)
    check_paged(w, lens, q, k, v, qw, kw, "in place", in_place=True)


def test_append_many_sequences():
    rng = np.random.default_rng(7)
    lens = rng.integers(0, 3000, size=1000).astype(np.int32)
    w, lens = paged_case(lens, 16, 32, 8, (8600,))
    q, k, v, qw, kw = inputs(1000, 32, 8, 8)
    check_paged(w, lens, q, k, v, qw, kw, "B=1000")


def test_append_contiguous():
    import paper_2609_12471_amd as kva
    t = torch()
    lens = np.array([0, 5, 255, 256, 100], np.int32)
    Lmax = 256
    w = W.make_contig(lens.clip(0, Lmax), Lmax, key=(8700,))
    q, k, v, qw, kw = inputs(5, 32, 8, 9)
    kc, vc = dev(w.k), dev(w.v)
    qo = t.empty_like(dev(q))
    nl = t.empty(5, dtype=t.int32, device="cuda")
    kva.kva_append(dev(q), dev(k), dev(v), qo, kc, vc, dev(lens), nl, q_norm_w=dev(qw),
                   k_norm_w=dev(kw), eps=EPS, rope_theta=THETA)
    t.cuda.synchronize()
    rq, rk, rv, dest, rnl = oracle.append(q, k, v, qw, kw, lens, Lmax=Lmax, eps=EPS, theta=THETA)
    assert np.array_equal(nl.cpu().numpy(), rnl)
    check_values(qo.cpu().numpy().view(np.uint16), rq, "contig q")
    kf = kc.cpu().numpy().view(np.uint16).reshape(-1, 8, 128)
    vf = vc.cpu().numpy().view(np.uint16).reshape(-1, 8, 128)
    wrote = dest >= 0
    assert list(wrote) == [True, True, True, False, True]
    check_values(kf[dest[wrote]], rk[wrote], "contig k")
    assert np.array_equal(vf[dest[wrote]], v[wrote])
    keep = np.ones(kf.shape[0], bool)
    keep[dest[wrote]] = False
    assert np.array_equal(kf[keep], w.k.reshape(-1, 8, 128)[keep])
    assert np.array_equal(vf[keep], w.v.reshape(-1, 8, 128)[keep])


def test_append_then_attention_end_to_end():
    """GPU: append, then attention over L + 1 positions with the appended
    query.  Oracle: the same two steps from the oracle's own rounded rows."""
    import paper_2609_12471_amd as kva
    t = torch()
    lens = np.array([511, 2047, 3000, 16, 0, 777], np.int32)
    w, lens = paged_case(lens, 16, 32, 8, (8800,))
    q, k, v, qw, kw = inputs(len(lens), 32, 8, 10)
    kp, vp, bt, sl = dev(w.k), dev(w.v), dev(w.block_table), dev(lens)
    qo = t.empty_like(dev(q))
    kva.kva_append_paged(dev(q), dev(k), dev(v), qo, kp, vp, bt, sl, sl, q_norm_w=dev(qw),
                         k_norm_w=dev(kw), eps=EPS, rope_theta=THETA)
    out = t.empty((len(lens), 32, 128), dtype=t.float32, device="cuda")
    lse = t.empty((len(lens), 32), dtype=t.float32, device="cuda")
    kva.kva_decode_attn_paged(qo, kp, vp, bt, sl, out, lse, scale=w.scale)
    t.cuda.synchronize()
    # oracle side
    rq, rk, rv, dest, rnl = oracle.append(q, k, v, qw, kw, lens, block_table=w.block_table,
                                          page_size=16, num_pages=w.num_pages, eps=EPS,
                                          theta=THETA)
    kpo, vpo = w.k.copy(), w.v.copy()
    kpo.reshape(-1, 8, 128)[dest] = oracle.round_bf16(rk)
    vpo.reshape(-1, 8, 128)[dest] = v
    ref, rlse = oracle.decode_attn_paged(oracle.round_bf16(rq), kpo, vpo, w.block_table, rnl,
                                         w.scale)
    assert np.array_equal(sl.cpu().numpy(), rnl)
    assert_parity(out.cpu().numpy(), ref, lse.cpu().numpy(), rlse, tag="append + attention")
