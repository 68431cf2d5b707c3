"""Pins of the oracle's chunked prefill.

* a chunk of one token is decode attention (bitwise);
* every new token equals a decode call over its causal prefix (bitwise), which
  checks the packing of queries and the position of each token;
* a whole prompt equals torch's causal scaled_dot_product_attention (a library
  routine, float64, grouped-query heads); with earlier context, the same
  routine with an explicit mask;
* empty chunks, and chunks longer than the sequence (tokens below position 0
  attend nothing)."""
import numpy as np
import pytest

import oracle
import workloads as W


def _decode_stack(p):
    c = p.cache
    out = np.empty(p.q.shape, np.float64)
    lse = np.empty(p.q.shape[:2], np.float64)
    for b in range(c.B):
        n = p.q_start[b + 1] - p.q_start[b]
        for i in range(n):
            row = p.q_start[b] + i
            L = int(c.seq_lens[b]) - n + i + 1
            o, l = oracle.decode_attn_paged(np.ascontiguousarray(p.q[row:row + 1]), c.k, c.v,
                                             np.ascontiguousarray(c.block_table[b:b + 1]),
                                             np.array([max(L, 0)], np.int32), c.scale)
            out[row], lse[row] = o[0], l[0]
    return out, lse


def _run(p):
    c = p.cache
    return oracle.prefill_paged(p.q, c.k, c.v, c.block_table, p.q_start, c.seq_lens, c.scale)


def test_one_token_chunk_is_decode_attention():
    p = W.make_prefill([100, 0, 37], [1, 1, 1], key=(6100,))
    out, lse = _run(p)
    c = p.cache
    ref, rlse = oracle.decode_attn_paged(p.q, c.k, c.v, c.block_table, c.seq_lens, c.scale)
    assert np.array_equal(out, ref) and np.array_equal(lse, rlse)


@pytest.mark.parametrize("P", [1, 16, 64])
def test_every_token_is_decode_over_its_causal_prefix(P):
    p = W.make_prefill([0, 50, 17, 200], [9, 33, 1, 16], page_size=P, key=(6200, P))
    out, lse = _run(p)
    ref, rlse = _decode_stack(p)
    assert np.array_equal(out, ref) and np.array_equal(lse, rlse)


def _sdpa(p, b):
    import torch
    c = p.cache
    n = int(p.q_start[b + 1] - p.q_start[b])
    L = int(c.seq_lens[b])
    P = c.page_size
    t = np.arange(L)
    k = W.bits_to_f32(c.k[c.block_table[b, t // P], t % P]).astype(np.float64)   # [L, Hkv, D]
    v = W.bits_to_f32(c.v[c.block_table[b, t // P], t % P]).astype(np.float64)
    q = W.bits_to_f32(p.q[p.q_start[b]:p.q_start[b + 1]]).astype(np.float64)      # [n, Hq, D]
    qt = torch.from_numpy(q).permute(1, 0, 2).unsqueeze(0)
    kt = torch.from_numpy(k).permute(1, 0, 2).unsqueeze(0).contiguous()
    vt = torch.from_numpy(v).permute(1, 0, 2).unsqueeze(0).contiguous()
    pos = (L - n) + np.arange(n)
    mask = torch.from_numpy(np.arange(L)[None, :] <= pos[:, None])
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask,
                                                         scale=float(np.float32(c.scale)),
                                                         enable_gqa=True)
    return o[0].permute(1, 0, 2).numpy()


def test_whole_prompt_matches_torch_causal_sdpa():
    p = W.make_prefill([0, 0], [120, 64], Hq=8, Hkv=2, key=(6300,))
    out, _ = _run(p)
    for b in range(2):
        ref = _sdpa(p, b)
        got = out[p.q_start[b]:p.q_start[b + 1]]
        np.testing.assert_allclose(got, ref, rtol=1e-10, atol=1e-12)
        # the causal form for a prompt with no earlier context is torch's is_causal
        import torch
        c = p.cache
        n = int(p.q_start[b + 1] - p.q_start[b])
        t = np.arange(n)
        k = W.bits_to_f32(c.k[c.block_table[b, t // 16], t % 16]).astype(np.float64)
        v = W.bits_to_f32(c.v[c.block_table[b, t // 16], t % 16]).astype(np.float64)
        q = W.bits_to_f32(p.q[p.q_start[b]:p.q_start[b + 1]]).astype(np.float64)
        o = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(q).permute(1, 0, 2).unsqueeze(0),
            torch.from_numpy(k).permute(1, 0, 2).unsqueeze(0).contiguous(),
            torch.from_numpy(v).permute(1, 0, 2).unsqueeze(0).contiguous(), is_causal=True,
            scale=float(np.float32(c.scale)), enable_gqa=True)[0].permute(1, 0, 2).numpy()
        np.testing.assert_allclose(got, o, rtol=1e-10, atol=1e-12)


def test_chunk_after_context_matches_masked_sdpa():
    p = W.make_prefill([300, 77], [40, 130], Hq=8, Hkv=2, key=(6400,))
    out, _ = _run(p)
    for b in range(2):
        np.testing.assert_allclose(out[p.q_start[b]:p.q_start[b + 1]], _sdpa(p, b), rtol=1e-10,
                                   atol=1e-12)


def test_empty_chunks_and_tokens_before_position_zero():
    p = W.make_prefill([10, 0, 5], [0, 3, 4], key=(6500,))
    c = p.cache
    # sequence 2 claims 4 new tokens but holds only 3 + ... : shorten it to 2
    lens = c.seq_lens.copy()
    lens[2] = 2
    out, lse = oracle.prefill_paged(p.q, c.k, c.v, c.block_table, p.q_start, lens, c.scale)
    rows = slice(p.q_start[2], p.q_start[3])
    # tokens at positions -2, -1 attend nothing; positions 0 and 1 attend 1 and 2 rows
    assert np.all(out[rows][:2] == 0) and np.all(np.isneginf(lse[rows][:2]))
    assert np.all(np.isfinite(lse[rows][2:]))
    assert out.shape[0] == 7
