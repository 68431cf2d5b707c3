"""Chunked prefill on the GPU (kva_prefill_paged) against the fp64 oracle,
under the same gate as decode (max-abs 2e-3, mean-abs 2e-4 on fp32 outputs,
and the paper's checker tolerance elementwise)."""
import numpy as np
import pytest

import oracle
import workloads as W
from kva_testlib import assert_parity, dev, torch

pytestmark = pytest.mark.gpu


def run(p, *, max_q_len=None, lse=True, seq_lens=None, scale=None):
    import paper_2609_12471_amd as kva
    t = torch()
    c = p.cache
    lens = c.seq_lens if seq_lens is None else seq_lens
    out = t.full((p.T, c.Hq, c.D), float("nan"), dtype=t.float32, device="cuda")
    ls = t.empty((p.T, c.Hq), dtype=t.float32, device="cuda") if lse else None
    mq = int(np.diff(p.q_start).max()) if max_q_len is None else max_q_len
    kva.kva_prefill_paged(dev(p.q), dev(c.k), dev(c.v), dev(c.block_table), dev(p.q_start),
                          dev(lens), out, ls, max_q_len=mq, scale=c.scale if scale is None else scale)
    t.cuda.synchronize()
    return out.cpu().numpy(), (ls.cpu().numpy() if lse else None)


def check(p, tag, **kw):
    print(f"[prefill] {tag}: B={p.cache.B} T={p.T} P={p.cache.page_size} Hq={p.cache.Hq}",
          flush=True)
    out, lse = run(p, **kw)
    c = p.cache
    lens = kw.get("seq_lens", c.seq_lens)
    scale = kw.get("scale")
    ref, rlse = oracle.prefill_paged(p.q, c.k, c.v, c.block_table, p.q_start, lens,
                                     c.scale if scale is None else scale)
    return assert_parity(out, ref, lse, rlse, tag=tag)


def test_prefill_small_chunks_over_context():
    check(W.make_prefill([0, 100, 1000, 31, 4096], [1, 7, 33, 64, 130], key=(7100,)),
          "small chunks")


@pytest.mark.parametrize("P", [1, 4, 16, 32, 64, 1024])
def test_prefill_page_sizes(P):
    check(W.make_prefill([0, 500, 77, 2000], [200, 64, 31, 96], page_size=P, key=(7200, P)),
          f"P={P}")


@pytest.mark.parametrize("Hq,Hkv", [(8, 8), (16, 8), (64, 8), (4, 1)])
def test_prefill_head_groups(Hq, Hkv):
    check(W.make_prefill([300, 0, 1500], [129, 256, 17], Hq=Hq, Hkv=Hkv, key=(7300, Hq)),
          f"Hq={Hq} Hkv={Hkv}")


def test_prefill_whole_prompts_and_empty_chunks():
    check(W.make_prefill([0, 0, 0, 0], [1000, 0, 1, 513], key=(7400,)), "prompts")


@pytest.mark.parametrize("scale", [0.0, -0.0883883476, 0.5])
def test_prefill_scales(scale):
    """Zero scale (every attended position weighs the same), a negative scale
    (the softmax favours the lowest scores) and a large one (peaked weights)."""
    check(W.make_prefill([0, 300, 1200], [70, 33, 129], key=(7600,)), f"scale={scale}", scale=scale)


def test_prefill_tokens_before_position_zero():
    p = W.make_prefill([0, 0], [40, 8], key=(7500,))
    lens = p.cache.seq_lens.copy()
    lens[0] = 25                        # 40 new tokens claimed, 25 in the cache
    check(p, "negative positions", seq_lens=lens)


def test_prefill_config_sample():
    """A sample of the benchmark workload (3 of its 64 rollouts), in the same
    launch shape: 512 new tokens over 512..7680 tokens of context."""
    p = W.make_prefill_config()
    b_keep = 3
    c = p.cache
    import dataclasses
    cache = dataclasses.replace(c, q=c.q[:b_keep], seq_lens=c.seq_lens[:b_keep].copy(),
                                block_table=np.ascontiguousarray(c.block_table[:b_keep]))
    q_start = np.ascontiguousarray(p.q_start[:b_keep + 1])
    sub = W.Prefill(cache, np.ascontiguousarray(p.q[:q_start[-1]]), q_start)
    check(sub, "config sample")


def test_prefill_full_config_sampled_rows():
    """The whole benchmark workload on the GPU; the oracle checks one new
    token at a seeded random offset in every 32-token tile of every rollout
    (every workgroup's tile of query rows is sampled), one by one."""
    from concurrent.futures import ThreadPoolExecutor
    p = W.make_prefill_config()
    out, lse = run(p)
    assert np.isfinite(out).all() and np.isfinite(lse).all()
    c = p.cache
    rng = np.random.default_rng(6100)
    rows = []
    for b in range(c.B):
        s0, s1 = int(p.q_start[b]), int(p.q_start[b + 1])
        for t0 in range(s0, s1, 32):
            rows.append(t0 + int(rng.integers(0, min(32, s1 - t0))))
    rows = np.array(rows, np.int64)
    # the oracle on single-token chunks: token row r of sequence b at its position
    b_of = np.searchsorted(p.q_start, rows, side="right") - 1
    n = np.diff(p.q_start)[b_of]
    pos = c.seq_lens[b_of] - n + (rows - p.q_start[b_of])
    ref = np.empty((rows.size, c.Hq, c.D))
    rlse = np.empty((rows.size, c.Hq))
    cuts = np.linspace(0, rows.size, 33).astype(int)

    def work(i):
        sl = slice(cuts[i], cuts[i + 1])
        ref[sl], rlse[sl] = oracle.decode_attn_paged(
            np.ascontiguousarray(p.q[rows[sl]]), c.k, c.v,
            np.ascontiguousarray(c.block_table[b_of[sl]]), (pos[sl] + 1).astype(np.int32), c.scale)

    with ThreadPoolExecutor(16) as ex:
        list(ex.map(work, range(32)))
    assert rows.size == c.B * 512 // 32
    assert_parity(out[rows], ref, lse[rows], rlse, tag="full config, one row per 32-token tile")


def test_prefill_is_deterministic():
    p = W.make_prefill([1000, 2000], [300, 77], key=(7600,))
    o1, l1 = run(p)
    o2, l2 = run(p)
    assert np.array_equal(o1.view(np.uint32), o2.view(np.uint32))
    assert np.array_equal(l1.view(np.uint32), l2.view(np.uint32))
