"""The entry points captured in a HIP graph (torch.cuda.CUDAGraph) and replayed.

A call issues kernel launches only: no allocation, no memset, no host
synchronisation, and grid shapes that depend on the batch's sizes but not on
its lengths (the kernels read seq_lens from device memory).  So one captured
decode step serves every later step of a serving loop: the lengths, q and the
cache change in place between replays.  Each graph is replayed several times
with eager work and synchronisations in between, and every replay is compared
with an eager call on the same inputs (bitwise: the kernels add in a fixed
order) and, where the inputs changed, with the oracle."""
import dataclasses

import numpy as np
import pytest

import oracle
import workloads as W
from kva_testlib import assert_parity, dev, run_oracle, torch

pytestmark = pytest.mark.gpu

LENS = [5, 130, 2049, 700, 33, 1024, 16, 17]


def capture(fn):
    """fn() captured on a side stream after two eager warm-up calls."""
    t = torch()
    s = t.cuda.Stream()
    s.wait_stream(t.cuda.current_stream())
    with t.cuda.stream(s):
        for _ in range(2):
            fn()
    t.cuda.current_stream().wait_stream(s)
    t.cuda.synchronize()
    g = t.cuda.CUDAGraph()
    with t.cuda.graph(g):
        fn()
    t.cuda.synchronize()
    return g


def replay_and_compare(g, outs, refs, tag, times=3):
    """Poison the outputs eagerly, replay, and compare bitwise with refs."""
    t = torch()
    for r in range(times):
        for o in outs:
            o.fill_(float("nan"))
        t.cuda.synchronize()
        g.replay()
        t.cuda.synchronize()
        for i, (o, ref) in enumerate(zip(outs, refs)):
            assert t.equal(o, ref), f"{tag}: replay {r}, output {i} differs from the eager call"


def test_graph_paged_decode_with_growing_lengths():
    import paper_2609_12471_amd as kva
    t = torch()
    w = W.make_paged(LENS, key=(9700,))
    full = np.asarray(LENS, np.int32)
    q, k, v, bt = dev(w.q), dev(w.k), dev(w.v), dev(w.block_table)
    lens = dev(np.maximum(full - 5, 0).astype(np.int32))    # five tokens short
    out = t.empty((w.B, w.Hq, w.D), dtype=t.float32, device="cuda")
    lse = t.empty((w.B, w.Hq), dtype=t.float32, device="cuda")
    ws = kva.kva_new_workspace(w.B, w.Hq, w.Hkv, w.D)

    def call(o=out, ls=lse):
        kva.kva_decode_attn_paged(q, k, v, bt, lens, o, ls, scale=w.scale, workspace=ws)

    g = capture(call)
    eo, el = t.empty_like(out), t.empty_like(lse)
    call(eo, el)
    t.cuda.synchronize()
    replay_and_compare(g, [out, lse], [eo, el], "paged, initial lengths")
    ref, rlse = run_oracle(dataclasses.replace(w, seq_lens=np.maximum(full - 5, 0).astype(np.int32)))
    assert_parity(out.cpu().numpy(), ref, lse.cpu().numpy(), rlse, tag="graph, initial lengths")

    # the next steps of the loop: the lengths grow in place, then q changes
    lens.copy_(dev(full))
    call(eo, el)
    t.cuda.synchronize()
    replay_and_compare(g, [out, lse], [eo, el], "paged, grown lengths")
    ref, rlse = run_oracle(w)
    assert_parity(out.cpu().numpy(), ref, lse.cpu().numpy(), rlse, tag="graph, grown lengths")

    w2 = W.make_paged(LENS, key=(9701,))
    q.copy_(dev(w2.q))
    call(eo, el)
    t.cuda.synchronize()
    replay_and_compare(g, [out, lse], [eo, el], "paged, new q")
    ref, rlse = run_oracle(dataclasses.replace(w, q=w2.q))
    assert_parity(out.cpu().numpy(), ref, lse.cpu().numpy(), rlse, tag="graph, new q")


def test_graph_noalloc_and_contiguous_and_fp8():
    import paper_2609_12471_amd as kva
    t = torch()
    wp = W.make_paged(LENS, key=(9710,))
    wc = W.make_contig(LENS, 2100, key=(9711,))
    w8 = W.quantize_fp8(W.make_paged(LENS, key=(9712,)))
    qp, kp, vp, btp, lp = dev(wp.q), dev(wp.k), dev(wp.v), dev(wp.block_table), dev(wp.seq_lens)
    qc, kc, vc, lc = dev(wc.q), dev(wc.k), dev(wc.v), dev(wc.seq_lens)
    k8 = t.from_numpy(w8.k).to("cuda").view(t.float8_e4m3fn)
    v8 = t.from_numpy(w8.v).to("cuda").view(t.float8_e4m3fn)
    q8, bt8, l8 = dev(w8.q), dev(w8.block_table), dev(w8.seq_lens)
    B, Hq, D, Hkv = wp.B, wp.Hq, wp.D, wp.Hkv
    outs = [t.empty((B, Hq, D), dtype=t.float32, device="cuda") for _ in range(3)]
    lses = [t.empty((B, Hq), dtype=t.float32, device="cuda") for _ in range(3)]
    ws_c = kva.kva_new_workspace(B, Hq, Hkv, D)
    ws_8 = kva.kva_new_workspace(B, Hq, Hkv, D)

    def calls(o=outs, ls=lses):
        kva.kva_decode_attn_paged_noalloc(qp, kp, vp, btp, lp, o[0], ls[0], scale=wp.scale)
        kva.kva_decode_attn(qc, kc, vc, lc, o[1], ls[1], scale=wc.scale, workspace=ws_c)
        kva.kva_decode_attn_paged_fp8(q8, k8, v8, bt8, l8, o[2], ls[2], scale=w8.scale,
                                      k_scale=w8.meta["k_scale"], v_scale=w8.meta["v_scale"],
                                      workspace=ws_8)

    g = capture(calls)
    eo = [t.empty_like(x) for x in outs]
    el = [t.empty_like(x) for x in lses]
    calls(eo, el)
    t.cuda.synchronize()
    replay_and_compare(g, outs + lses, eo + el, "noalloc + contiguous + fp8", times=4)
    for i, w in enumerate((wp, wc, w8)):
        ref, rlse = run_oracle(w)
        assert_parity(outs[i].cpu().numpy(), ref, lses[i].cpu().numpy(), rlse,
                      tag=f"graph replay, {w.layout} {w.meta.get('kv_dtype', 'bf16')}")


def test_graph_grouped_decode_and_new_token_step():
    """The grouped call (pass, attention, merge) and a whole decode step (append
    of the new token, then attention over the cache it extended) as graphs."""
    import paper_2609_12471_amd as kva
    t = torch()
    group, prefix = 4, 256
    lens = [300, 700, 290, 1000, 512, 260, 257, 900]
    w = W.make_paged(lens, key=(9720,), shared_prefix=(group, prefix))
    q, k, v, bt, sl = dev(w.q), dev(w.k), dev(w.v), dev(w.block_table), dev(w.seq_lens)
    out = t.empty((w.B, w.Hq, w.D), dtype=t.float32, device="cuda")
    lse = t.empty((w.B, w.Hq), dtype=t.float32, device="cuda")
    need = kva.kva_workspace_bytes_grouped(w.B, w.Hq, w.Hkv, w.D, group)
    ws = t.empty(need, dtype=t.uint8, device="cuda")

    def grouped(o=out, ls=lse):
        kva.kva_decode_attn_paged_grouped(q, k, v, bt, sl, o, ls, group=group, scale=w.scale,
                                          workspace=ws)

    g = capture(grouped)
    eo, el = t.empty_like(out), t.empty_like(lse)
    grouped(eo, el)
    t.cuda.synchronize()
    replay_and_compare(g, [out, lse], [eo, el], "grouped")
    ref, rlse = run_oracle(w)
    assert_parity(out.cpu().numpy(), ref, lse.cpu().numpy(), rlse, tag="graph, grouped")

    # decode step: the new token's row is written at position seq_lens[b] (the
    # lengths are those before the token), then attention runs over new_lens
    B, Hq, Hkv, D = w.B, w.Hq, w.Hkv, w.D
    base_lens = dev((np.asarray(lens, np.int32) - 1))
    q_in = dev(W.normal_bf16(np.random.SeedSequence((9721, 0)), B, Hq, D))
    k_in = dev(W.normal_bf16(np.random.SeedSequence((9721, 1)), B, Hkv, D))
    v_in = dev(W.normal_bf16(np.random.SeedSequence((9721, 2)), B, Hkv, D))
    q_out = t.empty_like(q_in)
    new_lens = t.empty_like(base_lens)
    k2, v2 = k.clone(), v.clone()
    ws2 = kva.kva_new_workspace(B, Hq, Hkv, D)

    def step(o=out, ls=lse):
        kva.kva_append_paged(q_in, k_in, v_in, q_out, k2, v2, bt, base_lens, new_lens)
        kva.kva_decode_attn_paged(q_out, k2, v2, bt, new_lens, o, ls, scale=w.scale,
                                  workspace=ws2)

    g2 = capture(step)
    step(eo, el)
    t.cuda.synchronize()
    replay_and_compare(g2, [out, lse], [eo, el], "append + attention")
    assert t.equal(new_lens, dev(np.asarray(lens, np.int32)))


def test_graph_prefill():
    import paper_2609_12471_amd as kva
    t = torch()
    p = W.make_prefill([0, 300, 1200, 64], [70, 33, 129, 1], key=(9730,))
    c = p.cache
    q, k, v, bt, qs, sl = (dev(p.q), dev(c.k), dev(c.v), dev(c.block_table), dev(p.q_start),
                           dev(c.seq_lens))
    out = t.empty((p.T, c.Hq, c.D), dtype=t.float32, device="cuda")
    lse = t.empty((p.T, c.Hq), dtype=t.float32, device="cuda")
    mq = int(np.diff(p.q_start).max())

    def call(o=out, ls=lse):
        kva.kva_prefill_paged(q, k, v, bt, qs, sl, o, ls, max_q_len=mq, scale=c.scale)

    g = capture(call)
    eo, el = t.empty_like(out), t.empty_like(lse)
    call(eo, el)
    t.cuda.synchronize()
    replay_and_compare(g, [out, lse], [eo, el], "prefill")
    ref, rlse = oracle.prefill_paged(p.q, c.k, c.v, c.block_table, p.q_start, c.seq_lens, c.scale)
    assert_parity(out.cpu().numpy(), ref, lse.cpu().numpy(), rlse, tag="graph, prefill")
