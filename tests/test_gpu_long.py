"""Long contexts.  A context of 2^20 tokens: one sequence of 1,048,573 tokens
(65,536 pages of 16, so page ids, table windows and flat granule indices all
run far past anything the other tests reach) beside one of 70,001 tokens, through the
paged call.  The oracle checks two of the eight KV heads (their four query
heads each) over the whole length: the heads are independent, so the oracle
runs on the cache sliced to one KV head.  And chunked prefill over 60,000
cached tokens."""
import numpy as np
import pytest

import oracle
import workloads as W
from kva_testlib import DeviceWorkload, assert_parity, run_gpu

pytestmark = pytest.mark.gpu


def test_million_token_context():
    lens = [(1 << 20) - 3, 70001]
    print(f"[long] paged P=16 lengths {lens}", flush=True)
    w = W.make_paged(lens, page_size=16, key=(9800,))
    out, lse = run_gpu(DeviceWorkload(w))
    G = w.Hq // w.Hkv
    for g in (0, w.Hkv - 1):
        print(f"[long] oracle for KV head {g}", flush=True)
        q = np.ascontiguousarray(w.q[:, G * g:G * (g + 1)])
        k = np.ascontiguousarray(w.k[:, :, g:g + 1])
        v = np.ascontiguousarray(w.v[:, :, g:g + 1])
        ref, rlse = oracle.decode_attn_paged(q, k, v, w.block_table, w.seq_lens, w.scale)
        assert_parity(out[:, G * g:G * (g + 1)], ref, lse[:, G * g:G * (g + 1)], rlse,
                      tag=f"2^20 tokens, KV head {g}")


def test_prefill_over_a_long_context():
    """Chunked prefill of 40 new tokens over 60,000 cached ones (470 staged
    blocks of 128 positions for every workgroup of that rollout), beside a short rollout; the
    oracle checks KV heads 0 and 5."""
    import paper_2609_12471_amd as kva
    from kva_testlib import dev, torch
    t = torch()
    p = W.make_prefill([60000, 3000], [40, 130], key=(9810,))
    c = p.cache
    print("[long] prefill ctx 60000+40, 3000+130", flush=True)
    out = t.full((p.T, c.Hq, c.D), float("nan"), dtype=t.float32, device="cuda")
    ls = t.empty((p.T, c.Hq), dtype=t.float32, device="cuda")
    kva.kva_prefill_paged(dev(p.q), dev(c.k), dev(c.v), dev(c.block_table), dev(p.q_start),
                          dev(c.seq_lens), out, ls, max_q_len=int(np.diff(p.q_start).max()),
                          scale=c.scale)
    t.cuda.synchronize()
    out, ls = out.cpu().numpy(), ls.cpu().numpy()
    G = c.Hq // c.Hkv
    for g in (0, 5):
        print(f"[long] prefill oracle for KV head {g}", flush=True)
        ref, rlse = oracle.prefill_paged(np.ascontiguousarray(p.q[:, G * g:G * (g + 1)]),
                                         np.ascontiguousarray(c.k[:, :, g:g + 1]),
                                         np.ascontiguousarray(c.v[:, :, g:g + 1]),
                                         c.block_table, p.q_start, c.seq_lens, c.scale)
        assert_parity(out[:, G * g:G * (g + 1)], ref, ls[:, G * g:G * (g + 1)], rlse,
                      tag=f"prefill over 60000 tokens, KV head {g}")
