"""A context of 2^20 tokens: one sequence of 1,048,573 tokens (65,536 pages of
16, so page ids, table windows and flat granule indices all run far past
anything the other tests reach) beside one of 70,001 tokens, through the
paged call.  The oracle checks two of the eight KV heads (their four query
heads each) over the whole length: the heads are independent, so the oracle
runs on the cache sliced to one KV head."""
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
