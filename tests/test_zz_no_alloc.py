"""kva_decode_attn_paged_noalloc (the entry point that allocates nothing: its
partial results live in the library's built-in device scratch array) against
kva_decode_attn_paged with a caller workspace, through the C ABI: bitwise the
same outputs on two calls in a row, the second with a smaller batch, and both
within the parity gate of the fp64 oracle."""
import numpy as np
import pytest

import workloads as W
from kva_testlib import DeviceWorkload, assert_parity, run_gpu, run_oracle, torch

pytestmark = pytest.mark.gpu


def _noalloc(dw):
    import paper_2609_12471_amd as kva
    t = torch()
    w = dw.w
    out = t.full((w.B, w.Hq, w.D), float("nan"), dtype=t.float32, device="cuda")
    lse = t.full((w.B, w.Hq), float("nan"), dtype=t.float32, device="cuda")
    kva.kva_decode_attn_paged_noalloc(dw.q, dw.k, dw.v, dw.block_table, dw.seq_lens, out, lse,
                                      scale=w.scale)
    t.cuda.synchronize()
    return out.cpu().numpy(), lse.cpu().numpy()


def test_noalloc_matches_the_workspace_call_on_two_calls_in_a_row():
    rng = np.random.default_rng(9100)
    big = W.make_paged(rng.integers(512, 8193, size=64), key=(9100, 0))
    small = W.make_paged(rng.integers(1, 3000, size=9), key=(9100, 1))
    for tag, w in (("B=64", big), ("B=9", small)):
        print(f"[noalloc] {tag}", flush=True)
        dw = DeviceWorkload(w)
        o_na, l_na = _noalloc(dw)
        o_ws, l_ws = run_gpu(dw)
        assert np.array_equal(o_na.view(np.uint32), o_ws.view(np.uint32)), tag
        assert np.array_equal(l_na.view(np.uint32), l_ws.view(np.uint32)), tag
        ref, rlse = run_oracle(w)
        assert_parity(o_na, ref, l_na, rlse, tag=f"noalloc {tag}")


def test_noalloc_rejects_a_batch_beyond_the_scratch():
    import paper_2609_12471_amd as kva
    t = torch()
    B, Hq, Hkv, D = 2048, 64, 8, 128
    q = t.zeros((B, Hq, D), dtype=t.int16, device="cuda")
    pool = t.zeros((4, 16, Hkv, D), dtype=t.int16, device="cuda")
    bt = t.zeros((B, 1), dtype=t.int32, device="cuda")
    lens = t.zeros((B,), dtype=t.int32, device="cuda")
    out = t.full((B, Hq, D), 7.0, dtype=t.float32, device="cuda")
    with pytest.raises(kva.KvaError) as e:
        kva.kva_decode_attn_paged_noalloc(q, pool, pool, bt, lens, out, scale=0.1)
    assert e.value.status == 7
    t.cuda.synchronize()
    assert bool((out == 7.0).all()), "a rejected call must leave the output untouched"
