"""GPU parity: the HIP path through the C ABI against the fp64 oracle on the
same seeded inputs.  Gate (fp32 outputs, all outputs of a case): max-abs <=
2e-3, mean-abs <= 2e-4, every output finite, plus the tight elementwise
diagnostic |err| <= 1e-4 + 1e-4 |ref|; lse under the same bounds.

The five rollout-shaped configs run at full size in the launch configuration
the benchmark times; smaller cases cover ragged lengths, every supported GQA
group, page sizes from 1 to 1024, contiguous caches and batch sizes up to 1000.
"""
import numpy as np
import pytest

import workloads as W
from kva_testlib import DeviceWorkload, assert_parity, run_gpu, run_oracle

pytestmark = pytest.mark.gpu

_CACHE = {}


def _config(k):
    if k not in _CACHE:
        _CACHE.clear()                      # keep at most one full-size config resident
        w = W.make_config(k)
        _CACHE[k] = (w, DeviceWorkload(w), run_oracle(w))
    return _CACHE[k]


@pytest.mark.timeout(600)
@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_config_parity_full_size(k):
    print(f"[parity] config {k} {W.CONFIG_NAMES[k]}", flush=True)
    w, dw, (ref, rlse) = _config(k)
    out, lse = run_gpu(dw)
    rep = assert_parity(out, ref, lse, rlse, tag=W.CONFIG_NAMES[k])
    print(f"[parity] config {k}: {rep}", flush=True)


def _case(layout, lens, Hq=32, Hkv=8, page_size=16, key=(500,), Lmax=None):
    if layout == "contig":
        return W.make_contig(lens, Lmax or max(max(lens), 1), Hq=Hq, Hkv=Hkv, key=key)
    return W.make_paged(lens, page_size=page_size, Hq=Hq, Hkv=Hkv, key=key)


RAGGED = [1, 2, 15, 16, 17, 31, 33, 64, 100, 255, 256, 257, 1000, 1023, 2049, 4097]


@pytest.mark.parametrize("layout", ["contig", "paged"])
@pytest.mark.parametrize("Hq,Hkv", [(32, 8), (32, 32), (32, 16), (32, 4), (4, 1), (8, 1)])
def test_ragged_lengths_every_group(layout, Hq, Hkv):
    print(f"[parity] ragged {layout} Hq={Hq} Hkv={Hkv}", flush=True)
    w = _case(layout, RAGGED, Hq=Hq, Hkv=Hkv, key=(501, Hq, Hkv))
    out, lse = run_gpu(DeviceWorkload(w))
    ref, rlse = run_oracle(w)
    assert_parity(out, ref, lse, rlse, tag=f"{layout} {Hq}/{Hkv}")


@pytest.mark.parametrize("page_size", [1, 2, 4, 8, 16, 32, 64, 256, 1024])
def test_page_sizes(page_size):
    print(f"[parity] page_size {page_size}", flush=True)
    lens = [1, 7, 16, 17, 300, 1025, 3000]
    w = _case("paged", lens, page_size=page_size, key=(502, page_size))
    out, lse = run_gpu(DeviceWorkload(w))
    ref, rlse = run_oracle(w)
    assert_parity(out, ref, lse, rlse, tag=f"P={page_size}")


def test_empty_sequences_and_zero_lengths():
    print("[parity] empty sequences", flush=True)
    for layout in ("contig", "paged"):
        w = _case(layout, [0, 5, 0, 0, 40, 0], key=(503,))
        out, lse = run_gpu(DeviceWorkload(w))
        ref, rlse = run_oracle(w)
        assert np.all(out[[0, 2, 3, 5]] == 0.0)
        assert np.all(np.isneginf(lse[[0, 2, 3, 5]]))
        assert_parity(out, ref, lse, rlse, tag=f"{layout} empties")
        w0 = _case(layout, [0, 0, 0], key=(504,), Lmax=16)
        out, lse = run_gpu(DeviceWorkload(w0))
        assert np.all(out == 0.0) and np.all(np.isneginf(lse))


def test_many_short_sequences():
    """1000 sequences: the per-wave search for its first sequence crosses many
    64-sequence chunks."""
    print("[parity] B=1000 short", flush=True)
    rng = np.random.default_rng(505)
    lens = rng.integers(0, 80, size=1000)
    w = _case("paged", lens, key=(505,))
    out, lse = run_gpu(DeviceWorkload(w))
    ref, rlse = run_oracle(w)
    assert_parity(out, ref, lse, rlse, tag="B=1000")


@pytest.mark.parametrize("layout,B", [("paged", 4500), ("contig", 2500)])
def test_batches_above_one_launch(layout, B):
    """Batches longer than one attention launch takes (2048 sequences) are
    split into several launches sharing one workspace."""
    print(f"[parity] {layout} B={B} (several launches)", flush=True)
    rng = np.random.default_rng(509)
    lens = rng.integers(0, 70, size=B)
    w = _case(layout, lens, key=(509, B), Lmax=72 if layout == "contig" else None)
    out, lse = run_gpu(DeviceWorkload(w))
    ref, rlse = run_oracle(w)
    assert_parity(out, ref, lse, rlse, tag=f"{layout} B={B}")


@pytest.mark.parametrize("weights,layout", [("1,1", "paged"), ("27,25", "paged"), ("64,1", "paged"),
                                            ("1,64", "contig"), ("5,3", "contig")])
def test_xcd_range_weights(weights, layout, monkeypatch):
    """Ranges weighted by the parity of the wave's XCD: every granule is still
    covered exactly once (parity), with ragged lengths that put range ends
    inside sequences.  At 64:1 either way the lightest range would be empty
    for this batch, which must take the equal-range fallback (an empty range
    would leave a merge slot between a sequence's pieces unwritten)."""
    monkeypatch.setenv("KVA_XCD_WEIGHTS", weights)
    print(f"[parity] xcd weights {weights} {layout}", flush=True)
    rng = np.random.default_rng(512)
    lens = rng.integers(1, 3000, size=37)
    lens[5] = 0
    w = _case(layout, lens, key=(512, 0 if layout == "paged" else 1))
    out, lse = run_gpu(DeviceWorkload(w))
    ref, rlse = run_oracle(w)
    assert_parity(out, ref, lse, rlse, tag=f"xcd {weights}")


@pytest.mark.parametrize("vgran,layout,page_size", [("0", "paged", 16), ("1", "contig", None),
                                                     ("7", "paged", 16), ("64", "paged", 16),
                                                     ("64", "contig", None), ("64", "paged", 4),
                                                     ("2", "paged", 4)])
def test_piece_granules(vgran, layout, page_size, monkeypatch):
    """Virtual granules ahead of every sequence in the work partition: ranges
    that cross into a sequence pay them, and at 64 many ranges hold nothing
    but virtual granules (no piece, no slot; such a wave must not load at all,
    which matters for pages smaller than a granule).  Every real granule must
    still be covered exactly once, with ragged and empty lengths."""
    monkeypatch.setenv("KVA_PIECE_GRANULES", vgran)
    print(f"[parity] piece granules {vgran} {layout} P={page_size}", flush=True)
    rng = np.random.default_rng(514)
    lens = rng.integers(0, 2500, size=41)
    lens[[3, 17]] = 0
    lens[9] = 1
    kw = {"page_size": page_size} if page_size else {}
    w = _case(layout, lens, key=(514, 0 if layout == "paged" else 1), **kw)
    out, lse = run_gpu(DeviceWorkload(w))
    ref, rlse = run_oracle(w)
    assert_parity(out, ref, lse, rlse, tag=f"vgran {vgran}")


@pytest.mark.parametrize("layout", ["paged", "contig"])
def test_plain_wave_order(layout, monkeypatch):
    """Equal ranges in wave order (the mapping of partitioned devices and of
    the fp8 kernels) for the bf16 kernel."""
    monkeypatch.setenv("KVA_XCD_MAP", "0")
    print(f"[parity] plain wave order {layout}", flush=True)
    rng = np.random.default_rng(513)
    lens = rng.integers(0, 5000, size=45)
    w = _case(layout, lens, key=(513, 0 if layout == "paged" else 1))
    out, lse = run_gpu(DeviceWorkload(w))
    ref, rlse = run_oracle(w)
    assert_parity(out, ref, lse, rlse, tag=f"plain order {layout}")


def test_single_long_sequence_max_length():
    """One 16384-token sequence (the longest rollout context): split over many
    waves and merged by the combine kernel."""
    print("[parity] B=1 L=16384", flush=True)
    w = _case("paged", [16384], key=(506,))
    out, lse = run_gpu(DeviceWorkload(w))
    ref, rlse = run_oracle(w)
    assert_parity(out, ref, lse, rlse, tag="L=16384")


def test_lengths_beyond_capacity_are_clamped():
    """Device lengths above the capacity are clamped to it, never read past."""
    print("[parity] clamped lengths", flush=True)
    w = _case("contig", [40, 64], key=(507,), Lmax=64)
    dw = DeviceWorkload(w)
    import torch
    dw.seq_lens = torch.tensor([40, 1000], dtype=torch.int32, device="cuda")
    out, lse = run_gpu(dw)
    ref, rlse = run_oracle(w)
    assert_parity(out, ref, lse, rlse, tag="clamp")


def test_no_lse_requested():
    w = _case("paged", [100, 200], key=(508,))
    out, _ = run_gpu(DeviceWorkload(w), lse=False)
    ref, _ = run_oracle(w)
    assert_parity(out, ref, tag="no lse")


@pytest.mark.parametrize("layout", ["paged", "contig"])
def test_negative_and_large_scales(layout):
    """A negative scale (weights favour the lowest scores) and a large one
    (peaked weights that move the running maximum often)."""
    w = _case(layout, [5, 130, 2049, 700], key=(511, 0 if layout == "paged" else 1))
    for scale in (-0.0883883476, 0.7):
        print(f"[parity] {layout} scale={scale}", flush=True)
        out, lse = run_gpu(DeviceWorkload(w), scale=scale)
        ref, rlse = run_oracle(w, scale=scale)
        assert_parity(out, ref, lse, rlse, tag=f"{layout} scale={scale}")


def test_scale_zero_gives_mean_of_values():
    w = _case("paged", [3, 50, 700], key=(509,))
    out, lse = run_gpu(DeviceWorkload(w), scale=0.0)
    ref, rlse = run_oracle(w, scale=0.0)
    assert_parity(out, ref, lse, rlse, tag="scale=0")
    np.testing.assert_allclose(lse, np.log(np.array([3, 50, 700]))[:, None] * np.ones((1, 32)),
                               rtol=0, atol=1e-5)


@pytest.mark.parametrize("S,D", [(1, 128), (3, 128), (70, 128), (5, 256), (4, 64), (0, 128)])
def test_combine_entry_point_matches_oracle(S, D):
    """kva_combine on fp32 parts (empty parts hold NaN and must be ignored)."""
    import torch
    import oracle
    import paper_2609_12471_amd as kva
    rng = np.random.default_rng(510 + S + D)
    B, Hq = 6, 8
    o = rng.standard_normal((S, B, Hq, D)).astype(np.float32)
    l = (rng.standard_normal((S, B, Hq)) * 3).astype(np.float32)
    l[rng.random((S, B, Hq)) < 0.2] = -np.inf
    if S:
        l[:, 0, 0] = -np.inf                         # every part of (0, 0) empty
    o[np.broadcast_to(np.isneginf(l)[..., None], o.shape)] = np.nan
    ref, rlse = oracle.combine(o.astype(np.float64), l.astype(np.float64))
    ref = np.nan_to_num(ref)                         # oracle skips empty parts too
    out = torch.empty((B, Hq, D), dtype=torch.float32, device="cuda")
    lse = torch.empty((B, Hq), dtype=torch.float32, device="cuda")
    kva.kva_combine(torch.from_numpy(o).cuda(), torch.from_numpy(l).cuda(), out, lse)
    torch.cuda.synchronize()
    assert_parity(out.cpu().numpy(), ref, lse.cpu().numpy(), rlse, tag=f"combine S={S} D={D}")


def test_context_shards_merge_to_the_whole():
    """One sequence split into two page-aligned shards (as context parallelism
    across GPUs would split it), each attended separately, then kva_combine:
    equal to attending the whole sequence."""
    import torch
    import paper_2609_12471_amd as kva
    from kva_testlib import dev
    L, cut = 5000, 2000
    w = W.make_paged([L], key=(511,))
    dw = DeviceWorkload(w)
    whole, wlse = run_gpu(dw)
    outs, lses = [], []
    for lo, hi in ((0, cut), (cut, L)):
        bt = np.full((1, w.max_pages), -1, np.int32)
        n = (hi - lo + 15) // 16
        bt[0, :n] = w.block_table[0, lo // 16: lo // 16 + n]
        o = torch.empty((1, 32, 128), dtype=torch.float32, device="cuda")
        ls = torch.empty((1, 32), dtype=torch.float32, device="cuda")
        kva.kva_decode_attn_paged(dw.q, dw.k, dw.v, dev(bt), dev(np.array([hi - lo], np.int32)),
                                  o, ls, scale=w.scale)
        outs.append(o); lses.append(ls)
    out = torch.empty((1, 32, 128), dtype=torch.float32, device="cuda")
    lse = torch.empty((1, 32), dtype=torch.float32, device="cuda")
    kva.kva_combine(torch.stack(outs).contiguous(), torch.stack(lses).contiguous(), out, lse)
    torch.cuda.synchronize()
    ref, rlse = run_oracle(w)
    assert_parity(out.cpu().numpy(), ref, lse.cpu().numpy(), rlse, tag="shards")
    np.testing.assert_allclose(out.cpu().numpy(), whole, rtol=0, atol=1e-6)


def test_workspace_reuse_across_calls():
    """One workspace, filled with garbage once, reused by consecutive calls of
    different shapes (whose layouts overlap differently): every call is
    correct, with no initialisation of the workspace at any point."""
    import torch
    import paper_2609_12471_amd as kva
    ws = kva.kva_new_workspace(300, 32, 8, 128)
    ws.copy_(torch.randint(0, 256, ws.shape, dtype=torch.uint8, device=ws.device))
    cases = [_case("paged", [16384], key=(520,)),
             _case("paged", RAGGED, key=(521,)),
             _case("contig", [5000, 3, 0, 900], key=(522,)),
             _case("paged", [16384, 40, 7000], key=(523,)),
             _case("paged", [16384], key=(520,))]
    for n, w in enumerate(cases):
        print(f"[parity] workspace reuse call {n}", flush=True)
        out, lse = run_gpu(DeviceWorkload(w), workspace=ws)
        ref, rlse = run_oracle(w)
        assert_parity(out, ref, lse, rlse, tag=f"reuse {n}")


def test_temporary_workspace_on_a_side_stream():
    """No workspace passed and the call queued on a side stream that is not
    the current one: the binding's temporary workspace is tied to that stream,
    so a tensor allocated and written on the current stream right after the
    call cannot take its memory while the kernels are still queued."""
    import torch
    import paper_2609_12471_amd as kva
    rng = np.random.default_rng(530)
    w = _case("paged", rng.integers(3000, 9000, size=48), key=(530,))
    dw = DeviceWorkload(w)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    outs = []
    for rep in range(3):
        out = torch.empty((w.B, w.Hq, w.D), dtype=torch.float32, device="cuda")
        lse = torch.empty((w.B, w.Hq), dtype=torch.float32, device="cuda")
        out.record_stream(side)
        lse.record_stream(side)
        # keep the side stream busy first, so the attention kernels are still queued
        with torch.cuda.stream(side):
            torch.cuda._sleep(2_000_000)
        kva.kva_decode_attn_paged(dw.q, dw.k, dw.v, dw.block_table, dw.seq_lens, out, lse,
                                  scale=w.scale, stream=side)
        # allocations of the same size on the current stream, filled at once
        junk = [torch.full((kva.kva_workspace_bytes(w.B, w.Hq, w.Hkv, w.D) // 4,), float("nan"),
                           dtype=torch.float32, device="cuda") for _ in range(2)]
        side.synchronize()
        torch.cuda.synchronize()
        del junk
        outs.append((out.cpu().numpy(), lse.cpu().numpy()))
    ref, rlse = run_oracle(w)
    for o, l in outs:
        assert_parity(o, ref, l, rlse, tag="side stream")
    with pytest.raises(ValueError):
        out = torch.empty((w.B, w.Hq, w.D), dtype=torch.float32, device="cuda")
        kva.kva_decode_attn_paged(dw.q, dw.k, dw.v, dw.block_table, dw.seq_lens, out,
                                  scale=w.scale, stream=side.cuda_stream)
