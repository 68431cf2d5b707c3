"""Shared-prefix (group) decode on the GPU against the fp64 oracle.

A grouped call must equal plain attention over each sequence's own block-table
row, so the reference is the same paged oracle as for kva_decode_attn_paged.
Cases cover the shared run being found (or not) on the device: full sharing,
group sizes that do not divide B, runs cut by a short member, tables that
diverge inside the prompt, no sharing, empty members, narrow and wide pages,
and every supported query-group size."""
import dataclasses

import numpy as np
import pytest

import workloads as W
from kva_testlib import DeviceWorkload, assert_parity, run_gpu, run_oracle, torch

pytestmark = pytest.mark.gpu


def run_grouped(dw, group, *, lse=True, workspace=None):
    import paper_2609_12471_amd as kva
    t = torch()
    w = dw.w
    out = t.empty((w.B, w.Hq, w.D), dtype=t.float32, device="cuda")
    ls = t.empty((w.B, w.Hq), dtype=t.float32, device="cuda") if lse else None
    kva.kva_decode_attn_paged_grouped(dw.q, dw.k, dw.v, dw.block_table, dw.seq_lens, out, ls,
                                      group=group, scale=w.scale, workspace=workspace)
    t.cuda.synchronize()
    return out.cpu().numpy(), (ls.cpu().numpy() if lse else None)


def check(w, group, tag):
    print(f"[grouped] {tag}: B={w.B} group={group} P={w.page_size} Hq={w.Hq} Hkv={w.Hkv}",
          flush=True)
    out, lse = run_grouped(DeviceWorkload(w), group)
    ref, rlse = run_oracle(w)
    return assert_parity(out, ref, lse, rlse, tag=tag)


def test_c5_grouped_parity():
    w = W.make_config(5)
    check(w, 8, "c5 grouped")


@pytest.mark.parametrize("lens,group,prefix,P,Hq,Hkv", [
    ([300, 500, 1000, 40 + 256], 4, 256, 16, 32, 8),
    ([700, 900, 650, 1200, 800, 777, 1500, 1111, 999, 640], 4, 512, 16, 32, 8),   # last group of 2
    ([100, 200, 300], 3, 96, 16, 32, 8),              # shared run = the shortest member
    ([256, 512, 700, 256], 4, 256, 16, 32, 8),        # two members have no tokens of their own
    ([1000, 1300, 1700, 1031], 4, 1000, 1, 32, 8),    # one-token pages
    ([600, 650, 700, 900, 333, 777], 6, 320, 4, 16, 4),
    ([2000, 2100, 2200, 2300], 4, 1920, 64, 32, 8),
    ([3000, 2500, 4000, 2600, 3500, 2900, 3100, 2700], 8, 2048, 128, 32, 8),
    ([900, 1000, 1100, 1200], 4, 768, 16, 64, 8),     # 8 query heads per KV head, 32 rows
    ([500] * 32, 32, 384, 16, 8, 8),                  # one query head per KV head, 32 members
    ([800, 820, 840, 860, 880, 900, 920, 940] * 2, 16, 640, 16, 16, 8),
    ([1024, 1500, 1200, 1800], 1, 0, 16, 32, 8),      # group 1: the plain path
    ([12, 9, 15, 7], 4, 0, 16, 32, 8),                # shorter than one granule
    ([4200, 4500, 5000, 4300], 4, 4096, 16, 32, 8),   # shared run past the first 192 table entries
    ([1500, 1600, 1700, 1800], 4, 1008, 16, 32, 8),   # odd granule count: a half block at the end
])
def test_grouped_shapes(lens, group, prefix, P, Hq, Hkv):
    key = (7100, len(lens), group, P, Hq)
    sp = (group, prefix) if prefix else None
    w = W.make_paged(lens, page_size=P, Hq=Hq, Hkv=Hkv, key=key, shared_prefix=sp)
    check(w, group, f"lens={lens[:4]}.. group={group} prefix={prefix} P={P} Hq={Hq}")


def _with(w, **kw):
    return dataclasses.replace(w, **kw)


def test_grouped_table_diverges_inside_the_prompt():
    lens = [1500, 1600, 1700, 1800, 1550, 1650, 1750, 1850]
    w = W.make_paged(lens, page_size=16, key=(7200,), shared_prefix=(4, 1024))
    bt = w.block_table.copy()
    # member 2 of group 0 takes page 37 from member 0's own (non-shared) pages
    bt[2, 37] = w.block_table[0, 70]
    # member 1 of group 1 differs already at page 0
    bt[5, 0] = w.block_table[4, 80]
    check(_with(w, block_table=bt), 4, "diverging tables")


def test_grouped_member_shorter_than_the_prompt():
    lens = [2000, 2100, 2200, 2300]
    w = W.make_paged(lens, page_size=16, key=(7300,), shared_prefix=(4, 1600))
    sl = w.seq_lens.copy()
    sl[3] = 901            # the shared run must stop at 896 tokens
    check(_with(w, seq_lens=sl), 4, "short member")


def test_grouped_without_shared_pages():
    lens = [800, 900, 1000, 1100, 1200, 1300, 1400, 1500]
    w = W.make_paged(lens, page_size=16, key=(7400,))
    check(w, 8, "no sharing")


def test_grouped_with_empty_members():
    lens = [1000, 0, 1200, 1300, 0, 0, 0, 0, 700, 800, 900, 1000]
    w = W.make_paged(lens, page_size=16, key=(7500,))
    bt = w.block_table.copy()
    # members 8..11 share their first 20 pages
    bt[9:12, :20] = bt[8, :20]
    check(_with(w, block_table=bt), 4, "empty members")


def test_grouped_is_deterministic_with_a_dirty_workspace():
    import paper_2609_12471_amd as kva
    t = torch()
    w = W.make_paged([1200, 1300, 1400, 1500, 1600, 1700, 1800, 1900], page_size=16, key=(7600,),
                     shared_prefix=(8, 1024))
    dw = DeviceWorkload(w)
    ws = t.full((kva.kva_workspace_bytes_grouped(w.B, w.Hq, w.Hkv, w.D, 8),), 0xFF,
                dtype=t.uint8, device="cuda")
    o1, l1 = run_grouped(dw, 8, workspace=ws)
    o2, l2 = run_grouped(dw, 8, workspace=ws)
    assert np.array_equal(o1.view(np.uint32), o2.view(np.uint32))
    assert np.array_equal(l1.view(np.uint32), l2.view(np.uint32))
    # and it agrees with the plain paged call to within fp32 rounding
    o3, l3 = run_gpu(dw)
    assert np.max(np.abs(o1 - o3)) < 1e-5 and np.max(np.abs(l1 - l3)) < 1e-5


def test_grouped_batch_above_one_launch():
    """B = 4200 sequences in groups of 8 (several attention launches): the
    launch slices are cut at group multiples, the shared-run lengths of later
    slices are read at their group offset, and each launch's merge reads its
    slots through the global plan.  Short lengths keep the oracle cheap."""
    rng = np.random.default_rng(7700)
    B = 4200
    lens = 32 + rng.integers(0, 60, size=B)
    lens[np.arange(3, B, 97)] = 32             # members as short as the shared run
    w = W.make_paged(lens, page_size=16, key=(7700,), shared_prefix=(8, 32))
    check(w, 8, "B=4200 group 8")


@pytest.mark.parametrize("weights", ["64,1", "1,64", "1,1"])
def test_grouped_part_weights(weights, monkeypatch):
    """The parts of a shared run take block ranges in proportion to the weight
    of their XCD parity; at 64:1 either way the light parts, and some waves of
    the heavy ones, get no block and write empty results, which the merge must
    skip."""
    monkeypatch.setenv("KVA_XCD_WEIGHTS", weights)
    lens = [1500, 1700, 1900, 2100, 1600, 1800, 2000, 2200]
    w = W.make_paged(lens, page_size=16, key=(7800,), shared_prefix=(8, 1024))
    check(w, 8, f"part weights {weights}")


def test_grouped_plain_order(monkeypatch):
    """Equal part ranges (the placement-agnostic order of partitioned devices)."""
    monkeypatch.setenv("KVA_XCD_MAP", "0")
    lens = [900, 1000, 1100, 1200, 1300, 1400, 1500, 1600] * 2
    w = W.make_paged(lens, page_size=16, key=(7900,), shared_prefix=(8, 768))
    check(w, 8, "plain order")
