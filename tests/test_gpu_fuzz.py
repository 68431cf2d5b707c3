"""Seeded random cases through every attention entry point against the oracle.

The other GPU tests pick their shapes by hand; these draw them: batch sizes,
length mixes (empty, shorter than a granule, a page, or a wave's share, and
long), page sizes, query-group sizes, cache types, scales, shared prefixes and
prefill chunks, each case printed before it runs.  Sizes stay small enough
for the oracle to finish every case in well under a second."""
import dataclasses

import numpy as np
import pytest

import oracle
import workloads as W
from kva_testlib import DeviceWorkload, assert_parity, dev, run_gpu, run_oracle, torch

pytestmark = pytest.mark.gpu

PAGES = [1, 2, 4, 8, 16, 32, 64, 128, 1024]
HEADS = [(32, 8), (16, 8), (8, 8), (64, 8), (4, 1), (32, 4), (16, 2)]


def draw_lengths(rng, B):
    kind = rng.integers(0, 4)
    if kind == 0:                                   # anything up to ~2.5K
        lens = rng.integers(0, 2500, size=B)
    elif kind == 1:                                 # short: around granule and page sizes
        lens = rng.choice([0, 1, 2, 15, 16, 17, 31, 32, 33, 63, 64, 65, 255, 256, 257], size=B)
    elif kind == 2:                                 # one long sequence among short ones
        lens = rng.integers(0, 40, size=B)
        lens[rng.integers(0, B)] = rng.integers(1500, 4000)
    else:                                           # log-normal around 600
        lens = np.clip(rng.lognormal(np.log(600), 0.8, size=B), 0, 4000).astype(np.int64)
    return [int(x) for x in lens]


def decode_cases(n=24, seed=9900):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        B = int(rng.integers(1, 25))
        Hq, Hkv = HEADS[rng.integers(0, len(HEADS))]
        out.append(dict(i=i, B=B, lens=draw_lengths(rng, B), Hq=Hq, Hkv=Hkv,
                        layout="paged" if rng.random() < 0.7 else "contig",
                        P=int(PAGES[rng.integers(0, len(PAGES))]),
                        fp8=bool(rng.random() < 0.35),
                        scale=float(rng.uniform(-0.3, 0.3))))
    return out


@pytest.mark.parametrize("c", decode_cases(), ids=lambda c: f"decode{c['i']}")
def test_fuzz_decode(c):
    print(f"[fuzz] {c}", flush=True)
    key = (9900, c["i"])
    if c["layout"] == "paged":
        w = W.make_paged(c["lens"], page_size=c["P"], Hq=c["Hq"], Hkv=c["Hkv"], key=key)
    else:
        w = W.make_contig(c["lens"], max(c["lens"]) + 3, Hq=c["Hq"], Hkv=c["Hkv"], key=key)
    if c["fp8"]:
        w = W.quantize_fp8(w)
    w = dataclasses.replace(w, scale=c["scale"])
    out, lse = run_gpu(DeviceWorkload(w))
    ref, rlse = run_oracle(w)
    assert_parity(out, ref, lse, rlse, tag=f"fuzz decode {c}")


def grouped_cases(n=10, seed=9910):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        Hq, Hkv = HEADS[rng.integers(0, len(HEADS))]
        G = Hq // Hkv
        group = int(rng.choice([g for g in (2, 3, 4, 5, 8) if g * G <= 32]))
        ngroups = int(rng.integers(1, 5))
        P = int(rng.choice([16, 32, 64]))
        prefix = P * int(rng.integers(1, 40))
        lens = []
        for _ in range(ngroups):
            lens += [prefix + int(x) for x in rng.integers(0, 900, size=group)]
        B = len(lens) - int(rng.integers(0, group))          # last group may be short
        out.append(dict(i=i, lens=lens[:B], group=group, prefix=prefix, P=P, Hq=Hq, Hkv=Hkv,
                        scale=float(rng.uniform(-0.3, 0.3))))
    return out


@pytest.mark.parametrize("c", grouped_cases(), ids=lambda c: f"grouped{c['i']}")
def test_fuzz_grouped(c):
    import paper_2609_12471_amd as kva
    print(f"[fuzz] {c}", flush=True)
    t = torch()
    w = W.make_paged(c["lens"], page_size=c["P"], Hq=c["Hq"], Hkv=c["Hkv"], key=(9910, c["i"]),
                     shared_prefix=(c["group"], c["prefix"]))
    w = dataclasses.replace(w, scale=c["scale"])
    dw = DeviceWorkload(w)
    out = t.empty((w.B, w.Hq, w.D), dtype=t.float32, device="cuda")
    ls = t.empty((w.B, w.Hq), dtype=t.float32, device="cuda")
    kva.kva_decode_attn_paged_grouped(dw.q, dw.k, dw.v, dw.block_table, dw.seq_lens, out, ls,
                                      group=c["group"], scale=w.scale)
    t.cuda.synchronize()
    ref, rlse = run_oracle(w)
    assert_parity(out.cpu().numpy(), ref, ls.cpu().numpy(), rlse, tag=f"fuzz grouped {c}")


def prefill_cases(n=8, seed=9920):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        B = int(rng.integers(1, 6))
        Hq, Hkv = HEADS[rng.integers(0, len(HEADS))]
        out.append(dict(i=i, ctx=[int(x) for x in rng.integers(0, 1500, size=B)],
                        n=[int(x) for x in rng.choice([0, 1, 7, 31, 64, 65, 200], size=B)],
                        P=int(PAGES[rng.integers(0, len(PAGES))]), Hq=Hq, Hkv=Hkv,
                        scale=float(rng.uniform(-0.3, 0.3))))
    return out


@pytest.mark.parametrize("c", prefill_cases(), ids=lambda c: f"prefill{c['i']}")
def test_fuzz_prefill(c):
    import paper_2609_12471_amd as kva
    print(f"[fuzz] {c}", flush=True)
    t = torch()
    p = W.make_prefill(c["ctx"], c["n"], page_size=c["P"], Hq=c["Hq"], Hkv=c["Hkv"],
                       key=(9920, c["i"]))
    cc = p.cache
    out = t.full((max(p.T, 1), cc.Hq, cc.D), float("nan"), dtype=t.float32, device="cuda")[:p.T]
    ls = t.empty((max(p.T, 1), cc.Hq), dtype=t.float32, device="cuda")[:p.T]
    mq = int(np.diff(p.q_start).max())
    kva.kva_prefill_paged(dev(p.q), dev(cc.k), dev(cc.v), dev(cc.block_table), dev(p.q_start),
                          dev(cc.seq_lens), out, ls, max_q_len=mq, scale=c["scale"])
    t.cuda.synchronize()
    if p.T == 0:
        return
    ref, rlse = oracle.prefill_paged(p.q, cc.k, cc.v, cc.block_table, p.q_start, cc.seq_lens,
                                     c["scale"])
    assert_parity(out.cpu().numpy(), ref, ls.cpu().numpy(), rlse, tag=f"fuzz prefill {c}")
