"""fp8 (e4m3fn) caches on the GPU against the fp64 oracle on the same codes
and scales, under the same gate as the bf16 path (max-abs 2e-3, mean-abs 2e-4,
and the paper's checker tolerance elementwise).  The kernels widen the codes
exactly, so the only differences from the oracle are fp32 rounding."""
import numpy as np
import pytest

import workloads as W
from kva_testlib import DeviceWorkload, assert_parity, run_gpu, run_oracle

pytestmark = pytest.mark.gpu


def check(w, tag):
    print(f"[fp8] {tag}: B={w.B} layout={w.layout} P={w.page_size}", flush=True)
    out, lse = run_gpu(DeviceWorkload(w))
    ref, rlse = run_oracle(w)
    return assert_parity(out, ref, lse, rlse, tag=tag)


@pytest.mark.parametrize("k", [2, 3, 4, 5])
def test_fp8_full_configs(k):
    check(W.quantize_fp8(W.make_config(k)), f"config {k} fp8")


@pytest.mark.parametrize("P", [1, 4, 16, 64, 1024])
def test_fp8_page_sizes(P):
    lens = [0, 1, 15, 16, 17, 500, 2049, 4000]
    check(W.quantize_fp8(W.make_paged(lens, page_size=P, key=(9100, P))), f"P={P}")


@pytest.mark.parametrize("P", [4, 16])
def test_fp8_ranges_of_virtual_granules_only(P, monkeypatch):
    """With many virtual granules per sequence in the work partition, many
    waves hold no real granule and must return before loading anything (the
    narrow-page loads would otherwise fall back to a row before the first)."""
    monkeypatch.setenv("KVA_PIECE_GRANULES", "64")
    rng = np.random.default_rng(9150)
    lens = rng.integers(0, 1500, size=29)
    lens[[2, 11]] = 0
    lens[5] = 1
    check(W.quantize_fp8(W.make_paged(lens, page_size=P, key=(9150, P))), f"vgran 64 P={P}")


@pytest.mark.parametrize("Hq,Hkv", [(8, 8), (16, 8), (64, 8), (4, 1)])
def test_fp8_head_groups(Hq, Hkv):
    lens = [33, 1000, 2500, 7]
    check(W.quantize_fp8(W.make_paged(lens, page_size=16, Hq=Hq, Hkv=Hkv, key=(9200, Hq))),
          f"Hq={Hq} Hkv={Hkv}")


def test_fp8_contiguous_ragged_with_poison_and_empties():
    lens = [0, 1, 31, 256, 0, 1000]
    check(W.quantize_fp8(W.make_contig(lens, 1024, key=(9300,))), "contig ragged")


@pytest.mark.parametrize("layout", ["paged", "contig"])
def test_fp8_negative_and_large_scales(layout):
    """The matrix-core engine's lazily moved maximum under a negative scale
    (weights favour the lowest scores) and a large one (peaked weights)."""
    lens = [5, 130, 2049, 700, 33]
    w = W.quantize_fp8(W.make_paged(lens, page_size=16, key=(9500,)) if layout == "paged"
                       else W.make_contig(lens, 2100, key=(9501,)))
    for scale in (-0.0883883476, 0.7):
        print(f"[fp8] {layout} scale={scale}", flush=True)
        out, lse = run_gpu(DeviceWorkload(w), scale=scale)
        ref, rlse = run_oracle(w, scale=scale)
        assert_parity(out, ref, lse, rlse, tag=f"fp8 {layout} scale={scale}")


def test_fp8_is_deterministic():
    w = W.quantize_fp8(W.make_paged([3000, 5000, 100], page_size=16, key=(9400,)))
    dw = DeviceWorkload(w)
    o1, l1 = run_gpu(dw)
    o2, l2 = run_gpu(dw)
    assert np.array_equal(o1.view(np.uint32), o2.view(np.uint32))
    assert np.array_equal(l1.view(np.uint32), l2.view(np.uint32))


def test_fp8_batch_above_one_launch():
    """B = 4500 paged fp8 sequences: several attention launches over one workspace."""
    rng = np.random.default_rng(9500)
    lens = rng.integers(0, 70, size=4500)
    check(W.quantize_fp8(W.make_paged(lens, page_size=16, key=(9500,))), "fp8 B=4500")
