"""Shared helpers for the GPU tests: device copies of seeded workloads, calls
through the C ABI (via the Python binding), the oracle run over independent
sequences in threads, and the parity gate."""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

import oracle
import workloads as W

# Parity gate on fp32 outputs against the fp64 oracle, over all outputs of a case.
MAX_ABS = 2e-3
MEAN_ABS = 2e-4
# Tight diagnostic: the elementwise tolerance of the paper's HIP checker
# (torch.allclose with rtol = atol = 1e-4, Unified Pipeline Architecture).
DIAG_ATOL = 1e-4
DIAG_RTOL = 1e-4

_THREADS = max(1, min(16, os.cpu_count() or 1))


def torch():
    import torch as t
    return t


def dev(a: np.ndarray):
    """numpy -> contiguous device tensor (uint16 bits travel as int16)."""
    t = torch()
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return t.from_numpy(np.ascontiguousarray(a)).to("cuda")


class DeviceWorkload:
    def __init__(self, w: W.Workload):
        self.w = w
        self.q = dev(w.q)
        self.k = dev(w.k)
        self.v = dev(w.v)
        self.seq_lens = dev(w.seq_lens)
        self.block_table = dev(w.block_table) if w.layout == "paged" else None


def is_fp8(w: W.Workload) -> bool:
    return w.meta.get("kv_dtype") == "fp8_e4m3fn"


def run_gpu(dw: DeviceWorkload, *, lse=True, workspace=None, scale=None, stream=None):
    import paper_2609_12471_amd as kva
    t = torch()
    w = dw.w
    out = t.empty((w.B, w.Hq, w.D), dtype=t.float32, device="cuda")
    ls = t.empty((w.B, w.Hq), dtype=t.float32, device="cuda") if lse else None
    s = w.scale if scale is None else scale
    if is_fp8(w):
        ks, vs = w.meta["k_scale"], w.meta["v_scale"]
        if w.layout == "contig":
            kva.kva_decode_attn_fp8(dw.q, dw.k, dw.v, dw.seq_lens, out, ls, scale=s, k_scale=ks,
                                    v_scale=vs, workspace=workspace, stream=stream)
        else:
            kva.kva_decode_attn_paged_fp8(dw.q, dw.k, dw.v, dw.block_table, dw.seq_lens, out, ls,
                                          scale=s, k_scale=ks, v_scale=vs, workspace=workspace,
                                          stream=stream)
    elif w.layout == "contig":
        kva.kva_decode_attn(dw.q, dw.k, dw.v, dw.seq_lens, out, ls, scale=s, workspace=workspace,
                            stream=stream)
    else:
        kva.kva_decode_attn_paged(dw.q, dw.k, dw.v, dw.block_table, dw.seq_lens, out, ls,
                                  scale=s, workspace=workspace, stream=stream)
    t.cuda.synchronize()
    return out.cpu().numpy(), (ls.cpu().numpy() if lse else None)


def run_oracle(w: W.Workload, scale=None):
    """fp64 oracle over the whole batch, sequences split over host threads
    (each call is the oracle on a contiguous slice of the batch)."""
    s = w.scale if scale is None else scale
    B = w.B
    out = np.empty((B, w.Hq, w.D), np.float64)
    lse = np.empty((B, w.Hq), np.float64)
    # balance by tokens: cut the batch into ~4 slices per thread
    n_parts = max(1, min(B, 4 * _THREADS))
    cuts = np.linspace(0, B, n_parts + 1).astype(int)

    def work(i):
        b0, b1 = cuts[i], cuts[i + 1]
        if b1 <= b0:
            return
        if is_fp8(w):
            ks, vs = w.meta["k_scale"], w.meta["v_scale"]
            if w.layout == "contig":
                o, l = oracle.decode_attn_fp8(w.q[b0:b1], w.k[b0:b1], w.v[b0:b1],
                                              w.seq_lens[b0:b1], s, ks, vs)
            else:
                o, l = oracle.decode_attn_fp8(w.q[b0:b1], w.k, w.v, w.seq_lens[b0:b1], s, ks, vs,
                                              block_table=w.block_table[b0:b1])
        elif w.layout == "contig":
            o, l = oracle.decode_attn(w.q[b0:b1], w.k[b0:b1], w.v[b0:b1], w.seq_lens[b0:b1], s)
        else:
            o, l = oracle.decode_attn_paged(w.q[b0:b1], w.k, w.v, w.block_table[b0:b1],
                                            w.seq_lens[b0:b1], s)
        out[b0:b1] = o
        lse[b0:b1] = l

    with ThreadPoolExecutor(_THREADS) as ex:
        list(ex.map(work, range(n_parts)))
    return out, lse


def parity_report(out, ref, lse=None, rlse=None):
    out = np.asarray(out, np.float64)
    err = np.abs(out - ref)
    rep = {
        "finite": bool(np.all(np.isfinite(out))),
        "max_abs": float(err.max()) if err.size else 0.0,
        "mean_abs": float(err.mean()) if err.size else 0.0,
        "diag_viol": int(np.sum(err > DIAG_ATOL + DIAG_RTOL * np.abs(ref))),
    }
    if lse is not None:
        lse = np.asarray(lse, np.float64)
        fin = np.isfinite(rlse)
        rep["lse_inf_match"] = bool(np.array_equal(np.isneginf(lse), np.isneginf(rlse)))
        le = np.abs(lse[fin] - rlse[fin])
        rep["lse_max_abs"] = float(le.max()) if le.size else 0.0
        rep["lse_mean_abs"] = float(le.mean()) if le.size else 0.0
        rep["lse_diag_viol"] = int(np.sum(le > DIAG_ATOL + DIAG_RTOL * np.abs(rlse[fin])))
    return rep


def assert_parity(out, ref, lse=None, rlse=None, tag="", diag=True):
    """The gate; `diag=False` drops the tight elementwise diagnostic (used only
    where fp32 scores of magnitude ~1e3 make it unreachable by construction)."""
    rep = parity_report(out, ref, lse, rlse)
    msg = f"{tag}: {rep}"
    assert rep["finite"], msg
    assert rep["max_abs"] <= MAX_ABS and rep["mean_abs"] <= MEAN_ABS, msg
    if diag:
        assert rep["diag_viol"] == 0, msg
    if lse is not None:
        assert rep["lse_inf_match"], msg
        assert rep["lse_max_abs"] <= MAX_ABS and rep["lse_mean_abs"] <= MEAN_ABS, msg
        if diag:
            assert rep["lse_diag_viol"] == 0, msg
    return rep


def bits_f64(h):
    return W.bits_to_f32(h).astype(np.float64)
