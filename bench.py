#!/usr/bin/env python3
"""Benchmark: batched grouped-query decode attention on one MI355X.

One step = one decode-attention call for the whole batch (one layer, one
decode step): the attention kernel and the merge of split partials, through
the C ABI.  Default workload: 64 rollouts (8 prompts x 8 samples), paged K/V
with 16-token pages in a shuffled pool, lengths uniform in [512, 8192], Qwen3-8B
attention shape (32 query heads, 8 KV heads, head_dim 128), bf16 cache, fp32
softmax/accumulation and output.  Inputs are seeded synthetic data resident in
HBM before timing starts.

Metric: effective KV HBM bandwidth = algorithmic K+V bytes of the step (4096 B
per cached token; a page shared by several sequences counts once) / step time,
next to MI355X's 8 TB/s; plus us per step.

    python bench.py [--steps K] [--warmup W] [--config 3] [--no-cpu-baseline]
    python bench.py --config 5 --group 8     # shared-prefix (group) decode call
    python bench.py --append                 # step = new-token append + attention
    python bench.py --kv fp8                 # fp8 (e4m3fn) caches, 2 KiB per token
    python bench.py --prefill                # chunked prefill (matrix-core bound): TFLOP/s

Prints one JSON line.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
PROFILE_TRAFFIC = os.path.join(ROOT, "profiles", "decode_attn_paged_c3_traffic.json")
# sources of the decode attention kernel: a counter profile is used only while
# these are unchanged
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2609_12471_amd", "csrc", f)
                  for f in ("kva_kernels.hip", "kva_device.h", "kva_internal.h")]


def kernel_source_hash() -> str:
    """Hash of the kernel sources' code: comments and whitespace are dropped,
    so a comment edit does not retire the counter profiles."""
    import re
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(f, encoding="utf-8") as fh:
            src = fh.read()
        src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
        src = re.sub(r"//[^\n]*", " ", src)
        h.update(" ".join(src.split()).encode())
    return h.hexdigest()[:16]


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", type=int, default=3, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--group", type=int, default=1,
                    help="paged configs: sequences per group for kva_decode_attn_paged_grouped "
                         "(1 = the plain paged call)")
    ap.add_argument("--kv", choices=["bf16", "fp8"], default="bf16",
                    help="cache element type (fp8: OCP e4m3fn codes, per-tensor scales)")
    ap.add_argument("--append", action="store_true",
                    help="paged configs: each step first runs kva_append_paged for the new "
                         "token (RMS norm + rotary + k/v append), then attention")
    ap.add_argument("--prefill", action="store_true",
                    help="chunked prefill: 64 rollouts x 512 new tokens over 512..7680 tokens "
                         "of context (kva_prefill_paged); reports TFLOP/s")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--stream-read-gib", type=int, default=4,
                    help="decode runs: also time a plain streaming read of this many GiB "
                         "(kva_debug_stream_read) as the achievable bandwidth; 0 = skip")
    ap.add_argument("--cold-calls", type=int, default=30,
                    help="extra calls timed one by one with a 1 GiB cache flush before each")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target CPU time of the oracle baseline sample")
    ap.add_argument("--prewarm-s", type=float, default=0.3,
                    help="seconds of untimed steps before the warm-up steps")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after timing, run one 1 GiB device-to-device copy (a kernel of known "
                         "traffic, used to scale hardware byte counters)")
    return ap.parse_args()


def cpu_baseline(w, target_s: float):
    """The fp64 oracle, single-threaded, on the first sequences of the same
    workload (a bounded sample), scaled to GB/s of K+V bytes."""
    import numpy as np
    import oracle
    # estimate cost from one short sequence, then take a prefix of the batch
    fp8 = w.meta.get("kv_dtype") == "fp8_e4m3fn"

    def run(n):
        if fp8:
            bt = w.block_table[:n] if w.layout == "paged" else None
            kk, vv = (w.k, w.v) if w.layout == "paged" else (w.k[:n], w.v[:n])
            oracle.decode_attn_fp8(w.q[:n], kk, vv, w.seq_lens[:n], w.scale, w.meta["k_scale"],
                                   w.meta["v_scale"], block_table=bt)
        elif w.layout == "paged":
            oracle.decode_attn_paged(w.q[:n], w.k, w.v, w.block_table[:n], w.seq_lens[:n], w.scale)
        else:
            oracle.decode_attn(w.q[:n], w.k[:n], w.v[:n], w.seq_lens[:n], w.scale)

    # single-threaded, pinned to one core of those this process may use
    pinned = None
    try:
        allowed = os.sched_getaffinity(0)
        core = min(allowed)
        os.sched_setaffinity(0, {core})
        pinned = core
    except (AttributeError, OSError):
        allowed = None
    t0 = time.perf_counter()
    run(1)
    per_tok = (time.perf_counter() - t0) / max(1, int(w.seq_lens[0]))
    budget_tok = target_s / max(per_tok, 1e-9)
    csum = np.cumsum(w.seq_lens.astype(np.int64))
    n = int(max(1, min(w.B, np.searchsorted(csum, budget_tok) + 1)))
    # a batch that takes less than the budget is run whole, repeatedly
    reps = 1 if n < w.B else max(1, int(round(budget_tok / max(1, int(csum[-1])))))
    t0 = time.perf_counter()
    for _ in range(reps):
        run(n)
    dt = time.perf_counter() - t0
    if allowed is not None:
        os.sched_setaffinity(0, allowed)
    toks = int(csum[n - 1])
    kv_bytes = toks * w.Hkv * w.D * w.kv_elem_bytes * 2 * reps
    return {
        "value": round(kv_bytes / dt / 1e9, 5),
        "unit": "GB/s",
        "cores": 1,
        "kind": "oracle",
        "sample": (f"first {n} of {w.B} sequences ({toks} cached tokens, "
                   f"{toks * w.Hkv * w.D * w.kv_elem_bytes * 2 / 1e6:.1f} MB of K+V)"
                   + (f", {reps} runs" if reps > 1 else "")
                   + f", fp64 single-threaded, {dt:.1f} s"),
        "seconds": round(dt, 2),
        "cpu_model": _cpu_model(),
        "host_cpus": os.cpu_count(),
        "pinned_core": pinned,
    }


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def load_traffic(src_hash: str):
    try:
        rec = json.load(open(PROFILE_TRAFFIC))
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_hash") != src_hash:
        return None
    return rec.get("hbm_bytes_per_launch")


MFMA_BF16_PEAK_TFLOPS = 2500.0     # MI355X dense bf16 matrix-core peak


def run_prefill(args):
    import numpy as np
    import torch
    import workloads as W
    import paper_2609_12471_amd as kva

    kva.lib()
    t_gen = time.perf_counter()
    p = W.make_prefill_config()
    print(f"[bench] generated {W.PREFILL_NAME} in {time.perf_counter() - t_gen:.1f}s",
          file=sys.stderr, flush=True)
    c = p.cache
    dev = torch.device("cuda:0")

    def d(a):
        return torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a).to(dev)

    q, k, v, bt, qs, lens = d(p.q), d(c.k), d(c.v), d(c.block_table), d(p.q_start), d(c.seq_lens)
    out = torch.empty((p.T, c.Hq, c.D), dtype=torch.float32, device=dev)
    lse = torch.empty((p.T, c.Hq), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()
    mq = int(np.diff(p.q_start).max())

    def step():
        kva.kva_prefill_paged(q, k, v, bt, qs, lens, out, lse, max_q_len=mq, scale=c.scale,
                              stream=stream)

    t_pre = time.perf_counter()
    while time.perf_counter() - t_pre < args.prewarm_s:
        step()
        torch.cuda.synchronize()
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ev_s = ev0.elapsed_time(ev1) / 1e3 / args.steps
    flops = p.flops()
    value = flops * args.steps / elapsed / 1e12
    rec = {
        "metric": "chunked-prefill attention TFLOP/s (% of MI355X bf16 matrix-core peak)",
        "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(elapsed / args.steps * 1e3, 5),
        "us_per_step": round(elapsed / args.steps * 1e6, 2),
        "pct_of_peak": round(100.0 * value / MFMA_BF16_PEAK_TFLOPS, 2),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": W.PREFILL_NAME, "batch": c.B, "new_tokens": p.T,
                   "context_tokens": int(c.seq_lens.sum()) - p.T, "heads_q": c.Hq,
                   "heads_kv": c.Hkv, "head_dim": c.D, "page_size": c.page_size,
                   "flops": flops, "call": "kva_prefill_paged",
                   "compute": "bf16 q/K/V on the matrix cores (softmax weights as two bf16 "
                              "parts), fp32 softmax and accumulation, fp32 output"},
        "roofline": {"bound": "mfma", "achieved": round(flops / ev_s / 1e12, 2),
                     "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(flops / ev_s / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
                     "traffic": None, "kernel": "prefill_kernel (one launch per step)",
                     "event_us_avg": round(ev_s * 1e6, 2),
                     "flops_note": "QK and PV multiply-adds of the causal prefixes, 2 flops "
                                   "each; the second bf16 part of P is not counted",
                     "profile": "profiles/prefill_kernel_trace.md"},
        "kernel_source_hash": kernel_source_hash(),
    }
    if not args.no_cpu_baseline:
        import oracle
        # the oracle on the first tokens of the first rollout, scaled to TFLOP/s
        n0 = int(p.q_start[1])
        m = 8
        while True:
            sub_q = np.ascontiguousarray(p.q[:m])
            qs1 = np.array([0, m], np.int32)
            lens1 = np.array([int(c.seq_lens[0]) - n0 + m], np.int32)
            t1 = time.perf_counter()
            oracle.prefill_paged(sub_q, c.k, c.v, np.ascontiguousarray(c.block_table[:1]), qs1,
                                 lens1, c.scale)
            dt = time.perf_counter() - t1
            if dt > args.cpu_seconds / 4 or m >= n0:
                break
            m = min(n0, m * 4)
        ctx0 = int(lens1[0]) - m
        fl = (m * ctx0 + m * (m + 1) // 2) * c.Hq * c.D * 4
        rec["cpu_baseline"] = {"value": round(fl / dt / 1e12, 6), "unit": "TFLOP/s", "cores": 1,
                               "kind": "oracle",
                               "sample": f"first {m} new tokens of rollout 0 over {ctx0} tokens "
                                         f"of context, fp64 single-threaded, {dt:.1f} s"}
    else:
        rec["cpu_baseline"] = None
    print(json.dumps(rec), flush=True)


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only: the decode-attention "
                                   "path has no multi-GPU mode (run with --gpus 1)"}))
        sys.exit(2)

    import numpy as np
    import torch
    import workloads as W
    import paper_2609_12471_amd as kva

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(1)
    if args.prefill:
        return run_prefill(args)
    kva.lib()                                   # fail loudly if the library is missing

    t_gen = time.perf_counter()
    w = W.make_config(args.config)
    fp8 = args.kv == "fp8"
    if fp8:
        w = W.quantize_fp8(w)
    gen_s = time.perf_counter() - t_gen
    print(f"[bench] generated {w.name} in {gen_s:.1f}s", file=sys.stderr, flush=True)

    dev = torch.device("cuda:0")

    def d(a):
        return torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a).to(dev)


    q, k, v, lens = d(w.q), d(w.k), d(w.v), d(w.seq_lens)
    bt = d(w.block_table) if w.layout == "paged" else None
    out = torch.empty((w.B, w.Hq, w.D), dtype=torch.float32, device=dev)
    lse = torch.empty((w.B, w.Hq), dtype=torch.float32, device=dev)
    grouped = args.group > 1
    if grouped and w.layout != "paged":
        print(json.dumps({"error": "--group needs a paged config"}))
        sys.exit(2)
    if fp8 and (grouped or args.append):
        print(json.dumps({"error": "--kv fp8 runs the plain decode call only"}))
        sys.exit(2)
    ws_bytes = (kva.kva_workspace_bytes_grouped(w.B, w.Hq, w.Hkv, w.D, args.group) if grouped
                else kva.kva_workspace_bytes(w.B, w.Hq, w.Hkv, w.D))
    ws = torch.zeros(ws_bytes, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()

    app = None
    if args.append:
        if w.layout != "paged":
            print(json.dumps({"error": "--append needs a paged config"}))
            sys.exit(2)
        gen = np.random.default_rng(17)
        q_new = d(W.normal_bf16(np.random.SeedSequence([17, 1]), w.B, w.Hq, w.D))
        k_new = d(W.normal_bf16(np.random.SeedSequence([17, 2]), w.B, w.Hkv, w.D))
        v_new = d(W.normal_bf16(np.random.SeedSequence([17, 3]), w.B, w.Hkv, w.D))
        gains = torch.from_numpy((1.0 + 0.1 * gen.standard_normal((2, w.D))).astype(np.float32))
        gains = gains.to(dev)
        # the new token goes to position L_b of the existing caches (the step is
        # repeated at the same position: lengths are written to a separate array)
        app = dict(q_new=q_new, k_new=k_new, v_new=v_new, q_out=torch.empty_like(q_new),
                   new_lens=torch.empty_like(lens), qw=gains[0], kw=gains[1])

    def append_step():
        kva.kva_append_paged(app["q_new"], app["k_new"], app["v_new"], app["q_out"], k, v, bt,
                             lens, app["new_lens"], q_norm_w=app["qw"], k_norm_w=app["kw"],
                             eps=1e-6, rope_theta=1e6, stream=stream)

    def step():
        if app is not None:
            append_step()
        if fp8:
            ks, vs = w.meta["k_scale"], w.meta["v_scale"]
            if w.layout == "paged":
                kva.kva_decode_attn_paged_fp8(q, k, v, bt, lens, out, lse, scale=w.scale,
                                              k_scale=ks, v_scale=vs, workspace=ws, stream=stream)
            else:
                kva.kva_decode_attn_fp8(q, k, v, lens, out, lse, scale=w.scale, k_scale=ks,
                                        v_scale=vs, workspace=ws, stream=stream)
        elif grouped:
            kva.kva_decode_attn_paged_grouped(q, k, v, bt, lens, out, lse, group=args.group,
                                              scale=w.scale, workspace=ws, stream=stream)
        elif w.layout == "paged":
            kva.kva_decode_attn_paged(q, k, v, bt, lens, out, lse, scale=w.scale, workspace=ws,
                                      stream=stream)
        else:
            kva.kva_decode_attn(q, k, v, lens, out, lse, scale=w.scale, workspace=ws, stream=stream)

    kv_logical = w.kv_bytes_logical()
    kv_unique = w.kv_bytes_unique()
    kv_bytes = kv_unique          # the metric's bytes: each physical page once

    # clocks and power state need ~0.1 s of sustained load to settle: run untimed
    # steps for a fixed time first, then the W warm-up steps
    t_pre = time.perf_counter()
    while time.perf_counter() - t_pre < args.prewarm_s:
        for _ in range(10):
            step()
        torch.cuda.synchronize()
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # timed region: exactly K steps back to back, bracketed by synchronisation;
    # one pair of HIP events on the stream the kernels run on brackets the same
    # K steps (GPU time of the region, without per-step marker overhead)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ev_avg_s = ev0.elapsed_time(ev1) / 1e3 / args.steps

    # the paper's timing protocol (median GPU-event time, cache flushed before
    # each measured call), outside the timed region above
    cold = []
    if args.cold_calls > 0:
        # reading 1 GiB replaces the L2 and memory-side cache contents with clean lines
        flush = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        for _ in range(args.cold_calls):
            sink = flush.sum()
            s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            s.record(stream)
            step()
            e.record(stream)
            torch.cuda.synchronize()
            cold.append(s.elapsed_time(e))
        del flush, sink

    # achievable read bandwidth, for context: a plain streaming read of 4 GiB
    # with the decode kernels' 16-byte non-temporal loads, median of 20 calls
    achievable = None
    if args.stream_read_gib > 0:
        nbytes = args.stream_read_gib << 30
        buf = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        sink_t = torch.zeros(512, dtype=torch.int32, device=dev)
        for _ in range(3):
            kva.kva_debug_stream_read(buf, sink_t, stream=stream)
        times = []
        for _ in range(20):
            s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            s.record(stream)
            kva.kva_debug_stream_read(buf, sink_t, stream=stream)
            e.record(stream)
            torch.cuda.synchronize()
            times.append(s.elapsed_time(e) / 1e3)
        t_med = statistics.median(times)
        achievable = {"kernel": "stream_read_kernel (kva_debug_stream_read)", "bytes": nbytes,
                      "calls": len(times), "us_median": round(t_med * 1e6, 2),
                      "gbps_median": round(nbytes / t_med / 1e9, 1),
                      "pct_of_hbm_peak": round(100.0 * nbytes / t_med / 1e9 / HBM_PEAK_GBS, 2)}
        del buf, sink_t

    if args.copy_calibration:
        src = torch.ones(1 << 28, dtype=torch.float32, device=dev)     # 1 GiB
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    append_rec = None
    if app is not None:
        # GPU time of the append kernel alone: queue a batch of calls behind a
        # long attention call, so the host has enqueued all of them before the
        # GPU reaches the first event (one call costs more host time than GPU time)
        batch, reps = 8, 10
        times = []
        for _ in range(reps):
            a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            app_on = app
            app = None
            step()                                   # attention only: keeps the GPU busy
            app = app_on
            a0.record(stream)
            for _ in range(batch):
                append_step()
            a1.record(stream)
            torch.cuda.synchronize()
            times.append(a0.elapsed_time(a1) * 1e3 / batch)
        a_us = statistics.median(times)
        a_bytes = 2 * w.B * (w.Hq + 2 * w.Hkv) * w.D * 2     # read + write, bf16
        append_rec = {"kernel": "append_kernel", "us_per_call": round(a_us, 2),
                      "bytes_per_call": a_bytes, "gbps": round(a_bytes / (a_us * 1e-6) / 1e9, 1),
                      "timing": f"GPU events over {batch} queued calls, median of {reps}"}

    value = kv_bytes * args.steps / elapsed / 1e9
    logical_gbs = kv_logical * args.steps / elapsed / 1e9
    achieved = kv_bytes / ev_avg_s / 1e9
    src_hash = kernel_source_hash()
    # the committed counter profile covers the default workload's plain call only
    traffic = load_traffic(src_hash) if (args.config == 3 and not grouped and not fp8) else None
    rec = {
        "metric": "decode-attn effective KV HBM GB/s (% of MI355X peak); us per layer-step",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 5),
        "us_per_step": round(elapsed / args.steps * 1e6, 2),
        "pct_of_hbm_peak": round(100.0 * value / HBM_PEAK_GBS, 2),
        "logical_gbs": round(logical_gbs, 2),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp8_e4m3fn" if fp8 else "bf16",
        "data": "synthetic",
        "config": {
            "workload": w.name,
            "batch": w.B,
            "layout": w.layout,
            "page_size": w.page_size or None,
            "heads_q": w.Hq, "heads_kv": w.Hkv, "head_dim": w.D,
            "tokens": int(w.seq_lens.sum()),
            "kv_bytes": kv_bytes,
            "kv_bytes_logical": kv_logical,
            "call": (("kva_decode_attn_paged_fp8" if w.layout == "paged" else "kva_decode_attn_fp8")
                     if fp8 else
                     f"kva_decode_attn_paged_grouped (group {args.group})" if grouped
                     else "kva_decode_attn_paged" if w.layout == "paged" else "kva_decode_attn"),
            "compute": ("fp8 e4m3fn K/V codes (per-tensor scales), bf16 q, fp32 softmax and "
                        "accumulation, fp32 output" if fp8 else
                        "bf16 K/V/q, fp32 softmax and accumulation, fp32 output"),
        },
        "roofline": {
            "bound": "hbm",
            "achieved": round(achieved, 2),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": traffic,
            "kernel": ("prefix_attn_kernel + decode_attn_kernel<4, paged> + merge_grouped_kernel"
                       if grouped else
                       f"decode_attn_kernel<4, {w.layout}, {args.kv}> + merge_split_kernel")
                      + " (one step)",
            "event_us_avg": round(ev_avg_s * 1e6, 2),
            "event_span": ("shared-run, attention and merge launches per step" if grouped else
                           "one attention launch + one merge launch per step"),
            "profile": ("profiles/decode_attn_fp8_c3_kernel_trace.md" if fp8 and args.config == 3
                        else "profiles/decode_attn_c3_kernel_trace.md"
                        if args.config == 3 and not grouped
                        else "profiles/grouped_decode_c5_kernel_trace.md" if grouped else None),
            "traffic_profile": ("profiles/decode_attn_paged_c3_traffic.json"
                                if args.config == 3 and not grouped and not fp8 else None),
        },
        "cold_cache": ({"calls": len(cold), "us_median": round(statistics.median(cold) * 1e3, 2),
                        "gbps_median": round(kv_bytes / (statistics.median(cold) / 1e3) / 1e9, 2)}
                       if cold else None),
        "achievable_read": achievable,
        "kernel_source_hash": src_hash,
    }
    if achievable is not None:
        achievable["decode_over_achievable"] = round(rec["value"] / achievable["gbps_median"], 4)
    if append_rec is not None:
        rec["append"] = append_rec
        rec["config"]["call"] = "kva_append_paged + " + rec["config"]["call"]
    if not args.no_cpu_baseline:
        print("[bench] cpu baseline (oracle) ...", file=sys.stderr, flush=True)
        rec["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
    else:
        rec["cpu_baseline"] = None
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
