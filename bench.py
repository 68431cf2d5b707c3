#!/usr/bin/env python3
"""Benchmark: batched grouped-query decode attention on one MI355X.

One step = one decode-attention call for the whole batch (one layer, one
decode step): the attention kernel and the merge of split partials, through
the C ABI.  Headline workload: 64 rollouts (8 prompts x 8 samples), paged K/V
with 16-token pages in a shuffled pool, lengths uniform in [512, 8192], Qwen3-8B
attention shape (32 query heads, 8 KV heads, head_dim 128), bf16 cache, fp32
softmax/accumulation and output.  Inputs are seeded synthetic data resident in
HBM before timing starts.

Metric: effective KV HBM bandwidth = algorithmic K+V bytes of the step (4096 B
per cached token; a page shared by several sequences counts once) / step time,
next to MI355X's 8 TB/s; plus us per step.

The default run also times every other workload and call of the library in
the same process (the `configs` list of the JSON line: configs 1, 2, 4, 5, the
shared-prefix call, fp8 caches, append + attention, chunked prefill), each with
its roofline fraction, its seeds and length statistics, and, from the oracle
leg, the parity of its last step's outputs on a bounded sample.

    python bench.py [--steps K] [--warmup W] [--config 3] [--no-cpu-baseline]
    python bench.py --config 5 --group 8     # shared-prefix (group) decode call alone
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
MFMA_BF16_PEAK_TFLOPS = 2500.0     # MI355X dense bf16 matrix-core peak
PROFILE_TRAFFIC = os.path.join(ROOT, "profiles", "decode_attn_paged_c3_traffic.json")
# sources of the decode attention kernel: a counter profile is used only while
# these are unchanged
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2609_12471_amd", "csrc", f)
                  for f in ("kva_kernels.hip", "kva_device.h", "kva_internal.h")]
# sources of the prefill kernel (same rule for its counter profile)
PREFILL_SOURCES = [os.path.join(ROOT, "paper_2609_12471_amd", "csrc", f)
                   for f in ("kva_prefill.hip", "kva_device.h", "kva_internal.h")]
PREFILL_TRAFFIC = os.path.join(ROOT, "profiles", "prefill_traffic.json")
# sources of the shared-run pass and merge of grouped calls, and of the append kernel
PREFIX_SOURCES = [os.path.join(ROOT, "paper_2609_12471_amd", "csrc", f)
                  for f in ("kva_prefix.hip", "kva_device.h", "kva_internal.h")]
APPEND_SOURCES = [os.path.join(ROOT, "paper_2609_12471_amd", "csrc", f)
                  for f in ("kva_append.hip", "kva_device.h", "kva_internal.h")]
# parity gate of the fp32 outputs against the fp64 oracle
GATE_MAX_ABS, GATE_MEAN_ABS = 2e-3, 2e-4


def kernel_source_hash(files=None) -> str:
    """Hash of the kernel sources' code (the decode sources unless `files`
    names others): comments and whitespace are dropped, so a comment edit does
    not retire the counter profiles."""
    import re
    h = hashlib.sha256()
    for f in (KERNEL_SOURCES if files is None else files):
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
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip the oracle leg (CPU baseline and parity samples)")
    ap.add_argument("--no-extras", action="store_true",
                    help="time the selected workload only (no `configs` list)")
    ap.add_argument("--extra-steps", type=int, default=100,
                    help="timed steps of each extra workload (at least --steps)")
    ap.add_argument("--stream-read-gib", type=int, default=4,
                    help="decode runs: also time a plain streaming read of this many GiB "
                         "(kva_debug_stream_read) as the achievable bandwidth; 0 = skip")
    ap.add_argument("--cold-calls", type=int, default=30,
                    help="extra calls timed one by one with a 1 GiB cache flush before each")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target CPU time of the oracle baseline sample of the headline")
    ap.add_argument("--extra-cpu-seconds", type=float, default=1.5,
                    help="target CPU time of each extra workload's oracle sample")
    ap.add_argument("--prewarm-s", type=float, default=0.3,
                    help="seconds of untimed steps before the warm-up steps")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after timing, run one 1 GiB device-to-device copy (a kernel of known "
                         "traffic, used to scale hardware byte counters)")
    return ap.parse_args()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


# ----------------------------------------------------------------------------- timing

def time_steps(step, stream, steps, warmup, prewarm_s):
    """Untimed steps for prewarm_s seconds and `warmup` more, then exactly
    `steps` steps back to back bracketed by synchronisation (wall clock) and by
    one pair of HIP events on the stream the kernels run on (GPU time)."""
    import torch
    t_pre = time.perf_counter()
    while time.perf_counter() - t_pre < prewarm_s:
        for _ in range(10):
            step()
        torch.cuda.synchronize()
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    return elapsed / steps, ev0.elapsed_time(ev1) / 1e3 / steps


def lengths_record(w, key, sigma=None):
    import numpy as np
    lens = np.ascontiguousarray(w.seq_lens, np.int32)
    rec = {"seed": {"entropy": [2609, 12471, *key], "generator": "numpy SeedSequence"},
           "n": int(lens.size), "min": int(lens.min()), "max": int(lens.max()),
           "mean": round(float(lens.mean()), 1), "tokens": int(lens.astype(np.int64).sum()),
           "sha16": hashlib.sha256(lens.tobytes()).hexdigest()[:16]}
    if sigma is not None:
        rec["lognormal_sigma"] = sigma
    return rec


# ----------------------------------------------------------------------------- oracle leg

def _pin_one_core():
    try:
        allowed = os.sched_getaffinity(0)
        core = min(allowed)
        os.sched_setaffinity(0, {core})
        return allowed, core
    except (AttributeError, OSError):
        return None, None


def _unpin(allowed):
    if allowed is not None:
        os.sched_setaffinity(0, allowed)


def _oracle_decode(w, idx):
    """The oracle on sequences `idx` of w (any subset; paged pools are shared)."""
    import numpy as np
    import oracle
    idx = np.asarray(idx)
    q = np.ascontiguousarray(w.q[idx])
    lens = np.ascontiguousarray(w.seq_lens[idx])
    fp8 = w.meta.get("kv_dtype") == "fp8_e4m3fn"
    if w.layout == "paged":
        bt = np.ascontiguousarray(w.block_table[idx])
        if fp8:
            return oracle.decode_attn_fp8(q, w.k, w.v, lens, w.scale, w.meta["k_scale"],
                                          w.meta["v_scale"], block_table=bt)
        return oracle.decode_attn_paged(q, w.k, w.v, bt, lens, w.scale)
    k, v = np.ascontiguousarray(w.k[idx]), np.ascontiguousarray(w.v[idx])
    if fp8:
        return oracle.decode_attn_fp8(q, k, v, lens, w.scale, w.meta["k_scale"], w.meta["v_scale"])
    return oracle.decode_attn(q, k, v, lens, w.scale)


def parity_of(out, ref, lse=None, rlse=None):
    """max-abs / mean-abs error of fp32 GPU outputs against the fp64 oracle."""
    import numpy as np
    o = np.asarray(out, np.float64)
    err = np.abs(o - ref)
    rec = {"max_abs": float(err.max()), "mean_abs": float(err.mean()),
           "finite": bool(np.isfinite(o).all())}
    if lse is not None:
        fin = np.isfinite(rlse)
        l = np.asarray(lse, np.float64)
        rec["lse_max_abs"] = float(np.abs(l[fin] - rlse[fin]).max()) if fin.any() else 0.0
        rec["lse_inf_match"] = bool(np.array_equal(np.isneginf(l), np.isneginf(rlse)))
    rec["gate"] = bool(rec["finite"] and rec["max_abs"] <= GATE_MAX_ABS
                       and rec["mean_abs"] <= GATE_MEAN_ABS
                       and rec.get("lse_max_abs", 0.0) <= GATE_MAX_ABS
                       and rec.get("lse_inf_match", True))
    return rec


def cpu_baseline(w, target_s: float, out=None, lse=None):
    """The fp64 oracle, single-threaded and pinned to one core, on the first
    sequences of the same workload (a bounded sample), scaled to GB/s of K+V
    bytes.  With the GPU's outputs of the same batch given, the oracle's results
    on that sample also give the parity of the GPU step."""
    import numpy as np
    allowed, pinned = _pin_one_core()
    t0 = time.perf_counter()
    _oracle_decode(w, [0])
    per_tok = (time.perf_counter() - t0) / max(1, int(w.seq_lens[0]))
    budget_tok = target_s / max(per_tok, 1e-9)
    csum = np.cumsum(w.seq_lens.astype(np.int64))
    n = int(max(1, min(w.B, np.searchsorted(csum, budget_tok) + 1)))
    # a batch that takes less than the budget is run whole, repeatedly
    reps = 1 if n < w.B else max(1, int(round(budget_tok / max(1, int(csum[-1])))))
    t0 = time.perf_counter()
    for _ in range(reps):
        ref, rlse = _oracle_decode(w, np.arange(n))
    dt = time.perf_counter() - t0
    _unpin(allowed)
    toks = int(csum[n - 1])
    kv_bytes = toks * w.Hkv * w.D * w.kv_elem_bytes * 2 * reps
    rec = {
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
    if out is not None:
        rec["parity"] = dict(parity_of(out[:n], ref, None if lse is None else lse[:n], rlse),
                             sample=f"sequences 0..{n - 1} of the last timed step")
    return rec


def oracle_sample(w, target_s, out, lse, rng_key):
    """Parity of the GPU's last step on a bounded, seeded sample of sequences
    (always including the longest, which is split over the most waves), with
    the oracle's single-core rate on that sample."""
    import numpy as np
    lens = w.seq_lens.astype(np.int64)
    allowed, _ = _pin_one_core()
    t0 = time.perf_counter()
    _oracle_decode(w, [int(np.argmin(lens))])
    per_tok = (time.perf_counter() - t0) / max(1, int(lens.min()))
    budget = target_s / max(per_tok, 1e-9)
    order = np.random.default_rng(rng_key).permutation(w.B)
    first = int(np.argmax(lens))
    order = np.concatenate([[first], order[order != first]])
    take, tot = [], 0
    for b in order:
        if take and tot + lens[b] > budget:
            continue
        take.append(int(b))
        tot += int(lens[b])
    idx = np.sort(np.array(take))
    t0 = time.perf_counter()
    ref, rlse = _oracle_decode(w, idx)
    dt = time.perf_counter() - t0
    _unpin(allowed)
    kvb = tot * w.Hkv * w.D * w.kv_elem_bytes * 2
    return dict(parity_of(out[idx], ref, lse[idx], rlse),
                sample=f"{len(idx)} of {w.B} sequences incl. the longest, {tot} tokens",
                cpu_oracle={"value": round(kvb / dt / 1e9, 5), "unit": "GB/s", "cores": 1,
                            "seconds": round(dt, 2)})


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def load_traffic(src_hash: str, path: str = PROFILE_TRAFFIC):
    try:
        rec = json.load(open(path))
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_hash") != src_hash:
        return None
    return rec.get("hbm_bytes_per_launch")


# ----------------------------------------------------------------------------- decode steps

class DecodeCase:
    """A workload resident on the device and the step of one library call over it."""

    def __init__(self, w, *, group=1, fp8=False, append=False, stream=None):
        import numpy as np
        import torch
        import workloads as W
        import paper_2609_12471_amd as kva
        self.w, self.group, self.fp8 = w, group, fp8
        dev = torch.device("cuda:0")

        def d(a):
            return torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a).to(dev)

        self.q, self.k, self.v, self.lens = d(w.q), d(w.k), d(w.v), d(w.seq_lens)
        self.bt = d(w.block_table) if w.layout == "paged" else None
        self.out = torch.empty((w.B, w.Hq, w.D), dtype=torch.float32, device=dev)
        self.lse = torch.empty((w.B, w.Hq), dtype=torch.float32, device=dev)
        grouped = group > 1
        ws_bytes = (kva.kva_workspace_bytes_grouped(w.B, w.Hq, w.Hkv, w.D, group) if grouped
                    else kva.kva_workspace_bytes(w.B, w.Hq, w.Hkv, w.D))
        self.ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
        self.stream = stream if stream is not None else torch.cuda.current_stream()
        self.app = None
        if append:
            gen = np.random.default_rng(17)
            q_new = d(W.normal_bf16(np.random.SeedSequence([17, 1]), w.B, w.Hq, w.D))
            k_new = d(W.normal_bf16(np.random.SeedSequence([17, 2]), w.B, w.Hkv, w.D))
            v_new = d(W.normal_bf16(np.random.SeedSequence([17, 3]), w.B, w.Hkv, w.D))
            gains = torch.from_numpy((1.0 + 0.1 * gen.standard_normal((2, w.D))).astype(np.float32))
            gains = gains.to(dev)
            # the new token goes to position L_b of the existing caches (the step is
            # repeated at the same position: lengths are written to a separate array)
            self.app = dict(q_new=q_new, k_new=k_new, v_new=v_new, q_out=torch.empty_like(q_new),
                            new_lens=torch.empty_like(self.lens), qw=gains[0], kw=gains[1])
        if fp8:
            self.call = "kva_decode_attn_paged_fp8" if w.layout == "paged" else "kva_decode_attn_fp8"
        elif grouped:
            self.call = f"kva_decode_attn_paged_grouped (group {group})"
        else:
            self.call = "kva_decode_attn_paged" if w.layout == "paged" else "kva_decode_attn"
        if append:
            self.call = "kva_append_paged + " + self.call

    def append_step(self):
        import paper_2609_12471_amd as kva
        a = self.app
        kva.kva_append_paged(a["q_new"], a["k_new"], a["v_new"], a["q_out"], self.k, self.v,
                             self.bt, self.lens, a["new_lens"], q_norm_w=a["qw"],
                             k_norm_w=a["kw"], eps=1e-6, rope_theta=1e6, stream=self.stream)

    def attention_step(self):
        import paper_2609_12471_amd as kva
        w, s = self.w, self.stream
        if self.fp8:
            ks, vs = w.meta["k_scale"], w.meta["v_scale"]
            if w.layout == "paged":
                kva.kva_decode_attn_paged_fp8(self.q, self.k, self.v, self.bt, self.lens, self.out,
                                              self.lse, scale=w.scale, k_scale=ks, v_scale=vs,
                                              workspace=self.ws, stream=s)
            else:
                kva.kva_decode_attn_fp8(self.q, self.k, self.v, self.lens, self.out, self.lse,
                                        scale=w.scale, k_scale=ks, v_scale=vs, workspace=self.ws,
                                        stream=s)
        elif self.group > 1:
            kva.kva_decode_attn_paged_grouped(self.q, self.k, self.v, self.bt, self.lens, self.out,
                                              self.lse, group=self.group, scale=w.scale,
                                              workspace=self.ws, stream=s)
        elif w.layout == "paged":
            kva.kva_decode_attn_paged(self.q, self.k, self.v, self.bt, self.lens, self.out,
                                      self.lse, scale=w.scale, workspace=self.ws, stream=s)
        else:
            kva.kva_decode_attn(self.q, self.k, self.v, self.lens, self.out, self.lse,
                                scale=w.scale, workspace=self.ws, stream=s)

    def step(self):
        if self.app is not None:
            self.append_step()
        self.attention_step()

    def append_kernel_time(self):
        """GPU time of the append kernel alone: a batch of calls queued behind a
        long attention call, so the host has enqueued all of them before the
        GPU reaches the first event (one call costs more host time than GPU
        time)."""
        import torch
        w = self.w
        batch, reps = 8, 10
        times = []
        for _ in range(reps):
            a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            self.attention_step()                 # keeps the GPU busy
            a0.record(self.stream)
            for _ in range(batch):
                self.append_step()
            a1.record(self.stream)
            torch.cuda.synchronize()
            times.append(a0.elapsed_time(a1) * 1e3 / batch)
        a_us = statistics.median(times)
        a_bytes = 2 * w.B * (w.Hq + 2 * w.Hkv) * w.D * 2     # read + write, bf16
        return {"kernel": "append_kernel", "us_per_call": round(a_us, 2),
                "bytes_per_call": a_bytes, "gbps": round(a_bytes / (a_us * 1e-6) / 1e9, 1),
                "timing": f"GPU events over {batch} queued calls, median of {reps}"}

    def results(self):
        return self.out.cpu().numpy(), self.lse.cpu().numpy()


def kernel_name(case):
    w = case.w
    if case.group > 1:
        return "prefix_attn_kernel + decode_attn_kernel<4, paged> + merge_grouped_kernel"
    kv = "fp8" if case.fp8 else "bf16"
    name = f"decode_attn_kernel<4, {w.layout}, {kv}> + merge_split_kernel"
    return ("append_kernel + " + name) if case.app is not None else name


# ----------------------------------------------------------------------------- extra workloads

def extra_decode(args, w, key, *, group=1, fp8=False, append=False, sigma=None, profile=None,
                 traffic_profile=None):
    import torch
    steps = max(args.steps, args.extra_steps)
    case = DecodeCase(w, group=group, fp8=fp8, append=append)
    wall_s, ev_s = time_steps(case.step, case.stream, steps, max(args.warmup, 5), args.prewarm_s)
    kvb = w.kv_bytes_unique()
    rec = {"workload": w.name, "call": case.call, "dtype": "fp8_e4m3fn" if fp8 else "bf16",
           "steps": steps, "us_per_step": round(wall_s * 1e6, 2),
           "event_us_avg": round(ev_s * 1e6, 2), "kv_bytes": kvb,
           "kv_bytes_logical": w.kv_bytes_logical(),
           "gbps": round(kvb / wall_s / 1e9, 2),
           "roofline": {"bound": "hbm", "achieved": round(kvb / ev_s / 1e9, 2),
                        "peak": HBM_PEAK_GBS, "unit": "GB/s",
                        "frac": round(kvb / ev_s / 1e9 / HBM_PEAK_GBS, 4),
                        "kernel": kernel_name(case), "profile": profile},
           "lengths": lengths_record(w, key, sigma)}
    if traffic_profile is not None:
        # HBM bytes of the step's attention kernel from the counter profile, while
        # the decode sources are those it was taken on
        t = load_traffic(kernel_source_hash(), os.path.join(ROOT, traffic_profile))
        rec["roofline"]["traffic"] = t
        rec["roofline"]["traffic_profile"] = traffic_profile if t is not None else None
    if append:
        rec["append"] = case.append_kernel_time()
    if not args.no_cpu_baseline:
        out, lse = case.results()
        rec["parity"] = oracle_sample(w, args.extra_cpu_seconds, out, lse, key)
    del case
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return rec


def prefill_case(args, steps, with_baseline, target_s, parity_rows=0):
    """Chunked prefill: TFLOP/s of kva_prefill_paged on the feedback-ingestion
    workload, optionally with the oracle's rate and the parity of sampled rows."""
    import numpy as np
    import torch
    import workloads as W
    import paper_2609_12471_amd as kva

    t_gen = time.perf_counter()
    p = W.make_prefill_config()
    log(f"generated {W.PREFILL_NAME} in {time.perf_counter() - t_gen:.1f}s")
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

    wall_s, ev_s = time_steps(step, stream, steps, max(args.warmup, 3), args.prewarm_s)
    flops = p.flops()
    rec = {"workload": W.PREFILL_NAME, "call": "kva_prefill_paged", "dtype": "bf16",
           "steps": steps, "us_per_step": round(wall_s * 1e6, 2),
           "event_us_avg": round(ev_s * 1e6, 2), "flops": flops,
           "tflops": round(flops / wall_s / 1e12, 2),
           "roofline": {"bound": "mfma", "achieved": round(flops / ev_s / 1e12, 2),
                        "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                        "frac": round(flops / ev_s / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
                        "traffic": load_traffic(kernel_source_hash(PREFILL_SOURCES), PREFILL_TRAFFIC),
                        "kernel": "prefill_kernel (one launch per step)",
                        "flops_note": "QK and PV multiply-adds of the causal prefixes, 2 flops "
                                      "each; the second bf16 part of P is not counted",
                        # the matrix-core work issued: P enters the PV products as
                        # two bf16 parts, so PV runs twice (QK and PV have equal
                        # flop counts): 1.5x the algorithmic flops, a lower bound
                        # (the masked positions of diagonal blocks are not counted)
                        "issued_mfma_tflops": round(1.5 * flops / ev_s / 1e12, 2),
                        "issued_frac": round(1.5 * flops / ev_s / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
                        "profile": "profiles/prefill_kernel_trace.md"},
           "batch": c.B, "new_tokens": p.T, "context_tokens": int(c.seq_lens.sum()) - p.T,
           "lengths": lengths_record(c, (6,))}
    if with_baseline:
        import oracle
        o_gpu = out.cpu().numpy()
        l_gpu = lse.cpu().numpy()
        allowed, _ = _pin_one_core()
        # the oracle on the first new tokens of rollout 0, scaled to TFLOP/s
        n0 = int(p.q_start[1])
        m = 8
        while True:
            sub_q = np.ascontiguousarray(p.q[:m])
            qs1 = np.array([0, m], np.int32)
            lens1 = np.array([int(c.seq_lens[0]) - n0 + m], np.int32)
            t1 = time.perf_counter()
            ref, rlse = oracle.prefill_paged(sub_q, c.k, c.v,
                                             np.ascontiguousarray(c.block_table[:1]), qs1, lens1,
                                             c.scale)
            dt = time.perf_counter() - t1
            if dt > target_s / 4 or m >= n0:
                break
            m = min(n0, m * 4)
        ctx0 = int(lens1[0]) - m
        fl = (m * ctx0 + m * (m + 1) // 2) * c.Hq * c.D * 4
        rec["cpu_baseline"] = {"value": round(fl / dt / 1e12, 6), "unit": "TFLOP/s", "cores": 1,
                               "kind": "oracle",
                               "sample": f"first {m} new tokens of rollout 0 over {ctx0} tokens "
                                         f"of context, fp64 single-threaded, {dt:.1f} s"}
        par = parity_of(o_gpu[:m], ref, l_gpu[:m], rlse)
        par["sample"] = f"new tokens 0..{m - 1} of rollout 0"
        if parity_rows > 0:
            # one row at a seeded offset in each of `parity_rows` evenly spaced
            # 32-token tiles: decode attention over its causal prefix
            rng = np.random.default_rng(6061)
            tiles = np.linspace(0, p.T // 32 - 1, parity_rows).astype(np.int64)
            rows = tiles * 32 + rng.integers(0, 32, size=tiles.size)
            b_of = np.searchsorted(p.q_start, rows, side="right") - 1
            n = np.diff(p.q_start)[b_of]
            pos = c.seq_lens[b_of] - n + (rows - p.q_start[b_of])
            r1, rl1 = oracle.decode_attn_paged(np.ascontiguousarray(p.q[rows]), c.k, c.v,
                                               np.ascontiguousarray(c.block_table[b_of]),
                                               (pos + 1).astype(np.int32), c.scale)
            par2 = parity_of(o_gpu[rows], r1, l_gpu[rows], rl1)
            par["rows"] = dict(par2, sample=f"{rows.size} rows, one per sampled 32-token tile")
            par["gate"] = bool(par["gate"] and par2["gate"])
        rec["parity"] = par
        _unpin(allowed)
    del q, k, v, bt, qs, lens, out, lse
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return rec


def run_extras(args, w3):
    """Every other workload and call, timed in this process (configs 1, 2, 4,
    5, the shared-prefix call, fp8 caches, append + attention, prefill)."""
    import workloads as W
    recs = []

    def guarded(tag, fn):
        log(f"extra: {tag}")
        try:
            recs.append(fn())
        except Exception as e:                    # keep the headline line whatever happens here
            recs.append({"workload": tag, "error": f"{type(e).__name__}: {e}"})

    guarded("c1", lambda: extra_decode(args, W.make_config(1), (1,)))
    guarded("c2", lambda: extra_decode(args, W.make_config(2), (2,),
                                       profile="profiles/decode_attn_c2_kernel_trace.md"))
    w4 = W.make_config(4)
    guarded("c4", lambda: extra_decode(args, w4, (4,), sigma=W.LOGNORMAL_SIGMA,
                                       profile="profiles/decode_attn_c4_kernel_trace.md",
                                       traffic_profile="profiles/decode_attn_paged_c4_traffic.json"))
    guarded("c4 fp8", lambda: extra_decode(args, W.quantize_fp8(w4), (4,), fp8=True,
                                           sigma=W.LOGNORMAL_SIGMA,
                                           profile="profiles/decode_attn_fp8_c4_kernel_trace.md"))
    del w4
    w5 = W.make_config(5)
    guarded("c5", lambda: extra_decode(args, w5, (5,),
                                       profile="profiles/decode_attn_c5_kernel_trace.md"))
    guarded("c5 grouped", lambda: extra_decode(args, w5, (5,), group=8,
                                               profile="profiles/grouped_decode_c5_kernel_trace.md",
                                               traffic_profile="profiles/grouped_decode_c5_traffic.json"))
    del w5
    guarded("c3 fp8", lambda: extra_decode(args, W.quantize_fp8(w3), (3,), fp8=True,
                                           profile="profiles/decode_attn_fp8_c3_kernel_trace.md",
                                           traffic_profile="profiles/decode_attn_paged_fp8_c3_traffic.json"))
    guarded("c3 append", lambda: extra_decode(args, w3, (3,), append=True,
                                              profile="profiles/append_c3_kernel_trace.md"))
    guarded("prefill", lambda: prefill_case(args, max(args.steps, 20), not args.no_cpu_baseline,
                                            4.0, parity_rows=32))
    return recs


# ----------------------------------------------------------------------------- main

def copy_calibration():
    """One 1 GiB device-to-device copy: a kernel of known traffic (1 GiB read,
    1 GiB written) whose byte counters scale those of the timed kernels."""
    import torch
    src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


def run_prefill(args):
    rec = prefill_case(args, args.steps, not args.no_cpu_baseline, args.cpu_seconds)
    if args.copy_calibration:
        copy_calibration()
    value = rec["tflops"]
    line = {
        "metric": "chunked-prefill attention TFLOP/s (% of MI355X bf16 matrix-core peak)",
        "value": value, "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(rec["us_per_step"] / 1e3, 5),
        "us_per_step": rec["us_per_step"],
        "pct_of_peak": round(100.0 * value / MFMA_BF16_PEAK_TFLOPS, 2),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": rec["workload"], "batch": rec["batch"],
                   "new_tokens": rec["new_tokens"], "context_tokens": rec["context_tokens"],
                   "heads_q": 32, "heads_kv": 8, "head_dim": 128, "page_size": 16,
                   "flops": rec["flops"], "call": "kva_prefill_paged",
                   "compute": "bf16 q/K/V on the matrix cores (softmax weights as two bf16 "
                              "parts), fp32 softmax and accumulation, fp32 output"},
        "roofline": dict(rec["roofline"], event_us_avg=rec["event_us_avg"]),
        "kernel_source_hash": kernel_source_hash(),
        "cpu_baseline": rec.get("cpu_baseline"),
        "parity": rec.get("parity"),
    }
    print(json.dumps(line), flush=True)


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only: the decode-attention "
                                   "path has no multi-GPU mode (run with --gpus 1)"}))
        sys.exit(2)

    import torch
    import workloads as W
    import paper_2609_12471_amd as kva

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(1)
    kva.lib()                                   # fail loudly if the library is missing
    if args.prefill:
        return run_prefill(args)

    t_gen = time.perf_counter()
    w3 = W.make_config(args.config)
    fp8 = args.kv == "fp8"
    w = W.quantize_fp8(w3) if fp8 else w3
    log(f"generated {w.name} in {time.perf_counter() - t_gen:.1f}s")
    grouped = args.group > 1
    if grouped and w.layout != "paged":
        print(json.dumps({"error": "--group needs a paged config"}))
        sys.exit(2)
    if fp8 and (grouped or args.append):
        print(json.dumps({"error": "--kv fp8 runs the plain decode call only"}))
        sys.exit(2)
    if args.append and w.layout != "paged":
        print(json.dumps({"error": "--append needs a paged config"}))
        sys.exit(2)
    case = DecodeCase(w, group=args.group, fp8=fp8, append=args.append)
    stream = case.stream
    dev = torch.device("cuda:0")

    kv_logical = w.kv_bytes_logical()
    kv_unique = w.kv_bytes_unique()
    kv_bytes = kv_unique          # the metric's bytes: each physical page once

    # timed region: exactly K steps back to back, bracketed by synchronisation;
    # one pair of HIP events on the stream the kernels run on brackets the same
    # K steps (GPU time of the region, without per-step marker overhead)
    wall_s, ev_avg_s = time_steps(case.step, stream, args.steps, args.warmup, args.prewarm_s)
    out_last, lse_last = case.results()

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
            case.step()
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
        copy_calibration()

    append_rec = case.append_kernel_time() if case.app is not None else None
    call = case.call
    del case
    torch.cuda.synchronize()
    torch.cuda.empty_cache()

    value = kv_bytes / wall_s / 1e9
    logical_gbs = kv_logical / wall_s / 1e9
    achieved = kv_bytes / ev_avg_s / 1e9
    src_hash = kernel_source_hash()
    # the committed counter profile covers the default workload's plain call only
    traffic = (load_traffic(src_hash)
               if (args.config == 3 and not grouped and not fp8 and not args.append) else None)
    kname = (("prefix_attn_kernel + decode_attn_kernel<4, paged> + merge_grouped_kernel"
              if grouped else
              f"decode_attn_kernel<4, {w.layout}, {args.kv}> + merge_split_kernel")
             + " (one step)")
    rec = {
        "metric": "decode-attn effective KV HBM GB/s (% of MI355X peak); us per layer-step",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall_s * 1e3, 5),
        "us_per_step": round(wall_s * 1e6, 2),
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
            "call": call,
            "compute": ("fp8 e4m3fn K/V codes (per-tensor scales), bf16 q, fp32 softmax and "
                        "accumulation, fp32 output" if fp8 else
                        "bf16 K/V/q, fp32 softmax and accumulation, fp32 output"),
            "lengths": lengths_record(w, (args.config,),
                                      W.LOGNORMAL_SIGMA if args.config == 4 else None),
        },
        "roofline": {
            "bound": "hbm",
            "achieved": round(achieved, 2),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": traffic,
            "kernel": kname,
            "event_us_avg": round(ev_avg_s * 1e6, 2),
            "event_span": ("shared-run, attention and merge launches per step" if grouped else
                           "one attention launch + one merge launch per step"),
            "profile": ("profiles/decode_attn_fp8_c3_kernel_trace.md" if fp8 and args.config == 3
                        else "profiles/decode_attn_c3_kernel_trace.md"
                        if args.config == 3 and not grouped
                        else "profiles/grouped_decode_c5_kernel_trace.md" if grouped else None),
            "traffic_profile": ("profiles/decode_attn_paged_c3_traffic.json"
                                if traffic is not None else None),
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
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle) ...")
        rec["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds, out_last, lse_last)
    else:
        rec["cpu_baseline"] = None
    default_line = (args.config == 3 and not grouped and not fp8 and not args.append)
    if default_line and not args.no_extras:
        rec["configs"] = run_extras(args, w3)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
