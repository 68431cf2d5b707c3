"""Seeded synthetic inputs for batched grouped-query decode attention.

This module only draws inputs; it holds none of the attention arithmetic.  Both
the fp64 oracle (``oracle/``) and the GPU library consume exactly the bf16 bit
patterns it produces.

Input recipe (stands in for the KV caches of RL rollouts; the paper's prompts,
trained weights and caches are not available):

* shape of Qwen3-8B attention: 32 query heads, 8 KV heads, head_dim 128;
* values i.i.d. N(0, 1) in fp32, RMS-normalised per 128-vector
  (x / sqrt(mean(x^2) + 1e-6), no gain), then rounded to bf16 (nearest-even);
  this applies to q, K and V;
* softmax scale 1/sqrt(128) as an fp32 number;
* unused cache memory (rows at or past a sequence's length, page tails, spare
  pages) holds bf16 NaN (0x7FC0), so any read of it that leaks into a result
  shows up as a non-finite output.

Rollout shapes come from the paper's hyperparameter table (group size G = 8
samples per prompt for multi-turn RL, 64 prompts per batch, sequence lengths of
8K for HIP RL and 16K for Triton RL) and its description of the rollout loop
(prompt sampled, G samples decoded for up to three turns).

Seeds: config k uses ``np.random.SeedSequence([2609, 12471, k])``, spawned into
child streams in a fixed order (lengths, page permutation, q, K, V).  Large
tensors are drawn in fixed-size chunks with one child seed per chunk, so the
bits do not depend on how many threads draw them.
"""
from __future__ import annotations

import dataclasses
import math
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

HQ, HKV, HEAD_DIM = 32, 8, 128
SCALE = float(np.float32(1.0 / math.sqrt(HEAD_DIM)))
BF16_NAN = np.uint16(0x7FC0)
SEED_ROOT = (2609, 12471)
LOGNORMAL_SIGMA = 0.7          # C4 length spread (unstated)
_CHUNK_ROWS = 8192             # rows of Hkv*D values drawn per child seed


@dataclasses.dataclass
class Workload:
    name: str
    layout: str                      # "contig" or "paged"
    q: np.ndarray                    # uint16 [B, Hq, D]
    k: np.ndarray                    # contig: [B, Lmax, Hkv, D]; paged: [num_pages, P, Hkv, D]
    v: np.ndarray
    seq_lens: np.ndarray             # int32 [B]
    scale: float = SCALE
    block_table: np.ndarray | None = None   # int32 [B, max_pages], -1 = unused
    page_size: int = 0
    meta: dict = dataclasses.field(default_factory=dict)

    @property
    def B(self): return self.q.shape[0]
    @property
    def Hq(self): return self.q.shape[1]
    @property
    def D(self): return self.q.shape[2]
    @property
    def Hkv(self): return self.k.shape[2]
    @property
    def Lmax(self):
        return self.k.shape[1] if self.layout == "contig" else self.block_table.shape[1] * self.page_size
    @property
    def num_pages(self): return self.k.shape[0] if self.layout == "paged" else 0
    @property
    def max_pages(self): return self.block_table.shape[1] if self.layout == "paged" else 0

    @property
    def kv_elem_bytes(self) -> int:
        """Bytes per cached element: 2 (bf16) or 1 (fp8 codes)."""
        return self.k.dtype.itemsize

    def kv_bytes_logical(self) -> int:
        """K+V bytes one decode step reads if every sequence reads its own rows."""
        return int(self.seq_lens.astype(np.int64).sum()) * self.Hkv * self.D * self.kv_elem_bytes * 2

    def kv_bytes_unique(self) -> int:
        """K+V bytes of distinct cache rows read (shared prefix pages counted once)."""
        if self.layout == "contig":
            return self.kv_bytes_logical()
        P = self.page_size
        rows = []
        for b in range(self.B):
            t = np.arange(int(self.seq_lens[b]), dtype=np.int64)
            rows.append(self.block_table[b, t // P].astype(np.int64) * P + t % P)
        rows = np.unique(np.concatenate(rows)) if rows else np.zeros(0)
        return len(rows) * self.Hkv * self.D * self.kv_elem_bytes * 2


# ----------------------------------------------------------------------------- bits

def bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round to nearest even (inputs are finite)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + r) >> 16).astype(np.uint16)


def bits_to_f32(h: np.ndarray) -> np.ndarray:
    return (h.astype(np.uint32) << 16).view(np.float32)


def _rms_normal(rng: np.random.Generator, shape) -> np.ndarray:
    x = rng.standard_normal(shape, dtype=np.float32)
    ms = np.mean(x * x, axis=-1, keepdims=True, dtype=np.float32)
    return x * (np.float32(1.0) / np.sqrt(ms + np.float32(1e-6)))


def _parallel(fn, n, threads=None):
    threads = threads or min(8, os.cpu_count() or 1)
    if n <= 1 or threads == 1:
        for i in range(n):
            fn(i)
    else:
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(fn, range(n)))


def fill_normal_bf16(seed: np.random.SeedSequence, dst: np.ndarray, rows: np.ndarray,
                     threads: int | None = None) -> None:
    """dst[rows[i]] = RMS-normalised N(0,1) bf16 values, for dst of shape
    [N, Hkv, D].  Values are drawn in chunks of _CHUNK_ROWS consecutive entries
    of `rows`, one child seed per chunk, so the bits depend only on the seed
    and the order of `rows`."""
    n_rows = rows.shape[0]
    n_chunks = max(1, (n_rows + _CHUNK_ROWS - 1) // _CHUNK_ROWS)
    kids = seed.spawn(n_chunks)
    shape = dst.shape[1:]

    def work(i):
        lo, hi = i * _CHUNK_ROWS, min(n_rows, (i + 1) * _CHUNK_ROWS)
        if hi > lo:
            rng = np.random.Generator(np.random.PCG64(kids[i]))
            dst[rows[lo:hi]] = bf16_bits(_rms_normal(rng, (hi - lo,) + shape))

    _parallel(work, n_chunks, threads)


def normal_bf16(seed: np.random.SeedSequence, n_rows: int, Hkv: int, D: int,
                threads: int | None = None) -> np.ndarray:
    """n_rows x Hkv x D RMS-normalised N(0,1) values as bf16 bits."""
    out = np.empty((n_rows, Hkv, D), np.uint16)
    fill_normal_bf16(seed, out, np.arange(n_rows, dtype=np.int64), threads)
    return out


def _filled(shape, value, threads=None) -> np.ndarray:
    """np.full, with the first touch of large arrays spread over threads."""
    a = np.empty(shape, np.uint16)
    flat = a.reshape(-1)
    n = flat.shape[0]
    parts = max(1, min(64, n >> 22))

    def work(i):
        flat[i * n // parts:(i + 1) * n // parts] = value

    _parallel(work, parts, threads)
    return a


def _seeds(key):
    ss = np.random.SeedSequence(list(SEED_ROOT) + list(key))
    return dict(zip(("lens", "perm", "q", "k", "v"), ss.spawn(5)))


# ----------------------------------------------------------------------------- builders

def make_contig(seq_lens, Lmax: int, *, Hq=HQ, Hkv=HKV, D=HEAD_DIM, key=(1000,),
                scale=SCALE, name="contig", poison=True) -> Workload:
    """Contiguous caches [B, Lmax, Hkv, D]; rows >= L_b hold NaN (if poison)."""
    lens = np.asarray(seq_lens, dtype=np.int32)
    B = lens.shape[0]
    if np.any(lens < 0) or np.any(lens > Lmax):
        raise ValueError("lengths outside [0, Lmax]")
    sd = _seeds(key)
    q = normal_bf16(sd["q"], B, Hq, D)
    fill = BF16_NAN if poison else np.uint16(0)
    k = _filled((B, Lmax, Hkv, D), fill)
    v = _filled((B, Lmax, Hkv, D), fill)
    rows = np.concatenate([b * Lmax + np.arange(int(lens[b]), dtype=np.int64) for b in range(B)]
                          ) if B else np.zeros(0, np.int64)
    fill_normal_bf16(sd["k"], k.reshape(B * Lmax, Hkv, D), rows)
    fill_normal_bf16(sd["v"], v.reshape(B * Lmax, Hkv, D), rows)
    return Workload(name, "contig", q, k, v, lens, scale, meta={"key": list(key)})


def make_paged(seq_lens, *, page_size=16, Hq=HQ, Hkv=HKV, D=HEAD_DIM, key=(2000,),
               scale=SCALE, max_pages=None, spare_num=1, spare_den=8, shared_prefix=None,
               name="paged", poison=True) -> Workload:
    """Paged pool [num_pages, P, Hkv, D] with a shuffled block table.

    shared_prefix = (group_size, prefix_tokens): sequences b = j*group_size ..
    (j+1)*group_size-1 map their first prefix_tokens/P table entries to the
    same physical pages (prefix_tokens must be a multiple of P and <= every L_b
    of the group).
    """
    lens = np.asarray(seq_lens, dtype=np.int32)
    B = lens.shape[0]
    P = int(page_size)
    if P <= 0 or (P & (P - 1)):
        raise ValueError("page_size must be a power of two")
    npg = (lens.astype(np.int64) + P - 1) // P
    if max_pages is None:
        max_pages = int(npg.max()) if B else 0
    if np.any(npg > max_pages):
        raise ValueError("a sequence needs more than max_pages pages")
    sd = _seeds(key)
    # logical page list: (b, j) -> unique logical id, shared prefix pages deduplicated
    logical = np.full((B, max_pages), -1, np.int64)
    nxt = 0
    gsz, pref_pages = (1, 0)
    if shared_prefix is not None:
        gsz, ptok = shared_prefix
        if ptok % P:
            raise ValueError("shared prefix must be page aligned")
        pref_pages = ptok // P
    for b in range(B):
        j0 = 0
        if pref_pages and b % gsz != 0:
            lead = b - b % gsz
            logical[b, :pref_pages] = logical[lead, :pref_pages]
            j0 = pref_pages
        for j in range(j0, int(npg[b])):
            logical[b, j] = nxt
            nxt += 1
    needed = nxt
    num_pages = needed + (needed * spare_num + spare_den - 1) // spare_den
    perm = np.random.Generator(np.random.PCG64(sd["perm"])).permutation(num_pages).astype(np.int64)
    table = np.where(logical >= 0, perm[np.maximum(logical, 0)], -1).astype(np.int32)
    # rows of the pool that hold live tokens, in order of first appearance
    rows = []
    seen = np.zeros(num_pages * P, bool) if num_pages else np.zeros(0, bool)
    for b in range(B):
        L = int(lens[b])
        t = np.arange(L, dtype=np.int64)
        r = table[b, t // P].astype(np.int64) * P + t % P
        fresh = r[~seen[r]]
        seen[fresh] = True
        rows.append(fresh)
    rows = np.concatenate(rows) if rows else np.zeros(0, np.int64)
    fill = BF16_NAN if poison else np.uint16(0)
    kp = _filled((num_pages * P, Hkv, D), fill)
    vp = _filled((num_pages * P, Hkv, D), fill)
    fill_normal_bf16(sd["k"], kp, rows)
    fill_normal_bf16(sd["v"], vp, rows)
    q = normal_bf16(sd["q"], B, Hq, D)
    return Workload(name, "paged", q, kp.reshape(num_pages, P, Hkv, D),
                    vp.reshape(num_pages, P, Hkv, D), lens, scale, table, P,
                    meta={"key": list(key), "needed_pages": needed})


# ----------------------------------------------------------------------------- chunked prefill

@dataclasses.dataclass
class Prefill:
    """Chunked prefill: sequence b holds ctx_b earlier tokens and n_b new ones
    (already in its cache, so cache.seq_lens[b] = ctx_b + n_b); the new tokens'
    queries are packed over the batch, rows q_start[b] .. q_start[b+1]-1."""
    cache: Workload                 # paged cache with the chunks appended; cache.q unused
    q: np.ndarray                   # uint16 [T, Hq, D]
    q_start: np.ndarray             # int32 [B + 1]

    @property
    def T(self): return self.q.shape[0]

    def flops(self) -> int:
        """QK and PV multiply-adds (2 flops each) of every new token over its causal prefix."""
        lens = self.cache.seq_lens.astype(np.int64)
        n = np.diff(self.q_start.astype(np.int64))
        # token i of b attends L_b - n_b + i + 1 positions; sum over i
        keys = (n * (lens - n) + n * (n + 1) // 2).sum()
        return int(keys) * self.cache.Hq * self.cache.D * 2 * 2


def make_prefill(ctx_lens, chunk_lens, *, page_size=16, Hq=HQ, Hkv=HKV, key=(3000,),
                 name="prefill", poison=True) -> Prefill:
    ctx = np.asarray(ctx_lens, np.int32)
    n = np.asarray(chunk_lens, np.int32)
    cache = make_paged(ctx + n, page_size=page_size, Hq=Hq, Hkv=Hkv, key=key, name=name,
                       poison=poison)
    q_start = np.concatenate([[0], np.cumsum(n)]).astype(np.int32)
    sd = _seeds(tuple(key) + (7,))
    q = normal_bf16(sd["q"], int(q_start[-1]), Hq, HEAD_DIM)
    return Prefill(cache, q, q_start)


PREFILL_NAME = "prefill_b64_chunk512_ctx512-7680_paged16"


def make_prefill_config() -> Prefill:
    """Feedback ingestion between turns: 64 rollouts, each with 512 new tokens
    on top of a context of U{512..7680} tokens (<= 8192 in all), paged 16."""
    rng = np.random.Generator(np.random.PCG64(_seeds((6,))["lens"]))
    ctx = rng.integers(512, 7680, size=64, endpoint=True).astype(np.int32)
    return make_prefill(ctx, np.full(64, 512, np.int32), key=(6,), name=PREFILL_NAME)


# ----------------------------------------------------------------------------- fp8 caches

# One scale per tensor, chosen from the data's bound rather than measured: the
# cached rows are RMS-normalised 128-vectors, so |x| <= sqrt(128), and x / s
# stays within e4m3fn's largest finite value (448).  K and V get different
# scales so that a swap of the two is visible.
FP8_K_SCALE = float(np.sqrt(128.0) / 448.0)
FP8_V_SCALE = float(np.sqrt(128.0) / 400.0)


def to_fp8_codes(bits: np.ndarray, scale: float, chunk: int = 1 << 24) -> np.ndarray:
    """bf16 bit patterns -> fp8 e4m3fn codes of x / scale (nearest, ties to
    even, via torch's conversion); NaN stays NaN."""
    import torch
    flat = bits.reshape(-1)
    out = np.empty(flat.shape[0], np.uint8)
    inv = np.float32(1.0 / scale)
    for i in range(0, flat.shape[0], chunk):
        x = torch.from_numpy(bits_to_f32(flat[i:i + chunk]) * inv)
        out[i:i + chunk] = x.to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    return out.reshape(bits.shape)


def quantize_fp8(w: Workload) -> Workload:
    """The same cache stored as fp8 codes (keys k_scale * fp8, values
    v_scale * fp8); q, lengths and the block table are unchanged."""
    meta = dict(w.meta, kv_dtype="fp8_e4m3fn", k_scale=FP8_K_SCALE, v_scale=FP8_V_SCALE)
    return dataclasses.replace(w, name=w.name + "_fp8", k=to_fp8_codes(w.k, FP8_K_SCALE),
                               v=to_fp8_codes(w.v, FP8_V_SCALE), meta=meta)


# ----------------------------------------------------------------------------- the five configs

CONFIG_NAMES = {
    1: "c1_single_seq_contig_L256",
    2: "c2_b8_contig_L1024-4096",
    3: "c3_b64_paged16_L512-8192",
    4: "c4_b256_paged16_lognormal3000",
    5: "c5_16x8_shared_prefix2048_paged16",
}


def config_lengths(k: int) -> np.ndarray:
    """Per-sequence lengths of config k (inclusive integer bounds)."""
    rng = np.random.Generator(np.random.PCG64(_seeds((k,))["lens"]))
    if k == 1:
        return np.array([256], np.int32)
    if k == 2:
        return rng.integers(1024, 4096, size=8, endpoint=True).astype(np.int32)
    if k == 3:
        return rng.integers(512, 8192, size=64, endpoint=True).astype(np.int32)
    if k == 4:
        x = np.exp(rng.normal(math.log(3000.0), LOGNORMAL_SIGMA, size=256))
        return np.clip(np.rint(x), 256, 16384).astype(np.int32)
    if k == 5:
        return (2048 + rng.integers(256, 8192, size=128, endpoint=True)).astype(np.int32)
    raise ValueError(f"no config {k}")


def make_config(k: int) -> Workload:
    lens = config_lengths(k)
    name = CONFIG_NAMES[k]
    if k == 1:
        return make_contig(lens, 256, key=(k,), name=name)
    if k == 2:
        return make_contig(lens, 4096, key=(k,), name=name)
    if k == 3:
        return make_paged(lens, page_size=16, max_pages=512, key=(k,), name=name)
    if k == 4:
        w = make_paged(lens, page_size=16, max_pages=1024, key=(k,), name=name)
        w.meta["lognormal_sigma"] = LOGNORMAL_SIGMA
        return w
    if k == 5:
        return make_paged(lens, page_size=16, max_pages=640, key=(k,), name=name,
                          shared_prefix=(8, 2048))
    raise ValueError(f"no config {k}")
