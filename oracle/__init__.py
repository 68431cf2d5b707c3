"""fp64 CPU oracle for batched grouped-query decode attention -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The GPU library never imports, links or
calls it, and the two share no code; the only thing both sides consume is the
bf16 bits produced by the seeded input generator.

The arithmetic lives in ``kva_oracle.c`` (plain C, binary64, single-threaded,
max-subtracted multi-pass softmax as in the paper's appendix of self-correction
examples, Examples 1 and 3).  This module only marshals numpy arrays through
ctypes.  Every array argument must be C-contiguous with the dtype named below;
bf16 tensors are passed as their raw ``uint16`` bit patterns.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "kva_oracle.c")
_LIB = os.path.join(_HERE, "libkva_oracle.so")

_ERRORS = {1: "bad argument", 2: "length or page id out of range", 3: "out of memory"}


def build() -> str:
    """Compile the oracle with gcc (binary64, no contraction, no fast-math)."""
    cmd = ["gcc", "-O2", "-std=c99", "-ffp-contract=off", "-fno-fast-math", "-fPIC",
           "-shared", "-o", _LIB + ".tmp", _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i32, i64, f64 = ctypes.c_int, ctypes.c_int64, ctypes.c_double
        lib.kvo_decode_attn.argtypes = [P, P, P, P, P, P, i32, i32, i32, i32, i32, f64]
        lib.kvo_decode_attn.restype = i32
        lib.kvo_decode_attn_paged.argtypes = [P, P, P, P, P, P, P, i32, i32, i32, i32, i32,
                                              i32, i64, f64]
        lib.kvo_decode_attn_paged.restype = i32
        lib.kvo_combine.argtypes = [P, P, P, P, i32, i32, i32, i32]
        lib.kvo_combine.restype = i32
        lib.kvo_append.argtypes = [P, P, P, P, P, P, P, i32, i32, i32, i32, i32, i32, i64, i32,
                                   f64, f64, P, P, P, P, P]
        lib.kvo_append.restype = i32
        lib.kvo_round_bf16.argtypes = [P, P, i64]
        lib.kvo_round_bf16.restype = i32
        lib.kvo_prefill_paged.argtypes = [P, P, P, P, P, P, P, P, i32, i32, i32, i32, i32, i32,
                                          i32, i64, f64]
        lib.kvo_prefill_paged.restype = i32
        lib.kvo_fp8_table.argtypes = [P]
        lib.kvo_fp8_table.restype = i32
        lib.kvo_decode_attn_fp8.argtypes = [P, P, P, P, P, P, P, i32, i32, i32, i32, i32, i32,
                                            i64, i32, f64, f64, f64]
        lib.kvo_decode_attn_fp8.restype = i32
        _lib = lib
    return _lib


def _ptr(a: np.ndarray | None):
    return None if a is None else a.ctypes.data


def _req(a, dtype, name, ndim=None):
    if not isinstance(a, np.ndarray) or a.dtype != dtype or not a.flags.c_contiguous:
        raise TypeError(f"{name}: expected a C-contiguous numpy array of {np.dtype(dtype)}")
    if ndim is not None and a.ndim != ndim:
        raise ValueError(f"{name}: expected {ndim} dims, got shape {a.shape}")
    return a


def _check(rc: int):
    if rc != 0:
        raise ValueError(f"oracle: {_ERRORS.get(rc, rc)}")


def decode_attn(q, k, v, seq_lens, scale: float):
    """Contiguous caches.  q uint16 [B,Hq,D]; k, v uint16 [B,Lmax,Hkv,D];
    seq_lens int32 [B].  Returns (out f64 [B,Hq,D], lse f64 [B,Hq])."""
    _req(q, np.uint16, "q", 3); _req(k, np.uint16, "k", 4); _req(v, np.uint16, "v", 4)
    _req(seq_lens, np.int32, "seq_lens", 1)
    B, Hq, D = q.shape
    _, Lmax, Hkv, Dk = k.shape
    if k.shape != v.shape or k.shape[0] != B or Dk != D or seq_lens.shape[0] != B:
        raise ValueError("shape mismatch")
    out = np.empty((B, Hq, D), np.float64)
    lse = np.empty((B, Hq), np.float64)
    _check(_load().kvo_decode_attn(_ptr(q), _ptr(k), _ptr(v), _ptr(seq_lens), _ptr(out),
                                   _ptr(lse), B, Hq, Hkv, D, Lmax, float(scale)))
    return out, lse


def decode_attn_paged(q, k_pool, v_pool, block_table, seq_lens, scale: float):
    """Paged caches.  k_pool, v_pool uint16 [num_pages,P,Hkv,D]; block_table
    int32 [B,max_pages]; position t of sequence b is slot t % P of page
    block_table[b, t // P].  Returns (out f64 [B,Hq,D], lse f64 [B,Hq])."""
    _req(q, np.uint16, "q", 3); _req(k_pool, np.uint16, "k_pool", 4)
    _req(v_pool, np.uint16, "v_pool", 4); _req(block_table, np.int32, "block_table", 2)
    _req(seq_lens, np.int32, "seq_lens", 1)
    B, Hq, D = q.shape
    num_pages, P, Hkv, Dk = k_pool.shape
    if k_pool.shape != v_pool.shape or Dk != D or block_table.shape[0] != B \
            or seq_lens.shape[0] != B:
        raise ValueError("shape mismatch")
    out = np.empty((B, Hq, D), np.float64)
    lse = np.empty((B, Hq), np.float64)
    _check(_load().kvo_decode_attn_paged(_ptr(q), _ptr(k_pool), _ptr(v_pool), _ptr(block_table),
                                         _ptr(seq_lens), _ptr(out), _ptr(lse), B, Hq, Hkv, D, P,
                                         block_table.shape[1], num_pages, float(scale)))
    return out, lse


def combine(o_parts, lse_parts):
    """Log-sum-exp merge of partial results over disjoint key sets.
    o_parts f64 [S,B,Hq,D]; lse_parts f64 [S,B,Hq] (-inf = empty part)."""
    _req(o_parts, np.float64, "o_parts", 4); _req(lse_parts, np.float64, "lse_parts", 3)
    S, B, Hq, D = o_parts.shape
    if lse_parts.shape != (S, B, Hq):
        raise ValueError("shape mismatch")
    out = np.empty((B, Hq, D), np.float64)
    lse = np.empty((B, Hq), np.float64)
    _check(_load().kvo_combine(_ptr(o_parts), _ptr(lse_parts), _ptr(out), _ptr(lse), S, B, Hq, D))
    return out, lse


def append(q_in, k_in, v_in, q_w, k_w, seq_lens, *, block_table=None, page_size=16,
           num_pages=0, Lmax=0, eps: float = 1e-6, theta: float = 1e6):
    """New-token preparation: RMS-normalise q and k per head (gains q_w, k_w
    float32 [D], or None to skip), rotate them at position L_b (theta <= 0 to
    skip), and find where the k/v rows go.  q_in uint16 [B,Hq,D]; k_in, v_in
    uint16 [B,Hkv,D]; paged if block_table (int32 [B,max_pages]) is given,
    else contiguous with Lmax rows per sequence.  Returns (q_out, k_out,
    v_out) as exact f64 arrays, dest_row int64 [B] (-1 = not written) and
    new_lens int32 [B]."""
    _req(q_in, np.uint16, "q_in", 3); _req(k_in, np.uint16, "k_in", 3)
    _req(v_in, np.uint16, "v_in", 3); _req(seq_lens, np.int32, "seq_lens", 1)
    for w, n in ((q_w, "q_w"), (k_w, "k_w")):
        if w is not None:
            _req(w, np.float32, n, 1)
    if block_table is not None:
        _req(block_table, np.int32, "block_table", 2)
    B, Hq, D = q_in.shape
    _, Hkv, Dk = k_in.shape
    if k_in.shape != v_in.shape or k_in.shape[0] != B or Dk != D or seq_lens.shape[0] != B:
        raise ValueError("shape mismatch")
    q_out = np.empty((B, Hq, D), np.float64)
    k_out = np.empty((B, Hkv, D), np.float64)
    v_out = np.empty((B, Hkv, D), np.float64)
    dest = np.empty(B, np.int64)
    new_lens = np.empty(B, np.int32)
    L = _load()
    maxp = block_table.shape[1] if block_table is not None else 0
    _check(L.kvo_append(_ptr(q_in), _ptr(k_in), _ptr(v_in), _ptr(q_w), _ptr(k_w),
                        _ptr(block_table), _ptr(seq_lens), B, Hq, Hkv, D, int(page_size), maxp,
                        int(num_pages), int(Lmax), float(eps), float(theta), _ptr(q_out),
                        _ptr(k_out), _ptr(v_out), _ptr(dest), _ptr(new_lens)))
    return q_out, k_out, v_out, dest, new_lens


def round_bf16(x):
    """Nearest bf16 (ties to even) of float64 values, as uint16 bit patterns."""
    x = np.ascontiguousarray(x, np.float64)
    out = np.empty(x.shape, np.uint16)
    _check(_load().kvo_round_bf16(_ptr(x), _ptr(out), int(x.size)))
    return out


def fp8_table():
    """The value of each of the 256 fp8 (e4m3fn) codes, f64 [256] (NaN codes -> nan)."""
    out = np.empty(256, np.float64)
    _check(_load().kvo_fp8_table(_ptr(out)))
    return out


def decode_attn_fp8(q, k, v, seq_lens, scale: float, k_scale: float, v_scale: float, *,
                    block_table=None):
    """fp8 (e4m3fn) caches: k, v uint8 codes, [B,Lmax,Hkv,D] contiguous or
    [num_pages,P,Hkv,D] with a block table; keys are k_scale * fp8(code),
    values v_scale * fp8(code).  q uint16 [B,Hq,D].  Returns (out, lse) f64."""
    _req(q, np.uint16, "q", 3); _req(k, np.uint8, "k", 4); _req(v, np.uint8, "v", 4)
    _req(seq_lens, np.int32, "seq_lens", 1)
    B, Hq, D = q.shape
    if k.shape != v.shape or k.shape[3] != D or seq_lens.shape[0] != B:
        raise ValueError("shape mismatch")
    Hkv = k.shape[2]
    if block_table is not None:
        _req(block_table, np.int32, "block_table", 2)
        num_pages, P = k.shape[0], k.shape[1]
        maxp, Lmax = block_table.shape[1], 0
    else:
        if k.shape[0] != B:
            raise ValueError("shape mismatch")
        num_pages, P, maxp, Lmax = 0, 1, 0, k.shape[1]
    out = np.empty((B, Hq, D), np.float64)
    lse = np.empty((B, Hq), np.float64)
    _check(_load().kvo_decode_attn_fp8(_ptr(q), _ptr(k), _ptr(v), _ptr(block_table),
                                       _ptr(seq_lens), _ptr(out), _ptr(lse), B, Hq, Hkv, D, P,
                                       maxp, num_pages, Lmax, float(scale), float(k_scale),
                                       float(v_scale)))
    return out, lse


def prefill_paged(q, k_pool, v_pool, block_table, q_start, seq_lens, scale: float):
    """Chunked prefill: q uint16 [T,Hq,D] holds n_b = q_start[b+1] - q_start[b]
    new tokens of sequence b, already in its cache at positions L_b - n_b ..
    L_b - 1 (L_b = seq_lens[b]); token i attends positions 0 .. L_b - n_b + i.
    Returns (out f64 [T,Hq,D], lse f64 [T,Hq])."""
    _req(q, np.uint16, "q", 3); _req(k_pool, np.uint16, "k_pool", 4)
    _req(v_pool, np.uint16, "v_pool", 4); _req(block_table, np.int32, "block_table", 2)
    _req(q_start, np.int32, "q_start", 1); _req(seq_lens, np.int32, "seq_lens", 1)
    T, Hq, D = q.shape
    num_pages, P, Hkv, Dk = k_pool.shape
    B = seq_lens.shape[0]
    if k_pool.shape != v_pool.shape or Dk != D or block_table.shape[0] != B \
            or q_start.shape[0] != B + 1:
        raise ValueError("shape mismatch")
    out = np.empty((T, Hq, D), np.float64)
    lse = np.empty((T, Hq), np.float64)
    _check(_load().kvo_prefill_paged(_ptr(q), _ptr(k_pool), _ptr(v_pool), _ptr(block_table),
                                     _ptr(q_start), _ptr(seq_lens), _ptr(out), _ptr(lse), B, T, Hq,
                                     Hkv, D, P, block_table.shape[1], num_pages, float(scale)))
    return out, lse
