"""Python binding of libkva (include/kva.h): batched grouped-query decode
attention over bf16 KV caches on MI355X.

Argument marshalling only: each function checks dtypes, devices, contiguity
and shapes of torch tensors, then calls the C entry point of the same name with
raw device pointers and torch's current HIP stream.  All computation runs in
the HIP kernels of libkva.so; there is no fallback path.  If the library has
not been built, every call raises.

bf16 inputs may be torch.bfloat16 tensors or int16/uint16 tensors holding the
raw bit patterns.
"""
from __future__ import annotations

import ctypes
import os

__all__ = [
    "KvaError", "lib", "kva_status_str", "kva_version", "kva_workspace_bytes", "kva_new_workspace",
    "kva_decode_attn", "kva_decode_attn_paged", "kva_combine", "kva_debug_gather_paged",
    "kva_workspace_bytes_grouped", "kva_decode_attn_paged_grouped", "kva_append",
    "kva_append_paged", "kva_decode_attn_fp8", "kva_decode_attn_paged_fp8", "kva_prefill_paged",
    "kva_debug_stream_read", "kva_decode_attn_paged_noalloc", "KVA_NOALLOC_SCRATCH_BYTES",
    "kva_debug_xcd_count", "kva_debug_xcd_ids",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libkva.so")

KVA_OK = 0
STATUS_NAMES = {0: "KVA_OK", 1: "KVA_ERR_NULL", 2: "KVA_ERR_SHAPE", 3: "KVA_ERR_ALIGN",
                4: "KVA_ERR_WORKSPACE", 5: "KVA_ERR_UNSUPPORTED", 6: "KVA_ERR_HIP",
                7: "KVA_ERR_SCRATCH"}
# Size of the device array kva_decode_attn_paged_noalloc works in (include/kva.h).
KVA_NOALLOC_SCRATCH_BYTES = 64 << 20

_lib = None


class KvaError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {STATUS_NAMES.get(status, status)} ({kva_status_str(status)})")


def lib() -> ctypes.CDLL:
    """The loaded libkva.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with "
                              "`python -m paper_2609_12471_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P, i32, i64, sz, f32 = (ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_size_t,
                                ctypes.c_float)
        L.kva_status_str.argtypes = [i32]
        L.kva_status_str.restype = ctypes.c_char_p
        L.kva_version.argtypes = []
        L.kva_version.restype = i32
        L.kva_workspace_bytes.argtypes = [i32, i32, i32, i32]
        L.kva_workspace_bytes.restype = sz
        L.kva_decode_attn.argtypes = [P, P, P, P, P, P, i32, i32, i32, i32, i32, f32, P, sz, P]
        L.kva_decode_attn.restype = i32
        L.kva_decode_attn_paged.argtypes = [P, P, P, P, P, P, P, i32, i32, i32, i32, i32, i32,
                                            i64, f32, P, sz, P]
        L.kva_decode_attn_paged.restype = i32
        L.kva_decode_attn_paged_noalloc.argtypes = [P, P, P, P, P, P, P, i32, i32, i32, i32, i32,
                                                    i32, i64, f32, P]
        L.kva_decode_attn_paged_noalloc.restype = i32
        L.kva_workspace_bytes_grouped.argtypes = [i32, i32, i32, i32, i32]
        L.kva_workspace_bytes_grouped.restype = sz
        L.kva_decode_attn_paged_grouped.argtypes = [P, P, P, P, P, P, P, i32, i32, i32, i32, i32,
                                                    i32, i64, i32, f32, P, sz, P]
        L.kva_decode_attn_paged_grouped.restype = i32
        f64 = ctypes.c_double
        L.kva_prefill_paged.argtypes = [P, P, P, P, P, P, P, P, i32, i32, i32, i32, i32, i32, i32,
                                        i32, i64, f32, P]
        L.kva_prefill_paged.restype = i32
        L.kva_decode_attn_fp8.argtypes = [P, P, P, P, P, P, i32, i32, i32, i32, i32, f32, f32,
                                          f32, P, sz, P]
        L.kva_decode_attn_fp8.restype = i32
        L.kva_decode_attn_paged_fp8.argtypes = [P, P, P, P, P, P, P, i32, i32, i32, i32, i32,
                                                i32, i64, f32, f32, f32, P, sz, P]
        L.kva_decode_attn_paged_fp8.restype = i32
        L.kva_append.argtypes = [P, P, P, P, P, P, P, P, P, P, i32, i32, i32, i32, i32, f32,
                                 f64, P]
        L.kva_append.restype = i32
        L.kva_append_paged.argtypes = [P, P, P, P, P, P, P, P, P, P, P, i32, i32, i32, i32, i32,
                                       i32, i64, f32, f64, P]
        L.kva_append_paged.restype = i32
        L.kva_combine.argtypes = [P, P, P, P, i32, i32, i32, i32, P]
        L.kva_combine.restype = i32
        L.kva_debug_gather_paged.argtypes = [P, P, P, P, i32, i32, i32, i32, i32, i64, i32, P]
        L.kva_debug_gather_paged.restype = i32
        L.kva_debug_stream_read.argtypes = [P, sz, P, i32, P]
        L.kva_debug_stream_read.restype = i32
        L.kva_debug_xcd_count.argtypes = [ctypes.POINTER(i32)]
        L.kva_debug_xcd_count.restype = i32
        L.kva_debug_xcd_ids.argtypes = [P, i32, P]
        L.kva_debug_xcd_ids.restype = i32
        _lib = L
    return _lib


def kva_status_str(status: int) -> str:
    return lib().kva_status_str(int(status)).decode()


def kva_version() -> int:
    return int(lib().kva_version())


def kva_workspace_bytes(B: int, Hq: int, Hkv: int, D: int) -> int:
    return int(lib().kva_workspace_bytes(B, Hq, Hkv, D))


def kva_workspace_bytes_grouped(B: int, Hq: int, Hkv: int, D: int, group: int) -> int:
    return int(lib().kva_workspace_bytes_grouped(B, Hq, Hkv, D, group))


# ----------------------------------------------------------------------------- marshalling

def _torch():
    import torch
    return torch


def _dev(t, name, dtypes, ndim=None):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name}: expected a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name}: must be a device tensor")
    if t.dtype not in dtypes:
        raise TypeError(f"{name}: dtype {t.dtype} not in {dtypes}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: must be contiguous")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name}: expected {ndim} dims, got {tuple(t.shape)}")
    return t


def _bf16_types():
    torch = _torch()
    return (torch.bfloat16, torch.int16, torch.uint16)


def _stream(stream):
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def kva_new_workspace(B: int, Hq: int, Hkv: int, D: int, device="cuda"):
    """A workspace for batches of up to B sequences, reusable by any number of
    calls (one call in flight at a time).  It needs no initialisation."""
    torch = _torch()
    return torch.empty(max(kva_workspace_bytes(B, Hq, Hkv, D), 1), dtype=torch.uint8, device=device)


def _workspace(workspace, need, device, stream):
    """The caller's workspace, or a temporary one.  A temporary is freed when
    the wrapper returns while the kernels may still be queued: torch's caching
    allocator may hand its memory to the next allocation on the stream it was
    allocated for, so it is tied to the stream the kernels run on
    (record_stream).  A raw integer stream handle cannot be tied: it needs an
    explicit workspace."""
    torch = _torch()
    if workspace is not None:
        _dev(workspace, "workspace", (torch.uint8,), 1)
        return workspace
    if stream is not None and not isinstance(stream, torch.cuda.Stream):
        raise ValueError("workspace: pass an explicit workspace with a raw stream handle")
    ws = torch.empty(max(need, 1), dtype=torch.uint8, device=device)
    if stream is not None and stream != torch.cuda.current_stream(device):
        ws.record_stream(stream)
    return ws


def _check(rc, where):
    if rc != KVA_OK:
        raise KvaError(rc, where)


def kva_decode_attn(q, k, v, seq_lens, out, lse=None, *, scale: float, workspace=None,
                    stream=None):
    """Contiguous caches.  q [B,Hq,D]; k, v [B,Lmax,Hkv,D] (bf16 bits);
    seq_lens int32 [B]; out float32 [B,Hq,D]; lse float32 [B,Hq] or None."""
    torch = _torch()
    bt = _bf16_types()
    _dev(q, "q", bt, 3); _dev(k, "k", bt, 4); _dev(v, "v", bt, 4)
    _dev(seq_lens, "seq_lens", (torch.int32,), 1); _dev(out, "out", (torch.float32,), 3)
    B, Hq, D = q.shape
    _, Lmax, Hkv, Dk = k.shape
    if tuple(v.shape) != tuple(k.shape) or k.shape[0] != B or Dk != D or seq_lens.shape[0] != B \
            or tuple(out.shape) != (B, Hq, D):
        raise ValueError("shape mismatch")
    if lse is not None:
        _dev(lse, "lse", (torch.float32,), 2)
        if tuple(lse.shape) != (B, Hq):
            raise ValueError("lse shape mismatch")
    need = kva_workspace_bytes(B, Hq, Hkv, D)
    ws = _workspace(workspace, need, q.device, stream)
    rc = lib().kva_decode_attn(q.data_ptr(), k.data_ptr(), v.data_ptr(), seq_lens.data_ptr(),
                               out.data_ptr(), None if lse is None else lse.data_ptr(),
                               B, Hq, Hkv, D, Lmax, float(scale), ws.data_ptr(), ws.numel(),
                               _stream(stream))
    _check(rc, "kva_decode_attn")
    return out, lse


def kva_decode_attn_paged(q, k_pool, v_pool, block_table, seq_lens, out, lse=None, *,
                          scale: float, workspace=None, stream=None):
    """Paged caches.  k_pool, v_pool [num_pages,P,Hkv,D] (bf16 bits);
    block_table int32 [B,max_pages]; other arguments as kva_decode_attn."""
    torch = _torch()
    bt = _bf16_types()
    _dev(q, "q", bt, 3); _dev(k_pool, "k_pool", bt, 4); _dev(v_pool, "v_pool", bt, 4)
    _dev(block_table, "block_table", (torch.int32,), 2)
    _dev(seq_lens, "seq_lens", (torch.int32,), 1); _dev(out, "out", (torch.float32,), 3)
    B, Hq, D = q.shape
    num_pages, P, Hkv, Dk = k_pool.shape
    if tuple(v_pool.shape) != tuple(k_pool.shape) or Dk != D or block_table.shape[0] != B \
            or seq_lens.shape[0] != B or tuple(out.shape) != (B, Hq, D):
        raise ValueError("shape mismatch")
    if lse is not None:
        _dev(lse, "lse", (torch.float32,), 2)
        if tuple(lse.shape) != (B, Hq):
            raise ValueError("lse shape mismatch")
    need = kva_workspace_bytes(B, Hq, Hkv, D)
    ws = _workspace(workspace, need, q.device, stream)
    rc = lib().kva_decode_attn_paged(q.data_ptr(), k_pool.data_ptr(), v_pool.data_ptr(),
                                     block_table.data_ptr(), seq_lens.data_ptr(), out.data_ptr(),
                                     None if lse is None else lse.data_ptr(), B, Hq, Hkv, D, P,
                                     block_table.shape[1], num_pages, float(scale),
                                     ws.data_ptr(), ws.numel(), _stream(stream))
    _check(rc, "kva_decode_attn_paged")
    return out, lse


def kva_decode_attn_paged_noalloc(q, k_pool, v_pool, block_table, seq_lens, out, lse=None, *,
                                  scale: float, stream=None):
    """kva_decode_attn_paged without a workspace: the library's built-in device
    scratch array holds the partial results (nothing is allocated, here or in
    the library).  Calls that overlap on one device race."""
    torch = _torch()
    bt = _bf16_types()
    _dev(q, "q", bt, 3); _dev(k_pool, "k_pool", bt, 4); _dev(v_pool, "v_pool", bt, 4)
    _dev(block_table, "block_table", (torch.int32,), 2)
    _dev(seq_lens, "seq_lens", (torch.int32,), 1); _dev(out, "out", (torch.float32,), 3)
    B, Hq, D = q.shape
    num_pages, P, Hkv, Dk = k_pool.shape
    if tuple(v_pool.shape) != tuple(k_pool.shape) or Dk != D or block_table.shape[0] != B \
            or seq_lens.shape[0] != B or tuple(out.shape) != (B, Hq, D):
        raise ValueError("shape mismatch")
    if lse is not None:
        _dev(lse, "lse", (torch.float32,), 2)
        if tuple(lse.shape) != (B, Hq):
            raise ValueError("lse shape mismatch")
    rc = lib().kva_decode_attn_paged_noalloc(
        q.data_ptr(), k_pool.data_ptr(), v_pool.data_ptr(), block_table.data_ptr(),
        seq_lens.data_ptr(), out.data_ptr(), None if lse is None else lse.data_ptr(), B, Hq, Hkv,
        D, P, block_table.shape[1], num_pages, float(scale), _stream(stream))
    _check(rc, "kva_decode_attn_paged_noalloc")
    return out, lse


def _fp8_types():
    torch = _torch()
    return (torch.uint8, torch.int8, torch.float8_e4m3fn)


def kva_decode_attn_fp8(q, k, v, seq_lens, out, lse=None, *, scale: float, k_scale: float,
                        v_scale: float, workspace=None, stream=None):
    """Contiguous fp8 (e4m3fn) caches: k, v [B,Lmax,Hkv,D] codes (uint8 or
    float8_e4m3fn); keys are k_scale * fp8, values v_scale * fp8."""
    torch = _torch()
    _dev(q, "q", _bf16_types(), 3); _dev(k, "k", _fp8_types(), 4); _dev(v, "v", _fp8_types(), 4)
    _dev(seq_lens, "seq_lens", (torch.int32,), 1); _dev(out, "out", (torch.float32,), 3)
    B, Hq, D = q.shape
    _, Lmax, Hkv, Dk = k.shape
    if tuple(v.shape) != tuple(k.shape) or k.shape[0] != B or Dk != D or seq_lens.shape[0] != B \
            or tuple(out.shape) != (B, Hq, D):
        raise ValueError("shape mismatch")
    if lse is not None:
        _dev(lse, "lse", (torch.float32,), 2)
        if tuple(lse.shape) != (B, Hq):
            raise ValueError("lse shape mismatch")
    ws = _workspace(workspace, kva_workspace_bytes(B, Hq, Hkv, D), q.device, stream)
    rc = lib().kva_decode_attn_fp8(q.data_ptr(), k.data_ptr(), v.data_ptr(), seq_lens.data_ptr(),
                                   out.data_ptr(), None if lse is None else lse.data_ptr(), B, Hq,
                                   Hkv, D, Lmax, float(scale), float(k_scale), float(v_scale),
                                   ws.data_ptr(), ws.numel(), _stream(stream))
    _check(rc, "kva_decode_attn_fp8")
    return out, lse


def kva_decode_attn_paged_fp8(q, k_pool, v_pool, block_table, seq_lens, out, lse=None, *,
                              scale: float, k_scale: float, v_scale: float, workspace=None,
                              stream=None):
    """Paged fp8 (e4m3fn) caches [num_pages,P,Hkv,D]; other arguments as
    kva_decode_attn_paged."""
    torch = _torch()
    _dev(q, "q", _bf16_types(), 3); _dev(k_pool, "k_pool", _fp8_types(), 4)
    _dev(v_pool, "v_pool", _fp8_types(), 4)
    _dev(block_table, "block_table", (torch.int32,), 2)
    _dev(seq_lens, "seq_lens", (torch.int32,), 1); _dev(out, "out", (torch.float32,), 3)
    B, Hq, D = q.shape
    num_pages, P, Hkv, Dk = k_pool.shape
    if tuple(v_pool.shape) != tuple(k_pool.shape) or Dk != D or block_table.shape[0] != B \
            or seq_lens.shape[0] != B or tuple(out.shape) != (B, Hq, D):
        raise ValueError("shape mismatch")
    if lse is not None:
        _dev(lse, "lse", (torch.float32,), 2)
        if tuple(lse.shape) != (B, Hq):
            raise ValueError("lse shape mismatch")
    ws = _workspace(workspace, kva_workspace_bytes(B, Hq, Hkv, D), q.device, stream)
    rc = lib().kva_decode_attn_paged_fp8(
        q.data_ptr(), k_pool.data_ptr(), v_pool.data_ptr(), block_table.data_ptr(),
        seq_lens.data_ptr(), out.data_ptr(), None if lse is None else lse.data_ptr(), B, Hq, Hkv,
        D, P, block_table.shape[1], num_pages, float(scale), float(k_scale), float(v_scale),
        ws.data_ptr(), ws.numel(), _stream(stream))
    _check(rc, "kva_decode_attn_paged_fp8")
    return out, lse


def kva_decode_attn_paged_grouped(q, k_pool, v_pool, block_table, seq_lens, out, lse=None, *,
                                  group: int, scale: float, workspace=None, stream=None):
    """Paged caches whose consecutive groups of `group` sequences may start
    with the same pages; arguments as kva_decode_attn_paged."""
    torch = _torch()
    bt = _bf16_types()
    _dev(q, "q", bt, 3); _dev(k_pool, "k_pool", bt, 4); _dev(v_pool, "v_pool", bt, 4)
    _dev(block_table, "block_table", (torch.int32,), 2)
    _dev(seq_lens, "seq_lens", (torch.int32,), 1); _dev(out, "out", (torch.float32,), 3)
    B, Hq, D = q.shape
    num_pages, P, Hkv, Dk = k_pool.shape
    if tuple(v_pool.shape) != tuple(k_pool.shape) or Dk != D or block_table.shape[0] != B \
            or seq_lens.shape[0] != B or tuple(out.shape) != (B, Hq, D):
        raise ValueError("shape mismatch")
    if lse is not None:
        _dev(lse, "lse", (torch.float32,), 2)
        if tuple(lse.shape) != (B, Hq):
            raise ValueError("lse shape mismatch")
    need = kva_workspace_bytes_grouped(B, Hq, Hkv, D, group)
    ws = _workspace(workspace, need, q.device, stream)
    rc = lib().kva_decode_attn_paged_grouped(
        q.data_ptr(), k_pool.data_ptr(), v_pool.data_ptr(), block_table.data_ptr(),
        seq_lens.data_ptr(), out.data_ptr(), None if lse is None else lse.data_ptr(), B, Hq, Hkv,
        D, P, block_table.shape[1], num_pages, int(group), float(scale), ws.data_ptr(), ws.numel(),
        _stream(stream))
    _check(rc, "kva_decode_attn_paged_grouped")
    return out, lse


def _opt_f32(t, name, n):
    torch = _torch()
    if t is None:
        return None
    _dev(t, name, (torch.float32,), 1)
    if t.shape[0] != n:
        raise ValueError(f"{name}: expected {n} values")
    return t.data_ptr()


def _append_check(q_in, k_in, v_in, q_out, seq_lens, new_lens):
    torch = _torch()
    bt = _bf16_types()
    _dev(q_in, "q_in", bt, 3); _dev(k_in, "k_in", bt, 3); _dev(v_in, "v_in", bt, 3)
    _dev(q_out, "q_out", bt, 3); _dev(seq_lens, "seq_lens", (torch.int32,), 1)
    B, Hq, D = q_in.shape
    _, Hkv, Dk = k_in.shape
    if tuple(v_in.shape) != tuple(k_in.shape) or k_in.shape[0] != B or Dk != D \
            or tuple(q_out.shape) != (B, Hq, D) or seq_lens.shape[0] != B:
        raise ValueError("shape mismatch")
    if new_lens is not None:
        _dev(new_lens, "new_lens", (torch.int32,), 1)
        if new_lens.shape[0] != B:
            raise ValueError("new_lens shape mismatch")
    return B, Hq, Hkv, D


def kva_append(q_in, k_in, v_in, q_out, k_cache, v_cache, seq_lens, new_lens=None, *,
               q_norm_w=None, k_norm_w=None, eps: float = 1e-6, rope_theta: float = 1e6,
               stream=None):
    """New-token step, contiguous caches [B, Lmax, Hkv, D]: RMS-normalise and
    rotate q and k, write q_out, append k and v at position seq_lens[b]."""
    B, Hq, Hkv, D = _append_check(q_in, k_in, v_in, q_out, seq_lens, new_lens)
    bt = _bf16_types()
    _dev(k_cache, "k_cache", bt, 4); _dev(v_cache, "v_cache", bt, 4)
    if tuple(k_cache.shape) != tuple(v_cache.shape) or k_cache.shape[0] != B \
            or k_cache.shape[2] != Hkv or k_cache.shape[3] != D:
        raise ValueError("cache shape mismatch")
    rc = lib().kva_append(q_in.data_ptr(), k_in.data_ptr(), v_in.data_ptr(),
                          _opt_f32(q_norm_w, "q_norm_w", D), _opt_f32(k_norm_w, "k_norm_w", D),
                          q_out.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(),
                          seq_lens.data_ptr(), None if new_lens is None else new_lens.data_ptr(),
                          B, Hq, Hkv, D, k_cache.shape[1], float(eps), float(rope_theta),
                          _stream(stream))
    _check(rc, "kva_append")


def kva_append_paged(q_in, k_in, v_in, q_out, k_pool, v_pool, block_table, seq_lens,
                     new_lens=None, *, q_norm_w=None, k_norm_w=None, eps: float = 1e-6,
                     rope_theta: float = 1e6, stream=None):
    """New-token step, paged caches [num_pages, P, Hkv, D] with a block table."""
    torch = _torch()
    B, Hq, Hkv, D = _append_check(q_in, k_in, v_in, q_out, seq_lens, new_lens)
    bt = _bf16_types()
    _dev(k_pool, "k_pool", bt, 4); _dev(v_pool, "v_pool", bt, 4)
    _dev(block_table, "block_table", (torch.int32,), 2)
    num_pages, P, Hkv2, D2 = k_pool.shape
    if tuple(v_pool.shape) != tuple(k_pool.shape) or Hkv2 != Hkv or D2 != D \
            or block_table.shape[0] != B:
        raise ValueError("pool shape mismatch")
    rc = lib().kva_append_paged(q_in.data_ptr(), k_in.data_ptr(), v_in.data_ptr(),
                                _opt_f32(q_norm_w, "q_norm_w", D),
                                _opt_f32(k_norm_w, "k_norm_w", D), q_out.data_ptr(),
                                k_pool.data_ptr(), v_pool.data_ptr(), block_table.data_ptr(),
                                seq_lens.data_ptr(),
                                None if new_lens is None else new_lens.data_ptr(), B, Hq, Hkv, D,
                                P, block_table.shape[1], num_pages, float(eps), float(rope_theta),
                                _stream(stream))
    _check(rc, "kva_append_paged")


def kva_prefill_paged(q, k_pool, v_pool, block_table, q_start, seq_lens, out, lse=None, *,
                      max_q_len: int, scale: float, stream=None):
    """Chunked prefill.  q [T,Hq,D] (bf16 bits): the new tokens of all
    sequences, sequence b's rows q_start[b] .. q_start[b+1]-1 (q_start int32
    [B+1]); their keys/values already sit at positions L_b - n_b .. L_b - 1 of
    the paged cache (L_b = seq_lens[b]); out float32 [T,Hq,D]."""
    torch = _torch()
    bt = _bf16_types()
    _dev(q, "q", bt, 3); _dev(k_pool, "k_pool", bt, 4); _dev(v_pool, "v_pool", bt, 4)
    _dev(block_table, "block_table", (torch.int32,), 2)
    _dev(q_start, "q_start", (torch.int32,), 1); _dev(seq_lens, "seq_lens", (torch.int32,), 1)
    _dev(out, "out", (torch.float32,), 3)
    T, Hq, D = q.shape
    num_pages, P, Hkv, Dk = k_pool.shape
    B = seq_lens.shape[0]
    if tuple(v_pool.shape) != tuple(k_pool.shape) or Dk != D or block_table.shape[0] != B \
            or q_start.shape[0] != B + 1 or tuple(out.shape) != (T, Hq, D):
        raise ValueError("shape mismatch")
    if lse is not None:
        _dev(lse, "lse", (torch.float32,), 2)
        if tuple(lse.shape) != (T, Hq):
            raise ValueError("lse shape mismatch")
    rc = lib().kva_prefill_paged(q.data_ptr(), k_pool.data_ptr(), v_pool.data_ptr(),
                                 block_table.data_ptr(), q_start.data_ptr(), seq_lens.data_ptr(),
                                 out.data_ptr(), None if lse is None else lse.data_ptr(), B, T,
                                 int(max_q_len), Hq, Hkv, D, P, block_table.shape[1], num_pages,
                                 float(scale), _stream(stream))
    _check(rc, "kva_prefill_paged")
    return out, lse


def kva_combine(o_parts, lse_parts, out, lse=None, *, stream=None):
    """o_parts float32 [S,B,Hq,D]; lse_parts float32 [S,B,Hq]; out [B,Hq,D]."""
    torch = _torch()
    _dev(o_parts, "o_parts", (torch.float32,), 4); _dev(lse_parts, "lse_parts", (torch.float32,), 3)
    _dev(out, "out", (torch.float32,), 3)
    S, B, Hq, D = o_parts.shape
    if tuple(lse_parts.shape) != (S, B, Hq) or tuple(out.shape) != (B, Hq, D):
        raise ValueError("shape mismatch")
    if lse is not None:
        _dev(lse, "lse", (torch.float32,), 2)
        if tuple(lse.shape) != (B, Hq):
            raise ValueError("lse shape mismatch")
    rc = lib().kva_combine(o_parts.data_ptr(), lse_parts.data_ptr(), out.data_ptr(),
                           None if lse is None else lse.data_ptr(), S, B, Hq, D, _stream(stream))
    _check(rc, "kva_combine")
    return out, lse


def kva_debug_gather_paged(pool, block_table, seq_lens, dst, *, stream=None):
    """pool [num_pages,P,Hkv,D] (bf16 bits) -> dst [B,Lcap,Hkv,D] via the block table."""
    torch = _torch()
    bt = _bf16_types()
    _dev(pool, "pool", bt, 4); _dev(dst, "dst", bt, 4)
    _dev(block_table, "block_table", (torch.int32,), 2); _dev(seq_lens, "seq_lens", (torch.int32,), 1)
    num_pages, P, Hkv, D = pool.shape
    B, Lcap, Hkv2, D2 = dst.shape
    if Hkv2 != Hkv or D2 != D or block_table.shape[0] != B or seq_lens.shape[0] != B:
        raise ValueError("shape mismatch")
    rc = lib().kva_debug_gather_paged(pool.data_ptr(), block_table.data_ptr(), seq_lens.data_ptr(),
                                      dst.data_ptr(), B, Hkv, D, P, block_table.shape[1],
                                      num_pages, Lcap, _stream(stream))
    _check(rc, "kva_debug_gather_paged")
    return dst


def kva_debug_stream_read(src, sink, *, stream=None):
    """Streaming read of the bytes of `src` (a contiguous CUDA tensor of a
    multiple of 16 bytes); block i XOR-reduces its share into sink[i] (int32)."""
    torch = _torch()
    if not (src.is_cuda and src.is_contiguous()):
        raise ValueError("src: contiguous CUDA tensor expected")
    _dev(sink, "sink", (torch.int32,), 1)
    rc = lib().kva_debug_stream_read(src.data_ptr(), src.numel() * src.element_size(), sink.data_ptr(),
                                     sink.shape[0], _stream(stream))
    _check(rc, "kva_debug_stream_read")
    return sink


def kva_debug_xcd_count() -> int:
    """XCDs of the current device as the runtime reports them (0: not reported)."""
    x = ctypes.c_int(0)
    _check(lib().kva_debug_xcd_count(ctypes.byref(x)), "kva_debug_xcd_count")
    return int(x.value)


def kva_debug_xcd_ids(out, *, stream=None):
    """Launch out.shape[0] one-wave workgroups; workgroup b writes the XCD it
    runs on to out[b] (int32 CUDA tensor)."""
    torch = _torch()
    _dev(out, "out", (torch.int32,), 1)
    rc = lib().kva_debug_xcd_ids(out.data_ptr(), out.shape[0], _stream(stream))
    _check(rc, "kva_debug_xcd_ids")
    return out
