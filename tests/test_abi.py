"""The C-ABI library on the host: it loads, exports every entry point that
include/kva.h declares, and rejects bad arguments before any launch.  No
compute call is made here; every rejected call returns before touching HIP."""
import ctypes
import os
import re

import pytest

import paper_2609_12471_amd as kva

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "kva.h")


def declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(kva_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    names = declared()
    assert {"kva_decode_attn", "kva_decode_attn_paged", "kva_combine", "kva_workspace_bytes",
            "kva_status_str", "kva_debug_gather_paged", "kva_version"} <= set(names)
    L = kva.lib()
    for n in names:
        assert hasattr(L, n), n
    nm = os.popen(f"nm -D --defined-only {kva.LIB_PATH}").read()
    for n in names:
        assert re.search(rf"\bT {n}$", nm, flags=re.M), f"{n} not exported with C linkage"


def test_status_strings_and_version():
    assert kva.kva_version() == 2
    for s in range(8):
        assert kva.kva_status_str(s) and kva.kva_status_str(s) != "unknown status"
    assert kva.kva_status_str(99) == "unknown status"


def test_workspace_needs_no_header_rule():
    """The workspace has no part that must be zero at first use: the header
    declares no such constant and the binding allocates workspaces uninitialised."""
    hdr = open(HEADER).read()
    assert "KVA_WORKSPACE_HEADER" not in hdr
    assert not hasattr(kva, "KVA_WORKSPACE_HEADER")


def test_workspace_bytes():
    a = kva.kva_workspace_bytes(64, 32, 8, 128)
    b = kva.kva_workspace_bytes(256, 32, 8, 128)
    assert 0 < a < b < 128 << 20
    assert kva.kva_workspace_bytes(-1, 32, 8, 128) == 0
    assert kva.kva_workspace_bytes(4, 30, 8, 128) == 0
    assert kva.kva_workspace_bytes(0, 32, 8, 128) > 0


FAKE = 1 << 20          # a 16-byte aligned non-NULL address; never dereferenced


def call_contig(**kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, lens=FAKE, out=FAKE, lse=None, B=2, Hq=32, Hkv=8, D=128,
             Lmax=64, scale=0.088, ws=FAKE, wsb=1 << 30, stream=None)
    a.update(kw)
    return kva.lib().kva_decode_attn(a["q"], a["k"], a["v"], a["lens"], a["out"], a["lse"], a["B"],
                                     a["Hq"], a["Hkv"], a["D"], a["Lmax"], a["scale"], a["ws"],
                                     a["wsb"], a["stream"])


def call_paged(**kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, bt=FAKE, lens=FAKE, out=FAKE, lse=None, B=2, Hq=32, Hkv=8,
             D=128, P=16, maxp=8, npages=100, scale=0.088, ws=FAKE, wsb=1 << 30, stream=None)
    a.update(kw)
    return kva.lib().kva_decode_attn_paged(a["q"], a["k"], a["v"], a["bt"], a["lens"], a["out"],
                                           a["lse"], a["B"], a["Hq"], a["Hkv"], a["D"], a["P"],
                                           a["maxp"], a["npages"], a["scale"], a["ws"], a["wsb"],
                                           a["stream"])


@pytest.mark.parametrize("kw,status", [
    (dict(D=64), 5), (dict(Hq=24, Hkv=8), 5), (dict(Hq=30, Hkv=8), 2), (dict(B=-1), 2),
    (dict(Lmax=-3), 2), (dict(q=None), 1), (dict(out=None), 1), (dict(k=FAKE + 2), 3),
    (dict(out=FAKE + 4), 3), (dict(lse=FAKE + 2), 3), (dict(ws=None), 4), (dict(wsb=100), 4),
    (dict(ws=FAKE + 16), 3), (dict(scale=float("nan")), 5), (dict(Lmax=1 << 29), 5),
    (dict(scale=3e38), 5), (dict(scale=-3e38), 5), (dict(B=0), 0),
])
def test_contig_argument_checks(kw, status):
    assert call_contig(**kw) == status


@pytest.mark.parametrize("kw,status", [
    (dict(P=24), 5), (dict(P=2048), 5), (dict(P=0), 2), (dict(maxp=-1), 2), (dict(npages=-1), 2),
    (dict(bt=None), 1), (dict(bt=FAKE + 2), 3), (dict(v=FAKE + 8), 3), (dict(D=256), 5),
    (dict(npages=(1 << 31) + 1), 5), (dict(maxp=1 << 25), 5), (dict(wsb=0), 4), (dict(B=0), 0),
    (dict(scale=3e38), 5), (dict(scale=float("-inf")), 5),
])
def test_paged_argument_checks(kw, status):
    assert call_paged(**kw) == status


def test_combine_and_gather_argument_checks():
    L = kva.lib()
    assert L.kva_combine(FAKE, FAKE, FAKE, None, 2, 3, 4, 127, None) == 5
    assert L.kva_combine(FAKE, FAKE, None, None, 2, 3, 4, 128, None) == 1
    assert L.kva_combine(FAKE + 4, FAKE, FAKE, None, 2, 3, 4, 128, None) == 3
    assert L.kva_combine(FAKE, FAKE, FAKE, None, -1, 3, 4, 128, None) == 2
    assert L.kva_combine(FAKE, FAKE, FAKE, None, 2, 0, 4, 128, None) == 0
    assert L.kva_debug_gather_paged(FAKE, FAKE, FAKE, FAKE, 2, 8, 128, 12, 4, 10, 64, None) == 5
    assert L.kva_debug_gather_paged(None, FAKE, FAKE, FAKE, 2, 8, 128, 16, 4, 10, 64, None) == 1
    assert L.kva_debug_gather_paged(FAKE, FAKE, FAKE, FAKE + 8, 2, 8, 128, 16, 4, 10, 64, None) == 3
    assert L.kva_debug_gather_paged(FAKE, FAKE, FAKE, FAKE, 2, 8, 128, 16, 4, 10, 0, None) == 0
    assert L.kva_debug_stream_read(FAKE, 1000, FAKE, 8, None) == 2          # not a multiple of 16
    assert L.kva_debug_stream_read(None, 1024, FAKE, 8, None) == 1
    assert L.kva_debug_stream_read(FAKE, 1024, FAKE, 0, None) == 1
    assert L.kva_debug_stream_read(FAKE + 8, 1024, FAKE, 8, None) == 3
    assert L.kva_debug_stream_read(FAKE, 0, None, 0, None) == 0             # nothing to read


def test_xcd_hook_argument_checks():
    L = kva.lib()
    assert L.kva_debug_xcd_count(None) == 1
    assert L.kva_debug_xcd_ids(FAKE, -1, None) == 2
    assert L.kva_debug_xcd_ids(FAKE, 65537, None) == 2
    assert L.kva_debug_xcd_ids(None, 8, None) == 1
    assert L.kva_debug_xcd_ids(FAKE + 2, 8, None) == 3
    assert L.kva_debug_xcd_ids(None, 0, None) == 0                         # nothing to launch


def call_grouped(**kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, bt=FAKE, lens=FAKE, out=FAKE, lse=None, B=16, Hq=32, Hkv=8,
             D=128, P=16, maxp=8, npages=100, group=8, scale=0.088, ws=FAKE, wsb=1 << 30,
             stream=None)
    a.update(kw)
    return kva.lib().kva_decode_attn_paged_grouped(
        a["q"], a["k"], a["v"], a["bt"], a["lens"], a["out"], a["lse"], a["B"], a["Hq"], a["Hkv"],
        a["D"], a["P"], a["maxp"], a["npages"], a["group"], a["scale"], a["ws"], a["wsb"],
        a["stream"])


@pytest.mark.parametrize("kw,status", [
    (dict(group=0), 2), (dict(group=-3), 2), (dict(group=9), 5), (dict(Hq=64, group=5), 5),
    (dict(Hq=8, Hkv=8, group=33), 5), (dict(P=24), 5), (dict(bt=None), 1), (dict(wsb=1000), 4),
    (dict(ws=FAKE + 64), 3), (dict(q=FAKE + 2), 3), (dict(B=0), 0), (dict(B=0, group=1), 0),
])
def test_grouped_argument_checks(kw, status):
    assert call_grouped(**kw) == status


def test_grouped_workspace_bytes():
    plain = kva.kva_workspace_bytes(128, 32, 8, 128)
    grouped = kva.kva_workspace_bytes_grouped(128, 32, 8, 128, 8)
    # plain part, one int32 per group, 4 prefix partials (129 floats) per (b, h)
    assert grouped >= plain + 4 * 128 * 32 * 129 * 4 + 16 * 4
    assert grouped < plain + 4 * 128 * 32 * 129 * 4 + 4096
    assert kva.kva_workspace_bytes_grouped(128, 32, 8, 128, 0) == 0
    assert kva.kva_workspace_bytes_grouped(-1, 32, 8, 128, 8) == 0
    assert kva.kva_workspace_bytes_grouped(128, 30, 8, 128, 8) == 0


def call_append_paged(**kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, qw=None, kw=None, qo=FAKE, kp=FAKE, vp=FAKE, bt=FAKE,
             lens=FAKE, nl=None, B=4, Hq=32, Hkv=8, D=128, P=16, maxp=8, npages=100, eps=1e-6,
             theta=1e6, stream=None)
    a.update(kw)
    return kva.lib().kva_append_paged(a["q"], a["k"], a["v"], a["qw"], a["kw"], a["qo"], a["kp"],
                                      a["vp"], a["bt"], a["lens"], a["nl"], a["B"], a["Hq"],
                                      a["Hkv"], a["D"], a["P"], a["maxp"], a["npages"], a["eps"],
                                      a["theta"], a["stream"])


@pytest.mark.parametrize("kw,status", [
    (dict(D=64), 5), (dict(Hq=24), 5), (dict(Hq=30), 2), (dict(B=-1), 2), (dict(P=12), 5),
    (dict(P=0), 2), (dict(npages=-1), 2), (dict(q=None), 1), (dict(qo=None), 1),
    (dict(lens=None), 1), (dict(bt=None), 1), (dict(kp=None), 1), (dict(qo=FAKE + 2), 3),
    (dict(qw=FAKE + 4), 3), (dict(nl=FAKE + 2), 3), (dict(eps=-1.0), 5),
    (dict(eps=float("inf")), 5), (dict(theta=float("nan")), 5), (dict(theta=1.0), 5),
    (dict(B=0), 0), (dict(B=0, q=None), 0),
])
def test_append_argument_checks(kw, status):
    assert call_append_paged(**kw) == status


def test_append_contiguous_argument_checks():
    L = kva.lib()
    args = [FAKE, FAKE, FAKE, None, None, FAKE, FAKE, FAKE, FAKE, None]
    assert L.kva_append(*args, 2, 32, 8, 128, -1, 1e-6, 1e6, None) == 2
    assert L.kva_append(*args, 2, 32, 8, 128, 1 << 29, 1e-6, 1e6, None) == 5
    assert L.kva_append(*args[:6], None, FAKE, FAKE, None, 2, 32, 8, 128, 16, 1e-6, 1e6,
                        None) == 1
    assert L.kva_append(*args, 0, 32, 8, 128, 16, 1e-6, 1e6, None) == 0


def test_fp8_argument_checks():
    L = kva.lib()
    base = [FAKE, FAKE, FAKE, FAKE, FAKE, None, 2, 32, 8, 128, 64]
    ok = [0.088, 0.03, 0.02, FAKE, 1 << 30, None]
    assert L.kva_decode_attn_fp8(*base[:6], 2, 32, 8, 64, 64, *ok) == 5
    assert L.kva_decode_attn_fp8(*base, 0.088, float("nan"), 0.02, FAKE, 1 << 30, None) == 5
    assert L.kva_decode_attn_fp8(*base, 0.088, 0.03, float("inf"), FAKE, 1 << 30, None) == 5
    # finite scales whose folded product (scale * k_scale * log2 e) overflows fp32
    assert L.kva_decode_attn_fp8(*base, 1.0, 3e38, 0.02, FAKE, 1 << 30, None) == 5
    assert L.kva_decode_attn_fp8(FAKE, FAKE + 2, FAKE, FAKE, FAKE, None, 2, 32, 8, 128, 64,
                                 *ok) == 3
    assert L.kva_decode_attn_fp8(*base, 0.088, 0.03, 0.02, FAKE, 100, None) == 4
    assert L.kva_decode_attn_fp8(FAKE, FAKE, FAKE, FAKE, FAKE, None, 0, 32, 8, 128, 64, *ok) == 0
    pbase = [FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, 2, 32, 8, 128, 16, 8, 100]
    assert L.kva_decode_attn_paged_fp8(*pbase, 0.088, float("nan"), 0.02, FAKE, 1 << 30,
                                       None) == 5
    assert L.kva_decode_attn_paged_fp8(*pbase[:11], 12, 8, 100, *ok) == 5
    assert L.kva_decode_attn_paged_fp8(*pbase, 100.0, 3e37, 0.02, FAKE, 1 << 30, None) == 5
    assert L.kva_decode_attn_paged_fp8(*pbase[:3], None, *pbase[4:], *ok) == 1
    assert L.kva_decode_attn_paged_fp8(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, 0, 32, 8, 128,
                                       16, 8, 100, *ok) == 0


def test_prefill_argument_checks():
    L = kva.lib()

    def call(**kw):
        a = dict(q=FAKE, k=FAKE, v=FAKE, bt=FAKE, qs=FAKE, lens=FAKE, out=FAKE, lse=None, B=4,
                 T=100, mq=64, Hq=32, Hkv=8, D=128, P=16, maxp=8, npages=100, scale=0.088)
        a.update(kw)
        return L.kva_prefill_paged(a["q"], a["k"], a["v"], a["bt"], a["qs"], a["lens"], a["out"],
                                   a["lse"], a["B"], a["T"], a["mq"], a["Hq"], a["Hkv"], a["D"],
                                   a["P"], a["maxp"], a["npages"], a["scale"], None)
    assert call(T=-1) == 2 and call(mq=-1) == 2 and call(Hq=30) == 2 and call(P=0) == 2
    assert call(D=64) == 5 and call(P=24) == 5 and call(scale=float("nan")) == 5
    assert call(scale=3e38) == 5
    assert call(Hq=24) == 5
    assert call(q=None) == 1 and call(qs=None) == 1 and call(out=None) == 1 and call(bt=None) == 1
    assert call(q=FAKE + 2) == 3 and call(qs=FAKE + 2) == 3 and call(lse=FAKE + 2) == 3
    assert call(B=0) == 0 and call(T=0) == 0 and call(mq=0) == 0


def call_noalloc(**kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, bt=FAKE, lens=FAKE, out=FAKE, lse=None, B=2, Hq=32, Hkv=8,
             D=128, P=16, maxp=8, npages=100, scale=0.088, stream=None)
    a.update(kw)
    return kva.lib().kva_decode_attn_paged_noalloc(
        a["q"], a["k"], a["v"], a["bt"], a["lens"], a["out"], a["lse"], a["B"], a["Hq"], a["Hkv"],
        a["D"], a["P"], a["maxp"], a["npages"], a["scale"], a["stream"])


@pytest.mark.parametrize("kw,status", [
    (dict(P=24), 5), (dict(bt=None), 1), (dict(q=FAKE + 2), 3), (dict(Hq=30), 2),
    (dict(B=0), 0), (dict(B=0, Hq=64), 0),
    # a workspace beyond the built-in scratch array: 8 query heads per KV head
    # and 2048 sequences need 2560 slots x 64 heads x 512 B > 64 MiB
    (dict(B=2048, Hq=64, Hkv=8), 7), (dict(B=5000, Hq=64, Hkv=8), 7),
])
def test_noalloc_argument_checks(kw, status):
    """Rejections happen on the host before any HIP call (a CPU-only host
    returns them too); a batch that fits returns before the scratch lookup
    only when it is empty."""
    assert call_noalloc(**kw) == status


def test_noalloc_scratch_limit_covers_every_batch_of_the_decode_shape():
    from paper_2609_12471_amd import KVA_NOALLOC_SCRATCH_BYTES
    hdr = open(HEADER).read()
    assert re.search(r"#define KVA_NOALLOC_SCRATCH_BYTES \(\(size_t\)64 << 20\)", hdr)
    assert KVA_NOALLOC_SCRATCH_BYTES == 64 << 20
    for B in (1, 64, 256, 2048, 100000):
        assert kva.kva_workspace_bytes(B, 32, 8, 128) <= KVA_NOALLOC_SCRATCH_BYTES
    assert kva.kva_workspace_bytes(2048, 64, 8, 128) > KVA_NOALLOC_SCRATCH_BYTES
