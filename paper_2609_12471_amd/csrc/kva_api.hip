// C-ABI entry points of libkva (declared in include/kva.h): host-side argument
// checks, workspace layout, launch sizing.  No device memory is allocated here:
// kva_decode_attn_paged_noalloc uses the file-scope device array `scratch`
// below, which the code object holds on every device the library runs on.

#include <atomic>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <mutex>

#include "kva.h"
#include "kva_internal.h"

namespace {

using namespace kva;

constexpr int kMaxDevices = 64;
constexpr int64_t kMaxCap = int64_t(1) << 28;     // longest supported sequence (tokens)
constexpr size_t kWsAlign = 256;

bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

int log2_exact(int x) {
    int l = 0;
    while ((1 << l) < x) ++l;
    return (1 << l) == x ? l : -1;
}

// The score multiplier in base 2 (scale * log2 e, times k_scale for fp8
// caches) as the kernels use it; false when it is not a finite float (a finite
// scale near the float limit overflows once folded).
bool fold_scale(double scale, float *out) {
    const float f = (float)(scale * 1.4426950408889634);
    if (!std::isfinite(scale) || !std::isfinite(f)) return false;
    *out = f;
    return true;
}

bool group_ok(int Hq, int Hkv) {
    if (Hq <= 0 || Hkv <= 0 || Hq % Hkv) return false;
    const int g = Hq / Hkv;
    return g == 1 || g == 2 || g == 4 || g == 8;
}

struct WsLayout {
    size_t plan, lse, o, total;
};

// [plan: B x int2][lse partials: slots x Hq floats][o partials: slots x Hq x D
// floats]; every byte the kernels read was written earlier in the same call,
// so the workspace needs no initialisation.
WsLayout ws_layout(int B, int Hq, int Hkv, int D) {
    const int64_t slots = max_slots(B, Hkv);
    WsLayout w;
    w.plan = 0;
    w.lse = w.plan + round_up(sizeof(int2) * (size_t)B, kWsAlign);
    w.o = w.lse + round_up(sizeof(float) * (size_t)slots * (size_t)Hq, kWsAlign);
    w.total = w.o + round_up(sizeof(float) * (size_t)slots * (size_t)Hq * (size_t)D, kWsAlign);
    return w;
}

// Workspace of kva_decode_attn_paged_noalloc, for callers that cannot
// allocate.  Each device holds its own copy for the life of the process.  In
// host code `scratch` is only a stand-in for the device array: its device
// address comes from hipGetSymbolAddress, once per device (scratch_address),
// and only that address is ever handed to kernels.  Every call on a device
// shares the array, so calls that overlap on one device race.
constexpr size_t kScratchBytes = KVA_NOALLOC_SCRATCH_BYTES;
static_assert(kScratchBytes % 256 == 0, "scratch size");
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::atomic<void *> g_scratch_addr[kMaxDevices];
std::mutex g_scratch_mu;

// Device address of `scratch` on the current device (looked up on the first
// call on each device, with that device current).
int scratch_address(void **addr) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return KVA_ERR_HIP;
    if (dev < 0 || dev >= kMaxDevices) return KVA_ERR_HIP;
    void *p = g_scratch_addr[dev].load(std::memory_order_acquire);
    if (!p) {
        std::lock_guard<std::mutex> lock(g_scratch_mu);
        p = g_scratch_addr[dev].load(std::memory_order_acquire);
        if (!p) {
            if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return KVA_ERR_HIP;
            g_scratch_addr[dev].store(p, std::memory_order_release);
        }
    }
    *addr = p;
    return KVA_OK;
}

// Resident attention waves per compute unit, cached per (device, kv type, layout, group).
std::atomic<int> g_waves_cache[kMaxDevices][2][3][4];
std::atomic<int> g_cu_cache[kMaxDevices];
std::atomic<int> g_xcd_cache[kMaxDevices];   // XCDs per device; -1: the runtime does not say

// XCDs of the current device, from the runtime (0 if it does not report them).
hipError_t device_xcds(int *xcds) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    int x = g_xcd_cache[dev].load(std::memory_order_relaxed);
    if (x == 0) {
        int v = 0;
        x = hipDeviceGetAttribute(&v, hipDeviceAttributeNumberOfXccs, dev) == hipSuccess && v > 0 ? v : -1;
        g_xcd_cache[dev].store(x, std::memory_order_relaxed);
    }
    *xcds = x > 0 ? x : 0;
    return hipSuccess;
}

int group_index(int group) { return group == 1 ? 0 : group == 2 ? 1 : group == 4 ? 2 : 3; }

// Optional override for tuning sweeps: KVA_WAVES_PER_CU (read per call; not cached).
int env_waves_per_cu() {
    const char *s = std::getenv("KVA_WAVES_PER_CU");
    if (!s || !*s) return 0;
    const int v = std::atoi(s);
    return v > 0 ? v : 0;
}

// Waves of one attention launch over B sequences: the resident waves per CU
// (registers, and the launch's LDS footprint), capped by the target.
hipError_t launch_waves(int layout, int group, int kv, int B, int *waves, int *cus_out = nullptr) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    int cus = g_cu_cache[dev].load(std::memory_order_relaxed);
    if (cus <= 0) {
        e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
        if (e != hipSuccess) return e;
        g_cu_cache[dev].store(cus, std::memory_order_relaxed);
    }
    std::atomic<int> &slot = g_waves_cache[dev][kv][layout][group_index(group)];
    int per_cu = slot.load(std::memory_order_relaxed);
    if (per_cu <= 0) {
        e = attn_waves_per_cu(layout, group, kv, &per_cu);
        if (e != hipSuccess) return e;
        if (per_cu <= 0) per_cu = kWavesPerBlock;
        slot.store(per_cu, std::memory_order_relaxed);
    }
    const int blocks_lds = kLdsPerCU / attn_lds_bytes(B > 0 ? B : 1, group, kv);
    if (per_cu > blocks_lds * kWavesPerBlock) per_cu = (blocks_lds > 0 ? blocks_lds : 1) * kWavesPerBlock;
    const int target = layout != kPagedNarrow
                           ? (kv == kKvFp8 ? kTargetWavesPerCUMfmaFp8 : kTargetWavesPerCUMfmaBf16)
                           : (kv == kKvFp8 ? kTargetWavesPerCUFp8 : kTargetWavesPerCU);
    if (per_cu > target) per_cu = target;
    const int over = env_waves_per_cu();
    if (over > 0) per_cu = over;
    if (cus_out) *cus_out = cus;
    int64_t w = (int64_t)cus * per_cu;
    if (w > kMaxWaves) w = kMaxWaves;
    if (w < 1) w = 1;
    *waves = (int)w;
    return hipSuccess;
}

// KVA_XCD_MAP=0 keeps equal ranges in wave order (tests, tuning sweeps; read per call).
bool xcd_map_allowed() {
    const char *s = std::getenv("KVA_XCD_MAP");
    return !(s && s[0] == '0');
}

// Virtual granules per sequence in the work partition; KVA_PIECE_GRANULES
// overrides the default for tuning sweeps (read per call; 0 .. 64).
int piece_granules() {
    const char *s = std::getenv("KVA_PIECE_GRANULES");
    if (!s || !*s) return kPieceGranules;
    const int v = std::atoi(s);
    return v >= 0 && v <= 64 ? v : kPieceGranules;
}

// XCD range weights; KVA_XCD_WEIGHTS="even,odd" overrides them for tuning
// sweeps (read per call; each in 1..64).
void xcd_weights(int *even, int *odd) {
    *even = kXcdWeightEven;
    *odd = kXcdWeightOdd;
    const char *s = std::getenv("KVA_XCD_WEIGHTS");
    if (!s || !*s) return;
    int e = 0, o = 0;
    if (std::sscanf(s, "%d,%d", &e, &o) == 2 && e >= 1 && e <= 64 && o >= 1 && o <= 64) {
        *even = e;
        *odd = o;
    }
}

// Sequences per attention launch: batches above kMaxSeqsPerLaunch are split,
// at multiples of the sharing group in grouped calls.
int launch_slice(int seq_group) {
    const int g = seq_group > 1 ? seq_group : 1;
    return kMaxSeqsPerLaunch - kMaxSeqsPerLaunch % g;
}

// Launch the attention kernel for sequences b0 .. b0 + nb - 1 of `base`, with
// the workspace's plan (entries b0 ..) and slots.
int launch_attention(const AttnArgs &base, int layout, int group, int kv, const WsLayout &wl,
                     char *ws, hipStream_t stream, float *out, float *lse, int b0, int nb,
                     AttnArgs *used) {
    int waves = 0, cus = 0;
    if (launch_waves(layout, group, kv, nb, &waves, &cus) != hipSuccess) return KVA_ERR_HIP;
    AttnArgs a = base;
    a.B = nb;
    a.q = base.q + (int64_t)b0 * base.Hq * kHeadDim;
    a.seq_lens = base.seq_lens + b0;
    if (layout == kContig) {
        const int64_t row_bytes = (int64_t)base.Hkv * kHeadDim * (kv == kKvFp8 ? 1 : 2);
        const int64_t off = (int64_t)b0 * base.seq_stride * row_bytes;
        a.k = reinterpret_cast<const uint16_t *>(reinterpret_cast<const char *>(base.k) + off);
        a.v = reinterpret_cast<const uint16_t *>(reinterpret_cast<const char *>(base.v) + off);
    } else if (base.block_table) {
        a.block_table = base.block_table + (int64_t)b0 * base.max_pages;
    }
    if (base.pref) a.pref = base.pref + b0 / base.group;
    a.out = out + (int64_t)b0 * base.Hq * kHeadDim;
    a.lse = lse ? lse + (int64_t)b0 * base.Hq : nullptr;
    a.plan = reinterpret_cast<int2 *>(ws + wl.plan) + b0;
    a.lse_ws = reinterpret_cast<float *>(ws + wl.lse);
    a.o_ws = reinterpret_cast<float *>(ws + wl.o);
    a.waves_per_head = waves / a.Hkv > 0 ? waves / a.Hkv : 1;
    a.vgran = piece_granules();
    int blocks = 0, xcds = 0;
    if (device_xcds(&xcds) != hipSuccess) return KVA_ERR_HIP;
    // (block id mod 8 is the XCD only on the whole 8-XCD device, 256 CUs)
    a.xcd_map = (kv == kKvBf16 && cus == kXcdDeviceCUs && xcds == kXcdCount && xcd_map_allowed()) ? 1 : 0;
    if (a.xcd_map) {
        xcd_weights(&a.w_even, &a.w_odd);
        // as many blocks of each parity as (KV heads) x (ranges of that parity) need
        const int64_t per_parity = (int64_t)a.Hkv * ((a.waves_per_head + 1) / 2);
        blocks = (int)(2 * ((per_parity + kWavesPerBlock - 1) / kWavesPerBlock));
    } else {
        a.w_even = a.w_odd = 1;
        const int64_t total_waves = (int64_t)a.waves_per_head * a.Hkv;
        blocks = (int)((total_waves + kWavesPerBlock - 1) / kWavesPerBlock);
    }
    if (launch_decode_attn(a, layout, group, kv, blocks, stream) != hipSuccess) return KVA_ERR_HIP;
    *used = a;
    return KVA_OK;
}

int decode_common(const AttnArgs &base, int layout, int group, void *workspace,
                  size_t workspace_bytes, hipStream_t stream, float *out, float *lse, int D,
                  int kv = kKvBf16) {
    const WsLayout wl = ws_layout(base.B, base.Hq, base.Hkv, D);
    if (!workspace) return KVA_ERR_WORKSPACE;
    if (workspace_bytes < wl.total) return KVA_ERR_WORKSPACE;
    if (!aligned(workspace, kWsAlign)) return KVA_ERR_ALIGN;
    if (base.B == 0) return KVA_OK;

    const int slice = launch_slice(1);
    for (int b0 = 0; b0 < base.B; b0 += slice) {
        const int nb = base.B - b0 < slice ? base.B - b0 : slice;
        AttnArgs a{};
        const int st = launch_attention(base, layout, group, kv, wl, static_cast<char *>(workspace),
                                        stream, out, lse, b0, nb, &a);
        if (st != KVA_OK) return st;
        MergeArgs m{};
        m.o_ws = a.o_ws;
        m.lse_ws = a.lse_ws;
        m.plan = a.plan;
        m.out = a.out;
        m.lse = a.lse;
        m.B = nb;
        m.Hq = a.Hq;
        if (launch_merge_split(m, stream) != hipSuccess) return KVA_ERR_HIP;
    }
    return KVA_OK;
}

// Workspace of a grouped call: the plain layout, then the shared granules per
// group and the partial results of the shared-prefix pass.
struct GroupWsLayout {
    WsLayout base;
    size_t pref, lse_pre, o_pre, total;
};

GroupWsLayout group_ws_layout(int B, int Hq, int Hkv, int D, int group) {
    GroupWsLayout w;
    w.base = ws_layout(B, Hq, Hkv, D);
    const size_t ngroups = (size_t)((B + group - 1) / group);
    const size_t rows = (size_t)kMaxPrefixParts * (size_t)B * (size_t)Hq;
    w.pref = w.base.total;
    w.lse_pre = w.pref + round_up(sizeof(int32_t) * ngroups, kWsAlign);
    w.o_pre = w.lse_pre + round_up(sizeof(float) * rows, kWsAlign);
    w.total = w.o_pre + round_up(sizeof(float) * rows * (size_t)D, kWsAlign);
    return w;
}

// Argument checks and kernel arguments shared by the paged entry points.
int paged_args(const void *q, const void *k_pool, const void *v_pool, const int32_t *block_table,
               const int32_t *seq_lens, float *out, float *lse, int B, int Hq, int Hkv, int D,
               int page_size, int max_pages_per_seq, int64_t num_pages, float scale, AttnArgs *a,
               int *layout) {
    if (B < 0 || Hq <= 0 || Hkv <= 0 || D <= 0 || page_size <= 0 || max_pages_per_seq < 0 ||
        num_pages < 0)
        return KVA_ERR_SHAPE;
    if (Hq % Hkv) return KVA_ERR_SHAPE;
    const int lp = log2_exact(page_size);
    if (D != kHeadDim || !group_ok(Hq, Hkv) || lp < 0 || page_size > 1024) return KVA_ERR_UNSUPPORTED;
    if ((int64_t)max_pages_per_seq * page_size > kMaxCap) return KVA_ERR_UNSUPPORTED;
    if (num_pages > (int64_t(1) << 31)) return KVA_ERR_UNSUPPORTED;
    float scale_log2 = 0.0f;
    if (!fold_scale(scale, &scale_log2)) return KVA_ERR_UNSUPPORTED;
    // an empty pool (num_pages == 0) or table (max_pages_per_seq == 0) may be NULL
    if (B > 0 && (!q || !seq_lens || !out || (num_pages > 0 && (!k_pool || !v_pool)) ||
                  (max_pages_per_seq > 0 && !block_table)))
        return KVA_ERR_NULL;
    if (!aligned(q, 16) || !aligned(k_pool, 16) || !aligned(v_pool, 16) || !aligned(out, 16) ||
        !aligned(block_table, 4) || !aligned(seq_lens, 4) || !aligned(lse, 4))
        return KVA_ERR_ALIGN;
    *a = AttnArgs{};
    a->q = static_cast<const uint16_t *>(q);
    a->k = static_cast<const uint16_t *>(k_pool);
    a->v = static_cast<const uint16_t *>(v_pool);
    a->block_table = block_table;
    a->seq_lens = seq_lens;
    a->num_pages = num_pages;
    a->B = B;
    a->Hq = Hq;
    a->Hkv = Hkv;
    a->cap = (num_pages == 0 || !block_table) ? 0 : max_pages_per_seq * page_size;
    a->seq_stride = 0;
    a->max_pages = max_pages_per_seq;
    a->log2_page = lp;
    a->scale_log2 = scale_log2;
    a->v_scale = 1.0f;
    *layout = page_size >= kGranule ? kPagedWide : kPagedNarrow;
    return KVA_OK;
}

// Shared checks of the append entry points.
int append_common(AppendArgs &a, const void *q_in, const void *k_in, const void *v_in,
                  const float *q_norm_w, const float *k_norm_w, void *q_out, void *k_cache,
                  void *v_cache, const int32_t *seq_lens, int32_t *new_lens, int B, int Hq,
                  int Hkv, int D, float eps, double rope_theta, hipStream_t stream) {
    if (B < 0 || Hq <= 0 || Hkv <= 0 || D <= 0 || Hq % Hkv) return KVA_ERR_SHAPE;
    if (D != kHeadDim || !group_ok(Hq, Hkv)) return KVA_ERR_UNSUPPORTED;
    if (!std::isfinite(eps) || eps < 0.0f || !std::isfinite(rope_theta) || rope_theta == 1.0)
        return KVA_ERR_UNSUPPORTED;
    if (B == 0) return KVA_OK;
    if (!q_in || !k_in || !v_in || !q_out || !seq_lens) return KVA_ERR_NULL;
    if (!aligned(q_in, 16) || !aligned(k_in, 16) || !aligned(v_in, 16) || !aligned(q_out, 16) ||
        !aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(q_norm_w, 16) ||
        !aligned(k_norm_w, 16) || !aligned(seq_lens, 4) || !aligned(new_lens, 4))
        return KVA_ERR_ALIGN;
    a.q_in = static_cast<const uint16_t *>(q_in);
    a.k_in = static_cast<const uint16_t *>(k_in);
    a.v_in = static_cast<const uint16_t *>(v_in);
    a.q_w = q_norm_w;
    a.k_w = k_norm_w;
    a.q_out = static_cast<uint16_t *>(q_out);
    a.k_cache = static_cast<uint16_t *>(k_cache);
    a.v_cache = static_cast<uint16_t *>(v_cache);
    a.seq_lens = seq_lens;
    a.new_lens = new_lens;
    a.B = B;
    a.Hq = Hq;
    a.Hkv = Hkv;
    a.eps = eps;
    a.rope = rope_theta > 0.0;
    a.log2_theta = a.rope ? std::log2(rope_theta) : 0.0;
    return launch_append(a, stream) == hipSuccess ? KVA_OK : KVA_ERR_HIP;
}

}  // namespace

extern "C" {

const char *kva_status_str(int status) {
    switch (status) {
        case KVA_OK: return "ok";
        case KVA_ERR_NULL: return "a required pointer is NULL";
        case KVA_ERR_SHAPE: return "invalid shape";
        case KVA_ERR_ALIGN: return "misaligned pointer";
        case KVA_ERR_WORKSPACE: return "workspace missing or too small";
        case KVA_ERR_UNSUPPORTED: return "unsupported configuration";
        case KVA_ERR_HIP: return "HIP runtime error";
        case KVA_ERR_SCRATCH: return "batch needs more than the built-in scratch buffer";
        default: return "unknown status";
    }
}

int kva_version(void) { return 2; }

size_t kva_workspace_bytes(int B, int Hq, int Hkv, int D) {
    if (B < 0 || Hq <= 0 || Hkv <= 0 || D <= 0 || Hq % Hkv) return 0;
    return ws_layout(B, Hq, Hkv, D).total;
}

int kva_decode_attn(const void *q, const void *k, const void *v, const int32_t *seq_lens,
                    float *out, float *lse, int B, int Hq, int Hkv, int D, int Lmax, float scale,
                    void *workspace, size_t workspace_bytes, void *stream) {
    if (B < 0 || Hq <= 0 || Hkv <= 0 || D <= 0 || Lmax < 0) return KVA_ERR_SHAPE;
    if (Hq % Hkv) return KVA_ERR_SHAPE;
    if (D != kHeadDim || !group_ok(Hq, Hkv) || Lmax > kMaxCap) return KVA_ERR_UNSUPPORTED;
    float scale_log2 = 0.0f;
    if (!fold_scale(scale, &scale_log2)) return KVA_ERR_UNSUPPORTED;
    // an empty cache (Lmax == 0) may come with NULL K/V pointers
    if (B > 0 && (!q || !seq_lens || !out || (Lmax > 0 && (!k || !v)))) return KVA_ERR_NULL;
    if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 16) ||
        !aligned(seq_lens, 4) || !aligned(lse, 4))
        return KVA_ERR_ALIGN;
    AttnArgs a{};
    a.q = static_cast<const uint16_t *>(q);
    a.k = static_cast<const uint16_t *>(k);
    a.v = static_cast<const uint16_t *>(v);
    a.block_table = nullptr;
    a.seq_lens = seq_lens;
    a.num_pages = 0;
    a.B = B;
    a.Hq = Hq;
    a.Hkv = Hkv;
    a.cap = Lmax;
    a.seq_stride = Lmax;
    a.max_pages = 0;
    a.log2_page = 0;
    a.scale_log2 = scale_log2;
    a.v_scale = 1.0f;
    return decode_common(a, kContig, Hq / Hkv, workspace, workspace_bytes,
                         static_cast<hipStream_t>(stream), out, lse, D);
}

int kva_decode_attn_fp8(const void *q, const void *k, const void *v, const int32_t *seq_lens,
                        float *out, float *lse, int B, int Hq, int Hkv, int D, int Lmax,
                        float scale, float k_scale, float v_scale, void *workspace,
                        size_t workspace_bytes, void *stream) {
    if (B < 0 || Hq <= 0 || Hkv <= 0 || D <= 0 || Lmax < 0) return KVA_ERR_SHAPE;
    if (Hq % Hkv) return KVA_ERR_SHAPE;
    if (D != kHeadDim || !group_ok(Hq, Hkv) || Lmax > kMaxCap) return KVA_ERR_UNSUPPORTED;
    float scale_log2 = 0.0f;
    if (!std::isfinite(k_scale) || !std::isfinite(v_scale) ||
        !fold_scale((double)scale * (double)k_scale, &scale_log2))
        return KVA_ERR_UNSUPPORTED;
    if (B > 0 && (!q || !seq_lens || !out || (Lmax > 0 && (!k || !v)))) return KVA_ERR_NULL;
    if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 16) ||
        !aligned(seq_lens, 4) || !aligned(lse, 4))
        return KVA_ERR_ALIGN;
    AttnArgs a{};
    a.q = static_cast<const uint16_t *>(q);
    a.k = static_cast<const uint16_t *>(k);
    a.v = static_cast<const uint16_t *>(v);
    a.seq_lens = seq_lens;
    a.B = B;
    a.Hq = Hq;
    a.Hkv = Hkv;
    a.cap = Lmax;
    a.seq_stride = Lmax;
    a.scale_log2 = scale_log2;
    a.v_scale = v_scale;
    return decode_common(a, kContig, Hq / Hkv, workspace, workspace_bytes,
                         static_cast<hipStream_t>(stream), out, lse, D, kKvFp8);
}

int kva_decode_attn_paged(const void *q, const void *k_pool, const void *v_pool,
                          const int32_t *block_table, const int32_t *seq_lens, float *out,
                          float *lse, int B, int Hq, int Hkv, int D, int page_size,
                          int max_pages_per_seq, int64_t num_pages, float scale,
                          void *workspace, size_t workspace_bytes, void *stream) {
    AttnArgs a{};
    int layout = 0;
    const int st = paged_args(q, k_pool, v_pool, block_table, seq_lens, out, lse, B, Hq, Hkv, D,
                              page_size, max_pages_per_seq, num_pages, scale, &a, &layout);
    if (st != KVA_OK) return st;
    return decode_common(a, layout, Hq / Hkv, workspace, workspace_bytes,
                         static_cast<hipStream_t>(stream), out, lse, D);
}

int kva_decode_attn_paged_noalloc(const void *q, const void *k_pool, const void *v_pool,
                                  const int32_t *block_table, const int32_t *seq_lens, float *out,
                                  float *lse, int B, int Hq, int Hkv, int D, int page_size,
                                  int max_pages_per_seq, int64_t num_pages, float scale,
                                  void *stream) {
    AttnArgs a{};
    int layout = 0;
    const int st = paged_args(q, k_pool, v_pool, block_table, seq_lens, out, lse, B, Hq, Hkv, D,
                              page_size, max_pages_per_seq, num_pages, scale, &a, &layout);
    if (st != KVA_OK) return st;
    if (ws_layout(B, Hq, Hkv, D).total > kScratchBytes) return KVA_ERR_SCRATCH;
    if (B == 0) return KVA_OK;
    void *ws = nullptr;
    const int sa = scratch_address(&ws);
    if (sa != KVA_OK) return sa;
    return decode_common(a, layout, Hq / Hkv, ws, kScratchBytes, static_cast<hipStream_t>(stream),
                         out, lse, D);
}

int kva_decode_attn_paged_fp8(const void *q, const void *k_pool, const void *v_pool,
                              const int32_t *block_table, const int32_t *seq_lens, float *out,
                              float *lse, int B, int Hq, int Hkv, int D, int page_size,
                              int max_pages_per_seq, int64_t num_pages, float scale,
                              float k_scale, float v_scale, void *workspace,
                              size_t workspace_bytes, void *stream) {
    if (!std::isfinite(k_scale) || !std::isfinite(v_scale)) return KVA_ERR_UNSUPPORTED;
    AttnArgs a{};
    int layout = 0;
    const int st = paged_args(q, k_pool, v_pool, block_table, seq_lens, out, lse, B, Hq, Hkv, D,
                              page_size, max_pages_per_seq, num_pages, scale, &a, &layout);
    if (st != KVA_OK) return st;
    if (!fold_scale((double)scale * (double)k_scale, &a.scale_log2)) return KVA_ERR_UNSUPPORTED;
    a.v_scale = v_scale;
    return decode_common(a, layout, Hq / Hkv, workspace, workspace_bytes,
                         static_cast<hipStream_t>(stream), out, lse, D, kKvFp8);
}

size_t kva_workspace_bytes_grouped(int B, int Hq, int Hkv, int D, int group) {
    if (B < 0 || Hq <= 0 || Hkv <= 0 || D <= 0 || Hq % Hkv || group < 1) return 0;
    return group_ws_layout(B, Hq, Hkv, D, group).total;
}

int kva_decode_attn_paged_grouped(const void *q, const void *k_pool, const void *v_pool,
                                  const int32_t *block_table, const int32_t *seq_lens, float *out,
                                  float *lse, int B, int Hq, int Hkv, int D, int page_size,
                                  int max_pages_per_seq, int64_t num_pages, int group, float scale,
                                  void *workspace, size_t workspace_bytes, void *stream) {
    if (group < 1) return KVA_ERR_SHAPE;
    AttnArgs base{};
    int layout = 0;
    const int st = paged_args(q, k_pool, v_pool, block_table, seq_lens, out, lse, B, Hq, Hkv, D,
                              page_size, max_pages_per_seq, num_pages, scale, &base, &layout);
    if (st != KVA_OK) return st;
    const int G = Hq / Hkv;
    if ((int64_t)group * G > kMaxGroupRows) return KVA_ERR_UNSUPPORTED;
    const GroupWsLayout wl = group_ws_layout(B, Hq, Hkv, D, group);
    if (!workspace || workspace_bytes < wl.total) return KVA_ERR_WORKSPACE;
    if (!aligned(workspace, kWsAlign)) return KVA_ERR_ALIGN;
    hipStream_t s = static_cast<hipStream_t>(stream);
    // one sequence per group, or pages smaller than a granule: the plain call
    if (group == 1 || page_size < kGranule)
        return decode_common(base, layout, G, workspace, workspace_bytes, s, out, lse, D);
    if (B == 0) return KVA_OK;

    char *ws = static_cast<char *>(workspace);
    int waves = 0, cus = 0, xcds = 0;
    if (launch_waves(layout, G, kKvBf16, B < kMaxSeqsPerLaunch ? B : kMaxSeqsPerLaunch, &waves, &cus) !=
            hipSuccess ||
        device_xcds(&xcds) != hipSuccess)
        return KVA_ERR_HIP;
    const int ngroups = (B + group - 1) / group;
    // shared-prefix pass: workgroups of kPrefixWaves waves per (group, KV head),
    // as many as the attention launch has waves in all
    int64_t parts = (int64_t)waves / ((int64_t)ngroups * Hkv * kPrefixWaves);
    if (parts < 1) parts = 1;
    if (parts > kMaxPrefixParts) parts = kMaxPrefixParts;

    PrefixArgs p{};
    p.q = base.q;
    p.k = base.k;
    p.v = base.v;
    p.block_table = base.block_table;
    p.seq_lens = base.seq_lens;
    p.pref = reinterpret_cast<int32_t *>(ws + wl.pref);
    p.o_pre = reinterpret_cast<float *>(ws + wl.o_pre);
    p.lse_pre = reinterpret_cast<float *>(ws + wl.lse_pre);
    p.num_pages = base.num_pages;
    p.B = B;
    p.Hq = Hq;
    p.Hkv = Hkv;
    p.cap = base.cap;
    p.max_pages = base.max_pages;
    p.log2_page = base.log2_page;
    p.group = group;
    p.ngroups = ngroups;
    p.parts = (int)parts;
    p.w_even = p.w_odd = 1;
    // on the whole device the pass's workgroups alternate between even and odd
    // XCDs: their ranges are weighted like the bf16 attention ranges
    if (cus == kXcdDeviceCUs && xcds == kXcdCount && xcd_map_allowed()) xcd_weights(&p.w_even, &p.w_odd);
    p.scale_log2 = base.scale_log2;
    if (launch_prefix(p, s) != hipSuccess) return KVA_ERR_HIP;

    AttnArgs sfx = base;
    sfx.pref = p.pref;
    sfx.group = group;
    const int slice = launch_slice(group);
    for (int b0 = 0; b0 < B; b0 += slice) {
        const int nb = B - b0 < slice ? B - b0 : slice;
        AttnArgs a{};
        const int st2 = launch_attention(sfx, layout, G, kKvBf16, wl.base, ws, s, out, lse, b0, nb,
                                         &a);
        if (st2 != KVA_OK) return st2;

        GroupMergeArgs m{};
        m.o_pre = p.o_pre;
        m.lse_pre = p.lse_pre;
        m.o_ws = a.o_ws;
        m.lse_ws = a.lse_ws;
        m.plan = reinterpret_cast<const int2 *>(ws + wl.base.plan);
        m.out = out;
        m.lse = lse;
        m.B = B;
        m.Hq = Hq;
        m.parts = (int)parts;
        m.b_off = b0;
        m.nb = nb;
        if (launch_merge_grouped(m, s) != hipSuccess) return KVA_ERR_HIP;
    }
    return KVA_OK;
}

int kva_append(const void *q_in, const void *k_in, const void *v_in, const float *q_norm_w,
               const float *k_norm_w, void *q_out, void *k_cache, void *v_cache,
               const int32_t *seq_lens, int32_t *new_lens, int B, int Hq, int Hkv, int D,
               int Lmax, float eps, double rope_theta, void *stream) {
    if (Lmax < 0) return KVA_ERR_SHAPE;
    if (Lmax > kMaxCap) return KVA_ERR_UNSUPPORTED;
    if (B > 0 && Lmax > 0 && (!k_cache || !v_cache)) return KVA_ERR_NULL;
    AppendArgs a{};
    a.paged = 0;
    a.block_table = nullptr;
    a.cap = Lmax;
    a.num_pages = 0;
    a.max_pages = 0;
    a.log2_page = 0;
    return append_common(a, q_in, k_in, v_in, q_norm_w, k_norm_w, q_out, k_cache, v_cache,
                         seq_lens, new_lens, B, Hq, Hkv, D, eps, rope_theta,
                         static_cast<hipStream_t>(stream));
}

int kva_append_paged(const void *q_in, const void *k_in, const void *v_in,
                     const float *q_norm_w, const float *k_norm_w, void *q_out, void *k_pool,
                     void *v_pool, const int32_t *block_table, const int32_t *seq_lens,
                     int32_t *new_lens, int B, int Hq, int Hkv, int D, int page_size,
                     int max_pages_per_seq, int64_t num_pages, float eps, double rope_theta,
                     void *stream) {
    if (page_size <= 0 || max_pages_per_seq < 0 || num_pages < 0) return KVA_ERR_SHAPE;
    const int lp = log2_exact(page_size);
    if (lp < 0 || page_size > 1024) return KVA_ERR_UNSUPPORTED;
    if ((int64_t)max_pages_per_seq * page_size > kMaxCap) return KVA_ERR_UNSUPPORTED;
    if (num_pages > (int64_t(1) << 31)) return KVA_ERR_UNSUPPORTED;
    if (B > 0 && ((num_pages > 0 && (!k_pool || !v_pool)) ||
                  (max_pages_per_seq > 0 && !block_table)))
        return KVA_ERR_NULL;
    if (!aligned(block_table, 4)) return KVA_ERR_ALIGN;
    AppendArgs a{};
    a.paged = 1;
    a.block_table = block_table;
    // no pool or no table: no room, every length clamps to 0 and nothing is written
    a.cap = (num_pages == 0 || !block_table) ? 0 : max_pages_per_seq * page_size;
    a.num_pages = num_pages;
    a.max_pages = max_pages_per_seq;
    a.log2_page = lp;
    return append_common(a, q_in, k_in, v_in, q_norm_w, k_norm_w, q_out, k_pool, v_pool,
                         seq_lens, new_lens, B, Hq, Hkv, D, eps, rope_theta,
                         static_cast<hipStream_t>(stream));
}

int kva_prefill_paged(const void *q, const void *k_pool, const void *v_pool,
                      const int32_t *block_table, const int32_t *q_start, const int32_t *seq_lens,
                      float *out, float *lse, int B, int T, int max_q_len, int Hq, int Hkv, int D,
                      int page_size, int max_pages_per_seq, int64_t num_pages, float scale,
                      void *stream) {
    if (B < 0 || T < 0 || max_q_len < 0 || Hq <= 0 || Hkv <= 0 || D <= 0 || page_size <= 0 ||
        max_pages_per_seq < 0 || num_pages < 0 || Hq % Hkv)
        return KVA_ERR_SHAPE;
    const int lp = log2_exact(page_size);
    if (D != kHeadDim || !group_ok(Hq, Hkv) || lp < 0 || page_size > 1024) return KVA_ERR_UNSUPPORTED;
    if ((int64_t)max_pages_per_seq * page_size > kMaxCap) return KVA_ERR_UNSUPPORTED;
    float scale_log2 = 0.0f;
    if (num_pages > (int64_t(1) << 31) || !fold_scale(scale, &scale_log2)) return KVA_ERR_UNSUPPORTED;
    const int G = Hq / Hkv;
    const int tpt = prefill_tokens_per_tile(G);
    const int64_t tiles = ((int64_t)max_q_len + tpt - 1) / tpt;
    if (tiles * ((int64_t)B * Hkv + kMaxXcds) > (int64_t(1) << 31) - 1) return KVA_ERR_UNSUPPORTED;
    if (B == 0 || T == 0 || max_q_len == 0) return KVA_OK;
    if (!q || !q_start || !seq_lens || !out || (num_pages > 0 && (!k_pool || !v_pool)) ||
        (max_pages_per_seq > 0 && !block_table))
        return KVA_ERR_NULL;
    if (!aligned(q, 16) || !aligned(k_pool, 16) || !aligned(v_pool, 16) || !aligned(out, 16) ||
        !aligned(block_table, 4) || !aligned(q_start, 4) || !aligned(seq_lens, 4) ||
        !aligned(lse, 4))
        return KVA_ERR_ALIGN;
    PrefillArgs a{};
    a.q = static_cast<const uint16_t *>(q);
    a.k = static_cast<const uint16_t *>(k_pool);
    a.v = static_cast<const uint16_t *>(v_pool);
    a.block_table = block_table;
    a.q_start = q_start;
    a.seq_lens = seq_lens;
    a.out = out;
    a.lse = lse;
    a.num_pages = num_pages;
    a.B = B;
    a.T = T;
    a.Hq = Hq;
    a.Hkv = Hkv;
    a.cap = (num_pages == 0 || !block_table) ? 0 : max_pages_per_seq * page_size;
    a.max_pages = max_pages_per_seq;
    a.log2_page = lp;
    a.tiles = (int)tiles;
    int xcds = 0;
    if (device_xcds(&xcds) != hipSuccess) return KVA_ERR_HIP;
    a.xcds = (xcds >= 1 && xcds <= kMaxXcds) ? xcds : 1;
    a.scale_log2 = scale_log2;
    return launch_prefill(a, static_cast<hipStream_t>(stream)) == hipSuccess ? KVA_OK : KVA_ERR_HIP;
}

int kva_combine(const float *o_parts, const float *lse_parts, float *out, float *lse, int S,
                int B, int Hq, int D, void *stream) {
    if (S < 0 || B < 0 || Hq <= 0 || D <= 0) return KVA_ERR_SHAPE;
    if (D % 2 || D > 256) return KVA_ERR_UNSUPPORTED;
    if (B == 0) return KVA_OK;
    if (!out || (S > 0 && (!o_parts || !lse_parts))) return KVA_ERR_NULL;
    if (!aligned(o_parts, 8) || !aligned(out, 8) || !aligned(lse_parts, 4) || !aligned(lse, 4))
        return KVA_ERR_ALIGN;
    CombineArgs c{};
    c.o_parts = o_parts;
    c.lse_parts = lse_parts;
    c.out = out;
    c.lse = lse;
    c.S = S;
    c.B = B;
    c.Hq = Hq;
    c.D = D;
    return launch_combine(c, static_cast<hipStream_t>(stream)) == hipSuccess ? KVA_OK : KVA_ERR_HIP;
}

int kva_debug_gather_paged(const void *pool, const int32_t *block_table,
                           const int32_t *seq_lens, void *dst, int B, int Hkv, int D,
                           int page_size, int max_pages_per_seq, int64_t num_pages, int Lcap,
                           void *stream) {
    if (B < 0 || Hkv <= 0 || D <= 0 || page_size <= 0 || max_pages_per_seq < 0 ||
        num_pages < 0 || Lcap < 0)
        return KVA_ERR_SHAPE;
    const int lp = log2_exact(page_size);
    if (D != kHeadDim || lp < 0 || page_size > 1024) return KVA_ERR_UNSUPPORTED;
    if ((int64_t)max_pages_per_seq * page_size > kMaxCap) return KVA_ERR_UNSUPPORTED;
    if (num_pages > (int64_t(1) << 31)) return KVA_ERR_UNSUPPORTED;
    if (B == 0 || Lcap == 0) return KVA_OK;
    if (!pool || !block_table || !seq_lens || !dst) return KVA_ERR_NULL;
    if (!aligned(pool, 16) || !aligned(dst, 16) || !aligned(block_table, 4) ||
        !aligned(seq_lens, 4))
        return KVA_ERR_ALIGN;
    GatherArgs g{};
    g.pool = static_cast<const uint16_t *>(pool);
    g.block_table = block_table;
    g.seq_lens = seq_lens;
    g.dst = static_cast<uint16_t *>(dst);
    g.num_pages = num_pages;
    g.B = B;
    g.Hkv = Hkv;
    g.D = D;
    g.max_pages = (num_pages == 0) ? 0 : max_pages_per_seq;
    g.log2_page = lp;
    g.Lcap = Lcap;
    return launch_gather(g, static_cast<hipStream_t>(stream)) == hipSuccess ? KVA_OK : KVA_ERR_HIP;
}

int kva_debug_stream_read(const void *src, size_t bytes, uint32_t *sink, int sink_words,
                          void *stream) {
    if (bytes % 16 != 0 || sink_words < 0) return KVA_ERR_SHAPE;
    if (bytes == 0) return KVA_OK;
    if (!src || !sink || sink_words == 0) return KVA_ERR_NULL;
    if (!aligned(src, 16) || !aligned(sink, 4)) return KVA_ERR_ALIGN;
    const int blocks = sink_words < 512 ? sink_words : 512;      // 2048 waves at most
    return launch_stream_read(src, (int64_t)bytes, sink, blocks, static_cast<hipStream_t>(stream)) ==
                   hipSuccess
               ? KVA_OK
               : KVA_ERR_HIP;
}

int kva_debug_xcd_count(int *xcds) {
    if (!xcds) return KVA_ERR_NULL;
    return device_xcds(xcds) == hipSuccess ? KVA_OK : KVA_ERR_HIP;
}

int kva_debug_xcd_ids(int32_t *out, int nblocks, void *stream) {
    if (nblocks < 0 || nblocks > kMaxXcdProbeBlocks) return KVA_ERR_SHAPE;
    if (nblocks == 0) return KVA_OK;
    if (!out) return KVA_ERR_NULL;
    if (!aligned(out, 4)) return KVA_ERR_ALIGN;
    return launch_xcd_ids(out, nblocks, static_cast<hipStream_t>(stream)) == hipSuccess ? KVA_OK
                                                                                       : KVA_ERR_HIP;
}

}  // extern "C"
