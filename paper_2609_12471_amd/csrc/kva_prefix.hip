// Shared-prefix (group) decode on gfx950: the pass over a group's shared
// prompt pages, and the merge of a grouped call.
//
// The samples of one prompt are consecutive sequences of the batch; their
// block-table rows start with the same page ids for the prompt's pages.  The
// prefix pass reads those pages once per KV head and attends them for every
// query head of every member of the group (group * Hq/Hkv rows, at most 32),
// which turns the step into a small dense contraction: per block of 32 cached
// tokens of KV head g,
//
//     S^T = K Q^T   (32 tokens x 32 rows, contraction over the 128 dims)
//     O^T += V^T P^T (128 dims x 32 rows, contraction over the 32 tokens)
//
// on the 32x32x16 bf16 matrix cores, with the online softmax of each row in
// fp32 between the two products.  P is handed to the second product as the
// sum of two bf16 numbers (high part and rounded remainder), which keeps its
// relative error near 2^-16 instead of bf16's 2^-8.
//
// Operand layout of v_mfma_f32_32x32x16_bf16 (lane l, h = l / 32): the A
// operand register holds A[l % 32][8h .. 8h+7], the B register B[8h .. 8h+7][l % 32],
// and output register r holds D[8(r/4) + 4h + r%4][l % 32].  The contraction
// index may be mapped to dims (first product) or tokens (second product) in any
// order, as long as both operands use the same map:
//   * first product: K-step kk, lane half h covers dims 64h + 8kk .. +7, so a
//     lane's K (A operand) and q (B operand) registers are 128 contiguous bytes
//     of one row;
//   * second product: the lane holds row l % 32's weights for tokens
//     8(r/4) + 4h + r%4 (the first product's output); K-step s2 uses its
//     registers 8s2 .. 8s2+7 as the B operand, which fixes the token order of
//     the V^T operand.
// K and V go from HBM straight into LDS (direct-to-LDS 16-byte loads, one
// instruction covering four whole 256-byte rows), row-major with swizzled
// 16-byte chunks (K) and 64-byte segments (V): each lane reads its K operand
// row directly and its V^T operands through transposing reads (read_tr16).
//
// Work split: one workgroup of four waves per (group, KV head, part); the
// parts' ranges of the shared run are weighted by the parity of their XCD,
// the four waves take consecutive runs of a part's blocks and merge their
// results through LDS, and each part writes one partial result per
// (sequence, query head) for the merge of the grouped call.

#include "kva_internal.h"
#include "kva_device.h"

namespace kva {
namespace {

using namespace dev;


constexpr int kBlockTokens = 32;         // tokens per matrix-core block
constexpr float kMaxSlack = 8.0f;        // log2 headroom before the running maximum moves

__device__ __forceinline__ int wave_min_i32(int x) {
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) x = min(x, __shfl_xor(x, d, 64));
    return x;
}


constexpr int kScanPages = 3;            // table pages per lane compared in the first round trip
constexpr int kScanMembers = 8;          // members compared per round trip
static_assert(kScanPages == 3, "page_of_gran selects among three registers");

// Shared granules of group j: leading pages whose (sanitised) ids agree in
// every member, capped by the shortest member, in whole granules.  The
// members' lengths and their table entries for the first 64 * kScanPages
// pages are loaded together (one round trip for groups of up to
// kScanMembers); member 0's entries are returned in id0 (page 64 k + lane in
// id0[k]) for the block loads.  Longer runs continue page window by window.
__device__ int shared_granules(const PrefixArgs &a, int j, int lane, int32_t (&id0)[kScanPages]) {
    const int b0 = j * a.group;
    const int members = min(a.group, a.B - b0);
    const int L = lane < members ? clamp_len(a.seq_lens[b0 + lane], a.cap) : 0x7fffffff;
    const int32_t *bt0 = a.block_table + (int64_t)b0 * a.max_pages;
    bool diff[kScanPages];
#pragma unroll
    for (int k = 0; k < kScanPages; ++k) {
        id0[k] = 0;
        diff[k] = false;
    }
    if (a.max_pages > 0) {
        // every load in flight at once: indexes clamped into the table (entries
        // past a member's pages are read, never used), results selected after
        int pc[kScanPages];
#pragma unroll
        for (int k = 0; k < kScanPages; ++k) {
            pc[k] = min(64 * k + lane, a.max_pages - 1);
            id0[k] = sanitize_page(bt0[pc[k]], a.num_pages);
        }
        for (int m0 = 1; m0 < members; m0 += kScanMembers) {
            int32_t idm[kScanMembers][kScanPages];
#pragma unroll
            for (int i = 0; i < kScanMembers; ++i) {
                const int64_t row = (int64_t)min(m0 + i, members - 1) * a.max_pages;
#pragma unroll
                for (int k = 0; k < kScanPages; ++k) idm[i][k] = bt0[row + pc[k]];
            }
#pragma unroll
            for (int i = 0; i < kScanMembers; ++i)
#pragma unroll
                for (int k = 0; k < kScanPages; ++k)
                    diff[k] |= sanitize_page(idm[i][k], a.num_pages) != id0[k];
        }
    }
    const int Lmin = uniform_i32(wave_min_i32(L));
    const int npg = (int)(((int64_t)Lmin + (1 << a.log2_page) - 1) >> a.log2_page);
    int shared = npg;
    bool found = false;
#pragma unroll
    for (int k = 0; k < kScanPages; ++k) {
        const uint64_t dm = __ballot(!found && diff[k] && 64 * k + lane < npg);
        if (dm && !found) {
            shared = 64 * k + (int)__builtin_ctzll(dm);
            found = true;
        }
    }
    for (int p0 = 64 * kScanPages; !found && p0 < npg; p0 += 64) {
        const int p = p0 + lane;
        bool diff = false;
        if (p < npg) {
            const int32_t first = sanitize_page(bt0[p], a.num_pages);
            for (int m = 1; m < members; ++m)
                diff |= sanitize_page(bt0[(int64_t)m * a.max_pages + p], a.num_pages) != first;
        }
        const uint64_t dm = __ballot(diff);
        if (dm) {
            shared = p0 + (int)__builtin_ctzll(dm);
            found = true;
        }
    }
    const int64_t T = min((int64_t)shared << a.log2_page, (int64_t)Lmin);
    return (int)(T / kGranule);
}

// Block slots in LDS (per wave): 32 K rows of 256 bytes, 16-byte chunk c of row
// r at chunk c ^ px_kswz(r) (the 16 rows a 16-lane phase of a score-operand
// read covers fall on 16 distinct chunks); 32 V rows of 256 bytes, 64-byte
// segment s of row r at segment s ^ px_vswz(r) (for the transposing reads).
constexpr int kSlotBytes = kBlockTokens * kHeadDim * 2;
constexpr int kDmaPolicy = 2;            // non-temporal, as the decode kernels' K/V loads
__device__ __forceinline__ int px_kswz(int r) { return ((r & 1) << 3) | ((r >> 1) & 7); }
__device__ __forceinline__ int px_vswz(int r) { return ((r & 1) << 1) | ((r >> 1) & 1); }

typedef __attribute__((address_space(3))) void lds_void_t;

// Direct-to-LDS loads of one 32-token block starting at token t0 (granules
// t0/16 and t0/16 + 1 live in pages pg0 and pg1) into a slot: instruction u
// fills rows 4u .. 4u + 3, lane l the 16-byte chunk at row 4u + l/16, chunk
// l % 16, with the cache chunk the swizzle puts there; tokens at or past `tend`
// read the last live row instead (finite data, weight 0).
__device__ __forceinline__ void dma_block(const PrefixArgs &a, int32_t pg0, int32_t pg1, int t0,
                                          int tend, int g, int lane, unsigned char *ks,
                                          unsigned char *vs) {
    const int rr = lane >> 4;
    const int p = lane & 15;
    const int pmask = (1 << a.log2_page) - 1;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        const int r = 4 * u + rr;
        const int t = min(t0 + r, tend - 1);
        // the clamped token lies in granule 1 only if granule 1 holds live tokens
        const int32_t pg = (u < 4 || t < t0 + kGranule) ? pg0 : pg1;
        const int64_t row = ((int64_t)pg << a.log2_page) + (t & pmask);
        const int64_t base = (row * a.Hkv + g) * kHeadDim;
        const int kc = p ^ px_kswz(r);
        const int vc = (((p >> 2) ^ px_vswz(r)) << 2) | (p & 3);
        __builtin_amdgcn_global_load_lds((const void *)(a.k + base + 8 * kc), (lds_void_t *)(ks + 1024 * u),
                                         16, 0, kDmaPolicy);
        __builtin_amdgcn_global_load_lds((const void *)(a.v + base + 8 * vc), (lds_void_t *)(vs + 1024 * u),
                                         16, 0, kDmaPolicy);
    }
}

__global__ __launch_bounds__(kPrefixWaves * 64) void prefix_attn_kernel(const PrefixArgs a) {
    // per wave, two block slots (K and V each); after the blocks the same
    // memory holds the wave's partial result for the workgroup's merge
    __shared__ __align__(16) unsigned char s_buf[kPrefixWaves][4 * kSlotBytes];
    const int lane = threadIdx.x & 63;
    const int wid = threadIdx.x >> 6;
    // workgroup: part `part` of (group j, KV head g); its waves split the
    // part's blocks in four consecutive runs and merge their results at the end
    const int pair = (int)(blockIdx.x / (unsigned)a.parts);
    const int part = (int)(blockIdx.x % (unsigned)a.parts);
    if (pair >= a.ngroups * a.Hkv) return;   // (uniform over the workgroup)
    const int g = pair % a.Hkv;
    const int j = pair / a.Hkv;

    int32_t id0[kScanPages];
    const int n = uniform_i32(shared_granules(a, j, lane, id0));
    if (g == 0 && part == 0 && wid == 0 && lane == 0) a.pref[j] = n;
    // the parts' block ranges, in proportion to the weight of their XCD parity
    // (workgroup blockIdx runs on XCD blockIdx mod 8); then four runs per part
    const int64_t nb = (n + 1) / 2;                      // 32-token blocks
    const int first = (int)blockIdx.x - part;            // block of part 0
    int64_t w_lo = 0, w_all = 0;
    for (int t = 0; t < a.parts; ++t) {
        const int64_t w = ((first + t) & 1) ? a.w_odd : a.w_even;
        if (t < part) w_lo += w;
        w_all += w;
    }
    const int64_t w_me = (((int)blockIdx.x) & 1) ? a.w_odd : a.w_even;
    const int64_t x0 = nb * w_lo / w_all, x1 = nb * (w_lo + w_me) / w_all;
    const int64_t y0 = x0 + (x1 - x0) * wid / kPrefixWaves;
    const int64_t y1 = x0 + (x1 - x0) * (wid + 1) / kPrefixWaves;
    const int gb = (int)(2 * y0);
    const int ge = (int)min(2 * y1, (int64_t)n);

    const int G = a.Hq / a.Hkv;
    const int b0 = j * a.group;
    const int rows = min(a.group, a.B - b0) * G;
    const int rho = lane & 31;   // query row held by this lane
    const int hh = lane >> 5;    // lane half
    const bool row_ok = rho < rows;
    const int bq = b0 + (row_ok ? rho / G : 0);
    const int hq = g * G + rho % G;

    f32x16_t acc[4];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[mt][r] = 0.0f;
    float m = -INFINITY;
    float l = 0.0f;                 // this lane's half of the row's weight sum

    if (gb < ge) {
    const int tbeg = gb * kGranule;
    const int tend = ge * kGranule;
    const int nblk = (tend - tbeg + kBlockTokens - 1) / kBlockTokens;
    const int32_t *bt = a.block_table + (int64_t)b0 * a.max_pages;
    // page of granule gi (clamped to the last live granule): from the scan's
    // registers when it lies in the scanned pages (the index is wave-uniform)
    auto page_of_gran = [&](int gi) -> int32_t {
        const int pi = uniform_i32((min(gi, ge - 1) * kGranule) >> a.log2_page);
        if (pi < 64 * kScanPages) {
            const int32_t v = (pi >> 6) == 0 ? id0[0] : (pi >> 6) == 1 ? id0[1] : id0[2];
            return __shfl(v, pi & 63, 64);
        }
        return sanitize_page(bt[pi], a.num_pages);
    };
    const int gbl = tbeg / kGranule;   // first granule of the item
    unsigned char *k0 = s_buf[wid], *v0 = k0 + kSlotBytes, *k1 = k0 + 2 * kSlotBytes,
                  *v1 = k0 + 3 * kSlotBytes;
    auto issue = [&](int blk, unsigned char *ks, unsigned char *vs) {
        dma_block(a, page_of_gran(gbl + 2 * blk), page_of_gran(gbl + 2 * blk + 1),
                  tbeg + blk * kBlockTokens, tend, g, lane, ks, vs);
    };
    // block 0 first, then q
    issue(0, k0, v0);

    // q rows (B operand of the first product): bytes 128h .. 128h+127 of row rho
    uint4 qf[8];
    {
        const uint4 *qp = (const uint4 *)(a.q + ((int64_t)bq * a.Hq + hq) * kHeadDim + 64 * hh);
#pragma unroll
        for (int kk = 0; kk < 8; ++kk) qf[kk] = row_ok ? qp[kk] : make_uint4(0u, 0u, 0u, 0u);
    }

    const float sl = a.scale_log2;
    // this lane's offsets: score-operand row rho, and V^T read sources
    const int kswz = px_kswz(rho);
    const int vrow = 4 * hh + ((lane & 15) >> 2);
    const int vcol = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
    const int vgr = px_vswz(vrow);

    // One 32-token block from its slot: scores, online softmax, V^T P^T.  All
    // the block's operands are read from LDS first (the compiler waits for
    // every outstanding direct-to-LDS load before them), then the next
    // block's loads are issued into the other slot, so they are in flight
    // during this block's arithmetic.
    auto consume = [&](int blk) {
        const unsigned char *ks = (blk & 1) ? k1 : k0;
        const unsigned char *vs = (blk & 1) ? v1 : v0;
        const int t0 = tbeg + blk * kBlockTokens;
        // scores: lane holds row rho, tokens t0 + 8(r/4) + 4h + r%4; the A
        // operand of K-step kk is dims 64h + 8kk .. +7 of K row rho
        uint4 ka[8];
#pragma unroll
        for (int kk = 0; kk < 8; ++kk) ka[kk] = *(const uint4 *)(ks + rho * 256 + 16 * ((8 * hh + kk) ^ kswz));
        // V^T operands (dim 32 mt + rho over tokens 16 s2 + 4h + 0..3 and
        // 16 s2 + 8 + 4h + 0..3, the B operand's token order), read now so that
        // their latency passes during the softmax
        uint4 va[4][2];
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
            for (int s2 = 0; s2 < 2; ++s2) {
                const uint16_t *src = (const uint16_t *)(vs + (16 * s2 + vrow) * 256) + 32 * (mt ^ vgr) + vcol;
                const uint2 lo4 = read_tr16(src);
                const uint2 hi4 = read_tr16(src + 8 * kHeadDim);
                va[mt][s2] = make_uint4(lo4.x, lo4.y, hi4.x, hi4.y);
            }
        if (blk + 1 < nblk) {
            // (the other slot was last read by the previous block, whose
            // operands were all in registers before its products)
            if (blk & 1) issue(blk + 1, k0, v0);
            else issue(blk + 1, k1, v1);
        }
        f32x16_t st0, st1;
#pragma unroll
        for (int r = 0; r < 16; ++r) { st0[r] = 0.0f; st1[r] = 0.0f; }
#pragma unroll
        for (int kk = 0; kk < 8; kk += 2) {
            st0 = mfma32(ka[kk], qf[kk], st0);
            st1 = mfma32(ka[kk + 1], qf[kk + 1], st1);
        }
        float p[16];
        float mx = -INFINITY;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int t = t0 + 8 * (r >> 2) + 4 * hh + (r & 3);
            p[r] = t < tend ? (st0[r] + st1[r]) * sl : -INFINITY;
            mx = fmaxf(mx, p[r]);
        }
        mx = pair_max(mx);
        // the running maximum moves (and the accumulators are rescaled) only
        // when some row's block maximum exceeds it by more than kMaxSlack: the
        // weights then stay below 2^kMaxSlack, and rescales are rare
        if (__ballot(mx > m + kMaxSlack)) {
            const float mn = fmaxf(m, mx);
            const float alpha = (mn == m) ? 1.0f : fast_exp2(m - mn);
            l *= alpha;
            m = mn;
#pragma unroll
            for (int mt = 0; mt < 4; ++mt)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[mt][r] *= alpha;
        }
        const float ms = (m == -INFINITY) ? 0.0f : m;
        float ps = 0.0f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            p[r] = fast_exp2(p[r] - ms);
            ps += p[r];
        }
        l += ps;
        // P^T operands, high and low bf16 parts: registers 8s2 .. 8s2+7
        uint4 phi[2], plo[2];
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
            uint32_t hw[4], lw[4];
#pragma unroll
            for (int e = 0; e < 4; ++e)
                split_bf16_pair(p[8 * s2 + 2 * e], p[8 * s2 + 2 * e + 1], hw[e], lw[e]);
            phi[s2] = make_uint4(hw[0], hw[1], hw[2], hw[3]);
            plo[s2] = make_uint4(lw[0], lw[1], lw[2], lw[3]);
        }
        // O^T += V^T P^T: tile mt covers dims 32mt .. 32mt+31
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) {
                acc[mt] = mfma32(va[mt][s2], phi[s2], acc[mt]);
                acc[mt] = mfma32(va[mt][s2], plo[s2], acc[mt]);
            }
    };

    for (int blk = 0; blk < nblk; ++blk) consume(blk);
    }

    // Merge of the workgroup's four results: each wave parks its accumulators
    // (lane-major in 16-byte chunks) and its rows' maximum and weight sum in
    // its own LDS region, then wave w combines dims 32w .. 32w+31 of every row.
    l = pair_sum(l);
    __syncthreads();                                     // every slot read
    float *mine = reinterpret_cast<float *>(s_buf[wid]);
    constexpr int kMl = 64 * 64;                          // floats of parked accumulators
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4)
            *(float4 *)(mine + ((4 * mt + r4) * 64 + lane) * 4) =
                make_float4(acc[mt][4 * r4], acc[mt][4 * r4 + 1], acc[mt][4 * r4 + 2], acc[mt][4 * r4 + 3]);
    if (hh == 0) {
        mine[kMl + rho] = m;
        mine[kMl + 32 + rho] = l;
    }
    __syncthreads();
    float mv[kPrefixWaves], lv[kPrefixWaves];
    float M = -INFINITY;
#pragma unroll
    for (int v = 0; v < kPrefixWaves; ++v) {
        const float *src = reinterpret_cast<const float *>(s_buf[v]);
        mv[v] = src[kMl + rho];
        lv[v] = src[kMl + 32 + rho];
        M = fmaxf(M, mv[v]);
    }
    float o[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) o[r] = 0.0f;
    float L = 0.0f;
#pragma unroll
    for (int v = 0; v < kPrefixWaves; ++v) {
        // a wave without tokens (m = -inf) has weight 0 and zero accumulators
        const float sc = mv[v] == -INFINITY ? 0.0f : fast_exp2(mv[v] - M);
        L = fmaf(sc, lv[v], L);
        const float *src = reinterpret_cast<const float *>(s_buf[v]);
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
            const float4 x = *(const float4 *)(src + ((4 * wid + r4) * 64 + lane) * 4);
            o[4 * r4] = fmaf(sc, x.x, o[4 * r4]);
            o[4 * r4 + 1] = fmaf(sc, x.y, o[4 * r4 + 1]);
            o[4 * r4 + 2] = fmaf(sc, x.z, o[4 * r4 + 2]);
            o[4 * r4 + 3] = fmaf(sc, x.w, o[4 * r4 + 3]);
        }
    }
    // partial result `part` of rows rho (every part writes one, empty or not):
    // lane holds dims 32 wid + 8(r/4) + 4h + r%4
    if (row_ok) {
        const int64_t prow = ((int64_t)part * a.B + bq) * a.Hq + hq;
        const float inv = L > 0.0f ? 1.0f / L : 0.0f;
        float *dst = a.o_pre + prow * kHeadDim + 32 * wid;
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4)
            *(float4 *)(dst + 8 * r4 + 4 * hh) =
                make_float4(o[4 * r4] * inv, o[4 * r4 + 1] * inv, o[4 * r4 + 2] * inv, o[4 * r4 + 3] * inv);
        if (wid == 0 && hh == 0) a.lse_pre[prow] = L > 0.0f ? (M + fast_log2(L)) * kLn2 : -INFINITY;
    }
}

// ---- merge of a grouped call: one wave per (sequence, query head); parts are
// the shared-prefix parts (every part writes one, lse = -inf if empty), then
// the sequence's own pieces

__global__ __launch_bounds__(256) void merge_grouped_kernel(const GroupMergeArgs a) {
    const int lane = threadIdx.x & 63;
    const int64_t wl = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (wl >= (int64_t)a.nb * a.Hq) return;
    const int b = a.b_off + (int)(wl / a.Hq);
    const int h = (int)(wl % a.Hq);
    const int64_t bh = (int64_t)b * a.Hq + h;
    const int2 pl = a.plan[b];
    // every part of the shared-prefix pass wrote a result (lse = -inf if empty)
    const PartList pre{a.o_pre + bh * kHeadDim, (int64_t)a.B * a.Hq * kHeadDim, a.lse_pre + bh,
                       (int64_t)a.B * a.Hq, a.parts};
    const PartList own{a.o_ws + ((int64_t)pl.x * a.Hq + h) * kHeadDim, (int64_t)a.Hq * kHeadDim,
                       a.lse_ws + (int64_t)pl.x * a.Hq + h, a.Hq, pl.y};
    merge_lists(pre, own, kHeadDim, a.out + bh * kHeadDim, a.lse ? a.lse + bh : nullptr, lane);
}

}  // namespace

hipError_t launch_prefix(const PrefixArgs &a, hipStream_t stream) {
    const int64_t blocks = (int64_t)a.ngroups * a.Hkv * a.parts;
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL(prefix_attn_kernel, dim3((unsigned)blocks), dim3(kPrefixWaves * 64), 0,
                       stream, a);
    return hipGetLastError();
}

hipError_t launch_merge_grouped(const GroupMergeArgs &a, hipStream_t stream) {
    const int64_t waves = (int64_t)a.nb * a.Hq;
    if (waves == 0) return hipSuccess;
    const int64_t blocks = (waves + 3) / 4;
    hipLaunchKernelGGL(merge_grouped_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, a);
    return hipGetLastError();
}

}  // namespace kva
