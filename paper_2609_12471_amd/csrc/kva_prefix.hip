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
// K and V are read from HBM as in the decode kernel (one 16-byte load per
// lane covers four whole 256-byte rows) and staged in LDS row-major with
// padded rows: each lane reads its K operand row directly and its V^T
// operands through transposing reads (read_tr16).

#include "kva_internal.h"
#include "kva_device.h"

namespace kva {
namespace {

using namespace dev;


constexpr int kBlockTokens = 32;         // tokens per matrix-core block
constexpr float kMaxSlack = 8.0f;        // log2 headroom before the running maximum moves
constexpr int kPrefixWaves = 4;          // waves per workgroup (independent items)

// Granules per split of a shared run of n granules: an even count (whole
// 32-token blocks).  Splits s < ceil(n / chunk) are the non-empty ones.
__device__ __forceinline__ int prefix_chunk(int n, int splits) {
    return ((n + splits - 1) / splits + 1) & ~1;
}

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

// Issue the loads of one 32-token block starting at token t0 (granules t0/16
// and t0/16 + 1 live in pages pg0 and pg1).  Load u of lane (r, c) = (lane / 16,
// lane % 16) reads 16 bytes (dims 8c .. 8c+7) of token t0 + 4u + r of head g;
// tokens at or past `tend` read the last live row instead.
__device__ __forceinline__ void load_block(const PrefixArgs &a, int32_t pg0, int32_t pg1, int t0,
                                           int tend, int g, int lane, uint4 (&kd)[8],
                                           uint4 (&vd)[8]) {
    const int r = lane >> 4;
    const int c = lane & 15;
    const int pmask = (1 << a.log2_page) - 1;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        const int t = min(t0 + 4 * u + r, tend - 1);
        // the clamped token lies in granule 1 only if granule 1 holds live tokens
        const int32_t pg = (u < 4 || t < t0 + kGranule) ? pg0 : pg1;
        const int64_t row = ((int64_t)pg << a.log2_page) + (t & pmask);
        const int64_t off = (row * a.Hkv + g) * kHeadDim + 8 * c;
        kd[u] = as_uint4(__builtin_nontemporal_load((const u32x4_t *)(a.k + off)));
        vd[u] = as_uint4(__builtin_nontemporal_load((const u32x4_t *)(a.v + off)));
    }
}

__global__ __launch_bounds__(kPrefixWaves * 64) void prefix_attn_kernel(const PrefixArgs a) {
    // per wave, a ring of two staged blocks (K rows, V rows)
    __shared__ uint32_t s_ks[kPrefixWaves][2][32 * kKsStride];
    __shared__ uint16_t s_vs[kPrefixWaves][2][32 * kVsStride];
    const int lane = threadIdx.x & 63;
    const int wid = threadIdx.x >> 6;
    const int wave = uniform_i32(blockIdx.x * kPrefixWaves + wid);
    if (wave >= a.ngroups * a.splits * a.Hkv) return;
    // consecutive waves: the KV heads of one token range
    const int g = wave % a.Hkv;
    const int s = (wave / a.Hkv) % a.splits;
    const int j = wave / (a.Hkv * a.splits);

    const int vsrc = vs_source(lane);


    int32_t id0[kScanPages];
    const int n = uniform_i32(shared_granules(a, j, lane, id0));
    if (g == 0 && s == 0 && lane == 0) a.pref[j] = n;
    const int chunk = prefix_chunk(n, a.splits);
    const int gb = s * chunk;
    const int ge = min(n, gb + chunk);
    if (gb >= ge) return;

    const int G = a.Hq / a.Hkv;
    const int b0 = j * a.group;
    const int rows = min(a.group, a.B - b0) * G;
    const int rho = lane & 31;   // query row held by this lane
    const int hh = lane >> 5;    // lane half
    const bool row_ok = rho < rows;
    const int bq = b0 + (row_ok ? rho / G : 0);
    const int hq = g * G + rho % G;

    // q rows (B operand of the first product): bytes 128h .. 128h+127 of row rho
    uint4 qf[8];
    {
        const uint4 *qp = (const uint4 *)(a.q + ((int64_t)bq * a.Hq + hq) * kHeadDim + 64 * hh);
#pragma unroll
        for (int kk = 0; kk < 8; ++kk) qf[kk] = row_ok ? qp[kk] : make_uint4(0u, 0u, 0u, 0u);
    }

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

    f32x16_t acc[4];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[mt][r] = 0.0f;
    float m = -INFINITY;
    float l = 0.0f;                 // this lane's half of the row's weight sum
    const float sl = a.scale_log2;

    // Stage a block's K and V rows as loaded into ring slot `slot` (rows past
    // the shared run are re-reads of its last live row, finite, and get
    // weight 0).
    auto stage = [&](int slot, const uint4 (&kc)[8], const uint4 (&vc)[8]) {
        uint32_t *ks = s_ks[wid][slot];
        uint16_t *vs = s_vs[wid][slot];
        const int r = lane >> 4;
        const int c = lane & 15;
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int tl = 4 * u + r;
            *(uint4 *)(ks + tl * kKsStride + 4 * c) = kc[u];
            *(uint4 *)(vs + tl * kVsStride + 8 * c) = vc[u];
        }
        __builtin_amdgcn_wave_barrier();
    };
    // One 32-token block from ring slot blk % 2: scores, online softmax, V^T P^T.
    auto consume = [&](int blk) {
        const int t0 = tbeg + blk * kBlockTokens;
        const uint32_t *ks = s_ks[wid][blk & 1];
        const uint16_t *vs = s_vs[wid][blk & 1];
        // scores: lane holds row rho, tokens t0 + 8(r/4) + 4h + r%4; the A
        // operand of K-step kk is bytes 128h + 16kk .. +15 of K row rho
        f32x16_t st;
#pragma unroll
        for (int r = 0; r < 16; ++r) st[r] = 0.0f;
#pragma unroll
        for (int kk = 0; kk < 8; ++kk) {
            const uint4 ka = *(const uint4 *)(ks + rho * kKsStride + 32 * hh + 4 * kk);
            st = mfma32(ka, qf[kk], st);
        }
        float p[16];
        float mx = -INFINITY;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int t = t0 + 8 * (r >> 2) + 4 * hh + (r & 3);
            p[r] = t < tend ? st[r] * sl : -INFINITY;
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
            for (int e = 0; e < 4; ++e) {
                const float x0 = p[8 * s2 + 2 * e], x1 = p[8 * s2 + 2 * e + 1];
                const uint32_t h0 = __float_as_uint(x0) >> 16, h1 = __float_as_uint(x1) >> 16;
                const uint32_t l0 = bf16_rne_bits(x0 - __uint_as_float(h0 << 16));
                const uint32_t l1 = bf16_rne_bits(x1 - __uint_as_float(h1 << 16));
                hw[e] = h0 | (h1 << 16);
                lw[e] = l0 | (l1 << 16);
            }
            phi[s2] = make_uint4(hw[0], hw[1], hw[2], hw[3]);
            plo[s2] = make_uint4(lw[0], lw[1], lw[2], lw[3]);
        }
        // O^T += V^T P^T: tile mt covers dims 32mt .. 32mt+31; the A operand of
        // K-step s2 holds dim 32mt + rho at tokens 16s2 + 4h + 0..3 and
        // 16s2 + 8 + 4h + 0..3 (the B operand's token order)
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
#pragma unroll
            for (int s2 = 0; s2 < 2; ++s2) {
                const uint2 lo4 = read_tr16(vs + vsrc + 16 * s2 * kVsStride + 32 * mt);
                const uint2 hi4 = read_tr16(vs + vsrc + (16 * s2 + 8) * kVsStride + 32 * mt);
                const uint4 va = make_uint4(lo4.x, lo4.y, hi4.x, hi4.y);
                acc[mt] = mfma32(va, phi[s2], acc[mt]);
                acc[mt] = mfma32(va, plo[s2], acc[mt]);
            }
        }
    };

    // Pipeline, two blocks in flight: while block b is consumed from its LDS
    // slot, the loads of block b + 1 (issued one step earlier) and of block
    // b + 2 (issued now) are outstanding; block b + 1 is staged into the other
    // slot after the step.  Two register sets alternate (no copies of loads
    // in flight); page ids come from the scan's registers; past the last
    // block the loads repeat it.
    uint4 ka[8], va[8], kb[8], vb[8];
    const int last = nblk - 1;
    const int gbl = tbeg / kGranule;   // first granule of the item
    auto issue = [&](int blk, uint4 (&kd)[8], uint4 (&vd)[8]) {
        const int bl = min(blk, last);
        load_block(a, page_of_gran(gbl + 2 * bl), page_of_gran(gbl + 2 * bl + 1),
                   tbeg + bl * kBlockTokens, tend, g, lane, kd, vd);
    };
    issue(0, ka, va);
    issue(1, kb, vb);
    stage(0, ka, va);
    for (int blk = 0; blk < nblk; blk += 2) {
        // block blk in slot 0 and block blk + 1 in (kb, vb)
        issue(blk + 2, ka, va);
        __builtin_amdgcn_sched_barrier(0);
        consume(blk);
        if (blk + 1 >= nblk) break;
        stage(1, kb, vb);
        issue(blk + 3, kb, vb);
        __builtin_amdgcn_sched_barrier(0);
        consume(blk + 1);
        if (blk + 2 >= nblk) break;
        stage(0, ka, va);
    }

    // partial result of rows rho: lane holds dims 32mt + 8(r/4) + 4h + r%4
    l = pair_sum(l);
    if (row_ok) {
        const int64_t prow = ((int64_t)s * a.B + bq) * a.Hq + hq;
        const float inv = l > 0.0f ? 1.0f / l : 0.0f;
        float *dst = a.o_pre + prow * kHeadDim;
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4)
                *(float4 *)(dst + 32 * mt + 8 * r4 + 4 * hh) =
                    make_float4(acc[mt][4 * r4] * inv, acc[mt][4 * r4 + 1] * inv,
                                acc[mt][4 * r4 + 2] * inv, acc[mt][4 * r4 + 3] * inv);
        if (hh == 0) a.lse_pre[prow] = l > 0.0f ? (m + fast_log2(l)) * kLn2 : -INFINITY;
    }
}

// ---- merge of a grouped call: one wave per (sequence, query head); parts are
// the non-empty prefix splits, then the sequence's own pieces

__global__ __launch_bounds__(256) void merge_grouped_kernel(const GroupMergeArgs a) {
    const int lane = threadIdx.x & 63;
    const int64_t wl = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (wl >= (int64_t)a.nb * a.Hq) return;
    const int b = a.b_off + (int)(wl / a.Hq);
    const int h = (int)(wl % a.Hq);
    const int64_t w = (int64_t)b * a.Hq + h;
    const int2 pl = a.plan[b];
    const int n = a.pref[b / a.group];
    const int chunk = prefix_chunk(n, a.splits);
    const int np = n > 0 ? (n + chunk - 1) / chunk : 0;
    const int64_t bh = (int64_t)b * a.Hq + h;
    const PartList pre{a.o_pre + bh * kHeadDim, (int64_t)a.B * a.Hq * kHeadDim, a.lse_pre + bh,
                       (int64_t)a.B * a.Hq, np};
    const PartList own{a.o_ws + ((int64_t)pl.x * a.Hq + h) * kHeadDim, (int64_t)a.Hq * kHeadDim,
                       a.lse_ws + (int64_t)pl.x * a.Hq + h, a.Hq, pl.y};
    merge_lists(pre, own, kHeadDim, a.out + w * kHeadDim, a.lse ? a.lse + w : nullptr, lane);
}

}  // namespace

hipError_t launch_prefix(const PrefixArgs &a, hipStream_t stream) {
    const int64_t waves = (int64_t)a.ngroups * a.splits * a.Hkv;
    if (waves == 0) return hipSuccess;
    const int64_t blocks = (waves + kPrefixWaves - 1) / kPrefixWaves;
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
