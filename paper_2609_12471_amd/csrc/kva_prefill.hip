// Chunked prefill on gfx950: the new tokens of each sequence (a prompt, or the
// feedback appended between turns) attend their causal prefix in a paged
// cache that already holds them.
//
// One workgroup of 8 waves per (sequence, KV head g, tile of new tokens).  The
// workgroup's 256 query rows are tile tokens x the Hq/Hkv query heads of g
// (64 tokens x 4 heads for Qwen3-8B), 32 rows per wave, so every K/V block it
// reads serves all heads that share it (8 waves per workgroup measured 6 %
// faster than 4: half the block loads and LDS writes per wave).  Per block of
// 128 cached positions the workgroup loads K and V once (coalesced: eight
// lanes per 256-byte row) into LDS, row-major, double-buffered (one barrier
// per block; 64-position blocks measured 1 % slower), and for each 32
// positions each wave runs the same matrix-core step as the shared-prefix
// pass:
//
//     S^T = K Q^T (8 x v_mfma_f32_32x32x16_bf16), causal mask, fp32 online
//     softmax per row, O^T += V^T P^T (P as high + low bf16 parts, 16 MFMAs).
//
// The V^T operands come straight from the row-major V block through
// transposing LDS reads (read_tr16).
//
// The staged V rows are 256 bytes, unpadded: 64-byte segment s of row r sits
// at segment s ^ v_swz(r), so the four rows that one 32-lane phase of a
// transposing read covers land on four different segments of gfx950's
// 64-bank LDS, and the two rows of a 16-lane write phase on opposite halves
// (no bank conflicts; rows padded to 288 bytes conflicted two-way on both).
// The K rows keep a 272-byte pitch: their operand reads are conflict-free.
//
// The softmax keeps a row's running maximum until a block's scores exceed it
// by more than 8 (base 2): the weights then stay below 2^8, well inside fp32,
// and the rescale of the 64 accumulators (which live in the matrix-core
// registers) happens only when a maximum really moves.  The causal compares
// run only on blocks that reach past the wave's first position.
//
// The next block's loads are issued before the current block is consumed (a
// deeper pipeline needs more registers and halves the resident waves, which
// measured slower).  A wave skips the blocks that lie entirely after its last
// row's position (the workgroup still loads them for the waves that need them).
//
// Every tile of a (sequence, KV head) pair re-reads the pair's cached K/V from
// position 0, so the launch order keeps those tiles together: workgroups are
// dealt to the N XCDs round-robin (block id mod N; N = 8 on MI355X, from the
// runtime), and XCD x takes pairs x, x + N, ..., all tiles of a pair in a row
// (longest prefix first).  The
// tiles of a pair then run at the same time on one XCD and walk the same K/V
// blocks through its L2 nearly in step.

#include "kva_internal.h"
#include "kva_device.h"

namespace kva {
namespace {

using namespace dev;

constexpr int kPfWaves = 8;
constexpr int kPfRows = 32 * kPfWaves;     // query rows (token x head) per workgroup
constexpr int kKeyBlock = 32;              // cached positions per matrix-core step
constexpr int kSteps = 4;                  // steps per staged block (one barrier each)
constexpr int kStageKeys = kKeyBlock * kSteps;
constexpr int kPassRows = kPfWaves * 64 / 8;   // block rows one load pass covers (8 lanes per row)
static_assert(kStageKeys % kPassRows == 0, "whole load passes per staged block");
constexpr int kPasses = kStageKeys / kPassRows;
constexpr float kMaxSlack = 8.0f;          // log2 headroom before the running maximum moves
constexpr int kRowV = kHeadDim;            // staged V row: 256 bytes in bf16
__device__ __forceinline__ int v_swz(int r) { return ((r & 1) << 1) | ((r >> 1) & 1); }
__device__ __forceinline__ int clamp_i(int x, int lo, int hi) { return x < lo ? lo : (x > hi ? hi : x); }

__global__ __launch_bounds__(kPfWaves * 64, 1) void prefill_kernel(const PrefillArgs a) {
    __shared__ uint32_t s_k[2][kStageKeys * kKsStride];
    __shared__ uint16_t s_v[2][kStageKeys * kRowV];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wid = tid >> 6;
    const int G = a.Hq / a.Hkv;
    const int tok_per_tile = kPfRows / G;
    // XCD-aware order (block id mod a.xcds selects the XCD)
    const int xcd = (int)(blockIdx.x % (unsigned)a.xcds);
    const int j = (int)(blockIdx.x / (unsigned)a.xcds);
    const int pair = (j / a.tiles) * a.xcds + xcd;
    if (pair >= a.B * a.Hkv) return;
    const int tile = a.tiles - 1 - j % a.tiles;
    const int b = pair / a.Hkv;
    const int g = pair % a.Hkv;
    const int qs = clamp_i(a.q_start[b], 0, a.T);
    const int n = clamp_i(a.q_start[b + 1], qs, a.T) - qs;     // new tokens of b
    const int L = clamp_len(a.seq_lens[b], a.cap);
    const int t0 = tile * tok_per_tile;
    if (t0 >= n) return;                                       // whole workgroup

    // this lane's query row: token t0 + row / G, head g*G + row % G
    const int rho = lane & 31;
    const int hh = lane >> 5;
    const int row = 32 * wid + rho;
    const int i = t0 + row / G;
    const bool row_ok = i < n;
    const int pos = L - n + i;                                 // attends positions 0 .. pos
    const int hq = g * G + row % G;
    const int64_t qrow = (int64_t)qs + (row_ok ? i : 0);

    uint4 qf[8];
    {
        const uint4 *qp = (const uint4 *)(a.q + (qrow * a.Hq + hq) * kHeadDim + 64 * hh);
#pragma unroll
        for (int kk = 0; kk < 8; ++kk) qf[kk] = row_ok ? qp[kk] : make_uint4(0u, 0u, 0u, 0u);
    }

    // positions the workgroup reads: 0 .. kend-1 (its last valid token's prefix)
    const int kend = L - n + min(t0 + tok_per_tile, n);
    // the last position any row of this wave attends, and the first
    const int wave_pos = L - n + min(t0 + (32 * wid + 31) / G, n - 1);
    const int wave_pos0 = L - n + t0 + (32 * wid) / G;
    const int nkb = kend > 0 ? (kend + kStageKeys - 1) / kStageKeys : 0;

    f32x16_t acc[4];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[mt][r] = 0.0f;
    float m = -INFINITY;
    float l = 0.0f;                 // this lane's half of the row's weight sum
    const float sl = a.scale_log2;

    // cooperative block load: thread -> keys kr + kPassRows u, 16-byte chunks cc and cc + 8
    const int kr = tid >> 3;
    const int cc = tid & 7;
    const int32_t *bt = a.block_table + (int64_t)b * a.max_pages;
    const int pmask = (1 << a.log2_page) - 1;
    uint4 kx[kPasses][2], vx[kPasses][2];
    // position this thread loads in step u of block kb; positions past kend-1
    // read the last one (a live row) and are masked
    auto key_pos = [&](int kb, int u) { return min(kb * kStageKeys + kPassRows * u + kr, kend - 1); };
    auto page_ids = [&](int kb, int32_t (&pid)[kPasses]) {
#pragma unroll
        for (int u = 0; u < kPasses; ++u) pid[u] = bt[key_pos(kb, u) >> a.log2_page];
    };
    auto load = [&](int kb, const int32_t (&pid)[kPasses]) {
#pragma unroll
        for (int u = 0; u < kPasses; ++u) {
            const int t = key_pos(kb, u);
            const int64_t page = sanitize_page(pid[u], a.num_pages);
            const int64_t off = (((page << a.log2_page) + (t & pmask)) * a.Hkv + g) * kHeadDim;
            const u32x4_t *kp = (const u32x4_t *)(a.k + off);
            const u32x4_t *vp = (const u32x4_t *)(a.v + off);
            kx[u][0] = as_uint4(__builtin_nontemporal_load(kp + cc));
            kx[u][1] = as_uint4(__builtin_nontemporal_load(kp + cc + 8));
            vx[u][0] = as_uint4(__builtin_nontemporal_load(vp + cc));
            vx[u][1] = as_uint4(__builtin_nontemporal_load(vp + cc + 8));
        }
    };
    // row kPassRows u + kr has the swizzle of kr (kPassRows is a multiple of 4)
    const int vgw = v_swz(kr);
    auto stage = [&](int buf) {
#pragma unroll
        for (int u = 0; u < kPasses; ++u) {
            uint32_t *ks = s_k[buf] + (kPassRows * u + kr) * kKsStride;
            uint16_t *vs = s_v[buf] + (kPassRows * u + kr) * kRowV;
            *(uint4 *)(ks + 4 * cc) = kx[u][0];
            *(uint4 *)(ks + 4 * (cc + 8)) = kx[u][1];
            *(uint4 *)(vs + 32 * ((cc >> 2) ^ vgw) + 8 * (cc & 3)) = vx[u][0];
            *(uint4 *)(vs + 32 * (((cc + 8) >> 2) ^ vgw) + 8 * (cc & 3)) = vx[u][1];
        }
    };
    // V^T operand reads: this lane's source row vrow (+ 16 s2, + 8) and bf16
    // column vcol of segment mt
    const int vrow = 4 * (lane >> 5) + ((lane & 15) >> 2);
    const int vcol = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
    const int vgr = v_swz(vrow);

    // One 32-key step at position k0: scores, causal mask, online softmax, V^T P^T.
    auto consume = [&](int k0, const uint32_t *ks, const uint16_t *vs) {
        f32x16_t st;
#pragma unroll
        for (int r = 0; r < 16; ++r) st[r] = 0.0f;
        uint4 ka[8];
#pragma unroll
        for (int kk = 0; kk < 8; ++kk) ka[kk] = *(const uint4 *)(ks + rho * kKsStride + 32 * hh + 4 * kk);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int kk = 0; kk < 8; ++kk) st = mfma32(ka[kk], qf[kk], st);
        // the V^T operands (dim 32 mt + rho over keys 16 s2 + 4 hh + 0..3 and
        // 16 s2 + 8 + 4 hh + 0..3) are read now, so their latency passes during
        // the softmax
        uint4 va[4][2];
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
            for (int s2 = 0; s2 < 2; ++s2) {
                const uint16_t *src = vs + (16 * s2 + vrow) * kRowV + 32 * (mt ^ vgr) + vcol;
                const uint2 lo4 = read_tr16(src);
                const uint2 hi4 = read_tr16(src + 8 * kRowV);
                va[mt][s2] = make_uint4(lo4.x, lo4.y, hi4.x, hi4.y);
            }
        float p[16];
        float mx = -INFINITY;
        if (k0 + kKeyBlock - 1 > wave_pos0) {
            // a block on the diagonal: mask positions after each row's own
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int t = k0 + 8 * (r >> 2) + 4 * hh + (r & 3);
                p[r] = t <= pos ? st[r] * sl : -INFINITY;
                mx = fmaxf(mx, p[r]);
            }
        } else {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                p[r] = st[r] * sl;
                mx = fmaxf(mx, p[r]);
            }
        }
        mx = pair_max(mx);
        // move the maximum (and rescale) only when some row's scores exceed it by
        // more than kMaxSlack; otherwise the weights stay below 2^kMaxSlack
        if (__ballot(mx > m + kMaxSlack)) {
            const float mn = fmaxf(m, mx);
            const float ms = (mn == -INFINITY) ? 0.0f : mn;
            const float alpha = fast_exp2(m - ms);
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
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
            for (int s2 = 0; s2 < 2; ++s2) {
                acc[mt] = mfma32(va[mt][s2], phi[s2], acc[mt]);
                acc[mt] = mfma32(va[mt][s2], plo[s2], acc[mt]);
            }
    };

    // Page ids run two blocks ahead of the K/V loads: the ids of block n+2 are
    // loaded before the K/V loads of block n+1, and the wait for those (at the
    // end of block n) covers them, so no load waits on an address.
    if (nkb > 0) {
        int32_t pid0[kPasses], pid1[kPasses], pid2[kPasses];
        page_ids(0, pid0);
        load(0, pid0);
        page_ids(min(1, nkb - 1), pid1);
        stage(0);
        __syncthreads();
        for (int kb = 0; kb < nkb; ++kb) {
            const bool more = kb + 1 < nkb;           // uniform over the workgroup
            if (more) {
                page_ids(min(kb + 2, nkb - 1), pid2);
                load(kb + 1, pid1);
            }
            const int buf = kb & 1;
#pragma unroll
            for (int u = 0; u < kSteps; ++u) {
                const int k0 = kb * kStageKeys + kKeyBlock * u;
                if (k0 <= wave_pos)
                    consume(k0, s_k[buf] + kKeyBlock * u * kKsStride, s_v[buf] + kKeyBlock * u * kRowV);
            }
            if (more) stage((kb + 1) & 1);
#pragma unroll
            for (int u = 0; u < kPasses; ++u) pid1[u] = pid2[u];
            __syncthreads();
        }
    }

    l = pair_sum(l);
    if (row_ok) {
        const int64_t orow = qrow * a.Hq + hq;
        const float inv = l > 0.0f ? 1.0f / l : 0.0f;
        float *dst = a.out + orow * kHeadDim;
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4)
                *(float4 *)(dst + 32 * mt + 8 * r4 + 4 * hh) =
                    make_float4(acc[mt][4 * r4] * inv, acc[mt][4 * r4 + 1] * inv,
                                acc[mt][4 * r4 + 2] * inv, acc[mt][4 * r4 + 3] * inv);
        if (a.lse && hh == 0) a.lse[orow] = l > 0.0f ? (m + fast_log2(l)) * kLn2 : -INFINITY;
    }
}

}  // namespace

hipError_t launch_prefill(const PrefillArgs &a, hipStream_t stream) {
    const int64_t pairs = (int64_t)a.B * a.Hkv;
    const int64_t blocks = (pairs + a.xcds - 1) / a.xcds * a.xcds * a.tiles;
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL(prefill_kernel, dim3((unsigned)blocks), dim3(kPfWaves * 64), 0, stream, a);
    return hipGetLastError();
}

int prefill_tokens_per_tile(int group) { return kPfRows / group; }

}  // namespace kva
