// Device helpers shared by the HIP kernel files of libkva (gfx950).  Not
// installed; not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kva_internal.h"

namespace kva {
namespace dev {

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                           __builtin_bit_cast(bf16x2_t, b), c, false);
}

__device__ __forceinline__ float bf16_lo(uint32_t x) { return __uint_as_float(x << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t x) { return __uint_as_float(x & 0xffff0000u); }

template <int CTRL>
__device__ __forceinline__ float dpp_f32(float x) {
    return __builtin_bit_cast(
        float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xf, 0xf, false));
}

// Sum over the 16 lanes of a DPP row.  Rotating by 8, 4, 2, 1 hands every lane
// of the row the same value: at each step both addends are already equal
// across the rotation orbit and fp addition commutes.
__device__ __forceinline__ float row_sum16(float x) {
    x += dpp_f32<0x128>(x);  // row_ror:8
    x += dpp_f32<0x124>(x);  // row_ror:4
    x += dpp_f32<0x122>(x);  // row_ror:2
    x += dpp_f32<0x121>(x);  // row_ror:1
    return x;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

__device__ __forceinline__ int uniform_i32(int x) { return __builtin_amdgcn_readfirstlane(x); }

__device__ __forceinline__ int64_t uniform_i64(int64_t x) {
    uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
    uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)x >> 32));
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ int64_t lane_i64(int64_t x, int lane) {
    uint32_t lo = __builtin_amdgcn_readlane((uint32_t)x, lane);
    uint32_t hi = __builtin_amdgcn_readlane((uint32_t)((uint64_t)x >> 32), lane);
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ int wave_incl_scan(int x, int lane) {
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        int y = __shfl_up(x, d, 64);
        if (lane >= d) x += y;
    }
    return x;
}

__device__ __forceinline__ int clamp_len(int L, int cap) { return L < 0 ? 0 : (L > cap ? cap : L); }

// ---- page-table addressing (shared by the attention kernels and the gather hook)

// Physical page holding position t of sequence b; ids outside [0, num_pages)
// are replaced by page 0 so that a bad table never reads out of bounds.
__device__ __forceinline__ int32_t sanitize_page(int32_t p, int64_t num_pages) {
    return ((int64_t)(uint32_t)p < num_pages) ? p : 0;
}

__device__ __forceinline__ int64_t page_of(const int32_t *__restrict__ bt, int b, int max_pages,
                                           int t, int log2_page, int64_t num_pages) {
    return sanitize_page(bt[(int64_t)b * max_pages + (t >> log2_page)], num_pages);
}

// Pool row (page * page_size + slot) of position t that lives in `page`.
__device__ __forceinline__ int64_t pool_row(int64_t page, int t, int log2_page) {
    return (page << log2_page) + (int64_t)(t & ((1 << log2_page) - 1));
}

// ---- raw buffer access

typedef __amdgpu_buffer_rsrc_t kv_rsrc_t;
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
// Fourth descriptor word for raw (untyped) buffer access on gfx9-family parts.
constexpr int kBufferFlags = 0x00020000;
// Cache policy of the K/V loads: non-temporal.  Every K/V byte is read once
// per call, so the stream should not displace anything in L2 or the
// memory-side cache; on MI355X this lifts the attention kernel from ~5.1 to
// ~5.9 TB/s.
constexpr int kKvLoadPolicy = 2;

__device__ __forceinline__ uint4 as_uint4(u32x4_t v) { return make_uint4(v.x, v.y, v.z, v.w); }

// ---- matrix-core blocks (shared-prefix pass, prefill)
//
// v_mfma_f32_32x32x16_bf16, lane l, h = l / 32: the A register holds
// A[l % 32][8h .. 8h+7], the B register B[8h .. 8h+7][l % 32], output
// register r holds D[8(r/4) + 4h + r%4][l % 32] (checked on the GPU).

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

__device__ __forceinline__ f32x16_t mfma32(const uint4 &a, const uint4 &b, const f32x16_t &c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                   __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

// K block in LDS: 32 token rows of 256 bytes, padded to 272 (the operand
// reads of one instruction, 32 rows at one column, then spread over the banks).
constexpr int kKsStride = 68;   // dwords
// V block in LDS: 32 token rows of 256 bytes, padded to 288, read as V^T
// operands through ds_read_b64_tr_b16.  Within each 16-lane group that read
// gives lane 4a + j element j of the 8-byte chunks lanes a, a + 4, a + 8,
// a + 12 point at (checked on the GPU), so four lanes pointing at four
// consecutive tokens (4 dims each) give sixteen lanes one dim each over those
// tokens; with 288-byte rows a group's four rows fall on disjoint banks.
constexpr int kVsStride = 144;  // bf16

typedef short s16x4v_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint2 read_tr16(const uint16_t *p) {
    const s16x4v_t r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4v_t *)p);
    return __builtin_bit_cast(uint2, r);
}

// For the A operand of v_mfma_f32_32x32x16_bf16 over a V block (dim 32 mt +
// l % 32, tokens 16 s2 + 4h + 0..3 and 16 s2 + 8 + 4h + 0..3): this lane's
// source offset (bf16) as a pointer of the transposing reads; add
// (16 s2 + 8 q) * kVsStride + 32 mt for half q of K-step s2 of tile mt.
__device__ __forceinline__ int vs_source(int lane) {
    return (4 * (lane >> 5) + ((lane & 15) >> 2)) * kVsStride + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
}

// Sum or maximum of this lane's value and that of lane l ^ 32 (the other half
// of a 32x32 output column).
__device__ __forceinline__ float pair_sum(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float pair_max(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// bf16 nearest-even of x (finite x), as bits.
__device__ __forceinline__ uint32_t bf16_rne_bits(float x) {
    const uint32_t u = __float_as_uint(x);
    return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

// Softmax weights as two bf16 parts for a matrix-core product: for x0, x1
// (lanes' weights of two consecutive operand positions) the high parts are
// x truncated to bf16, the low parts the exact remainder truncated to bf16;
// hi + lo carries x to a relative 2^-16.  Packed two per dword.
__device__ __forceinline__ void split_bf16_pair(float x0, float x1, uint32_t &hi, uint32_t &lo) {
    const uint32_t u0 = __float_as_uint(x0), u1 = __float_as_uint(x1);
    hi = __builtin_amdgcn_perm(u1, u0, 0x07060302u);
    const float r0 = x0 - __uint_as_float(u0 & 0xffff0000u);
    const float r1 = x1 - __uint_as_float(u1 & 0xffff0000u);
    lo = __builtin_amdgcn_perm(__float_as_uint(r1), __float_as_uint(r0), 0x07060302u);
}

// ---- merge of partial results over disjoint key ranges (one wave, one row)
//
// A list of parts: part s has normalised output o[s * os + d] (d < D <= 256)
// and log-sum-exp l[s * ls] (natural log; -inf = empty part).  A merge takes
// the parts of two lists, the first list's in index order, then the second's.
// Lane s holds the log-sum-exp of part s (64 parts per round), so the maximum
// and the weight sum are wave reductions; the outputs are then accumulated two
// dims per lane with eight part loads in flight.  Parts are always added in
// the same order, so the result does not depend on which wave merges or when.

struct PartList {
    const float *o;
    int64_t os;
    const float *l;
    int64_t ls;
    int n;
};

__device__ __forceinline__ const float *part_o(const PartList &p1, const PartList &p2, int s) {
    return s < p1.n ? p1.o + (int64_t)s * p1.os : p2.o + (int64_t)(s - p1.n) * p2.os;
}

__device__ __forceinline__ float part_lse(const PartList &p1, const PartList &p2, int s) {
    return s < p1.n ? p1.l[(int64_t)s * p1.ls] : p2.l[(int64_t)(s - p1.n) * p2.ls];
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) x = fmaxf(x, __shfl_xor(x, d, 64));
    return x;
}

constexpr int kMergeFast = 32;   // parts merged with all loads in flight at once

__device__ inline void merge_lists(const PartList &p1, const PartList &p2, int D, float *out,
                                   float *lse_out, int lane) {
    constexpr float kLog2e = 1.4426950408889634f;
    const int n = p1.n + p2.n;
    if (n <= kMergeFast && D <= 128) {
        // Up to kMergeFast parts: every load (lse per lane, outputs two dims
        // per lane) is issued before any is used, so the merge costs one
        // round trip.
        const float ls = lane < n ? part_lse(p1, p2, lane) : -INFINITY;
        const int d = 2 * lane;
        float2 o[kMergeFast];
#pragma unroll
        for (int s = 0; s < kMergeFast; ++s)
            o[s] = (s < n && d < D) ? *(const float2 *)(part_o(p1, p2, s) + d)
                                     : make_float2(0.0f, 0.0f);
        const float M = wave_max(ls);
        if (M == -INFINITY) {
            if (d < D) *(float2 *)(out + d) = make_float2(0.0f, 0.0f);
            if (lse_out && lane == 0) *lse_out = -INFINITY;
            return;
        }
        const float wl = (ls == -INFINITY) ? 0.0f : fast_exp2((ls - M) * kLog2e);
        float wsum = 0.0f;
        float2 acc = make_float2(0.0f, 0.0f);
#pragma unroll
        for (int s = 0; s < kMergeFast; ++s) {
            if (s < n) {
                const float ws = __shfl(wl, s, 64);
                wsum += ws;
                // an empty part's outputs are never read into the sum
                if (ws != 0.0f) {
                    acc.x = fmaf(ws, o[s].x, acc.x);
                    acc.y = fmaf(ws, o[s].y, acc.y);
                }
            }
        }
        if (d < D) *(float2 *)(out + d) = make_float2(acc.x / wsum, acc.y / wsum);
        if (lse_out && lane == 0) *lse_out = M + fast_log2(wsum) * kLn2;
        return;
    }
    float M = -INFINITY;
    for (int s0 = 0; s0 < n; s0 += 64) {
        const float ls = (s0 + lane < n) ? part_lse(p1, p2, s0 + lane) : -INFINITY;
        M = fmaxf(M, wave_max(ls));
    }
    if (M == -INFINITY) {
        for (int d = 2 * lane; d < D; d += 128) *(float2 *)(out + d) = make_float2(0.0f, 0.0f);
        if (lse_out && lane == 0) *lse_out = -INFINITY;
        return;
    }
    float wsum = 0.0f;
    float2 acc[2] = {make_float2(0.0f, 0.0f), make_float2(0.0f, 0.0f)};   // dims 2*lane (+128)
    for (int s0 = 0; s0 < n; s0 += 64) {
        const float ls = (s0 + lane < n) ? part_lse(p1, p2, s0 + lane) : -INFINITY;
        // empty parts (lse = -inf) get weight exactly 0 and are skipped below
        const float wl = (ls == -INFINITY) ? 0.0f : fast_exp2((ls - M) * kLog2e);
        const int cnt = min(64, n - s0);
        for (int i = 0; i < cnt; ++i) wsum += __shfl(wl, i, 64);
        for (int dd = 0; dd < 2; ++dd) {
            const int d = 2 * lane + 128 * dd;
            if (d >= D) break;
            int i = 0;
            for (; i + 8 <= cnt; i += 8) {
                float2 o[8];
                float ws[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    ws[u] = __shfl(wl, i + u, 64);
                    o[u] = ws[u] != 0.0f ? *(const float2 *)(part_o(p1, p2, s0 + i + u) + d)
                                         : make_float2(0.0f, 0.0f);
                }
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    acc[dd].x = fmaf(ws[u], o[u].x, acc[dd].x);
                    acc[dd].y = fmaf(ws[u], o[u].y, acc[dd].y);
                }
            }
            for (; i < cnt; ++i) {
                const float ws = __shfl(wl, i, 64);
                if (ws != 0.0f) {
                    const float2 o = *(const float2 *)(part_o(p1, p2, s0 + i) + d);
                    acc[dd].x = fmaf(ws, o.x, acc[dd].x);
                    acc[dd].y = fmaf(ws, o.y, acc[dd].y);
                }
            }
        }
    }
    for (int dd = 0; dd < 2; ++dd) {
        const int d = 2 * lane + 128 * dd;
        if (d < D) *(float2 *)(out + d) = make_float2(acc[dd].x / wsum, acc[dd].y / wsum);
    }
    if (lse_out && lane == 0) *lse_out = M + fast_log2(wsum) * kLn2;
}

__device__ __forceinline__ void merge_parts(const float *o_p, int64_t o_stride, const float *lse_p,
                                            int64_t l_stride, int n, int D, float *out,
                                            float *lse_out, int lane) {
    const PartList p1{o_p, o_stride, lse_p, l_stride, n};
    const PartList p2{o_p, 0, lse_p, 0, 0};
    merge_lists(p1, p2, D, out, lse_out, lane);
}

}  // namespace dev
}  // namespace kva
