// The step before attention for each sequence's newly decoded token, on
// gfx950: per-head RMS normalisation of its query and key, rotary position
// embedding at its position, and the append of its key and value to the cache.
//
// One workgroup per sequence.  The loads of the head rows are issued first
// (they do not depend on the position).  The 64 rotation angles of the
// sequence's position are formed in binary64 (the angle of the lowest pair
// grows with the position, up to ~1e4 radians, where fp32 would lose ~1e-3),
// reduced modulo 2 pi in binary64 (2 pi in two parts, each product taken
// inside a fused multiply-add), and only the remainder goes through fp32
// sincos; the cosines and sines sit in LDS.  Each head row (128 bf16) is held by
// 16 lanes, 8 dims per lane: the sum of squares is a DPP row sum, and the
// rotation partner of dim i (dim i +- 64) sits in the lane 8 positions away in
// the same DPP row.  Arithmetic is fp32; each output is rounded once to bf16
// (nearest even).  The kernel moves ~2 x (Hq + 2 Hkv) x 256 bytes per
// sequence: it is bound by launch latency, not by bandwidth.

#include "kva_internal.h"
#include "kva_device.h"

namespace kva {
namespace {

using namespace dev;

constexpr int kRowsPerPass = 16;     // head rows per workgroup pass (16 lanes each)
constexpr int kPreloadPasses = 4;    // passes whose row loads are issued up front

// 2 pi = kTwoPiHi + kTwoPiLo: the binary64 nearest 2 pi, and the remainder.
constexpr double kTwoPiHi = 6.28318530717958623200e+00;
constexpr double kTwoPiLo = 2.44929359829470635446e-16;

// cos and sin of the binary64 angle x >= 0.  fma(-k, hi, x) is x - k hi
// rounded once (the product is exact inside the fma), so the remainder is
// accurate to a few ulp of pi for any k below 2^50.
__device__ __forceinline__ void cos_sin(double x, float &c, float &s) {
    const double k = rint(x * 0.15915494309189533577);   // x / (2 pi)
    const double r = fma(-k, kTwoPiLo, fma(-k, kTwoPiHi, x));
    sincosf((float)r, &s, &c);
}

// fp32 -> bf16 bits, nearest even (finite values).
__device__ __forceinline__ uint32_t to_bf16_rne(float x) {
    const uint32_t u = __float_as_uint(x);
    return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

__global__ __launch_bounds__(256) void append_kernel(const AppendArgs a) {
    __shared__ float s_cos[kHeadDim / 2], s_sin[kHeadDim / 2];
    const int b = blockIdx.x;
    const int tid = threadIdx.x;
    const int c = tid & 15;          // 8 dims: 8c .. 8c+7
    const int rows = a.Hq + 2 * a.Hkv;

    // head row r of this sequence: q rows, then k rows, then v rows
    auto row_src = [&](int r) {
        return r < a.Hq ? a.q_in + ((int64_t)b * a.Hq + r) * kHeadDim
             : (r < a.Hq + a.Hkv ? a.k_in + ((int64_t)b * a.Hkv + (r - a.Hq)) * kHeadDim
                                 : a.v_in + ((int64_t)b * a.Hkv + (r - a.Hq - a.Hkv)) * kHeadDim);
    };
    uint4 pre[kPreloadPasses];
#pragma unroll
    for (int it = 0; it < kPreloadPasses; ++it) {
        const int r = (tid >> 4) + kRowsPerPass * it;
        if (r < rows) pre[it] = *(const uint4 *)(row_src(r) + 8 * c);
    }

    const int L = clamp_len(a.seq_lens[b], a.cap);

    // destination row of the new key and value, or -1: no room, or a page id
    // outside the pool (a write is never redirected)
    int64_t row = -1;
    if (L < a.cap) {
        if (a.paged) {
            const int32_t pg = a.block_table[(int64_t)b * a.max_pages + (L >> a.log2_page)];
            if ((int64_t)(uint32_t)pg < a.num_pages)
                row = ((int64_t)pg << a.log2_page) + (L & ((1 << a.log2_page) - 1));
        } else {
            row = (int64_t)b * a.cap + L;
        }
    }
    if (a.rope && tid < kHeadDim / 2) {
        // theta^(-2i/D) and the angle in binary64
        const double inv = exp2(-(2.0 * tid / kHeadDim) * a.log2_theta);
        cos_sin((double)L * inv, s_cos[tid], s_sin[tid]);
    }
    // every thread has read seq_lens[b] before it may be overwritten (new_lens
    // may alias seq_lens)
    __syncthreads();
    if (tid == 0 && a.new_lens) a.new_lens[b] = row >= 0 ? L + 1 : L;

    const float inv_d = 1.0f / kHeadDim;
    int it = 0;
    for (int r = tid >> 4; r < rows; r += kRowsPerPass, ++it) {
        const int kind = r < a.Hq ? 0 : (r < a.Hq + a.Hkv ? 1 : 2);   // q, k, v
        const int h = kind == 0 ? r : (kind == 1 ? r - a.Hq : r - a.Hq - a.Hkv);
        uint4 raw;
        if (it < kPreloadPasses) {
#pragma unroll
            for (int j = 0; j < kPreloadPasses; ++j)
                if (j == it) raw = pre[j];
        } else {
            raw = *(const uint4 *)(row_src(r) + 8 * c);
        }
        if (kind != 0 && row < 0) continue;     // nowhere to put this sequence's k/v
        uint4 res = raw;
        if (kind != 2) {
            const uint32_t w4[4] = {raw.x, raw.y, raw.z, raw.w};
            float x[8];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                x[2 * e] = bf16_lo(w4[e]);
                x[2 * e + 1] = bf16_hi(w4[e]);
            }
            const float *gain = kind == 0 ? a.q_w : a.k_w;
            if (gain) {
                float ss = 0.0f;
#pragma unroll
                for (int e = 0; e < 8; ++e) ss = fmaf(x[e], x[e], ss);
                ss = row_sum16(ss);
                const float rinv = 1.0f / sqrtf(ss * inv_d + a.eps);
                const float4 g0 = *(const float4 *)(gain + 8 * c);
                const float4 g1 = *(const float4 *)(gain + 8 * c + 4);
                const float gw[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
#pragma unroll
                for (int e = 0; e < 8; ++e) x[e] = (x[e] * rinv) * gw[e];
            }
            if (a.rope) {
                // lanes c < 8 hold dims i < 64 (partner i + 64), lanes c >= 8 the
                // upper halves (partner i - 64): y_lo = x c - p s, y_hi = x c + p s
                const float sgn = c < 8 ? -1.0f : 1.0f;
                float y[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float p = dpp_f32<0x128>(x[e]);   // row_ror:8 -> lane c ^ 8
                    const int i = (8 * c + e) & (kHeadDim / 2 - 1);
                    y[e] = fmaf(sgn * p, s_sin[i], x[e] * s_cos[i]);
                }
#pragma unroll
                for (int e = 0; e < 8; ++e) x[e] = y[e];
            }
            res = make_uint4(to_bf16_rne(x[0]) | (to_bf16_rne(x[1]) << 16),
                             to_bf16_rne(x[2]) | (to_bf16_rne(x[3]) << 16),
                             to_bf16_rne(x[4]) | (to_bf16_rne(x[5]) << 16),
                             to_bf16_rne(x[6]) | (to_bf16_rne(x[7]) << 16));
        }
        uint16_t *dst = kind == 0 ? a.q_out + ((int64_t)b * a.Hq + h) * kHeadDim
                      : (kind == 1 ? a.k_cache : a.v_cache) + (row * a.Hkv + h) * kHeadDim;
        *(uint4 *)(dst + 8 * c) = res;
    }
}

}  // namespace

hipError_t launch_append(const AppendArgs &a, hipStream_t stream) {
    if (a.B == 0) return hipSuccess;
    hipLaunchKernelGGL(append_kernel, dim3((unsigned)a.B), dim3(256), 0, stream, a);
    return hipGetLastError();
}

}  // namespace kva
