// HIP kernels for batched grouped-query decode attention on gfx950 (MI355X).
//
// Work decomposition.  The granules (16-token steps) of all sequences are laid
// end to end in one flat index space of length Gtot, each non-empty sequence
// after a few virtual granules that carry no work (a range pays them for every
// sequence it enters, the cost of starting a piece).  Each KV head g gets Wh
// waves; wave (i, g) takes a contiguous granule range (range i of Wh, sized
// by the speed of the wave's XCD), which may start inside one sequence and
// end inside another.  Every piece of a sequence a wave covers becomes one
// partial result (normalised output + log-sum-exp) for the G query heads of g,
// stored in slot i + b; a second kernel merges the partials of each sequence
// in slot order.  Every wave thus streams a fixed share of the K/V bytes
// whatever the mix of lengths, and the grid is sized to the waves the device
// keeps resident, so there is no tail of idle compute units.
//
// Inside a wave.  The granules of a wave's range form one continuous stream
// (the next granule's K/V loads are issued before the current one is
// consumed); the arithmetic of a granule is a compute engine chosen per cache
// type and layout: on the matrix cores (MfmaBf16Engine, MfmaFp8Engine: K
// through an LDS tile into S^T = K Q^T, granule pairs per softmax update,
// O^T += V^T P^T with V^T by transposing LDS reads) for pages of 16+ tokens
// and contiguous caches, on the vector ALU (DotEngine: dot2 products summed
// over DPP rows, one online softmax per token row) for smaller pages.

#include "kva_internal.h"
#include "kva_device.h"

namespace kva {
namespace {

using namespace dev;

// ---- cache element types: one 16-lane row slice per token row
//
// bf16: a lane's 8 dims are 16 bytes; fp8 (OCP e4m3fn codes): 8 bytes.  The
// compute step widens fp8 keys to bf16 pairs (exact: e4m3fn values have 4
// significant bits) for the same dot2 products, and fp8 values to fp32; the
// per-tensor scales are folded in by the caller (keys into the score scale,
// values into the final output).

template <int KV> struct KvChunk;
template <> struct KvChunk<kKvBf16> { typedef uint4 type; static constexpr int kBytes = 2; };
template <> struct KvChunk<kKvFp8> { typedef uint2 type; static constexpr int kBytes = 1; };

typedef __bf16 bf16x2v_t __attribute__((ext_vector_type(2)));
typedef float f32x2v_t __attribute__((ext_vector_type(2)));

// Key chunk as four bf16 pairs.
__device__ __forceinline__ uint4 key_bf16(const uint4 &k) { return k; }
__device__ __forceinline__ uint4 key_bf16(const uint2 &k) {
    return make_uint4(
        __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(k.x, 1.0f, false)),
        __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(k.x, 1.0f, true)),
        __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(k.y, 1.0f, false)),
        __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(k.y, 1.0f, true)));
}

// Value chunk as 8 floats.
__device__ __forceinline__ void value_f32(const uint4 &v, float (&vf)[8]) {
    vf[0] = bf16_lo(v.x); vf[1] = bf16_hi(v.x); vf[2] = bf16_lo(v.y); vf[3] = bf16_hi(v.y);
    vf[4] = bf16_lo(v.z); vf[5] = bf16_hi(v.z); vf[6] = bf16_lo(v.w); vf[7] = bf16_hi(v.w);
}
__device__ __forceinline__ void value_f32(const uint2 &v, float (&vf)[8]) {
    const f32x2v_t a = __builtin_amdgcn_cvt_pk_f32_fp8(v.x, false);
    const f32x2v_t b = __builtin_amdgcn_cvt_pk_f32_fp8(v.x, true);
    const f32x2v_t c = __builtin_amdgcn_cvt_pk_f32_fp8(v.y, false);
    const f32x2v_t d = __builtin_amdgcn_cvt_pk_f32_fp8(v.y, true);
    vf[0] = a.x; vf[1] = a.y; vf[2] = b.x; vf[3] = b.y;
    vf[4] = c.x; vf[5] = c.y; vf[6] = d.x; vf[7] = d.y;
}

__device__ __forceinline__ void zero_chunk(uint4 &v) { v = make_uint4(0u, 0u, 0u, 0u); }
__device__ __forceinline__ void zero_chunk(uint2 &v) { v = make_uint2(0u, 0u); }

// ---- one granule step of one wave

template <int G, bool MASK, typename C>
__device__ __forceinline__ void attend_step(const uint32_t (&qv)[G][4], const C (&kd)[4],
                                            C (&vd)[4], float (&m)[G], float (&l)[G],
                                            float (&acc)[G][8], float scale_log2, int r,
                                            int nvalid) {
    float s[G][4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const uint4 kb = key_bf16(kd[u]);
#pragma unroll
        for (int j = 0; j < G; ++j) {
            float d = dot2_bf16(qv[j][0], kb.x, 0.0f);
            d = dot2_bf16(qv[j][1], kb.y, d);
            d = dot2_bf16(qv[j][2], kb.z, d);
            d = dot2_bf16(qv[j][3], kb.w, d);
            s[j][u] = row_sum16(d) * scale_log2;
        }
    }
    if (MASK) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const bool ok = (4 * u + r) < nvalid;
#pragma unroll
            for (int j = 0; j < G; ++j) s[j][u] = ok ? s[j][u] : -INFINITY;
            // poisoned rows past the length must not reach the sum: 0 * NaN = NaN
            if (!ok) zero_chunk(vd[u]);
        }
    }
    float p[G][4];
#pragma unroll
    for (int j = 0; j < G; ++j) {
        const float mx = fmaxf(fmaxf(s[j][0], s[j][1]), fmaxf(s[j][2], s[j][3]));
        const float mn = fmaxf(m[j], mx);
        const float ms = (mn == -INFINITY) ? 0.0f : mn;
        const float alpha = fast_exp2(m[j] - ms);
#pragma unroll
        for (int u = 0; u < 4; ++u) p[j][u] = fast_exp2(s[j][u] - ms);
        l[j] = fmaf(l[j], alpha, (p[j][0] + p[j][1]) + (p[j][2] + p[j][3]));
        m[j] = mn;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[j][e] *= alpha;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        float vf[8];
        value_f32(vd[u], vf);
#pragma unroll
        for (int j = 0; j < G; ++j) {
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[j][e] = fmaf(p[j][u], vf[e], acc[j][e]);
        }
    }
}


// ---- batch tables (LDS, one copy per block)
//
// pre[b] = first flat granule of sequence b (granules of one KV head, all
// sequences end to end, each non-empty one after a.vgran virtual granules),
// pre[B] = total; len[b] = the clamped length.

// First granule of sequence b this kernel attends: past the group's shared
// run in grouped calls, else 0.
__device__ __forceinline__ int gran_lo(const AttnArgs &a, int b) {
    return a.pref ? a.pref[b / a.group] : 0;
}

__device__ __forceinline__ int64_t shfl_up_i64(int64_t x, int d) {
    const int lo = __shfl_up((int)(uint32_t)x, d, 64);
    const int hi = __shfl_up((int)((uint64_t)x >> 32), d, 64);
    return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

// Whole block: lengths are read once (kPer per thread, all loads in flight),
// then a block-wide scan of the granule counts.
__device__ void build_tables(const AttnArgs &a, int64_t *pre, int32_t *len, int64_t *wsum) {
    constexpr int kPer = kMaxSeqsPerLaunch / (kWavesPerBlock * 64);
    const int tid = threadIdx.x;
    int Ls[kPer], lo[kPer];
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
        const int b = tid * kPer + k;
        Ls[k] = b < a.B ? a.seq_lens[b] : 0;
        lo[k] = b < a.B ? gran_lo(a, b) : 0;
    }
    int n[kPer];
    int64_t run = 0;
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
        const int b = tid * kPer + k;
        const int L = clamp_len(Ls[k], a.cap);
        n[k] = b < a.B ? max(0, (L + kGranule - 1) / kGranule - lo[k]) : 0;
        if (n[k] > 0) n[k] += a.vgran;
        if (b < a.B) len[b] = L;
        run += n[k];
    }
    const int lane = tid & 63;
    int64_t incl = run;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int64_t y = shfl_up_i64(incl, d);
        if (lane >= d) incl += y;
    }
    if (lane == 63) wsum[tid >> 6] = incl;
    __syncthreads();
    int64_t x = incl - run;
    for (int w = 0; w < (tid >> 6); ++w) x += wsum[w];
    if (tid == 0) pre[0] = 0;
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
        const int b = tid * kPer + k;
        x += n[k];
        if (b < a.B) pre[b + 1] = x;
    }
    __syncthreads();
}

// ---- work decomposition of one KV head's flat granule space
//
// The space [0, gtot) is cut into wh ranges, one per wave of the head, in
// proportion to weights wa (even range index: waves on even XCDs) and wb
// (odd index); with wa = wb the ranges are equal.  Range i is the producer of
// partial results with index i: the piece of sequence b it covers goes to
// slot i + b.  Slots are unique (a later range only covers the same or later
// sequences), and a sequence's pieces occupy consecutive slots.
// floor(a / b) for 0 <= a < 2^53, 0 < b < 2^53.  The fp64 quotient of the
// (exact) operands is correctly rounded, so its integer part is the floor or
// one more; one integer check fixes it.  (64-bit integer division would be
// expanded into a long vector sequence.)
__device__ __forceinline__ int64_t fdiv(int64_t a, int64_t b) {
    int64_t q = (int64_t)((double)a / (double)b);
    if (q * b > a) --q;
    return q;
}

struct Split {
    int64_t gtot;   // granules per KV head
    int64_t wh;     // ranges per KV head
    int64_t wa, wb; // weights of the ranges with even / odd index

    // total weight of ranges 0 .. i-1, and range i's first granule
    __device__ int64_t wsum(int64_t i) const { return ((i + 1) >> 1) * wa + (i >> 1) * wb; }
    __device__ int64_t x(int64_t i) const { return fdiv(gtot * wsum(i), wsum(wh)); }
    // the range holding granule y: the largest i with x(i) <= y, i.e. with
    // wsum(i) <= floor(((y + 1) wsum(wh) - 1) / gtot)
    __device__ int64_t range_of(int64_t y) const {
        const int64_t v = fdiv((y + 1) * wsum(wh) - 1, gtot);
        const int64_t k = fdiv(v, wa + wb);
        const int64_t i = 2 * k + (v - k * (wa + wb) >= wa ? 1 : 0);
        return i < wh - 1 ? i : wh - 1;
    }
    __device__ int64_t producer_of(int64_t y) const { return range_of(y); }
};

// Merge plan for the second kernel, written by wave (g, i) = (0, 0): per sequence {first
// slot, number of pieces}; 0 pieces for sequences written directly (one
// piece, or empty).  Grouped calls send every piece to a slot.
__device__ void write_plan(const AttnArgs &a, const Split &sp, const int64_t *pre, int lane) {
    for (int b = lane; b < a.B; b += 64) {
        const int64_t en = pre[b + 1];
        const int64_t st = pre[b] + (en > pre[b] ? a.vgran : 0);   // first real granule
        int2 pl = make_int2(0, 0);
        if (en > st) {
            const int64_t first = sp.producer_of(st);
            const int64_t last = sp.producer_of(en - 1);
            if (last > first || a.pref) pl = make_int2((int)(first + b), (int)(last - first + 1));
        }
        a.plan[b] = pl;
    }
}

// Largest b with pre[b] <= u (u < pre[B]): the sequence holding flat granule u.
__device__ __forceinline__ int find_seq(const int64_t *pre, int B, int64_t u) {
    int lo = 0, hi = B;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (uniform_i64(pre[mid]) <= u) lo = mid;
        else hi = mid;
    }
    return lo;
}

// ---- the granule stream of one wave
//
// A wave works through a list of segments: runs of granules of one piece that
// share one window of page ids.  Loads run one granule ahead of the
// arithmetic, across segment and piece boundaries: the next segment is
// resolved a few granules before it is needed, its page ids are fetched into
// the second of two LDS windows, and its q rows into a two-slot LDS ring, so a
// piece boundary costs no memory round trip.

enum SegFlags : int { kSegValid = 1, kSegFirst = 2, kSegLast = 4 };

struct Seg {
    int b, g;          // sequence and KV head
    int gl0, gl1;      // granules [gl0, gl1) of the sequence
    int L;             // sequence length
    int pbase;         // paged: block-table index of the window's first page
    int nseg;          // pieces of the sequence (1: written to the output directly)
    int flags;         // kSegValid | kSegFirst (first of its piece) | kSegLast (last of its piece)
    int64_t slot;      // partial-result slot of the piece
};

// Per-granule tag of a loaded buffer, read by the compute step.
struct Tag {
    int nvalid;        // live rows (16 except for a sequence's last granule)
    int flags;         // kSegValid; kSegFirst: first granule of a piece; kSegLast: last
    int b, g, nseg, qpar;
    int64_t slot;
};

// Sum (or maximum) of x over the four 16-lane rows of the wave (lanes l, l^16,
// l^32, l^48), via the gfx950 row-swap permutes: the lower row's value is
// always the first addend, so every lane gets the same result.
__device__ __forceinline__ float rows_sum4(float x) {
    auto t = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = __uint_as_float(t[0]) + __uint_as_float(t[1]);
    auto u = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(u[0]) + __uint_as_float(u[1]);
}
__device__ __forceinline__ float rows_max4(float x) {
    auto t = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = fmaxf(__uint_as_float(t[0]), __uint_as_float(t[1]));
    auto u = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(u[0]), __uint_as_float(u[1]));
}

// ---- compute engines of the granule stream
//
// An engine owns the per-piece arithmetic state and knows how its lanes map
// onto a granule's K/V rows; the stream (segments, windows, look-ahead)
// drives it one granule at a time: load, start (new piece), step, finish.

// Vector-ALU engine (pages below 16 tokens, where a granule's rows are
// gathered one by one).  Lane (r, c) = (lane / 16, lane % 16) owns dims
// 8c..8c+7 of token rows r, r+4, r+8, r+12; q.K by bf16 dot2 and DPP row sums,
// each token row with its own online softmax, rows merged at the end.
template <int G, int KV>
struct DotEngine {
    typedef typename KvChunk<KV>::type C;
    static constexpr int EB = KvChunk<KV>::kBytes;
    struct Buf { C k[4], v[4]; };
    typedef uint32_t Q[G][4];

    int lane, r, c;
    uint32_t qv[G][4];
    float m[G], l[G], acc[G][8];

    __device__ void setup(int ln, unsigned char *) {
        lane = ln;
        r = ln >> 4;
        c = ln & 15;
    }

    // Granule rows through range-limited buffer descriptors (rows past the
    // length read zeros).
    __device__ void load(const kv_rsrc_t &rk, const kv_rsrc_t &rv, int row_bytes, Buf &b) const {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int off = (4 * u + r) * row_bytes + 8 * EB * c;
            if constexpr (KV == kKvBf16) {
                b.k[u] = as_uint4(__builtin_amdgcn_raw_buffer_load_b128(rk, off, 0, kKvLoadPolicy));
                b.v[u] = as_uint4(__builtin_amdgcn_raw_buffer_load_b128(rv, off, 0, kKvLoadPolicy));
            } else {
                const u32x2_t k2 = __builtin_amdgcn_raw_buffer_load_b64(rk, off, 0, kKvLoadPolicy);
                const u32x2_t v2 = __builtin_amdgcn_raw_buffer_load_b64(rv, off, 0, kKvLoadPolicy);
                b.k[u] = make_uint2(k2.x, k2.y);
                b.v[u] = make_uint2(v2.x, v2.y);
            }
        }
    }

    // Pages smaller than a granule: one page lookup per row; rows past the
    // length re-read the last live row (masked later).
    __device__ void load_rows(const AttnArgs &a, const int32_t *ids, int pbase, int t0, int nvalid,
                              int g, int lp, Buf &b) const {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int tt = t0 + min(4 * u + r, nvalid - 1);
            const int64_t page = ids[(tt >> lp) - pbase];
            const int64_t off = ((pool_row(page, tt, lp) * a.Hkv + g) * kHeadDim + 8 * c) * EB;
            b.k[u] = *(const C *)((const char *)a.k + off);
            b.v[u] = *(const C *)((const char *)a.v + off);
        }
    }

    __device__ void load_q(const AttnArgs &a, int bb, int g, Q &qd) const {
#pragma unroll
        for (int j = 0; j < G; ++j) {
            const uint4 t = *(const uint4 *)(a.q + ((int64_t)bb * a.Hq + g * G + j) * kHeadDim + 8 * c);
            qd[j][0] = t.x; qd[j][1] = t.y; qd[j][2] = t.z; qd[j][3] = t.w;
        }
    }

    // q rows into a ring slot of G rows of 256 bytes (the four lanes of a
    // column write the same bytes), and back at the start of the piece.
    __device__ void park_q(const Q &q, unsigned char *slot) const {
#pragma unroll
        for (int j = 0; j < G; ++j)
            *(uint4 *)(slot + j * kQRowBytes + 16 * c) = make_uint4(q[j][0], q[j][1], q[j][2], q[j][3]);
    }

    __device__ void start(const unsigned char *slot) {
#pragma unroll
        for (int j = 0; j < G; ++j) {
            m[j] = -INFINITY;
            l[j] = 0.0f;
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[j][e] = 0.0f;
            const uint4 t = *(const uint4 *)(slot + j * kQRowBytes + 16 * c);
            qv[j][0] = t.x; qv[j][1] = t.y; qv[j][2] = t.z; qv[j][3] = t.w;
        }
    }

    template <bool MASK>
    __device__ void step(Buf &b, float sl, int nvalid) {
        attend_step<G, MASK>(qv, b.k, b.v, m, l, acc, sl, r, nvalid);
    }

    // Merge the four token rows and store the piece's result.  The per-row
    // maxima and sums are combined with row swaps; the accumulators with a
    // reduce-scatter over the rows (rows r and r+2, then r and r+1, always the
    // lower row first), after which row r holds the totals of flat outputs
    // [2G r, 2G r + 2G) (index 8 j + e) and every lane stores a contiguous run.
    __device__ void finish(float v_scale, float *o_base, float *l_base, int h0) {
        float w[G], inv[G], lse[G];
#pragma unroll
        for (int j = 0; j < G; ++j) {
            const float M = rows_max4(m[j]);
            const float Ms = (M == -INFINITY) ? 0.0f : M;
            w[j] = fast_exp2(m[j] - Ms);
            const float lj = rows_sum4(l[j] * w[j]);
            inv[j] = lj > 0.0f ? 1.0f / lj : 0.0f;
            if constexpr (KV == kKvFp8) inv[j] *= v_scale;
            lse[j] = lj > 0.0f ? (M + fast_log2(lj)) * kLn2 : -INFINITY;
        }
        constexpr int NV = 8 * G;
        float s1[NV / 2];
#pragma unroll
        for (int k = 0; k < NV / 2; ++k) {
            const float x = acc[k / 8][k % 8] * w[k / 8];
            const float y = acc[(k + NV / 2) / 8][(k + NV / 2) % 8] * w[(k + NV / 2) / 8];
            auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(y), false, false);
            s1[k] = __uint_as_float(p[0]) + __uint_as_float(p[1]);
        }
        float s2[NV / 4];
#pragma unroll
        for (int k = 0; k < NV / 4; ++k) {
            auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(s1[k]), __float_as_uint(s1[k + NV / 4]),
                                                      false, false);
            s2[k] = __uint_as_float(p[0]) + __uint_as_float(p[1]);
        }
        // this lane's outputs: flat indices 2G r + k, k < 2G
#pragma unroll
        for (int k = 0; k < NV / 4; ++k) {
            // head of flat index 2G r + k (a lane's run spans whole heads for G >= 4)
            float sc = inv[0];
#pragma unroll
            for (int j = 1; j < G; ++j)
                if (((2 * G * r + k) >> 3) == j) sc = inv[j];
            s2[k] *= sc;
        }
        if constexpr (G >= 4) {
#pragma unroll
            for (int q = 0; q < G / 4; ++q) {
                const int j = (G / 4) * r + q;
                float4 *dst = (float4 *)(o_base + (h0 + j) * kHeadDim + 8 * c);
                dst[0] = make_float4(s2[8 * q], s2[8 * q + 1], s2[8 * q + 2], s2[8 * q + 3]);
                dst[1] = make_float4(s2[8 * q + 4], s2[8 * q + 5], s2[8 * q + 6], s2[8 * q + 7]);
            }
        } else if constexpr (G == 2) {
            *(float4 *)(o_base + (h0 + (r >> 1)) * kHeadDim + 8 * c + 4 * (r & 1)) =
                make_float4(s2[0], s2[1], s2[2], s2[3]);
        } else {
            *(float2 *)(o_base + h0 * kHeadDim + 8 * c + 2 * r) = make_float2(s2[0], s2[1]);
        }
        if (lane == 0 && l_base) {
#pragma unroll
            for (int j = 0; j < G; ++j) l_base[h0 + j] = lse[j];
        }
    }
};

typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef int i32x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ f32x4_t mfma16k32(const uint4 &a, const uint4 &b, const f32x4_t &c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                   __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}
__device__ __forceinline__ f32x4_t mfma16k16(const uint2 &a, const uint2 &b, const f32x4_t &c) {
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4_t, a),
                                                     __builtin_bit_cast(s16x4_t, b), c, 0, 0, 0);
}
// Four fp8 (e4m3fn) codes as four bf16 (exact: e4m3fn values have 4 significant bits).
__device__ __forceinline__ uint2 fp8x4_to_bf16(uint32_t x) {
    return make_uint2(
        __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(x, 1.0f, false)),
        __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(x, 1.0f, true)));
}

static_assert(kKtOffset == 2 * kGranule * kVtRow + 16 && kKtOffset % 16 == 0, "fp8 tile layout");

// Matrix-core engine for fp8 caches.  Per granule and KV head the products
// are 16 tokens x 128 dims x (G <= 16) query heads:
//  * loads: a granule's K (and V) rows are 16 rows of 128 codes; eight lanes
//    read one whole row (lane l: bytes 16 (l % 8).. of rows l / 8 and 8 + l / 8),
//    so every load instruction fetches whole 128-byte lines.  (Loading in the
//    matrix operand's layout instead, half a line per row per instruction,
//    measured 20% slower: the kernel is bound by its loads, not its arithmetic.)
//  * S^T = K Q^T on v_mfma_f32_16x16x32_bf16 (4 products over the 128 dims):
//    the K rows pass through the wave's LDS tile, from which lane l reads 32
//    codes of token l % 16 (bytes 16h..16h+15 and 64+16h..64+16h+15, h = l / 16)
//    and widens them to bf16 as the A operand; the B operand holds the same
//    dims of q for head l % 16 (columns of heads >= G are computed but never
//    stored).  The result gives lane l the scores of tokens 4h..4h+3 for head
//    l % 16.
//  * online softmax per head: maxima over the four lane groups by row swaps;
//    the running maximum moves only when a block exceeds it by more than 2^8,
//    so the accumulators are rarely rescaled.
//  * O^T = V^T P^T on v_mfma_f32_16x16x16bf16_1k (8 dim blocks, P as two bf16
//    parts): the score layout is exactly the B operand (tokens 4h..4h+3 of
//    head l % 16), so P never moves between lanes; V^T comes from the V rows
//    staged in LDS through ds_read_b64_tr_b8, whose result gives lane l the
//    bytes of one dim for the eight rows its 16-lane group pointed at (lane
//    l % 16 = 8a + j receives byte j from the lanes 2s + a, s < 8): one read
//    serves two dim blocks.
template <int G>
struct MfmaFp8Engine {
    static_assert(G <= 16, "query heads per KV head");
    struct Buf { uint4 k[2], v[2]; };
    typedef u32x4_t Q[4];           // (a native vector type keeps the temp in registers)

    int lane, hq;
    unsigned char *vt;            // this wave's V tile in LDS
    uint4 qv[4];
    f32x4_t o[8];                 // O^T blocks: lane l holds dims 16 db + 4 h + i of head l % 16
    float m, l;

    __device__ void setup(int ln, unsigned char *tile) {
        lane = ln;
        hq = ln >> 4;
        vt = tile;
    }

    // Rows l / 8 and 8 + l / 8, bytes 16 (l % 8)..+15: whole lines per instruction.
    __device__ void load(const kv_rsrc_t &rk, const kv_rsrc_t &rv, int row_bytes, Buf &b) const {
        const int off = (lane >> 3) * row_bytes + 16 * (lane & 7);
        b.k[0] = as_uint4(__builtin_amdgcn_raw_buffer_load_b128(rk, off, 0, kKvLoadPolicy));
        b.k[1] = as_uint4(__builtin_amdgcn_raw_buffer_load_b128(rk, off + 8 * row_bytes, 0, kKvLoadPolicy));
        b.v[0] = as_uint4(__builtin_amdgcn_raw_buffer_load_b128(rv, off, 0, kKvLoadPolicy));
        b.v[1] = as_uint4(__builtin_amdgcn_raw_buffer_load_b128(rv, off + 8 * row_bytes, 0, kKvLoadPolicy));
    }

    __device__ void load_rows(const AttnArgs &, const int32_t *, int, int, int, int, int, Buf &) const {}

    // B operands of the four q.K products: dims 16h + 8(kk & 1) + 64(kk >> 1)
    // + s (s < 8) of head l % 16, the dims the A operand holds for token l % 16.
    // Columns of heads >= G (never stored) repeat head G - 1.
    __device__ void load_q(const AttnArgs &a, int bb, int g, Q &qd) const {
        const int n = min(lane & 15, G - 1);
        const uint16_t *row = a.q + ((int64_t)bb * a.Hq + g * G + n) * kHeadDim;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) qd[kk] = *(const u32x4_t *)(row + 16 * hq + 8 * (kk & 1) + 64 * (kk >> 1));
    }

    // q rows into a ring slot of G rows of 256 bytes (lanes of the repeated
    // column G - 1 write the same bytes), and back at the start of the piece.
    __device__ void park_q(const Q &q, unsigned char *slot) const {
        unsigned char *row = slot + min(lane & 15, G - 1) * kQRowBytes + 32 * hq;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) *(u32x4_t *)(row + 16 * (kk & 1) + 128 * (kk >> 1)) = q[kk];
    }

    __device__ void start(const unsigned char *slot) {
        const unsigned char *row = slot + min(lane & 15, G - 1) * kQRowBytes + 32 * hq;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) qv[kk] = *(const uint4 *)(row + 16 * (kk & 1) + 128 * (kk >> 1));
#pragma unroll
        for (int db = 0; db < 8; ++db) o[db] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
        m = -INFINITY;
        l = 0.0f;
        pending = false;
    }

    // Granules are processed in pairs: the first of a pair only gets its
    // scores and stages its V rows; the second runs one softmax update over
    // both (32 tokens) and P.V with 16x16x32 products.  A piece's odd last
    // granule is processed alone (16x16x16 products) by finish().
    bool pending;
    float xp[4];                  // scaled, masked scores of the pending granule

    // V rows of a granule into tile half `half` (rows of half 1 start 16
    // bytes further, so the two halves fall on different banks).
    __device__ void stage_v(const Buf &b, int half) {
        unsigned char *row = vt + half * kVtHalf1 + (lane >> 3) * kVtRow + 16 * (lane & 7);
        *(uint4 *)row = b.v[0];
        *(uint4 *)(row + 8 * kVtRow) = b.v[1];
    }

    template <bool MASK>
    __device__ void scores(const Buf &b, float sl, int nvalid, float (&x)[4]) const {
        // K rows through the LDS tile into the A operand layout
        unsigned char *kt = vt + kKtOffset;
        unsigned char *wr = kt + (lane >> 3) * kKtRow + 16 * (lane & 7);
        __builtin_amdgcn_wave_barrier();
        *(uint4 *)wr = b.k[0];
        *(uint4 *)(wr + 8 * kKtRow) = b.k[1];
        __builtin_amdgcn_wave_barrier();
        const unsigned char *rd = kt + (lane & 15) * kKtRow + 16 * hq;
        const uint4 k0 = *(const uint4 *)rd;
        const uint4 k1 = *(const uint4 *)(rd + 64);
        __builtin_amdgcn_wave_barrier();
        // 4 products over the 128 dims, in two independent chains
        f32x4_t s0 = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f}, s1 = s0;
        const uint32_t kw[8] = {k0.x, k0.y, k0.z, k0.w, k1.x, k1.y, k1.z, k1.w};
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            const uint2 lo = fp8x4_to_bf16(kw[2 * kk]);
            const uint2 hi = fp8x4_to_bf16(kw[2 * kk + 1]);
            if (kk & 1) s1 = mfma16k32(make_uint4(lo.x, lo.y, hi.x, hi.y), qv[kk], s1);
            else s0 = mfma16k32(make_uint4(lo.x, lo.y, hi.x, hi.y), qv[kk], s0);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            x[i] = (s0[i] + s1[i]) * sl;
            if (MASK && 4 * hq + i >= nvalid) x[i] = -INFINITY;
        }
    }

    // Online-softmax update with a block maximum mx (the same in the four lane
    // groups of a head): the running maximum moves only when the block exceeds
    // it by 2^8.
    __device__ void rescale(float mx) {
        const bool up = mx > m + 8.0f;
        if (__ballot(up)) {
            const float mn = up ? mx : m;
            const float alpha = fast_exp2(m - mn);
            m = mn;
            l *= alpha;
#pragma unroll
            for (int db = 0; db < 8; ++db)
#pragma unroll
                for (int i = 0; i < 4; ++i) o[db][i] *= alpha;
        }
    }

    template <bool MASK>
    __device__ void step(Buf &b, float sl, int nvalid) {
        float x[4];
        scores<MASK>(b, sl, nvalid, x);
        if (!pending) {
            stage_v(b, 0);
#pragma unroll
            for (int i = 0; i < 4; ++i) xp[i] = x[i];
            pending = true;
            return;
        }
        stage_v(b, 1);
        pending = false;
        rescale(rows_max4(fmaxf(fmaxf(fmaxf(xp[0], xp[1]), fmaxf(xp[2], xp[3])),
                                fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])))));
        // P operand, k = 8h + s: tokens 4h + s of the first granule (s < 4),
        // 4h + s - 4 of the second
        float p[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            p[i] = fast_exp2(xp[i] - m);
            p[4 + i] = fast_exp2(x[i] - m);
        }
        l += ((p[0] + p[1]) + (p[2] + p[3])) + ((p[4] + p[5]) + (p[6] + p[7]));
        uint32_t ph[4], pl[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) split_bf16_pair(p[2 * i], p[2 * i + 1], ph[i], pl[i]);
        const uint4 bh = make_uint4(ph[0], ph[1], ph[2], ph[3]);
        const uint4 bl = make_uint4(pl[0], pl[1], pl[2], pl[3]);
        // V^T operands: as a source of the transposing read this lane points at
        // row 4h + (s & 3) of half s >> 2, dims 16 db + 8a (s = (l % 16) / 2,
        // a = l & 1), so receiving lane 8a + j gets dim 16 db + 8a + j of the
        // 8 tokens in P's k order
        __builtin_amdgcn_wave_barrier();
        const int s16 = (lane & 15) >> 1;
        const unsigned char *src = vt + (s16 >> 2) * kVtHalf1 + (4 * hq + (s16 & 3)) * kVtRow + 8 * (lane & 1);
        uint4 av[8];
#pragma unroll
        for (int db = 0; db < 8; ++db) {
            const i32x2_t t = __builtin_amdgcn_ds_read_tr8_b64_v2i32(
                (__attribute__((address_space(3))) i32x2_t *)(src + 16 * db));
            const uint2 a0 = fp8x4_to_bf16((uint32_t)t[0]);
            const uint2 a1 = fp8x4_to_bf16((uint32_t)t[1]);
            av[db] = make_uint4(a0.x, a0.y, a1.x, a1.y);
        }
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int db = 0; db < 8; ++db) o[db] = mfma16k32(av[db], bh, o[db]);
#pragma unroll
        for (int db = 0; db < 8; ++db) o[db] = mfma16k32(av[db], bl, o[db]);
    }

    // The pending granule alone: P.V over its 16 tokens.
    __device__ void flush() {
        if (!pending) return;
        pending = false;
        rescale(rows_max4(fmaxf(fmaxf(xp[0], xp[1]), fmaxf(xp[2], xp[3]))));
        float p[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) p[i] = fast_exp2(xp[i] - m);
        l += (p[0] + p[1]) + (p[2] + p[3]);
        uint32_t ph[2], pl[2];
        split_bf16_pair(p[0], p[1], ph[0], pl[0]);
        split_bf16_pair(p[2], p[3], ph[1], pl[1]);
        const uint2 bh = make_uint2(ph[0], ph[1]), bl = make_uint2(pl[0], pl[1]);
        // V^T operands of half 0: source row 4h + (s & 3), dims 16 (2 db2 +
        // (s >> 2)) + 8a; one read serves two dim blocks
        __builtin_amdgcn_wave_barrier();
        const int s16 = (lane & 15) >> 1;
        const unsigned char *src = vt + (4 * hq + (s16 & 3)) * kVtRow + 16 * (s16 >> 2) + 8 * (lane & 1);
        uint2 av[8];
#pragma unroll
        for (int db2 = 0; db2 < 4; ++db2) {
            const i32x2_t t = __builtin_amdgcn_ds_read_tr8_b64_v2i32(
                (__attribute__((address_space(3))) i32x2_t *)(src + 32 * db2));
            av[2 * db2] = fp8x4_to_bf16((uint32_t)t[0]);
            av[2 * db2 + 1] = fp8x4_to_bf16((uint32_t)t[1]);
        }
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int db = 0; db < 8; ++db) o[db] = mfma16k16(av[db], bh, o[db]);
#pragma unroll
        for (int db = 0; db < 8; ++db) o[db] = mfma16k16(av[db], bl, o[db]);
    }

    __device__ void finish(float v_scale, float *o_base, float *l_base, int h0) {
        flush();
        const int n = lane & 15;
        const float lt = rows_sum4(l);
        const float inv = lt > 0.0f ? v_scale / lt : 0.0f;
        if (n < G) {
            float *dst = o_base + (h0 + n) * kHeadDim + 4 * hq;
#pragma unroll
            for (int db = 0; db < 8; ++db)
                *(float4 *)(dst + 16 * db) = make_float4(o[db][0] * inv, o[db][1] * inv, o[db][2] * inv,
                                                          o[db][3] * inv);
            if (hq == 0 && l_base) l_base[h0 + n] = lt > 0.0f ? (m + fast_log2(lt)) * kLn2 : -INFINITY;
        }
    }
};

// Matrix-core engine for bf16 caches: the fp8 engine's products without the
// widening.  Per granule and KV head, 16 tokens x 128 dims x (G <= 16) heads:
//  * loads: sixteen lanes read one whole 256-byte row (lane l: bytes
//    16 (l % 16).. of rows l / 16 + 4u, u < 4), whole lines per instruction;
//  * S^T = K Q^T on four v_mfma_f32_16x16x32_bf16 (two chains): the K rows
//    pass through the wave's LDS tile, from which lane l reads dims
//    32 kk + 8h .. +7 of token l % 16 (h = l / 16) as the A operand of step kk;
//    the B operand holds the same dims of q for head l % 16.  Lane l gets the
//    scores of tokens 4h..4h+3 for head l % 16;
//  * the online softmax and granule pairs of the fp8 engine (32-token softmax
//    updates, lazily moved maximum, P as two bf16 parts);
//  * O^T = V^T P^T on v_mfma_f32_16x16x32_bf16 over a pair (k = 8h + s: token
//    4h + s of the first granule for s < 4, 4h + s - 4 of the second): the V
//    rows of both granules sit in the tile, and ds_read_b64_tr_b16 gives lane
//    l (within its 16-lane group, the lanes of one h) dim 16 db + l % 16 of
//    tokens 4h..4h+3 when source lane 4s + a points at row 4h + s, dims
//    16 db + 4a .. +3.  An odd last granule runs on 16x16x16 products.
template <int G>
struct MfmaBf16Engine {
    static_assert(G <= 16, "query heads per KV head");
    struct Buf { uint4 k[4], v[4]; };
    typedef u32x4_t Q[4];

    int lane, hq;
    unsigned char *vt;            // this wave's tile in LDS
    uint4 qv[4];
    f32x4_t o[8];                 // O^T blocks: lane l holds dims 16 db + 4 h + i of head l % 16
    float m, l;
    bool pending;
    float xp[4];                  // scaled, masked scores of the pending granule

    __device__ void setup(int ln, unsigned char *tile) {
        lane = ln;
        hq = ln >> 4;
        vt = tile;
    }

    __device__ void load(const kv_rsrc_t &rk, const kv_rsrc_t &rv, int row_bytes, Buf &b) const {
        const int off = (lane >> 4) * row_bytes + 16 * (lane & 15);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            b.k[u] = as_uint4(__builtin_amdgcn_raw_buffer_load_b128(rk, off + 4 * u * row_bytes, 0, kKvLoadPolicy));
            b.v[u] = as_uint4(__builtin_amdgcn_raw_buffer_load_b128(rv, off + 4 * u * row_bytes, 0, kKvLoadPolicy));
        }
    }

    __device__ void load_rows(const AttnArgs &, const int32_t *, int, int, int, int, int, Buf &) const {}

    // B operands of the four q.K products: dims 32 kk + 8h .. +7 of head l % 16.
    // Columns of heads >= G (never stored) repeat head G - 1.
    __device__ void load_q(const AttnArgs &a, int bb, int g, Q &qd) const {
        const int n = min(lane & 15, G - 1);
        const uint16_t *row = a.q + ((int64_t)bb * a.Hq + g * G + n) * kHeadDim;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) qd[kk] = *(const u32x4_t *)(row + 32 * kk + 8 * hq);
    }

    // q rows into a ring slot of G rows of 256 bytes, and back at piece start.
    __device__ void park_q(const Q &q, unsigned char *slot) const {
        unsigned char *row = slot + min(lane & 15, G - 1) * kQRowBytes + 16 * hq;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) *(u32x4_t *)(row + 64 * kk) = q[kk];
    }

    __device__ void start(const unsigned char *slot) {
        const unsigned char *row = slot + min(lane & 15, G - 1) * kQRowBytes + 16 * hq;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) qv[kk] = *(const uint4 *)(row + 64 * kk);
#pragma unroll
        for (int db = 0; db < 8; ++db) o[db] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
        m = -INFINITY;
        l = 0.0f;
        pending = false;
    }

    // V rows of a granule into tile half `half`.
    __device__ void stage_v(const Buf &b, int half) {
        unsigned char *row = vt + half * kVbHalf1 + (lane >> 4) * kVbRow + 16 * (lane & 15);
#pragma unroll
        for (int u = 0; u < 4; ++u) *(uint4 *)(row + 4 * u * kVbRow) = b.v[u];
    }

    template <bool MASK>
    __device__ void scores(const Buf &b, float sl, int nvalid, float (&x)[4]) const {
        unsigned char *kt = vt + kKbOffset;
        unsigned char *wr = kt + (lane >> 4) * kKbRow + 16 * (lane & 15);
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int u = 0; u < 4; ++u) *(uint4 *)(wr + 4 * u * kKbRow) = b.k[u];
        __builtin_amdgcn_wave_barrier();
        const unsigned char *rd = kt + (lane & 15) * kKbRow + 16 * hq;
        uint4 ka[4];
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) ka[kk] = *(const uint4 *)(rd + 64 * kk);
        __builtin_amdgcn_wave_barrier();
        f32x4_t s0 = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f}, s1 = s0;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            if (kk & 1) s1 = mfma16k32(ka[kk], qv[kk], s1);
            else s0 = mfma16k32(ka[kk], qv[kk], s0);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            x[i] = (s0[i] + s1[i]) * sl;
            if (MASK && 4 * hq + i >= nvalid) x[i] = -INFINITY;
        }
    }

    __device__ void rescale(float mx) {
        const bool up = mx > m + 8.0f;
        if (__ballot(up)) {
            const float mn = up ? mx : m;
            const float alpha = fast_exp2(m - mn);
            m = mn;
            l *= alpha;
#pragma unroll
            for (int db = 0; db < 8; ++db)
#pragma unroll
                for (int i = 0; i < 4; ++i) o[db][i] *= alpha;
        }
    }

    // this lane as a source of the transposing reads: row 4h + (l % 16) / 4 of
    // a half, dims 4 (l % 4) of a 16-dim block
    __device__ const unsigned char *tr_source() const {
        return vt + (4 * hq + ((lane & 15) >> 2)) * kVbRow + 8 * (lane & 3);
    }

    template <bool MASK>
    __device__ void step(Buf &b, float sl, int nvalid) {
        float x[4];
        scores<MASK>(b, sl, nvalid, x);
        if (!pending) {
            stage_v(b, 0);
#pragma unroll
            for (int i = 0; i < 4; ++i) xp[i] = x[i];
            pending = true;
            return;
        }
        stage_v(b, 1);
        pending = false;
        rescale(rows_max4(fmaxf(fmaxf(fmaxf(xp[0], xp[1]), fmaxf(xp[2], xp[3])),
                                fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])))));
        float p[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            p[i] = fast_exp2(xp[i] - m);
            p[4 + i] = fast_exp2(x[i] - m);
        }
        l += ((p[0] + p[1]) + (p[2] + p[3])) + ((p[4] + p[5]) + (p[6] + p[7]));
        uint32_t ph[4], pl[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) split_bf16_pair(p[2 * i], p[2 * i + 1], ph[i], pl[i]);
        const uint4 bh = make_uint4(ph[0], ph[1], ph[2], ph[3]);
        const uint4 bl = make_uint4(pl[0], pl[1], pl[2], pl[3]);
        __builtin_amdgcn_wave_barrier();
        const unsigned char *src = tr_source();
#pragma unroll
        for (int db = 0; db < 8; ++db) {
            const uint2 lo = read_tr16((const uint16_t *)(src + 32 * db));
            const uint2 hi = read_tr16((const uint16_t *)(src + kVbHalf1 + 32 * db));
            const uint4 av = make_uint4(lo.x, lo.y, hi.x, hi.y);
            o[db] = mfma16k32(av, bh, o[db]);
            o[db] = mfma16k32(av, bl, o[db]);
        }
        __builtin_amdgcn_wave_barrier();
    }

    // The pending granule alone: P.V over its 16 tokens.
    __device__ void flush() {
        if (!pending) return;
        pending = false;
        rescale(rows_max4(fmaxf(fmaxf(xp[0], xp[1]), fmaxf(xp[2], xp[3]))));
        float p[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) p[i] = fast_exp2(xp[i] - m);
        l += (p[0] + p[1]) + (p[2] + p[3]);
        uint32_t ph[2], pl[2];
        split_bf16_pair(p[0], p[1], ph[0], pl[0]);
        split_bf16_pair(p[2], p[3], ph[1], pl[1]);
        const uint2 bh = make_uint2(ph[0], ph[1]), bl = make_uint2(pl[0], pl[1]);
        __builtin_amdgcn_wave_barrier();
        const unsigned char *src = tr_source();
#pragma unroll
        for (int db = 0; db < 8; ++db) {
            const uint2 av = read_tr16((const uint16_t *)(src + 32 * db));
            o[db] = mfma16k16(av, bh, o[db]);
            o[db] = mfma16k16(av, bl, o[db]);
        }
        __builtin_amdgcn_wave_barrier();
    }

    __device__ void finish(float v_scale, float *o_base, float *l_base, int h0) {
        flush();
        const int n = lane & 15;
        const float lt = rows_sum4(l);
        const float inv = lt > 0.0f ? v_scale / lt : 0.0f;
        if (n < G) {
            float *dst = o_base + (h0 + n) * kHeadDim + 4 * hq;
#pragma unroll
            for (int db = 0; db < 8; ++db)
                *(float4 *)(dst + 16 * db) = make_float4(o[db][0] * inv, o[db][1] * inv, o[db][2] * inv,
                                                          o[db][3] * inv);
            if (hq == 0 && l_base) l_base[h0 + n] = lt > 0.0f ? (m + fast_log2(lt)) * kLn2 : -INFINITY;
        }
    }
};

template <int G, int LAYOUT, int KV> struct EngineFor { typedef DotEngine<G, KV> type; };
template <int G> struct EngineFor<G, kContig, kKvFp8> { typedef MfmaFp8Engine<G> type; };
template <int G> struct EngineFor<G, kPagedWide, kKvFp8> { typedef MfmaFp8Engine<G> type; };
template <int G> struct EngineFor<G, kContig, kKvBf16> { typedef MfmaBf16Engine<G> type; };
template <int G> struct EngineFor<G, kPagedWide, kKvBf16> { typedef MfmaBf16Engine<G> type; };

template <int G, int LAYOUT, int KV>
__device__ __forceinline__ void stream_work(const AttnArgs &a, const Split &sp, const int64_t *pre,
                                            const int32_t *len, const int32_t *nseg, int32_t *win,
                                            unsigned char *tile, unsigned char *qring, int g0, int64_t i0,
                                            int lane) {
    typedef typename EngineFor<G, LAYOUT, KV>::type E;
    typedef typename E::Buf Buf;
    constexpr int EB = KvChunk<KV>::kBytes;
    constexpr bool kPaged = LAYOUT != kContig;
    const int Hkv = a.Hkv;
    E eng;
    eng.setup(lane, tile);
    const int lp = a.log2_page;
    const int row_bytes = Hkv * kHeadDim * EB;
    const float sl = a.scale_log2;

    // ---- resolver: pieces of the wave's range, cut into window segments
    int64_t ru, ru1;                  // flat part of the range still to cut
    const int64_t rprod = i0;         // producer index of the range
    const int rg = g0;
    // (64-bit divisions are expanded into vector code: keep their results in
    // scalar registers, or every address derived from them would be treated
    // as per-lane)
    ru = uniform_i64(sp.x(i0));
    ru1 = uniform_i64(sp.x(i0 + 1));
    int rb = find_seq(pre, a.B, ru);
    // piece being cut
    int pb = 0, pgl = 0, pgl1 = 0, pL = 0, pnseg = 0;
    bool have_piece = false, pfirst = false;
    int64_t pslot = 0;

    // Next piece; false when the wave's work is done.
    auto next_piece = [&]() -> bool {
        int64_t st, en;
        for (;;) {
            if (ru >= ru1) return false;
            st = uniform_i64(pre[rb]);
            en = uniform_i64(pre[rb + 1]);
            while (en <= ru && rb + 1 < a.B) {
                ++rb;
                st = en;
                en = uniform_i64(pre[rb + 1]);
            }
            // the sequence's virtual granules come first and carry no work
            st += en > st ? a.vgran : 0;
            if (ru >= st) break;
            ru = min(st, ru1);
        }
        pb = rb;
        pL = uniform_i32(len[rb]);
        const int lo = (pL + kGranule - 1) / kGranule - (int)(en - st);
        const int64_t pe = min(ru1, en);
        pgl = (int)(ru - st) + lo;
        pgl1 = (int)(pe - st) + lo;
        pslot = rprod + rb;
        pnseg = a.pref ? 0 : uniform_i32(nseg[rb]);
        ru = pe;
        have_piece = true;
        pfirst = true;
        return true;
    };

    // Next segment (kSegValid clear when none is left).
    auto next_segment = [&]() -> Seg {
        Seg s{};
        if (!have_piece && !next_piece()) return s;
        s.b = pb;
        s.g = rg;
        s.gl0 = pgl;
        s.L = pL;
        s.nseg = pnseg;
        s.slot = pslot;
        int end = pgl1;
        if (kPaged) {
            s.pbase = (pgl * kGranule) >> lp;
            // granules the window's pages hold
            const int64_t wend = lp >= 4 ? ((int64_t)(s.pbase + kPageWin) << (lp - 4))
                                         : (int64_t)pgl + ((int64_t)kPageWin << lp) / kGranule;
            if (wend < end) end = (int)wend;
        }
        s.gl1 = end;
        s.flags = kSegValid | (pfirst ? kSegFirst : 0) | (end == pgl1 ? kSegLast : 0);
        pgl = end;
        pfirst = false;
        if (end == pgl1) have_piece = false;
        return s;
    };

    // Page ids of a segment's window, sanitised: into registers (four per lane) ...
    auto fetch_window = [&](const Seg &s, int32_t (&w)[kPageWin / 64]) {
#pragma unroll
        for (int k = 0; k < kPageWin / 64; ++k) {
            const int e = s.pbase + 64 * k + lane;
            const int32_t p = e < a.max_pages ? a.block_table[(int64_t)s.b * a.max_pages + e] : 0;
            w[k] = sanitize_page(p, a.num_pages);
        }
    };
    // ... and from registers into LDS buffer `buf`.
    auto store_window = [&](int buf, const int32_t (&w)[kPageWin / 64]) {
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int k = 0; k < kPageWin / 64; ++k) win[buf * kPageWin + 64 * k + lane] = w[k];
        __builtin_amdgcn_wave_barrier();
    };

    // ---- load cursor: segment Ln, granule gl.  The values the loads need are
    // kept apart: head byte offset, window base, length.
    Seg Ln = next_segment();
    // a range of virtual granules only holds no work (and its invalid segment
    // has no live row for the narrow-page loads to fall back on)
    if (!(Ln.flags & kSegValid)) return;
    int wb = 0;
    int32_t wv[kPageWin / 64];
    if (kPaged) {
        fetch_window(Ln, wv);
        store_window(0, wv);
    }
    // q ring: the q rows of a piece are loaded into qt when the load cursor
    // enters it and parked in LDS slot qpar at the end of the next compute
    // step.  That step always belongs to an earlier piece (computing trails
    // loading by at least one granule, and every entry is followed by a
    // compute step before the next one), and the piece two entries back,
    // which used the same slot, is finished by then.
    typename E::Q qt;
    int qpar = 0;
    bool q_park = false;
    eng.load_q(a, Ln.b, Ln.g, qt);
    int gl = Ln.gl0;
    Seg N{};
    bool n_ready = false;

    // Issue the K/V loads of granule x of the load segment.  Rows past the
    // length are not read: the buffer range stops after the last live row
    // (out-of-range lanes read zeros), and the narrow-page path re-reads the
    // last live row; the compute step masks them.
    auto load_gran = [&](int x, Buf &buf) {
        const int t0 = x * kGranule;
        const int nvalid = min(kGranule, Ln.L - t0);
        if (LAYOUT == kPagedNarrow) {
            eng.load_rows(a, win + wb * kPageWin, Ln.pbase, t0, nvalid, Ln.g, lp, buf);
        } else {
            int64_t row0;
            if (LAYOUT == kContig) {
                row0 = (int64_t)Ln.b * a.seq_stride + t0;
            } else {
                const int64_t page = uniform_i32(win[wb * kPageWin + ((t0 >> lp) - Ln.pbase)]);
                row0 = pool_row(page, t0, lp);
            }
            // (uniform by construction; made explicit so the descriptor stays in
            // scalar registers)
            const int64_t base = uniform_i64(row0 * row_bytes + (int64_t)Ln.g * kHeadDim * EB);
            // (a load issued after the wave's last granule, which only keeps
            // the pipeline's shape, gets an empty range: nothing is fetched)
            const int range = uniform_i32((Ln.flags & kSegValid) ? (nvalid - 1) * row_bytes + kHeadDim * EB : 0);
            const kv_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(
                (void *)((const char *)a.k + base), 0, range, kBufferFlags);
            const kv_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
                (void *)((const char *)a.v + base), 0, range, kBufferFlags);
            eng.load(rk, rv, row_bytes, buf);
        }
    };

    auto make_tag = [&]() -> Tag {
        Tag t;
        t.flags = Ln.flags & kSegValid;
        t.nvalid = min(kGranule, Ln.L - gl * kGranule);
        if (gl == Ln.gl0 && (Ln.flags & kSegFirst)) t.flags |= kSegFirst;
        if (gl == Ln.gl1 - 1 && (Ln.flags & kSegLast)) t.flags |= kSegLast;
        t.b = Ln.b;
        t.g = Ln.g;
        t.nseg = Ln.nseg;
        t.slot = Ln.slot;
        t.qpar = qpar;
        return t;
    };

    // ---- look-ahead.  The segment after Ln is resolved (and its page ids
    // fetched) as soon as Ln is entered.
    auto resolve = [&]() {
        N = next_segment();
        if (kPaged && (N.flags & kSegValid)) fetch_window(N, wv);
        n_ready = true;
    };
    // Look-ahead action due with the load cursor at gl.
    auto events = [&]() {
        if (!n_ready && gl >= Ln.gl0) resolve();
    };
    // Load index of the next look-ahead action (INT_MAX if none).
    auto next_event = [&]() -> int { return n_ready ? 0x7fffffff : Ln.gl0; };

    // Move the load cursor one granule on (after each compute step of the
    // general path).
    auto advance = [&]() {
        if (!(Ln.flags & kSegValid)) return;
        ++gl;
        events();
        if (gl >= Ln.gl1) {
            if (!n_ready) resolve();
            if (N.flags & kSegValid) {
                if (kPaged) {
                    wb ^= 1;
                    store_window(wb, wv);
                }
                if (N.flags & kSegFirst) {
                    qpar ^= 1;
                    eng.load_q(a, N.b, N.g, qt);
                    q_park = true;
                }
                Ln = N;
                gl = N.gl0;
                n_ready = false;
                events();
            } else {
                // no work left: further loads repeat the last granule, untagged
                Ln.flags = 0;
                gl = Ln.gl1 - 1;
            }
        }
    };

    // General compute step: starts and ends pieces, masks partial granules.
    auto compute = [&](const Tag &t, Buf &buf) {
        if (t.flags & kSegFirst) eng.start(qring + t.qpar * G * kQRowBytes);
        eng.template step<true>(buf, sl, t.nvalid);
        if (t.flags & kSegLast) {
            // a sequence covered by one piece is written to the output directly
            const bool single = t.nseg == 1;
            float *o_base = single ? a.out + (int64_t)t.b * a.Hq * kHeadDim : a.o_ws + t.slot * a.Hq * kHeadDim;
            float *l_base = single ? (a.lse ? a.lse + (int64_t)t.b * a.Hq : nullptr) : a.lse_ws + t.slot * a.Hq;
            eng.finish(a.v_scale, o_base, l_base, t.g * G);
        }
        if (q_park) {
            eng.park_q(qt, qring + qpar * G * kQRowBytes);
            q_park = false;
        }
    };

    // ---- the stream: the loads of the next granule are issued before the
    // current one is consumed.  At the top of the loop the current granule is
    // in (ka, va) with tag ta, and gl is the next granule to load.
    Buf A, B;
    Tag ta = make_tag(), tb;
    load_gran(gl, A);
    eng.park_q(qt, qring);
    events();
    advance();
    // a wave never handles more granules than the whole batch holds: a bound
    // every wave reaches even if the decomposition were inconsistent
    int64_t budget = sp.gtot * Hkv + 2;
    while (--budget > 0) {
        // Plain pairs (no tags, no branches; loads one granule ahead) while both
        // loads stay inside Ln and neither is its piece's first or last
        // granule; look-ahead actions run between pairs.
        if (ta.flags == kSegValid && ta.nvalid == kGranule && (Ln.flags & kSegValid)) {
            const int first_gl = uniform_i32((Ln.flags & kSegFirst) ? Ln.gl0 : -1);
            const int lim = uniform_i32(Ln.gl1 - 3);
            gl = uniform_i32(gl);
            while (gl > first_gl && gl <= lim) {
                const int stop = uniform_i32(min(lim, next_event() - 1));
                while (gl <= stop) {
                    load_gran(gl, B);
                    __builtin_amdgcn_sched_barrier(0);
                    eng.template step<false>(A, sl, kGranule);
                    load_gran(gl + 1, A);
                    __builtin_amdgcn_sched_barrier(0);
                    eng.template step<false>(B, sl, kGranule);
                    gl += 2;
                }
                if (gl <= lim) events();
            }
        }
        // a pair of general steps (the buffers are used in turn, so the current
        // granule is back in (ka, va) afterwards)
        tb = make_tag();
        load_gran(gl, B);
        __builtin_amdgcn_sched_barrier(0);
        if (!(ta.flags & kSegValid)) break;
        compute(ta, A);
        advance();
        ta = make_tag();
        load_gran(gl, A);
        __builtin_amdgcn_sched_barrier(0);
        if (!(tb.flags & kSegValid)) break;
        compute(tb, B);
        advance();
    }
}

// The matrix-core kernels are held to 256 registers (two waves per SIMD; fp8
// runs two per SIMD, and bf16, at one wave per SIMD, measured slower
// compiled without the cap: 183.2 vs 181.9 us on 64 rollouts of 512-8192
// tokens).
template <int LAYOUT, int KV> constexpr int attn_waves_per_simd() {
    return LAYOUT != kPagedNarrow ? 2 : 1;
}

template <int G, int LAYOUT, int KV>
__global__ __launch_bounds__(kWavesPerBlock * 64)
__attribute__((amdgpu_waves_per_eu(attn_waves_per_simd<LAYOUT, KV>()))) void decode_attn_kernel(const AttnArgs a) {
    extern __shared__ __align__(16) unsigned char s_dyn[];
    __shared__ int64_t s_wsum[kWavesPerBlock];
    int64_t *pre = reinterpret_cast<int64_t *>(s_dyn);
    int32_t *len = reinterpret_cast<int32_t *>(s_dyn + attn_lds_len_offset(a.B));
    int32_t *nseg = reinterpret_cast<int32_t *>(s_dyn + attn_lds_nseg_offset(a.B));
    build_tables(a, pre, len, s_wsum);

    Split sp;
    sp.gtot = uniform_i64(pre[a.B]);
    // at least two granules per range, so tiny batches are not shredded (larger
    // minimum ranges measured slower on every config: parallelism wins)
    sp.wh = uniform_i64(min((int64_t)a.waves_per_head, (sp.gtot + 1) / 2));
    sp.wa = a.w_even;
    sp.wb = a.w_odd;
    // weighted ranges only while the lightest still holds a granule (range i
    // has at least floor(gtot w_i / wsum(wh)) granules): an empty range would
    // leave a merge slot between a sequence's pieces unwritten
    if (sp.gtot * min(sp.wa, sp.wb) < sp.wsum(sp.wh)) sp.wa = sp.wb = 1;
    // pieces of each sequence (1: its result goes straight to the output)
    for (int b = threadIdx.x; b < a.B; b += kWavesPerBlock * 64) {
        const int64_t en = pre[b + 1];
        const int64_t st = pre[b] + (en > pre[b] ? a.vgran : 0);   // first real granule
        nseg[b] = en > st ? (int)(sp.producer_of(en - 1) - sp.producer_of(st) + 1) : 0;
    }
    __syncthreads();

    const int lane = threadIdx.x & 63;
    int32_t *win = reinterpret_cast<int32_t *>(s_dyn + attn_lds_win_offset(a.B)) +
                   (threadIdx.x >> 6) * 2 * kPageWin;
    // Blocks go to the XCDs round-robin (block id mod 8).  With xcd_map the
    // waves of the even blocks and those of the odd blocks are each numbered
    // (KV head, range pair), and a wave's range index has its block's parity,
    // so every KV head has half its ranges on even XCDs and half on odd ones;
    // otherwise waves are numbered (range, KV head) in block order.
    int g, i;
    if (a.xcd_map) {
        const int wp = uniform_i32((int)(blockIdx.x >> 1) * kWavesPerBlock + (threadIdx.x >> 6));
        g = wp % a.Hkv;
        i = 2 * (wp / a.Hkv) + (int)(blockIdx.x & 1);
    } else {
        const int wave = uniform_i32((int)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6));
        g = wave % a.Hkv;
        i = wave / a.Hkv;
    }
    if (i >= a.waves_per_head) return;

    // Empty sequences own no granule: the first wave of each KV head writes
    // their outputs (zeros, lse = -inf) for that head's query heads.  (In
    // grouped calls the merge kernel writes every output.)
    if (i == 0 && !a.pref) {
        for (int b0 = 0; b0 < a.B; b0 += 64) {
            const int b = b0 + lane;
            uint64_t empty = __ballot(b < a.B && len[b] == 0);
            while (empty) {
                const int be = b0 + (int)__builtin_ctzll(empty);
                empty &= empty - 1;
                for (int j = 0; j < G; ++j) {
                    const int64_t row = (int64_t)be * a.Hq + g * G + j;
                    *(float2 *)(a.out + row * kHeadDim + 2 * lane) = make_float2(0.0f, 0.0f);
                    if (a.lse && lane == 0) a.lse[row] = -INFINITY;
                }
            }
        }
    }
    if (g == 0 && i == 0) write_plan(a, sp, pre, lane);
    if ((int64_t)i >= sp.wh) return;
    unsigned char *tile = s_dyn + attn_lds_tile_offset(a.B) + (threadIdx.x >> 6) * attn_tile_bytes(KV);
    unsigned char *qring = s_dyn + attn_lds_q_offset(a.B, KV) + (threadIdx.x >> 6) * 2 * G * kQRowBytes;
    stream_work<G, LAYOUT, KV>(a, sp, pre, len, nseg, win, tile, qring, g, i, lane);
}

// ---- merge of split sequences after the attention kernel: one wave per
// (sequence, query head); sequences with no plan entry were written directly

__global__ __launch_bounds__(256) void merge_split_kernel(const MergeArgs a) {
    const int lane = threadIdx.x & 63;
    const int64_t w = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (w >= (int64_t)a.B * a.Hq) return;
    const int b = (int)(w / a.Hq);
    const int h = (int)(w % a.Hq);
    const int2 pl = a.plan[b];
    if (pl.y == 0) return;
    merge_parts(a.o_ws + ((int64_t)pl.x * a.Hq + h) * kHeadDim, (int64_t)a.Hq * kHeadDim,
                a.lse_ws + (int64_t)pl.x * a.Hq + h, a.Hq, pl.y, kHeadDim,
                a.out + w * kHeadDim, a.lse ? a.lse + w : nullptr, lane);
}

// ---- public merge entry point: one wave per (sequence, query head)

__global__ __launch_bounds__(256) void combine_kernel(const CombineArgs a) {
    const int lane = threadIdx.x & 63;
    const int64_t w = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (w >= (int64_t)a.B * a.Hq) return;
    const int64_t bh = w;
    merge_parts(a.o_parts + bh * a.D, (int64_t)a.B * a.Hq * a.D, a.lse_parts + bh,
                (int64_t)a.B * a.Hq, a.S, a.D, a.out + bh * a.D, a.lse ? a.lse + bh : nullptr, lane);
}

// ---- page-table gather hook: one thread per 16-byte chunk of the dense output

__global__ __launch_bounds__(256) void gather_kernel(const GatherArgs a) {
    const int chunks = a.D / 8;
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t total = (int64_t)a.B * a.Lcap * a.Hkv * chunks;
    if (idx >= total) return;
    const int c = (int)(idx % chunks);
    int64_t rest = idx / chunks;
    const int g = (int)(rest % a.Hkv);
    rest /= a.Hkv;
    const int t = (int)(rest % a.Lcap);
    const int b = (int)(rest / a.Lcap);
    const int cap = (int)min((int64_t)a.max_pages << a.log2_page, (int64_t)a.Lcap);
    const int L = clamp_len(a.seq_lens[b], cap);
    uint4 val = make_uint4(0u, 0u, 0u, 0u);
    if (t < L) {
        const int64_t page = page_of(a.block_table, b, a.max_pages, t, a.log2_page, a.num_pages);
        val = *(const uint4 *)(a.pool + (pool_row(page, t, a.log2_page) * a.Hkv + g) * a.D + 8 * c);
    }
    *(uint4 *)(a.dst + (((int64_t)b * a.Lcap + t) * a.Hkv + g) * a.D + 8 * c) = val;
}

template <int G, int LAYOUT, int KV>
const void *attn_kernel_ptr() {
    return (const void *)&decode_attn_kernel<G, LAYOUT, KV>;
}

template <int LAYOUT, int KV>
const void *attn_kernel_for_group(int group) {
    switch (group) {
        case 1: return attn_kernel_ptr<1, LAYOUT, KV>();
        case 2: return attn_kernel_ptr<2, LAYOUT, KV>();
        case 4: return attn_kernel_ptr<4, LAYOUT, KV>();
        case 8: return attn_kernel_ptr<8, LAYOUT, KV>();
        default: return nullptr;
    }
}

template <int KV>
const void *attn_kernel_for_layout(int layout, int group) {
    switch (layout) {
        case kContig: return attn_kernel_for_group<kContig, KV>(group);
        case kPagedWide: return attn_kernel_for_group<kPagedWide, KV>(group);
        case kPagedNarrow: return attn_kernel_for_group<kPagedNarrow, KV>(group);
        default: return nullptr;
    }
}

const void *attn_kernel(int layout, int group, int kv) {
    switch (kv) {
        case kKvBf16: return attn_kernel_for_layout<kKvBf16>(layout, group);
        case kKvFp8: return attn_kernel_for_layout<kKvFp8>(layout, group);
        default: return nullptr;
    }
}

}  // namespace

hipError_t launch_decode_attn(const AttnArgs &a, int layout, int group, int kv, int blocks,
                              hipStream_t stream) {
    const void *fn = attn_kernel(layout, group, kv);
    if (!fn) return hipErrorInvalidValue;
    void *args[] = {(void *)&a};
    return hipLaunchKernel(fn, dim3(blocks), dim3(kWavesPerBlock * 64), args,
                           (size_t)attn_lds_bytes(a.B, group, kv), stream);
}

hipError_t launch_combine(const CombineArgs &a, hipStream_t stream) {
    const int64_t waves = (int64_t)a.B * a.Hq;
    if (waves == 0) return hipSuccess;
    const int64_t blocks = (waves + 3) / 4;
    hipLaunchKernelGGL(combine_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, a);
    return hipGetLastError();
}

hipError_t launch_merge_split(const MergeArgs &a, hipStream_t stream) {
    const int64_t waves = (int64_t)a.B * a.Hq;
    if (waves == 0) return hipSuccess;
    const int64_t blocks = (waves + 3) / 4;
    hipLaunchKernelGGL(merge_split_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, a);
    return hipGetLastError();
}

hipError_t launch_gather(const GatherArgs &a, hipStream_t stream) {
    const int64_t total = (int64_t)a.B * a.Lcap * a.Hkv * (a.D / 8);
    if (total == 0) return hipSuccess;
    const int64_t blocks = (total + 255) / 256;
    hipLaunchKernelGGL(gather_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, a);
    return hipGetLastError();
}

hipError_t attn_waves_per_cu(int layout, int group, int kv, int *waves) {
    const void *fn = attn_kernel(layout, group, kv);
    if (!fn) return hipErrorInvalidValue;
    int blocks = 0;
    hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
        &blocks, fn, kWavesPerBlock * 64, (size_t)attn_lds_bytes(1, group, kv));
    if (e != hipSuccess) return e;
    *waves = blocks * kWavesPerBlock;
    return hipSuccess;
}

}  // namespace kva
