// HIP kernels for batched grouped-query decode attention on gfx950 (MI355X).
//
// Work decomposition.  The granules (16-token steps) of all sequences are laid
// end to end in one flat index space of length Gtot.  Each KV head g gets Wh
// waves; wave (i, g) takes the contiguous granule range
// [i*Gtot/Wh, (i+1)*Gtot/Wh), which may start inside one sequence and end
// inside another.  Every piece of a sequence a wave covers becomes one partial
// result (normalised output + log-sum-exp) for the G query heads of g, stored
// in slot i + b; a second kernel merges the partials of each sequence in slot
// order.  Every wave thus streams the same number of K/V bytes whatever the
// mix of lengths, and the grid is sized to the waves the device keeps
// resident, so there is no tail of idle compute units.
//
// Inside a wave.  Lane (r, c) = (lane / 16, lane % 16) owns 16 bytes (8 bf16,
// dims 8c..8c+7) of the 256-byte K and V rows of tokens r, r+4, r+8, r+12 of
// the current granule: one 16-byte load per lane fetches four whole rows with
// full 64-byte segments per row quarter.  q.K partials are formed with the
// bf16 dot2 instruction and summed over the 16 lanes of a DPP row; each of the
// four token rows runs its own online softmax (running max m, sum l, output
// accumulator) in fp32 so no cross-row exchange sits in the inner loop.  The
// four row states are merged once per piece with the log-sum-exp identity.
// The next granule's K/V loads are issued before the current one is consumed.

#include "kva_internal.h"
#include "kva_device.h"

namespace kva {
namespace {

using namespace dev;

// First granule of sequence b this kernel attends: past the group's shared
// run in grouped calls, else 0.
__device__ __forceinline__ int gran_lo(const AttnArgs &a, int b) {
    return a.pref ? a.pref[b / a.group] : 0;
}

// Granules of sequence b this kernel attends.
__device__ __forceinline__ int seq_granules(const AttnArgs &a, int b) {
    return (clamp_len(a.seq_lens[b], a.cap) + kGranule - 1) / kGranule - gran_lo(a, b);
}


// ---- merge plan for the second kernel, written by wave 0: per sequence
// {first slot, number of pieces}; 0 pieces for sequences written directly
// (one piece, or empty)

__device__ void write_plan(const AttnArgs &a, int64_t gtot, int64_t wh, int lane) {
    int64_t base = 0;
    for (int b0 = 0; b0 < a.B; b0 += 64) {
        const int b = b0 + lane;
        const int n = b < a.B ? seq_granules(a, b) : 0;
        const int64_t incl = base + wave_incl_scan(n, lane);
        const int64_t st = incl - n;
        if (b < a.B) {
            int2 pl = make_int2(0, 0);
            if (n > 0) {
                // the wave holding granule y is ((y + 1) * wh - 1) / gtot
                const int64_t first = ((st + 1) * wh - 1) / gtot;
                const int64_t last = (incl * wh - 1) / gtot;
                if (last > first || a.pref) pl = make_int2((int)(first + b), (int)(last - first + 1));
            }
            a.plan[b] = pl;
        }
        base = lane_i64(incl, 63);
    }
}

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


// Page ids of the current chunk of a piece: a per-wave window of kPageWin
// consecutive block-table entries in LDS, filled before the chunk's granule
// loop starts.  LDS reads are counted apart from vector-memory loads, so a page
// lookup never forces a wait on K/V loads in flight, and the hot loop holds no
// branch around a vector-memory load.
constexpr int kPageWin = 256;

// Fill ids[0 .. kPageWin) with (sanitised) entries first .. first+kPageWin-1
// of sequence b's block-table row.
__device__ __forceinline__ void window_fill(const AttnArgs &a, int32_t *ids, int b, int first,
                                            int lane) {
    __builtin_amdgcn_wave_barrier();           // every lane is done with the old window
#pragma unroll
    for (int k = 0; k < kPageWin / 64; ++k) {
        const int e = first + 64 * k + lane;
        const int32_t p = e < a.max_pages ? a.block_table[(int64_t)b * a.max_pages + e] : 0;
        ids[64 * k + lane] = sanitize_page(p, a.num_pages);
    }
    __builtin_amdgcn_wave_barrier();
}

// Issue the K and V loads of granule gl (tokens gl*16 .. gl*16+15) of sequence b.
// Positions at or past L are redirected to L-1 (always a live row) and masked
// later.  Paged layouts read page ids from the window (page index `pbase` at ids[0]).
// FULL: the granule is known to hold 16 live positions, so the per-lane
// offsets do not depend on the length and stay in registers across granules.
template <int LAYOUT, bool FULL, int KV>
__device__ __forceinline__ void load_granule(const AttnArgs &a, const int32_t *ids, int pbase,
                                             int b, int g, int gl, int L, int lane,
                                             typename KvChunk<KV>::type (&kd)[4],
                                             typename KvChunk<KV>::type (&vd)[4]) {
    typedef typename KvChunk<KV>::type C;
    constexpr int EB = KvChunk<KV>::kBytes;
    const int r = lane >> 4;
    const int c = lane & 15;
    const int t0 = gl * kGranule;
    const int lim = FULL ? kGranule - 1 : L - 1 - t0;  // >= 0 for every granule of the sequence
    const int Hkv = a.Hkv;
    if (LAYOUT == kPagedNarrow) {
        const int lp = a.log2_page;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int tt = t0 + min(4 * u + r, lim);
            const int64_t page = ids[(tt >> lp) - pbase];
            const int64_t off = ((pool_row(page, tt, lp) * Hkv + g) * kHeadDim + 8 * c) * EB;
            kd[u] = *(const C *)((const char *)a.k + off);
            vd[u] = *(const C *)((const char *)a.v + off);
        }
    } else {
        int64_t row0;
        if (LAYOUT == kContig) {
            row0 = (int64_t)b * a.seq_stride + t0;
        } else {
            const int64_t page = __builtin_amdgcn_readfirstlane(ids[(t0 >> a.log2_page) - pbase]);
            row0 = pool_row(page, t0, a.log2_page);
        }
        // Buffer loads: a descriptor (in scalar registers) whose base is the
        // granule's first row of head g and whose range is the granule's 16
        // rows, plus a per-lane byte offset that is the same for every full
        // granule.  An offset outside the range would read zeros, not fault.
        const int64_t row_bytes = (int64_t)Hkv * kHeadDim * EB;
        const int64_t base = row0 * row_bytes + (int64_t)g * kHeadDim * EB;
        const int range = (int)(kGranule * row_bytes);
        const kv_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc((void *)((const char *)a.k + base), 0,
                                                               range, kBufferFlags);
        const kv_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc((void *)((const char *)a.v + base), 0,
                                                               range, kBufferFlags);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int off = min(4 * u + r, lim) * (int)row_bytes + 8 * EB * c;
            if constexpr (KV == kKvBf16) {
                kd[u] = as_uint4(__builtin_amdgcn_raw_buffer_load_b128(rk, off, 0, kKvLoadPolicy));
                vd[u] = as_uint4(__builtin_amdgcn_raw_buffer_load_b128(rv, off, 0, kKvLoadPolicy));
            } else {
                const u32x2_t k2 = __builtin_amdgcn_raw_buffer_load_b64(rk, off, 0, kKvLoadPolicy);
                const u32x2_t v2 = __builtin_amdgcn_raw_buffer_load_b64(rv, off, 0, kKvLoadPolicy);
                kd[u] = make_uint2(k2.x, k2.y);
                vd[u] = make_uint2(v2.x, v2.y);
            }
        }
    }
}

// Granules [gl0, gl1) of sequence b for KV head g; result into slot `slot`,
// or, if the sequence is covered by this one piece (nseg == 1), into the output.
template <int G, int LAYOUT, int KV>
__device__ __forceinline__ void attend_piece(const AttnArgs &a, int32_t *ids, int b, int g,
                                             int gl0, int gl1, int L, int64_t slot, int nseg,
                                             int lane) {
    const int r = lane >> 4;
    const int c = lane & 15;
    const int h0 = g * G;

    uint32_t qv[G][4];
#pragma unroll
    for (int j = 0; j < G; ++j) {
        const uint4 t = *(const uint4 *)(a.q + ((int64_t)b * a.Hq + h0 + j) * kHeadDim + 8 * c);
        qv[j][0] = t.x; qv[j][1] = t.y; qv[j][2] = t.z; qv[j][3] = t.w;
    }
    float m[G], l[G], acc[G][8];
#pragma unroll
    for (int j = 0; j < G; ++j) {
        m[j] = -INFINITY;
        l[j] = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[j][e] = 0.0f;
    }
    const float sl = a.scale_log2;
    // The last granule of the sequence is partly empty unless L is a multiple
    // of 16; it can only be the last granule of the piece.
    const bool has_tail = (L % kGranule) != 0 && gl1 == (L + kGranule - 1) / kGranule;
    const int full_end = has_tail ? gl1 - 1 : gl1;
    // granules per chunk: one window of page ids (every granule of a contiguous
    // cache in one chunk)
    const int chunk = (LAYOUT == kContig) ? (1 << 30) : ((kPageWin << a.log2_page) / kGranule);

    typename KvChunk<KV>::type ka[4], va[4], kb[4], vb[4];
    for (int c0 = gl0; c0 < gl1; c0 += chunk) {
        const int c1 = min(gl1, c0 + chunk);
        const int cfull = min(c1, full_end);
        int pbase = 0;
        if (LAYOUT != kContig) {
            pbase = (c0 * kGranule) >> a.log2_page;
            window_fill(a, ids, b, pbase, lane);
        }
        // Pipelined loop over the chunk's full granules: the loads of the next
        // granule (clamped to the chunk's last one) are issued before the
        // current granule is consumed.
        if (c0 < cfull)
            load_granule<LAYOUT, true, KV>(a, ids, pbase, b, g, c0, L, lane, ka, va);
        else
            load_granule<LAYOUT, false, KV>(a, ids, pbase, b, g, c0, L, lane, ka, va);
        int gl = c0;
        for (; gl + 2 <= cfull; gl += 2) {
            load_granule<LAYOUT, true, KV>(a, ids, pbase, b, g, gl + 1, L, lane, kb, vb);
            // keep the scheduler from sinking the loads below the arithmetic
            __builtin_amdgcn_sched_barrier(0);
            attend_step<G, false>(qv, ka, va, m, l, acc, sl, r, kGranule);
            load_granule<LAYOUT, true, KV>(a, ids, pbase, b, g, min(gl + 2, cfull - 1), L, lane, ka, va);
            __builtin_amdgcn_sched_barrier(0);
            attend_step<G, false>(qv, kb, vb, m, l, acc, sl, r, kGranule);
        }
        // At most one full granule (held in ka/va) and the masked tail remain.
        if (gl < cfull) {
            load_granule<LAYOUT, false, KV>(a, ids, pbase, b, g, min(gl + 1, c1 - 1), L, lane, kb, vb);
            __builtin_amdgcn_sched_barrier(0);
            attend_step<G, false>(qv, ka, va, m, l, acc, sl, r, kGranule);
            if (gl + 1 < c1)
                attend_step<G, true>(qv, kb, vb, m, l, acc, sl, r, L - (gl + 1) * kGranule);
        } else if (gl < c1) {
            // only the tail is left; unless it is the chunk's first granule, ka/va
            // hold a prefetch clamped to the last full granule: load the tail
            if (gl != c0) load_granule<LAYOUT, false, KV>(a, ids, pbase, b, g, gl, L, lane, ka, va);
            attend_step<G, true>(qv, ka, va, m, l, acc, sl, r, L - gl * kGranule);
        }
    }

    // Merge the four token rows and store this piece's partial result.  A
    // sequence covered by one piece is written to the output directly.
    const bool single = nseg == 1;
    float *o_base = single ? a.out + (int64_t)b * a.Hq * kHeadDim : a.o_ws + slot * a.Hq * kHeadDim;
    float *l_base = single ? (a.lse ? a.lse + (int64_t)b * a.Hq : nullptr) : a.lse_ws + slot * a.Hq;
#pragma unroll
    for (int j = 0; j < G; ++j) {
        float M = fmaxf(m[j], __shfl_xor(m[j], 16, 64));
        M = fmaxf(M, __shfl_xor(M, 32, 64));
        const float Ms = (M == -INFINITY) ? 0.0f : M;
        const float w = fast_exp2(m[j] - Ms);
        float lj = l[j] * w;
        lj += __shfl_xor(lj, 16, 64);
        lj += __shfl_xor(lj, 32, 64);
        float o[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            float t = acc[j][e] * w;
            t += __shfl_xor(t, 16, 64);
            t += __shfl_xor(t, 32, 64);
            o[e] = lj > 0.0f ? t / lj : 0.0f;
            if constexpr (KV == kKvFp8) o[e] *= a.v_scale;
        }
        if (r == 0) {
            float4 *dst = (float4 *)(o_base + (h0 + j) * kHeadDim + 8 * c);
            dst[0] = make_float4(o[0], o[1], o[2], o[3]);
            dst[1] = make_float4(o[4], o[5], o[6], o[7]);
        }
        if (lane == 0 && l_base) l_base[h0 + j] = lj > 0.0f ? (M + fast_log2(lj)) * kLn2 : -INFINITY;
    }
}

template <int G, int LAYOUT, int KV>
__global__ __launch_bounds__(kWavesPerBlock * 64) void decode_attn_kernel(const AttnArgs a) {
    __shared__ int32_t s_page_ids[kWavesPerBlock][kPageWin];
    const int lane = threadIdx.x & 63;
    const int wave = uniform_i32(blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6));
    int32_t *page_ids = s_page_ids[threadIdx.x >> 6];
    const int g = wave % a.Hkv;
    const int i = wave / a.Hkv;
    if (i >= a.waves_per_head) return;

    // Total granules over the batch; lengths are read 256 at a time (four per
    // lane, loads issued together).
    int64_t gtot = 0;
    for (int b0 = 0; b0 < a.B; b0 += 256) {
        int n[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int b = b0 + 64 * k + lane;
            n[k] = b < a.B ? seq_granules(a, b) : 0;
        }
        int t = (n[0] + n[1]) + (n[2] + n[3]);
#pragma unroll
        for (int d = 32; d >= 1; d >>= 1) t += __shfl_xor(t, d, 64);
        gtot += t;
    }
    gtot = uniform_i64(gtot);
    // Empty sequences own no granule: the first wave of each KV head writes
    // their outputs (zeros, lse = -inf) for that head's query heads.  (In
    // grouped calls the merge kernel writes every output.)
    if (i == 0 && !a.pref) {
        for (int b0 = 0; b0 < a.B; b0 += 64) {
            const int b = b0 + lane;
            uint64_t empty = __ballot(b < a.B && clamp_len(a.seq_lens[b], a.cap) == 0);
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
    // At least two granules per wave, so tiny batches are not shredded.
    const int64_t wh = min((int64_t)a.waves_per_head, (gtot + 1) / 2);
    if (wave == 0) write_plan(a, gtot, wh, lane);
    if ((int64_t)i >= wh) return;

    const int64_t x0 = (int64_t)i * gtot / wh;
    const int64_t x1 = (int64_t)(i + 1) * gtot / wh;

    // First sequence whose granules reach past x0, and where it starts.
    int b = 0;
    int64_t start = 0;
    {
        int64_t base = 0;
        bool found = false;
        for (int b0 = 0; b0 < a.B && !found; b0 += 256) {
            int n[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int bb = b0 + 64 * k + lane;
                n[k] = bb < a.B ? seq_granules(a, bb) : 0;
            }
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int bb = b0 + 64 * k + lane;
                const int64_t incl = base + wave_incl_scan(n[k], lane);
                const uint64_t below = __ballot(bb < a.B && incl <= x0);
                const int cnt = __popcll(below);
                if (!found && cnt < 64) {
                    b = b0 + 64 * k + cnt;
                    start = lane_i64(incl - n[k], cnt);
                    found = true;
                }
                base = lane_i64(incl, 63);
            }
        }
    }
    b = uniform_i32(b);
    start = uniform_i64(start);

    int64_t x = x0;
    while (x < x1 && b < a.B) {
        const int L = uniform_i32(clamp_len(a.seq_lens[b], a.cap));
        const int lo = uniform_i32(gran_lo(a, b));
        const int64_t end = start + (L + kGranule - 1) / kGranule - lo;
        if (end > x) {
            const int64_t stop = min(x1, end);
            // waves holding the first and last granule of the sequence: the
            // wave holding granule y is ((y + 1) * wh - 1) / gtot
            const int64_t first = ((start + 1) * wh - 1) / gtot;
            const int64_t last = (end * wh - 1) / gtot;
            // grouped calls send even single pieces to a slot (nseg 0)
            const int nseg = a.pref ? 0 : (int)(last - first + 1);
            attend_piece<G, LAYOUT, KV>(a, page_ids, b, g, (int)(x - start) + lo, (int)(stop - start) + lo,
                                    L, (int64_t)i + b, nseg, lane);
            x = stop;
        }
        start = end;
        ++b;
    }
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
    return hipLaunchKernel(fn, dim3(blocks), dim3(kWavesPerBlock * 64), args, 0, stream);
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
    hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, fn, kWavesPerBlock * 64, 0);
    if (e != hipSuccess) return e;
    *waves = blocks * kWavesPerBlock;
    return hipSuccess;
}

}  // namespace kva
