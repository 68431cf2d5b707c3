// Internal interface between the C-ABI entry points (kva_api.hip) and the
// kernels (kva_kernels.hip).  Not installed; not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kva {

constexpr int kHeadDim = 128;        // the only supported head size
constexpr int kGranule = 16;         // tokens per inner-loop step of one wave
constexpr int kWavesPerBlock = 4;    // attention kernel: 256 threads per block
constexpr int kMaxWaves = 4096;      // upper bound on waves of one attention launch (256 CUs x 16)
// Resident attention waves per compute unit the launch aims for (capped by
// occupancy and by the launch's LDS footprint).
//  * matrix-core engines (pages of 16+ tokens, contiguous caches): bf16 at
//    four waves per CU (64 rollouts of 512-8192 tokens in 16-token pages on
//    MI355X: 180 us at 4, 185 us at 8); fp8, a granule being half the bytes,
//    at eight (98 us at 8, 106 us at 4, 113 us at 12), its kernels held to
//    two waves per SIMD;
//  * vector-ALU engine (pages below 16 tokens): bf16 at four (the vector ALU
//    is the busy unit), fp8 at eight.
constexpr int kTargetWavesPerCU = 4;
constexpr int kTargetWavesPerCUFp8 = 8;
constexpr int kTargetWavesPerCUMfmaBf16 = 4;
constexpr int kTargetWavesPerCUMfmaFp8 = 8;
// Sequences of one attention launch: each block keeps the batch's granule
// prefix sums and lengths in LDS; longer batches are split into launches.
constexpr int kMaxSeqsPerLaunch = 2048;
constexpr int kPageWin = 256;        // page ids per window (two windows per wave)
// XCD-weighted ranges (bf16 caches): a wave's range index has the parity of
// its XCD, and ranges on even XCDs are kXcdWeightEven / kXcdWeightOdd times
// longer.  On MI355X the odd XCDs stream 8-16 % slower than the even ones, so
// equal ranges leave the kernel waiting for the odd ones (64 rollouts of
// 512-8192 tokens: 188.5 -> 185.5 us when first measured, 256 rollouts of
// log-normal lengths: 631 -> 616 us).  The fp8 kernels (two blocks per CU)
// measured ~2 % slower with this placement and keep equal ranges in wave
// order.
constexpr int kXcdWeightEven = 28;   // (matrix-core engine; swept 1:1 .. 31:25 on the benchmark workloads)
constexpr int kXcdWeightOdd = 25;
constexpr int kXcdDeviceCUs = 256;   // the whole MI355X (8 XCDs x 32 CUs); partitions keep equal ranges
constexpr int kPieceGranules = 2;    // virtual granules per sequence (AttnArgs::vgran)
constexpr int kXcdCount = 8;         // XCDs of the whole MI355X: workgroups go to them round-robin
constexpr int kMaxXcds = 16;         // XCD counts the prefill launch order accepts
constexpr int kMaxXcdProbeBlocks = 65536;   // blocks of one kva_debug_xcd_ids launch

enum KvLayout : int {
    kContig = 0,      // [B][Lmax][Hkv][D]
    kPagedWide = 1,   // paged, page_size >= kGranule: one page per granule
    kPagedNarrow = 2  // paged, page_size <  kGranule: several pages per granule
};

enum KvType : int {
    kKvBf16 = 0,      // bf16 cache
    kKvFp8 = 1        // OCP fp8 e4m3fn codes with per-tensor scales
};

// LDS of one attention block for a launch of B sequences:
// [pre: B+1 int64][len: B int32][nseg: B int32][windows: waves x 2 x kPageWin int32]
// [engine tiles: waves x attn_tile_bytes(kv)][q rings: waves x 2 x G x kQRowBytes].
__host__ __device__ inline int attn_lds_len_offset(int B) { return ((B + 1) * 8 + 15) / 16 * 16; }
__host__ __device__ inline int attn_lds_nseg_offset(int B) {
    return attn_lds_len_offset(B) + (B * 4 + 15) / 16 * 16;
}
__host__ __device__ inline int attn_lds_win_offset(int B) {
    return attn_lds_nseg_offset(B) + (B * 4 + 15) / 16 * 16;
}
// Per-wave tile of the matrix-core fp8 engine: V rows of two granules (16 rows
// of 128 codes each, rows padded to 160 bytes, so a 16-lane transposing read
// touches 32 distinct banks), then the K rows of one granule (rows padded to
// 144 bytes: eight lanes reading 16 bytes of eight rows cover the 32 banks).
constexpr int kVtRow = 160;
constexpr int kVtHalf1 = 16 * kVtRow + 16;      // second granule's rows (shifted by 4 banks)
constexpr int kKtRow = 144;
constexpr int kKtOffset = kVtHalf1 + 16 * kVtRow;
constexpr int kVtTileBytes = kKtOffset + 16 * kKtRow;
// Per-wave tile of the matrix-core bf16 engine: V rows of two granules (16
// rows of 256 bytes each, padded to 288: the four rows of a 16-lane
// transposing read fall on disjoint banks), then the K rows of one granule
// (padded to 272: eight lanes reading 16 bytes of eight rows cover the banks).
constexpr int kVbRow = 288;
constexpr int kVbHalf1 = 16 * kVbRow;
constexpr int kKbRow = 272;
constexpr int kKbOffset = 2 * 16 * kVbRow;
constexpr int kBf16TileBytes = kKbOffset + 16 * kKbRow;
__host__ __device__ inline int attn_tile_bytes(int kv) { return kv == kKvBf16 ? kBf16TileBytes : kVtTileBytes; }
__host__ __device__ inline int attn_lds_tile_offset(int B) {
    return attn_lds_win_offset(B) + kWavesPerBlock * 2 * kPageWin * 4;
}
// Per-wave q ring: two slots, each the G query rows (128 bf16, 256 bytes) of a
// piece, so a piece's q can be parked while the previous piece still computes.
constexpr int kQRowBytes = kHeadDim * 2;
__host__ __device__ inline int attn_lds_q_offset(int B, int kv) {
    return attn_lds_tile_offset(B) + kWavesPerBlock * attn_tile_bytes(kv);
}
__host__ __device__ inline int attn_lds_bytes(int B, int G, int kv) {
    return attn_lds_q_offset(B, kv) + kWavesPerBlock * 2 * G * kQRowBytes;
}
constexpr int kLdsPerCU = 160 * 1024;  // MI355X

struct AttnArgs {
    const uint16_t *q;            // bf16 [B][Hq][D]
    const uint16_t *k;            // contiguous cache or page pool
    const uint16_t *v;
    const int32_t *block_table;   // [B][max_pages] (paged only)
    const int32_t *seq_lens;      // [B]
    float *out;                   // [B][Hq][D]       result
    float *lse;                   // [B][Hq]          result log-sum-exp, or NULL
    float *o_ws;                  // [slots][Hq][D]   partial outputs
    float *lse_ws;                // [slots][Hq]      partial log-sum-exp (natural log)
    int2 *plan;                   // [B]              {first slot, pieces} of split sequences
    int64_t num_pages;            // paged: pool size in pages
    int B, Hq, Hkv;
    int cap;                      // max length: Lmax (contiguous) or max_pages * page_size
    int seq_stride;               // contiguous: Lmax (rows per sequence)
    int max_pages;                // paged: block-table row length
    int log2_page;                // paged: log2(page_size)
    int waves_per_head;           // Wh: waves given to each KV head
    int xcd_map;                  // 1: range index parity = XCD parity, weights below apply
    int w_even, w_odd;            // range weights of even / odd range indices (xcd_map = 1)
    float scale_log2;             // scale * log2(e) (fp8: times the key scale)
    float v_scale;                // fp8: value scale, applied to the output
    // grouped calls: sequence b starts at granule pref[b / group] (the shared
    // run is attended by the prefix kernel) and every piece, single or not,
    // goes to a workspace slot; the merge kernel writes all outputs
    const int32_t *pref;          // [ngroups] or NULL
    int group;
    // work partition: every non-empty sequence's granules are preceded by this
    // many virtual granules in the flat space, which carry no loads; a range
    // that crosses into a sequence pays them, so ranges with more pieces get
    // fewer real granules (a piece costs about two granules' time)
    int vgran;
};

struct CombineArgs {
    const float *o_parts;         // [S][B][Hq][D]
    const float *lse_parts;       // [S][B][Hq]
    float *out;
    float *lse;                   // may be NULL
    int S, B, Hq, D;
};

struct MergeArgs {
    const float *o_ws;
    const float *lse_ws;
    const int2 *plan;
    float *out;
    float *lse;                   // may be NULL
    int B, Hq;
};

// Shared-prefix pass of a grouped call: one wave per (group, KV head, split).
struct PrefixArgs {
    const uint16_t *q;
    const uint16_t *k;
    const uint16_t *v;
    const int32_t *block_table;
    const int32_t *seq_lens;
    int32_t *pref;                // [ngroups]  shared granules per group (written)
    float *o_pre;                 // [parts][B][Hq][D] partial outputs
    float *lse_pre;               // [parts][B][Hq]    partial log-sum-exp
    int64_t num_pages;
    int B, Hq, Hkv, cap, max_pages, log2_page, group, ngroups;
    int parts;                    // workgroups (partial results) per (group, KV head)
    int w_even, w_odd;            // range weights of workgroups on even / odd XCDs
    float scale_log2;
};

struct GroupMergeArgs {
    const float *o_pre;
    const float *lse_pre;
    const float *o_ws;
    const float *lse_ws;
    const int2 *plan;
    float *out;
    float *lse;                   // may be NULL
    int B, Hq, parts;
    int b_off, nb;                // sequences b_off .. b_off + nb - 1 of the batch
};

// New-token step: RMS-normalise q and k per head, rotate them at the new
// position, write q out and append k, v to the cache.
struct AppendArgs {
    const uint16_t *q_in;         // [B][Hq][D]
    const uint16_t *k_in;         // [B][Hkv][D]
    const uint16_t *v_in;         // [B][Hkv][D]
    const float *q_w;             // [D] RMS gains, or NULL (no normalisation)
    const float *k_w;
    uint16_t *q_out;              // [B][Hq][D]
    uint16_t *k_cache;            // pool [num_pages][P][Hkv][D] or [B][Lmax][Hkv][D]
    uint16_t *v_cache;
    const int32_t *block_table;   // [B][max_pages] (paged)
    const int32_t *seq_lens;      // [B] current lengths = the new token's position
    int32_t *new_lens;            // [B] or NULL; may alias seq_lens
    int64_t num_pages;
    int B, Hq, Hkv, cap, max_pages, log2_page;
    int paged;                    // 1: pool + block table, 0: contiguous [B][cap][Hkv][D]
    float eps;
    double log2_theta;            // log2(rotary base)
    int rope;                     // 0: no rotation
};

// Chunked prefill: new tokens attend their causal prefix in a paged cache.
struct PrefillArgs {
    const uint16_t *q;            // [T][Hq][D], sequence b's rows q_start[b] .. q_start[b+1]-1
    const uint16_t *k;            // pool [num_pages][P][Hkv][D]
    const uint16_t *v;
    const int32_t *block_table;   // [B][max_pages]
    const int32_t *q_start;       // [B + 1]
    const int32_t *seq_lens;      // [B] lengths including the new tokens
    float *out;                   // [T][Hq][D]
    float *lse;                   // [T][Hq] or NULL
    int64_t num_pages;
    int B, T, Hq, Hkv, cap, max_pages, log2_page;
    int tiles;                    // query tiles per (sequence, KV head)
    int xcds;                     // XCDs workgroups are dealt to round-robin (1 if unknown)
    float scale_log2;
};

struct GatherArgs {
    const uint16_t *pool;
    const int32_t *block_table;
    const int32_t *seq_lens;
    uint16_t *dst;
    int64_t num_pages;
    int B, Hkv, D, max_pages, log2_page, Lcap;
};

constexpr int kPrefixWaves = 4;        // shared-prefix pass: waves per workgroup
constexpr int kMaxPrefixParts = 4;     // shared-prefix pass: workgroups per (group, KV head)
constexpr int kMaxGroupRows = 32;      // shared-prefix pass: group * (Hq / Hkv) query rows

// Slots of partial results a launch may write: the piece of sequence b that
// range i covers goes to slot i + b, so at most (ranges per head) + B - 1,
// with B the launch's sequences.
inline int64_t max_slots(int B, int Hkv) {
    const int64_t Bl = B < kMaxSeqsPerLaunch ? B : kMaxSeqsPerLaunch;
    return (int64_t)(kMaxWaves / Hkv) + Bl;
}

hipError_t launch_decode_attn(const AttnArgs &a, int layout, int group, int kv, int blocks,
                              hipStream_t stream);
hipError_t launch_combine(const CombineArgs &a, hipStream_t stream);
hipError_t launch_merge_split(const MergeArgs &a, hipStream_t stream);
hipError_t launch_gather(const GatherArgs &a, hipStream_t stream);
hipError_t launch_prefix(const PrefixArgs &a, hipStream_t stream);
hipError_t launch_merge_grouped(const GroupMergeArgs &a, hipStream_t stream);
hipError_t launch_append(const AppendArgs &a, hipStream_t stream);
hipError_t launch_prefill(const PrefillArgs &a, hipStream_t stream);
hipError_t launch_xcd_ids(int32_t *out, int nblocks, hipStream_t stream);
int prefill_tokens_per_tile(int group);   // new tokens per prefill workgroup

// Resident attention waves per compute unit for (layout, group, kv) on the current device.
hipError_t attn_waves_per_cu(int layout, int group, int kv, int *waves);
hipError_t launch_stream_read(const void *src, int64_t bytes, uint32_t *sink, int blocks,
                              hipStream_t stream);

}  // namespace kva
