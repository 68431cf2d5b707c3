/*
 * kva.h -- C ABI of libkva: batched grouped-query decode attention over bf16
 * KV caches, hand-written HIP for gfx950 (MI355X).
 *
 * The operation is the attention step of autoregressive decoding that the
 * paper's RL rollouts spend their time in (appendix "Training Details",
 * subsection "Implementation Components": prompts are sampled, the policy
 * decodes code and reflections for up to three turns, G samples per prompt;
 * hyperparameter table: group size 8, 64 prompts, 8K/16K sequence lengths).
 * For one decode step of one layer, every sequence b and query head h:
 *
 *   g   = h / (Hq / Hkv)                          consecutive query heads share a KV head
 *   s_t = scale * <q[b,h,:], K[b,t,g,:]>          t = 0 .. L_b-1 (no mask inside the cache)
 *   out[b,h,:] = sum_t softmax(s)_t * V[b,t,g,:]  softmax with the maximum subtracted
 *   lse[b,h]   = ln sum_t exp(s_t)                (natural log of the scaled scores)
 *   L_b = 0   ->  out = 0, lse = -inf
 *
 * The softmax is the max-subtracted form the paper's appendix of self-correction
 * examples arrives at (Example 1; Example 3 for rows longer than one block);
 * the kernels evaluate it in one pass as an online softmax, and merge the
 * results of disjoint key ranges with the log-sum-exp identity (the
 * multi-stage reduction the experiments section lists among generated-kernel
 * failure modes).  Results match the exact definition up to fp32 rounding.
 *
 * Conventions shared by every entry point
 *   - All data pointers are DEVICE pointers; the caller owns every buffer.
 *     The library allocates no device memory and keeps no pointer after a
 *     call returns.
 *   - bf16 tensors are passed as 16-bit storage (raw bit patterns).
 *   - Calls are enqueued on `stream` (a hipStream_t, NULL = the default
 *     stream) and return without synchronising; inputs must stay alive and
 *     unmodified until the stream has passed the call.
 *   - Host-side argument checks (NULL pointers, shapes, alignment, workspace
 *     size, supported configuration) run before anything is launched.  On
 *     failure the call returns a nonzero kva_status, launches nothing and
 *     leaves every output untouched.  A launch error reported by the HIP
 *     runtime returns KVA_ERR_HIP.
 *   - Device-resident integers are not inspected by the host.  The kernels
 *     clamp each length to [0, capacity]; a block-table entry outside
 *     [0, num_pages) is replaced by page 0 (never read out of bounds), which
 *     gives unspecified values for that sequence.
 *   - Supported: D = 128; Hq % Hkv == 0 with Hq / Hkv in {1, 2, 4, 8};
 *     page_size a power of two in [1, 1024].  Others: KVA_ERR_UNSUPPORTED.
 *   - Results are deterministic: the same inputs on the same device give
 *     bitwise identical outputs (no floating-point atomics; the merge order
 *     of partial results is fixed).
 *   - The library's mutable global state: per-device caches (resident waves
 *     per compute unit, compute-unit and XCD counts, the address of the
 *     scratch array) filled on first use, and the scratch array of
 *     kva_decode_attn_paged_noalloc.  Calls may come from several host
 *     threads, but two calls in flight at once must not share a workspace.
 *   - One decode call is two kernel launches on `stream`: the attention kernel, then
 *     a small kernel that merges the pieces of sequences split over waves
 *     (three for kva_decode_attn_paged_grouped with group > 1).
 *   - A call is kernel launches only (no allocation, no memset, no host
 *     synchronisation), so it can be captured in a HIP graph once its
 *     per-device caches are filled (one eager call on the device first).  The
 *     launch shapes depend on the sizes passed (B, Hq, Hkv, group, max_q_len)
 *     and on the device, never on device data: lengths, block tables, q and
 *     the caches may change in place between replays of a captured call.
 */
#ifndef KVA_H_
#define KVA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    KVA_OK = 0,
    KVA_ERR_NULL = 1,          /* a required pointer is NULL                         */
    KVA_ERR_SHAPE = 2,         /* a size is negative, zero where it must not be, ... */
    KVA_ERR_ALIGN = 3,         /* a pointer is not aligned as documented             */
    KVA_ERR_WORKSPACE = 4,     /* workspace missing or smaller than required         */
    KVA_ERR_UNSUPPORTED = 5,   /* valid but unsupported configuration                */
    KVA_ERR_HIP = 6,           /* the HIP runtime reported an error                  */
    KVA_ERR_SCRATCH = 7        /* batch too large for the built-in scratch buffer    */
} kva_status;

/* Static text for a status code (never NULL). */
const char *kva_status_str(int status);

/* Library ABI version, currently 2 (2: the workspace needs no initialised
 * header; kva_decode_attn_paged_noalloc and the placement hooks added; the
 * grouped workspace holds 4 shared-prefix partial results per row, not 16). */
int kva_version(void);

/*
 * Bytes of workspace kva_decode_attn / kva_decode_attn_paged (and their fp8
 * variants) need for a batch of B sequences with Hq query heads, Hkv KV heads
 * and head size D.  The bound depends on neither the lengths nor the device:
 * the kernels cut the batch's tokens into at most 4096 / Hkv ranges per KV
 * head, whatever the lengths, so no length hint is needed.  Returns 0 when
 * the arguments are invalid.
 *
 * The workspace holds a per-sequence merge plan and the partial results of
 * sequences split over several waves.  It needs no initialisation (every byte
 * a call reads was written earlier in the same call) and may be reused by
 * consecutive calls of any shape that fits.  Batches of more than 2048
 * sequences run as several kernel launches over the same workspace.
 */
size_t kva_workspace_bytes(int B, int Hq, int Hkv, int D);

/*
 * Decode attention over contiguous caches.
 *   q          bf16 [B][Hq][D], 16-byte aligned
 *   k, v       bf16 [B][Lmax][Hkv][D], 16-byte aligned; row t of sequence b
 *              is read only for t < seq_lens[b]
 *   seq_lens   int32 [B] (device); each clamped to [0, Lmax] by the kernel
 *   out        fp32 [B][Hq][D], 16-byte aligned (written)
 *   lse        fp32 [B][Hq] (written) or NULL
 *   scale      multiplier of q.K (typically 1/sqrt(D)); finite, and finite
 *              once folded into base 2 (|scale| * log2 e <= FLT_MAX), else
 *              KVA_ERR_UNSUPPORTED
 *   workspace  >= kva_workspace_bytes(B, Hq, Hkv, D) bytes, 256-byte aligned
 * B = 0 is a valid no-op.  Lmax may be 0 (all lengths then clamp to 0; k and v
 * may then be NULL).
 */
int kva_decode_attn(const void *q, const void *k, const void *v, const int32_t *seq_lens,
                    float *out, float *lse, int B, int Hq, int Hkv, int D, int Lmax,
                    float scale, void *workspace, size_t workspace_bytes, void *stream);

/*
 * Decode attention over a paged cache: position t of sequence b lives in
 * physical page block_table[b][t / page_size], slot t % page_size.
 *   k_pool, v_pool  bf16 [num_pages][page_size][Hkv][D], 16-byte aligned;
 *                   several sequences may map the same physical page (a
 *                   shared prompt prefix)
 *   block_table     int32 [B][max_pages_per_seq] (device); entries past a
 *                   sequence's last page may be read (every row is read
 *                   only within its max_pages_per_seq entries) but are never
 *                   used, so they may hold any value
 *   seq_lens        int32 [B] (device); each clamped to
 *                   [0, max_pages_per_seq * page_size], and to 0 when
 *                   num_pages == 0 (the pools may then be NULL; the table
 *                   may be NULL when max_pages_per_seq == 0)
 * Other arguments as for kva_decode_attn.
 */
int kva_decode_attn_paged(const void *q, const void *k_pool, const void *v_pool,
                          const int32_t *block_table, const int32_t *seq_lens, float *out,
                          float *lse, int B, int Hq, int Hkv, int D, int page_size,
                          int max_pages_per_seq, int64_t num_pages, float scale,
                          void *workspace, size_t workspace_bytes, void *stream);

/*
 * kva_decode_attn_paged without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  The partial results live in a device
 * array built into the library, KVA_NOALLOC_SCRATCH_BYTES bytes, one copy on
 * every device the library runs on, held until the process ends.  The call
 * allocates nothing: the array's device address is looked up once per device
 * (on the first call with that device current) and every later call only
 * launches kernels.
 *   - Same arguments (minus workspace), semantics, results (bitwise) and
 *     status codes as kva_decode_attn_paged.
 *   - A batch whose workspace (kva_workspace_bytes(B, Hq, Hkv, D)) exceeds
 *     KVA_NOALLOC_SCRATCH_BYTES returns KVA_ERR_SCRATCH and launches nothing
 *     (every B fits at Hq = 32, Hkv = 8, D = 128).
 *   - Every call on one device shares the array: calls that overlap on one
 *     device (two streams, or two host threads) race and give undefined
 *     results.  Calls in order on one stream are safe; nothing in the array
 *     needs to be cleared between calls.
 */
#define KVA_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int kva_decode_attn_paged_noalloc(const void *q, const void *k_pool, const void *v_pool,
                                  const int32_t *block_table, const int32_t *seq_lens, float *out,
                                  float *lse, int B, int Hq, int Hkv, int D, int page_size,
                                  int max_pages_per_seq, int64_t num_pages, float scale,
                                  void *stream);

/*
 * The same two calls over 8-bit floating-point caches: K and V hold OCP FP8
 * E4M3 codes ("e4m3fn": sign, 4 exponent bits with bias 7, 3 mantissa bits,
 * largest finite 448, S.1111.111 = NaN), one byte per element, with one scale
 * per tensor: the key at a code c is k_scale * fp8(c), the value v_scale *
 * fp8(c).  Half the bytes of a bf16 cache per token (2 KiB per token per layer
 * at Hkv = 8, D = 128).  The result is attention over those values, as above:
 * the kernels widen the codes exactly (to bf16 for the q.K products, to fp32
 * for the weighted sum), fold k_scale into the score scale and apply v_scale
 * to the normalised output (lse is that of the scaled scores).
 *   k, v / k_pool, v_pool  uint8 codes, layouts as for the bf16 calls,
 *                          16-byte aligned
 *   k_scale, v_scale       finite, with scale * k_scale * log2 e finite in fp32
 *                          (else KVA_ERR_UNSUPPORTED)
 * Workspace: kva_workspace_bytes(B, Hq, Hkv, D).  Other arguments and
 * conventions as for kva_decode_attn / kva_decode_attn_paged.
 */
int kva_decode_attn_fp8(const void *q, const void *k, const void *v, const int32_t *seq_lens,
                        float *out, float *lse, int B, int Hq, int Hkv, int D, int Lmax,
                        float scale, float k_scale, float v_scale, void *workspace,
                        size_t workspace_bytes, void *stream);

int kva_decode_attn_paged_fp8(const void *q, const void *k_pool, const void *v_pool,
                              const int32_t *block_table, const int32_t *seq_lens, float *out,
                              float *lse, int B, int Hq, int Hkv, int D, int page_size,
                              int max_pages_per_seq, int64_t num_pages, float scale,
                              float k_scale, float v_scale, void *workspace,
                              size_t workspace_bytes, void *stream);

/*
 * Bytes of workspace kva_decode_attn_paged_grouped needs: the amount of
 * kva_workspace_bytes(B, Hq, Hkv, D) plus room for the shared-prefix pass (4
 * partial results per sequence and query head, one int32 per group).  Returns
 * 0 when the arguments are invalid (group < 1 included).  No initialisation
 * is needed.
 */
size_t kva_workspace_bytes_grouped(int B, int Hq, int Hkv, int D, int group);

/*
 * Shared-prefix (group) decode over a paged cache.  The samples drawn for one
 * prompt (the paper samples a group of outputs per prompt: appendix "Training
 * Details", hyperparameter table, group size 8) decode from the same prompt
 * tokens, so their caches start with the same physical pages.  This call
 * computes what kva_decode_attn_paged computes for the same arguments (equal
 * up to fp32 rounding), but reads those pages once per group instead of once
 * per sample:
 *   - sequences are taken in groups of `group` consecutive sequences (the
 *     last group may be smaller);
 *   - on the device, each group's shared run is found: the leading pages
 *     whose block-table entries (after the bad-id replacement) are equal in
 *     every member, cut at the shortest member's length and rounded down to a
 *     multiple of 16 tokens.  Nothing is assumed about the table: a group
 *     with no common leading page simply has an empty shared run;
 *   - the shared run is attended once per KV head for all group * Hq/Hkv
 *     query heads that read it, on the matrix cores (bf16 products, fp32
 *     accumulation; the softmax weights enter the second product as a sum of
 *     two bf16 parts); the rest of each sequence is attended as by
 *     kva_decode_attn_paged; the partial results are merged with the
 *     log-sum-exp identity.
 *   group      >= 1 (else KVA_ERR_SHAPE); group * (Hq / Hkv) <= 32 (else
 *              KVA_ERR_UNSUPPORTED); group = 1, or page_size < 16, runs
 *              kva_decode_attn_paged (nothing is read once per group then)
 *   workspace  >= kva_workspace_bytes_grouped(B, Hq, Hkv, D, group) bytes,
 *              256-byte aligned
 * Other arguments, conventions and status codes as for kva_decode_attn_paged.
 */
int kva_decode_attn_paged_grouped(const void *q, const void *k_pool, const void *v_pool,
                                  const int32_t *block_table, const int32_t *seq_lens, float *out,
                                  float *lse, int B, int Hq, int Hkv, int D, int page_size,
                                  int max_pages_per_seq, int64_t num_pages, int group, float scale,
                                  void *workspace, size_t workspace_bytes, void *stream);

/*
 * The step before attention for the token each sequence has just decoded:
 * per-head RMS normalisation of its query and key, rotary position embedding
 * at its position, and the append of its key and value to the cache.  The
 * paper names Qwen3-8B as its policy model (section "Compact AMD Kernel LLMs")
 * but defines neither operation; the arithmetic below is this library's
 * reading of that model's attention input (per-head RMS norm with a shared
 * gain vector, rotate-half rotary embedding, base 1e6), not something the
 * paper states.  RMS normalisation is one of the kernel families the paper's
 * experiments section lists.
 * For every sequence b (L_b = seq_lens[b] clamped to [0, capacity]: the new
 * token's position):
 *   q rows (Hq per sequence) and k rows (Hkv):
 *     x_d <- x_d / sqrt(mean_e x_e^2 + eps) * w_d       (w = q_norm_w or k_norm_w;
 *                                                       skipped when NULL)
 *     for i < D/2, a_i = L_b * rope_theta^(-2i/D):       (skipped when rope_theta <= 0)
 *       y_i = x_i cos a_i - x_{i+D/2} sin a_i,   y_{i+D/2} = x_{i+D/2} cos a_i + x_i sin a_i
 *   q_out[b] = rotated q rows; the rotated k rows and the unchanged v rows are
 *   written at position L_b of sequence b's cache; new_lens[b] = L_b + 1.
 * If position L_b does not exist (L_b = capacity, or, paged, the block-table
 * entry is outside [0, num_pages)), nothing is written to the cache for that
 * sequence and new_lens[b] = L_b; q_out is written regardless.
 *   q_in       bf16 [B][Hq][D];  k_in, v_in bf16 [B][Hkv][D] (finite values)
 *   q_norm_w, k_norm_w  fp32 [D] or NULL
 *   q_out      bf16 [B][Hq][D]; may be q_in itself (in place)
 *   seq_lens   int32 [B];  new_lens int32 [B] or NULL, may be seq_lens itself
 *   eps        >= 0 (1e-6 for Qwen3);  rope_theta  base of the rotary
 *              frequencies (1e6 for Qwen3), <= 0 for no rotation
 * Angles are formed in binary64; normalisation and rotation run in fp32 and
 * each output is rounded once to bf16 (nearest even).  All pointers 16-byte
 * aligned (seq_lens, new_lens, block_table: 4).  One kernel launch; moves
 * about 2 * (Hq + 2 Hkv) * D * 2 bytes per sequence.  Same conventions as the
 * attention calls; D = 128, Hq / Hkv in {1, 2, 4, 8}; eps and rope_theta finite
 * and rope_theta != 1 (else KVA_ERR_UNSUPPORTED).
 */
int kva_append(const void *q_in, const void *k_in, const void *v_in, const float *q_norm_w,
               const float *k_norm_w, void *q_out, void *k_cache, void *v_cache,
               const int32_t *seq_lens, int32_t *new_lens, int B, int Hq, int Hkv, int D,
               int Lmax, float eps, double rope_theta, void *stream);
/* k_cache, v_cache: bf16 [B][Lmax][Hkv][D]; capacity Lmax. */

int kva_append_paged(const void *q_in, const void *k_in, const void *v_in,
                     const float *q_norm_w, const float *k_norm_w, void *q_out, void *k_pool,
                     void *v_pool, const int32_t *block_table, const int32_t *seq_lens,
                     int32_t *new_lens, int B, int Hq, int Hkv, int D, int page_size,
                     int max_pages_per_seq, int64_t num_pages, float eps, double rope_theta,
                     void *stream);
/* k_pool, v_pool, block_table, page_size, max_pages_per_seq, num_pages as for
 * kva_decode_attn_paged; capacity max_pages_per_seq * page_size (0 when
 * num_pages == 0). */

/*
 * Chunked prefill over a paged cache: the prompt, or the feedback appended
 * between turns (the paper's multi-turn reflection rollouts ingest the
 * execution feedback of each turn before decoding the next: appendix "More
 * Details of Compact LLM Training", "Multi-Turn On-Policy Reflection"), as a
 * chunk of n_b new tokens per sequence whose keys and values are already in
 * the cache at positions L_b - n_b .. L_b - 1 (L_b = seq_lens[b]).  New token
 * i of sequence b sits at position p = L_b - n_b + i and attends positions
 * 0 .. p (causal): the same attention as above with length p + 1; p < 0
 * attends nothing (out = 0, lse = -inf).
 *   q          bf16 [T][Hq][D]: the new tokens of all sequences, sequence b's
 *              rows q_start[b] .. q_start[b+1]-1
 *   q_start    int32 [B + 1] (device), nondecreasing from 0 to T; the kernels
 *              clamp each entry to [previous entry, T]
 *   seq_lens   int32 [B] (device), including the new tokens
 *   out        fp32 [T][Hq][D] (written);  lse fp32 [T][Hq] (written) or NULL
 *   max_q_len  host bound on every n_b (the grid is sized from it); new tokens
 *              past it are not computed and their outputs are left unwritten
 * Pools, block table, page size, scale: as for kva_decode_attn_paged.  No
 * workspace.  One kernel launch; the q.K and P.V products run on the matrix
 * cores (bf16 inputs, fp32 accumulation; the softmax weights enter P.V as the
 * sum of two bf16 parts), the softmax in fp32.
 */
int kva_prefill_paged(const void *q, const void *k_pool, const void *v_pool,
                      const int32_t *block_table, const int32_t *q_start, const int32_t *seq_lens,
                      float *out, float *lse, int B, int T, int max_q_len, int Hq, int Hkv, int D,
                      int page_size, int max_pages_per_seq, int64_t num_pages, float scale,
                      void *stream);

/*
 * Merge S partial attention results over disjoint key sets of the same
 * queries (split-K, or context shards computed elsewhere):
 *   o_parts    fp32 [S][B][Hq][D], each part normalised by its own softmax sum
 *   lse_parts  fp32 [S][B][Hq], natural-log sum of exp of the part's scores;
 *              -inf marks an empty part (its o_parts values are ignored)
 *   out        fp32 [B][Hq][D] (written);  lse fp32 [B][Hq] (written) or NULL
 * With M = max_i lse_i:  out = sum_i e^(lse_i - M) o_i / sum_i e^(lse_i - M),
 * lse = M + ln sum_i e^(lse_i - M); all parts empty -> out = 0, lse = -inf.
 * Parts are merged in index order.  o_parts, out: 8-byte aligned.  D even and
 * at most 256 (else KVA_ERR_UNSUPPORTED).
 */
int kva_combine(const float *o_parts, const float *lse_parts, float *out, float *lse, int S,
                int B, int Hq, int D, void *stream);

/*
 * Test hook for page-table indexing: copies, through the same address
 * computation the attention kernels use, the rows of a paged pool into a
 * dense cache.
 *   pool   bf16 [num_pages][page_size][Hkv][D], 16-byte aligned
 *   dst    bf16 [B][Lcap][Hkv][D], 16-byte aligned (written): row t of
 *          sequence b is the pool row of position t for t < min(L_b, Lcap),
 *          zero for min(L_b, Lcap) <= t < Lcap
 */
int kva_debug_gather_paged(const void *pool, const int32_t *block_table,
                           const int32_t *seq_lens, void *dst, int B, int Hkv, int D,
                           int page_size, int max_pages_per_seq, int64_t num_pages, int Lcap,
                           void *stream);

/*
 * Measurement hook: a plain streaming read of `bytes` bytes at `src` with the
 * decode kernels' 16-byte non-temporal loads, the achievable HBM read
 * bandwidth reported beside the decode figures.  Block i of
 * min(sink_words, 512) blocks (four waves each, every wave a contiguous
 * share) XOR-reduces its share of the 32-bit words of the buffer and writes
 * the result to sink[i]; entries past the block count are left untouched
 * (the XOR of all entries of a zeroed sink is the XOR of every word).
 *   src    device, 16-byte aligned, bytes a multiple of 16 (else
 *          KVA_ERR_ALIGN / KVA_ERR_SHAPE); bytes = 0 launches nothing
 *   sink   device uint32 [sink_words], sink_words >= 1
 * Asynchronous on `stream`, like every call.
 */
int kva_debug_stream_read(const void *src, size_t bytes, uint32_t *sink, int sink_words,
                          void *stream);

/*
 * Placement hooks.  The bf16 decode launches size their ranges for the XCD
 * each workgroup lands on, and the prefill launch orders its tiles by XCD,
 * both assuming that workgroups are dealt to the XCDs round-robin (block id
 * mod the XCD count); these report what the device does.
 *
 * kva_debug_xcd_count: *xcds = the XCDs of the current device as the runtime
 * reports them (8 on a whole MI355X), 0 if it does not report them; the
 * decode ranges are weighted only when this is 8 on a 256-CU device.
 *   xcds   host int; NULL gives KVA_ERR_NULL
 *
 * kva_debug_xcd_ids: launches nblocks one-wave workgroups; workgroup b writes
 * the XCD it runs on (the XCC_ID hardware register) to out[b].
 *   out      device int32 [nblocks], 4-byte aligned
 *   nblocks  0 .. 65536 (else KVA_ERR_SHAPE); 0 launches nothing
 * Asynchronous on `stream`.
 */
int kva_debug_xcd_count(int *xcds);
int kva_debug_xcd_ids(int32_t *out, int nblocks, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* KVA_H_ */
