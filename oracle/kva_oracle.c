/*
 * kva_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, single-threaded binary64 reference for batched grouped-query
 * decode attention over bf16 KV caches.  Only the test suite, the smoke check
 * and the benchmark's CPU-baseline leg may load this library; the product path
 * never links, loads or calls it, and this file shares no code with the GPU
 * library.
 *
 * What it computes, for every sequence b and query head h:
 *
 *   g   = h / (Hq / Hkv)                 (consecutive query heads share a KV head)
 *   s_t = scale * sum_d q[b,h,d] * K_t[d]          t = 0 .. L_b-1
 *   m   = max_t s_t
 *   w_t = exp(s_t - m)
 *   l   = sum_t w_t
 *   out = (sum_t w_t * V_t) / l ,   lse = m + ln(l)
 *   L_b = 0  ->  out = 0, lse = -inf
 *
 * The softmax is the max-subtracted ("numerically stable") form, evaluated in
 * separate passes (maximum; exponentials and their sum; normalised weighted
 * sum), which is how the paper's appendix of multi-turn self-correction
 * examples repairs a softmax (Example 1: subtract the row maximum before
 * exponentiating; Example 3: a max pass, an exp-and-sum pass and a normalise
 * pass for rows longer than one block).  Decode attention is exact up to
 * rounding order, so this file is that definition written out, with no
 * blocking, fusion or online rescaling.
 *
 * The split-K combine is the log-sum-exp identity for merging softmax results
 * computed over disjoint key sets (the "multi-stage reductions" the paper's
 * experiments section names as a failure class for generated kernels).
 *
 * Precision: every bf16 input is widened exactly to binary64 (bits << 16 ->
 * float -> double); sums run in a fixed order (t ascending, d ascending);
 * build with -ffp-contract=off and without fast-math.
 *
 * Pins: see tests/test_oracle_pins.py (closed forms, invariants, reduction to
 * torch's scaled_dot_product_attention, and mpmath at 50 digits).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define KVO_OK 0
#define KVO_ERR_ARG 1
#define KVO_ERR_RANGE 2
#define KVO_ERR_NOMEM 3

static double bf16_to_f64(uint16_t h) {
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/*
 * One (sequence, query head) pair.  krow[t] / vrow[t] point at the D bf16
 * values of cache position t for this head's KV head.  s is scratch of L
 * doubles.
 */
static void attend_one(const uint16_t *qh, const uint16_t *const *krow,
                       const uint16_t *const *vrow, int L, int D, double scale,
                       double *out, double *lse, double *s) {
    if (L == 0) {
        for (int d = 0; d < D; ++d) out[d] = 0.0;
        *lse = -INFINITY;
        return;
    }
    /* scores */
    for (int t = 0; t < L; ++t) {
        double dot = 0.0;
        for (int d = 0; d < D; ++d) dot += bf16_to_f64(qh[d]) * bf16_to_f64(krow[t][d]);
        s[t] = scale * dot;
    }
    /* pass 1: maximum */
    double m = s[0];
    for (int t = 1; t < L; ++t)
        if (s[t] > m) m = s[t];
    /* pass 2: exponentials and their sum */
    double l = 0.0;
    for (int t = 0; t < L; ++t) {
        s[t] = exp(s[t] - m);
        l += s[t];
    }
    /* pass 3: normalised weighted sum of values */
    for (int d = 0; d < D; ++d) {
        double acc = 0.0;
        for (int t = 0; t < L; ++t) acc += s[t] * bf16_to_f64(vrow[t][d]);
        out[d] = acc / l;
    }
    *lse = m + log(l);
}

static int check_heads(int B, int Hq, int Hkv, int D) {
    if (B < 0 || Hq <= 0 || Hkv <= 0 || D <= 0) return 0;
    if (Hq % Hkv != 0) return 0;
    return 1;
}

/*
 * Contiguous caches.
 *   q      bf16 [B][Hq][D]
 *   k, v   bf16 [B][Lmax][Hkv][D]
 *   lens   int32 [B], 0 <= lens[b] <= Lmax
 *   out    f64 [B][Hq][D];  lse f64 [B][Hq] (may be NULL)
 */
int kvo_decode_attn(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                    const int32_t *lens, double *out, double *lse, int B, int Hq,
                    int Hkv, int D, int Lmax, double scale) {
    if (!check_heads(B, Hq, Hkv, D) || Lmax < 0) return KVO_ERR_ARG;
    for (int b = 0; b < B; ++b)
        if (lens[b] < 0 || lens[b] > Lmax) return KVO_ERR_RANGE;
    const int group = Hq / Hkv;
    double *s = (double *)malloc(sizeof(double) * (size_t)(Lmax > 0 ? Lmax : 1));
    const uint16_t **kr = (const uint16_t **)malloc(sizeof(void *) * (size_t)(Lmax > 0 ? Lmax : 1));
    const uint16_t **vr = (const uint16_t **)malloc(sizeof(void *) * (size_t)(Lmax > 0 ? Lmax : 1));
    if (!s || !kr || !vr) {
        free(s); free(kr); free(vr);
        return KVO_ERR_NOMEM;
    }
    for (int b = 0; b < B; ++b) {
        for (int h = 0; h < Hq; ++h) {
            const int g = h / group;
            for (int t = 0; t < lens[b]; ++t) {
                size_t row = ((size_t)b * (size_t)Lmax + (size_t)t) * (size_t)Hkv + (size_t)g;
                kr[t] = k + row * (size_t)D;
                vr[t] = v + row * (size_t)D;
            }
            double l_out;
            attend_one(q + ((size_t)b * Hq + h) * D, kr, vr, lens[b], D, scale,
                       out + ((size_t)b * Hq + h) * D, &l_out, s);
            if (lse) lse[(size_t)b * Hq + h] = l_out;
        }
    }
    free(s); free(kr); free(vr);
    return KVO_OK;
}

/*
 * Paged caches: position t of sequence b lives in physical page
 * block_table[b][t / page_size], slot t % page_size.
 *   k_pool, v_pool  bf16 [num_pages][page_size][Hkv][D]
 *   block_table     int32 [B][max_pages]
 * Returns KVO_ERR_RANGE if a page needed by some position is outside
 * [0, num_pages) or a length exceeds max_pages * page_size.
 */
int kvo_decode_attn_paged(const uint16_t *q, const uint16_t *k_pool, const uint16_t *v_pool,
                          const int32_t *block_table, const int32_t *lens, double *out,
                          double *lse, int B, int Hq, int Hkv, int D, int page_size,
                          int max_pages, int64_t num_pages, double scale) {
    if (!check_heads(B, Hq, Hkv, D) || page_size <= 0 || max_pages < 0 || num_pages < 0)
        return KVO_ERR_ARG;
    int64_t cap = (int64_t)page_size * (int64_t)max_pages;
    int lmax = 0;
    for (int b = 0; b < B; ++b) {
        if (lens[b] < 0 || (int64_t)lens[b] > cap) return KVO_ERR_RANGE;
        if (lens[b] > lmax) lmax = lens[b];
        for (int t = 0; t < lens[b]; t += page_size) {
            int32_t p = block_table[(size_t)b * max_pages + t / page_size];
            if (p < 0 || (int64_t)p >= num_pages) return KVO_ERR_RANGE;
        }
    }
    const int group = Hq / Hkv;
    double *s = (double *)malloc(sizeof(double) * (size_t)(lmax > 0 ? lmax : 1));
    const uint16_t **kr = (const uint16_t **)malloc(sizeof(void *) * (size_t)(lmax > 0 ? lmax : 1));
    const uint16_t **vr = (const uint16_t **)malloc(sizeof(void *) * (size_t)(lmax > 0 ? lmax : 1));
    if (!s || !kr || !vr) {
        free(s); free(kr); free(vr);
        return KVO_ERR_NOMEM;
    }
    for (int b = 0; b < B; ++b) {
        for (int h = 0; h < Hq; ++h) {
            const int g = h / group;
            for (int t = 0; t < lens[b]; ++t) {
                int32_t page = block_table[(size_t)b * max_pages + t / page_size];
                size_t row = ((size_t)page * (size_t)page_size + (size_t)(t % page_size)) * (size_t)Hkv
                             + (size_t)g;
                kr[t] = k_pool + row * (size_t)D;
                vr[t] = v_pool + row * (size_t)D;
            }
            double l_out;
            attend_one(q + ((size_t)b * Hq + h) * D, kr, vr, lens[b], D, scale,
                       out + ((size_t)b * Hq + h) * D, &l_out, s);
            if (lse) lse[(size_t)b * Hq + h] = l_out;
        }
    }
    free(s); free(kr); free(vr);
    return KVO_OK;
}

/*
 * Merge S partial results computed over disjoint key sets.
 *   o_parts   f64 [S][B][Hq][D], each part already normalised by its own sum
 *   lse_parts f64 [S][B][Hq],   -inf marks an empty part
 *   out       f64 [B][Hq][D];   lse f64 [B][Hq] (may be NULL)
 * With w_i = exp(lse_i - M), M = max over non-empty parts:
 *   out = sum_i w_i * o_i / sum_i w_i,   lse = M + ln(sum_i w_i).
 * All parts empty -> out = 0, lse = -inf.
 */
int kvo_combine(const double *o_parts, const double *lse_parts, double *out, double *lse,
                int S, int B, int Hq, int D) {
    if (S < 0 || B < 0 || Hq <= 0 || D <= 0) return KVO_ERR_ARG;
    const size_t BH = (size_t)B * (size_t)Hq;
    for (size_t bh = 0; bh < BH; ++bh) {
        double M = -INFINITY;
        for (int i = 0; i < S; ++i) {
            double li = lse_parts[(size_t)i * BH + bh];
            if (li > M) M = li;
        }
        double *o = out + bh * (size_t)D;
        if (M == -INFINITY) {
            for (int d = 0; d < D; ++d) o[d] = 0.0;
            if (lse) lse[bh] = -INFINITY;
            continue;
        }
        double wsum = 0.0;
        for (int i = 0; i < S; ++i) {
            double li = lse_parts[(size_t)i * BH + bh];
            if (li == -INFINITY) continue;
            wsum += exp(li - M);
        }
        for (int d = 0; d < D; ++d) {
            double acc = 0.0;
            for (int i = 0; i < S; ++i) {
                double li = lse_parts[(size_t)i * BH + bh];
                if (li == -INFINITY) continue;
                acc += exp(li - M) * o_parts[((size_t)i * BH + bh) * (size_t)D + d];
            }
            o[d] = acc / wsum;
        }
        if (lse) lse[bh] = M + log(wsum);
    }
    return KVO_OK;
}
