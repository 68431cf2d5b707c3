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
 * The softmax is the max-subtracted form (stable against overflow), evaluated in
 * separate passes (maximum; exponentials and their sum; normalised weighted
 * sum), which is how the paper's appendix of multi-turn self-correction
 * examples repairs a softmax (Example 1: subtract the row maximum before
 * exponentiating; Example 3: a max pass, an exp-and-sum pass and a normalise
 * pass for rows longer than one block).  Decode attention is exact up to
 * rounding order, so this file is that definition written out, with no
 * blocking, fusion or online rescaling.
 *
 * The split-K combine is the log-sum-exp identity for merging softmax results
 * computed over disjoint key sets (reductions done in several stages, which the
 * paper's experiments section names as a failure class for generated kernels).
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

/*
 * The step before attention for the newly decoded token of every sequence:
 * per-head RMS normalisation of its query and key, rotary position embedding
 * at its position, and the append of its key and value to the cache.  The
 * paper names Qwen3-8B as its policy model (section "Compact AMD Kernel LLMs"
 * and the training appendix) but defines neither operation: the formulas
 * below are this build's reading of that model's attention input (per-head
 * RMS norm with one gain vector shared by the heads, eps inside the square
 * root; rotate-half rotary embedding at the current length), the standard
 * textbook forms, not a statement of the paper.  RMS normalisation is among
 * the kernel families the experiments section lists.
 *
 *   pos_b = L_b (the current length, clamped to [0, cap]): the new token's position
 *   RMS:    x_d <- x_d / sqrt(mean_e x_e^2 + eps) * w_d       (skipped if w == NULL)
 *   rotary: for i < D/2, a_i = pos_b * theta^(-2i/D),
 *           y_i       = x_i       cos a_i - x_{i+D/2} sin a_i
 *           y_{i+D/2} = x_{i+D/2} cos a_i + x_i       sin a_i   (skipped if theta <= 0)
 *   q rows: RMS with w_q, then rotary.  k rows: RMS with w_k, then rotary.
 *   v rows: unchanged.
 *   Destination of the k and v rows of sequence b:
 *     paged (block_table != NULL): pool row page * P + pos % P, page =
 *       block_table[b][pos / P]; no write if pos >= cap or the page id is
 *       outside [0, num_pages)
 *     contiguous (block_table == NULL): row b * cap + pos (cap = Lmax); no
 *       write if pos >= cap
 *   new_lens[b] = pos + 1 if the rows are written, else pos.
 *
 * Outputs are the exact (binary64) values; their rounding to bf16 is left to
 * the comparison.  dest_row[b] is the pool/cache row index, or -1.
 *   q_in [B][Hq][D], k_in / v_in [B][Hkv][D]: bf16 bits
 *   q_out [B][Hq][D], k_out / v_out [B][Hkv][D]: binary64
 */
static void rms_rotate(const uint16_t *x, const float *w, int D, double eps, int pos,
                       double theta, double *y) {
    double tmp[1024];
    for (int d = 0; d < D; ++d) tmp[d] = bf16_to_f64(x[d]);
    if (w) {
        double ss = 0.0;
        for (int d = 0; d < D; ++d) ss += tmp[d] * tmp[d];
        const double r = 1.0 / sqrt(ss / (double)D + eps);
        for (int d = 0; d < D; ++d) tmp[d] = tmp[d] * r * (double)w[d];
    }
    if (theta > 0.0) {
        const int half = D / 2;
        for (int i = 0; i < half; ++i) {
            const double a = (double)pos * pow(theta, -2.0 * (double)i / (double)D);
            const double c = cos(a), s = sin(a);
            y[i] = tmp[i] * c - tmp[i + half] * s;
            y[i + half] = tmp[i + half] * c + tmp[i] * s;
        }
    } else {
        for (int d = 0; d < D; ++d) y[d] = tmp[d];
    }
}

int kvo_append(const uint16_t *q_in, const uint16_t *k_in, const uint16_t *v_in,
               const float *q_w, const float *k_w, const int32_t *block_table,
               const int32_t *seq_lens, int B, int Hq, int Hkv, int D, int page_size,
               int max_pages, int64_t num_pages, int Lmax, double eps, double theta,
               double *q_out, double *k_out, double *v_out, int64_t *dest_row,
               int32_t *new_lens) {
    if (!check_heads(B, Hq, Hkv, D) || D > 1024 || D % 2) return KVO_ERR_ARG;
    const int paged = block_table != NULL;
    if (paged && (page_size <= 0 || max_pages < 0 || num_pages < 0)) return KVO_ERR_ARG;
    if (!paged && Lmax < 0) return KVO_ERR_ARG;
    const int64_t cap = paged ? (int64_t)max_pages * page_size : (int64_t)Lmax;
    for (int b = 0; b < B; ++b) {
        int64_t L = seq_lens[b];
        if (L < 0) L = 0;
        if (L > cap) L = cap;
        const int pos = (int)L;
        for (int h = 0; h < Hq; ++h) {
            const size_t o = ((size_t)b * Hq + h) * (size_t)D;
            rms_rotate(q_in + o, q_w, D, eps, pos, theta, q_out + o);
        }
        for (int g = 0; g < Hkv; ++g) {
            const size_t o = ((size_t)b * Hkv + g) * (size_t)D;
            rms_rotate(k_in + o, k_w, D, eps, pos, theta, k_out + o);
            for (int d = 0; d < D; ++d) v_out[o + d] = bf16_to_f64(v_in[o + d]);
        }
        int64_t row = -1;
        if (pos < cap) {
            if (paged) {
                const int32_t page = block_table[(size_t)b * max_pages + pos / page_size];
                if (page >= 0 && (int64_t)page < num_pages)
                    row = (int64_t)page * page_size + pos % page_size;
            } else {
                row = (int64_t)b * cap + pos;
            }
        }
        dest_row[b] = row;
        new_lens[b] = row >= 0 ? pos + 1 : pos;
    }
    return KVO_OK;
}

/*
 * Round binary64 values to the nearest bf16 (ties to even), directly from the
 * exact value (no intermediate float, so no double rounding).  Finite inputs
 * within bf16's range; results as bf16 bit patterns.
 */
static uint16_t f64_to_bf16(double x) {
    const uint16_t sign = signbit(x) ? 0x8000u : 0u;
    double ax = fabs(x);
    if (ax == 0.0) return sign;
    int e;
    frexp(ax, &e);                          /* ax = m * 2^e, m in [0.5, 1) */
    int step = e - 8;                       /* 8 significant bits */
    if (step < -133) step = -133;           /* below the smallest normal: subnormal grid */
    const double r = ldexp(rint(ldexp(ax, -step)), step);  /* rint: nearest, ties to even */
    const float f = (float)r;               /* exact: r has at most 9 significant bits */
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    return (uint16_t)((u >> 16) | sign);
}

int kvo_round_bf16(const double *x, uint16_t *out, int64_t n) {
    if (n < 0) return KVO_ERR_ARG;
    for (int64_t i = 0; i < n; ++i) out[i] = f64_to_bf16(x[i]);
    return KVO_OK;
}

/*
 * 8-bit floating-point caches (OCP FP8 E4M3, "e4m3fn": 1 sign bit, 4 exponent
 * bits with bias 7, 3 mantissa bits, no infinities, S.1111.111 = NaN; largest
 * finite value 448).  The cache stores codes c; the values they stand for are
 * k_scale * fp8(c) for keys and v_scale * fp8(c) for values, one scale per
 * tensor.  Attention is then exactly the definition above over those values.
 */
static double fp8_e4m3_to_f64(uint8_t c) {
    const int sign = c >> 7, e = (c >> 3) & 15, m = c & 7;
    if (e == 15 && m == 7) return NAN;
    const double v = e == 0 ? ldexp((double)m, -9)          /* subnormal: m * 2^-3 * 2^(1-7) */
                            : ldexp((double)(8 + m), e - 10); /* (1 + m/8) * 2^(e-7) */
    return sign ? -v : v;
}

/* The value of every code, for the pins. */
int kvo_fp8_table(double *out256) {
    for (int c = 0; c < 256; ++c) out256[c] = fp8_e4m3_to_f64((uint8_t)c);
    return KVO_OK;
}

static void attend_one_fp8(const uint16_t *qh, const uint8_t *const *krow,
                           const uint8_t *const *vrow, int L, int D, double scale,
                           double k_scale, double v_scale, double *out, double *lse, double *s) {
    if (L == 0) {
        for (int d = 0; d < D; ++d) out[d] = 0.0;
        *lse = -INFINITY;
        return;
    }
    for (int t = 0; t < L; ++t) {
        double dot = 0.0;
        for (int d = 0; d < D; ++d)
            dot += bf16_to_f64(qh[d]) * (k_scale * fp8_e4m3_to_f64(krow[t][d]));
        s[t] = scale * dot;
    }
    double m = s[0];
    for (int t = 1; t < L; ++t)
        if (s[t] > m) m = s[t];
    double l = 0.0;
    for (int t = 0; t < L; ++t) {
        s[t] = exp(s[t] - m);
        l += s[t];
    }
    for (int d = 0; d < D; ++d) {
        double acc = 0.0;
        for (int t = 0; t < L; ++t) acc += s[t] * (v_scale * fp8_e4m3_to_f64(vrow[t][d]));
        out[d] = acc / l;
    }
    *lse = m + log(l);
}

/*
 * fp8 caches, contiguous (block_table == NULL: k, v uint8 [B][Lmax][Hkv][D])
 * or paged (k, v uint8 [num_pages][page_size][Hkv][D], block_table as for
 * kvo_decode_attn_paged).  q stays bf16; out, lse as for the bf16 calls.
 */
int kvo_decode_attn_fp8(const uint16_t *q, const uint8_t *k, const uint8_t *v,
                        const int32_t *block_table, const int32_t *lens, double *out,
                        double *lse, int B, int Hq, int Hkv, int D, int page_size,
                        int max_pages, int64_t num_pages, int Lmax, double scale,
                        double k_scale, double v_scale) {
    if (!check_heads(B, Hq, Hkv, D)) return KVO_ERR_ARG;
    const int paged = block_table != NULL;
    if (paged && (page_size <= 0 || max_pages < 0 || num_pages < 0)) return KVO_ERR_ARG;
    if (!paged && Lmax < 0) return KVO_ERR_ARG;
    const int64_t cap = paged ? (int64_t)page_size * max_pages : (int64_t)Lmax;
    int lmax = 0;
    for (int b = 0; b < B; ++b) {
        if (lens[b] < 0 || (int64_t)lens[b] > cap) return KVO_ERR_RANGE;
        if (lens[b] > lmax) lmax = lens[b];
        if (paged)
            for (int t = 0; t < lens[b]; t += page_size) {
                const int32_t p = block_table[(size_t)b * max_pages + t / page_size];
                if (p < 0 || (int64_t)p >= num_pages) return KVO_ERR_RANGE;
            }
    }
    const int group = Hq / Hkv;
    const size_t n = (size_t)(lmax > 0 ? lmax : 1);
    double *s = (double *)malloc(sizeof(double) * n);
    const uint8_t **kr = (const uint8_t **)malloc(sizeof(void *) * n);
    const uint8_t **vr = (const uint8_t **)malloc(sizeof(void *) * n);
    if (!s || !kr || !vr) {
        free(s); free(kr); free(vr);
        return KVO_ERR_NOMEM;
    }
    for (int b = 0; b < B; ++b) {
        for (int h = 0; h < Hq; ++h) {
            const int g = h / group;
            for (int t = 0; t < lens[b]; ++t) {
                size_t row;
                if (paged) {
                    const int32_t page = block_table[(size_t)b * max_pages + t / page_size];
                    row = ((size_t)page * (size_t)page_size + (size_t)(t % page_size)) *
                              (size_t)Hkv + (size_t)g;
                } else {
                    row = ((size_t)b * (size_t)Lmax + (size_t)t) * (size_t)Hkv + (size_t)g;
                }
                kr[t] = k + row * (size_t)D;
                vr[t] = v + row * (size_t)D;
            }
            double l_out;
            attend_one_fp8(q + ((size_t)b * Hq + h) * D, kr, vr, lens[b], D, scale, k_scale,
                           v_scale, out + ((size_t)b * Hq + h) * D, &l_out, s);
            if (lse) lse[(size_t)b * Hq + h] = l_out;
        }
    }
    free(s); free(kr); free(vr);
    return KVO_OK;
}

/*
 * Chunked prefill over a paged cache: every sequence b brings n_b new tokens
 * (rows q_start[b] .. q_start[b+1]-1 of q, packed over the batch), whose keys
 * and values already occupy positions L_b - n_b .. L_b - 1 of its cache
 * (L_b = lens[b]).  New token i sits at position p = L_b - n_b + i and, with
 * the causal mask, attends positions 0 .. p: exactly decode attention with
 * length p + 1 (no position below 0: p < 0 attends nothing).
 *   q        bf16 [T][Hq][D],  T = q_start[B]
 *   out      f64 [T][Hq][D];  lse f64 [T][Hq] (may be NULL)
 * q_start must be nondecreasing from 0 to T; page ids as for
 * kvo_decode_attn_paged (KVO_ERR_RANGE otherwise).
 */
int kvo_prefill_paged(const uint16_t *q, const uint16_t *k_pool, const uint16_t *v_pool,
                      const int32_t *block_table, const int32_t *q_start, const int32_t *lens,
                      double *out, double *lse, int B, int T, int Hq, int Hkv, int D,
                      int page_size, int max_pages, int64_t num_pages, double scale) {
    if (!check_heads(B, Hq, Hkv, D) || T < 0 || page_size <= 0 || max_pages < 0 ||
        num_pages < 0)
        return KVO_ERR_ARG;
    if (q_start[0] != 0 || q_start[B] != T) return KVO_ERR_RANGE;
    const int64_t cap = (int64_t)page_size * (int64_t)max_pages;
    int lmax = 0;
    for (int b = 0; b < B; ++b) {
        if (q_start[b + 1] < q_start[b]) return KVO_ERR_RANGE;
        if (lens[b] < 0 || (int64_t)lens[b] > cap) return KVO_ERR_RANGE;
        if (lens[b] > lmax) lmax = lens[b];
        for (int t = 0; t < lens[b]; t += page_size) {
            const int32_t p = block_table[(size_t)b * max_pages + t / page_size];
            if (p < 0 || (int64_t)p >= num_pages) return KVO_ERR_RANGE;
        }
    }
    const int group = Hq / Hkv;
    const size_t n = (size_t)(lmax > 0 ? lmax : 1);
    double *s = (double *)malloc(sizeof(double) * n);
    const uint16_t **kr = (const uint16_t **)malloc(sizeof(void *) * n);
    const uint16_t **vr = (const uint16_t **)malloc(sizeof(void *) * n);
    if (!s || !kr || !vr) {
        free(s); free(kr); free(vr);
        return KVO_ERR_NOMEM;
    }
    for (int b = 0; b < B; ++b) {
        const int nb = q_start[b + 1] - q_start[b];
        for (int i = 0; i < nb; ++i) {
            const int pos = lens[b] - nb + i;
            const int Lq = pos >= 0 ? pos + 1 : 0;
            const size_t row_q = (size_t)q_start[b] + (size_t)i;
            for (int h = 0; h < Hq; ++h) {
                const int g = h / group;
                for (int t = 0; t < Lq; ++t) {
                    const int32_t page = block_table[(size_t)b * max_pages + t / page_size];
                    const size_t row = ((size_t)page * (size_t)page_size +
                                        (size_t)(t % page_size)) * (size_t)Hkv + (size_t)g;
                    kr[t] = k_pool + row * (size_t)D;
                    vr[t] = v_pool + row * (size_t)D;
                }
                double l_out;
                attend_one(q + (row_q * Hq + h) * D, kr, vr, Lq, D, scale,
                           out + (row_q * Hq + h) * D, &l_out, s);
                if (lse) lse[row_q * Hq + h] = l_out;
            }
        }
    }
    free(s); free(kr); free(vr);
    return KVO_OK;
}
