/*
 * Reference (oracle) for batched decode attention over a paged KV cache.
 *
 * TEST INFRASTRUCTURE ONLY. This file is the slow, plainly written CPU
 * definition that the GPU library is checked against. Only the test suite,
 * the smoke check and the benchmark's CPU-baseline leg may load it; the GPU
 * library never links, calls or includes anything from here, and this file
 * includes nothing from the GPU library.
 *
 * What it computes (the decode step of the generation stage, StreamRL
 * Section 2.1 "Background": each in-flight sample's newest token attends over
 * the key-value cache of its own context, which grows by one token per step;
 * the cache is stored in fixed-size pages addressed through a per-sequence
 * block table as in PagedAttention, cited in Section 8; batches are ragged
 * because continuous batching releases finished samples early, Section 6):
 *
 *   for every sequence b and query head h, with G = Hq / Hkv and g = h / G,
 *   L = seq_lens[b]:
 *     token t (0 <= t < L) lives in page  block_table[b][t / P]  at slot t % P
 *     s_t   = scale * sum_d q[b][h][d] * K[page][g][slot][d]
 *     m     = max_t s_t
 *     w_t   = exp(s_t - m)
 *     out[b][h][:] = sum_t w_t * V[page][g][slot][:] / sum_t w_t
 *   and out[b][h][:] = 0 when L == 0.
 *
 * This is the textbook softmax(q K^T * scale) V; the paper does not write
 * the formula down. Everything is carried in double precision and the
 * softmax is the plain two-pass form (max first, then weights): there is no
 * blocking, no online rescaling and no split of the token range, so a reader
 * can compare each loop with the definition above.
 *
 * Cache layout: K and V are separate arrays of shape
 * [num_pages][Hkv][P][D]; one page holds P consecutive tokens of every KV
 * head. kv_kind 0: bf16 (stored as the upper 16 bits of an IEEE binary32).
 * kv_kind 1: OCP FP8 E4M3 ("e4m3fn": exponent bias 7, no infinities, the
 * all-ones code is NaN, largest finite 448) with one fp32 scale per
 * (page, KV head) for K and another for V; the cached value is
 * decode(byte) * scale.
 *
 * Status: 0 on success, -1 on an argument the definition cannot be applied
 * to (null pointer, Hq not a multiple of Hkv, negative or too-long length,
 * page id outside [0, num_pages), a bad row index). On -1 nothing is
 * guaranteed about `out`.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* bf16 -> double: a bf16 value is the high half of a binary32; widening is exact. */
double sl_oracle_bf16_to_double(uint16_t bits)
{
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/*
 * OCP 8-bit floating point, E4M3 variant: 1 sign bit, 4 exponent bits
 * (bias 7), 3 mantissa bits. Exponent field 0 encodes subnormals
 * m/8 * 2^(1-7). Exponent field 15 is an ordinary binade except for
 * mantissa 7, which is NaN; there are no infinities.
 */
double sl_oracle_e4m3_to_double(uint8_t code)
{
    int sign = (code >> 7) & 1;
    int e = (code >> 3) & 0xF;
    int m = code & 0x7;
    double mag;
    if (e == 0xF && m == 0x7)
        return NAN;
    if (e == 0)
        mag = ldexp((double)m / 8.0, 1 - 7);
    else
        mag = ldexp(1.0 + (double)m / 8.0, e - 7);
    return sign ? -mag : mag;
}

/* Cached value of element d of token `slot` of (page, head g). */
static double kv_value(int kv_kind, const void *pages, const float *scales,
                       int Hkv, int P, int D, int page, int g, int slot, int d)
{
    size_t idx = (((size_t)page * Hkv + g) * P + slot) * D + d;
    if (kv_kind == 0)
        return sl_oracle_bf16_to_double(((const uint16_t *)pages)[idx]);
    return sl_oracle_e4m3_to_double(((const uint8_t *)pages)[idx]) *
           (double)scales[(size_t)page * Hkv + g];
}

/* One (sequence, query head) row of the definition above. */
static int attend_row(int kv_kind, int Hq, int Hkv, int D, int P, int max_blocks,
                      int num_pages, const uint16_t *q, const void *k_pages,
                      const void *v_pages, const float *k_scales,
                      const float *v_scales, const int32_t *block_table,
                      const int32_t *seq_lens, double scale, int b, int h,
                      double *out_row)
{
    int G = Hq / Hkv;
    int g = h / G;
    int L = seq_lens[b];
    const uint16_t *qrow = q + ((size_t)b * Hq + h) * D;
    double *s;
    double m, z;
    int t, d;

    for (d = 0; d < D; ++d)
        out_row[d] = 0.0;
    if (L == 0)
        return 0;
    if (L < 0 || L > max_blocks * P)
        return -1;

    s = (double *)malloc((size_t)L * sizeof(double));
    if (!s)
        return -1;

    /* Pass 1: every score, then their maximum. */
    for (t = 0; t < L; ++t) {
        int page = block_table[(size_t)b * max_blocks + t / P];
        int slot = t % P;
        double dot = 0.0;
        if (page < 0 || page >= num_pages) {
            free(s);
            return -1;
        }
        for (d = 0; d < D; ++d)
            dot += sl_oracle_bf16_to_double(qrow[d]) *
                   kv_value(kv_kind, k_pages, k_scales, Hkv, P, D, page, g, slot, d);
        s[t] = scale * dot;
    }
    m = s[0];
    for (t = 1; t < L; ++t)
        if (s[t] > m)
            m = s[t];

    /* Pass 2: weights, their sum, and the weighted sum of value rows. */
    z = 0.0;
    for (t = 0; t < L; ++t) {
        int page = block_table[(size_t)b * max_blocks + t / P];
        int slot = t % P;
        double w = exp(s[t] - m);
        z += w;
        for (d = 0; d < D; ++d)
            out_row[d] += w * kv_value(kv_kind, v_pages, v_scales, Hkv, P, D,
                                       page, g, slot, d);
    }
    for (d = 0; d < D; ++d)
        out_row[d] /= z;
    free(s);
    return 0;
}

/*
 * Decode attention for the sequences listed in `rows` (all B sequences when
 * rows == NULL, in which case nrows must equal B). out has shape
 * [nrows][Hq][D]; row i of out belongs to sequence rows[i].
 * nthreads <= 0 uses the OpenMP default.
 */
int sl_oracle_decode_attn(int kv_kind, int B, int Hq, int Hkv, int D, int P,
                          int max_blocks, int num_pages, const uint16_t *q,
                          const void *k_pages, const void *v_pages,
                          const float *k_scales, const float *v_scales,
                          const int32_t *block_table, const int32_t *seq_lens,
                          float scale, const int32_t *rows, int nrows,
                          double *out, int nthreads)
{
    int status = 0;
    long n, i;

    if (B < 0 || Hq <= 0 || Hkv <= 0 || D <= 0 || P <= 0 || max_blocks < 0 ||
        num_pages < 0 || nrows < 0)
        return -1;
    if (Hq % Hkv != 0)
        return -1;
    if (kv_kind != 0 && kv_kind != 1)
        return -1;
    if (!q || !k_pages || !v_pages || !block_table || !seq_lens || !out)
        return -1;
    if (kv_kind == 1 && (!k_scales || !v_scales))
        return -1;
    if (!rows && nrows != B)
        return -1;
    for (i = 0; rows && i < nrows; ++i)
        if (rows[i] < 0 || rows[i] >= B)
            return -1;

#ifdef _OPENMP
    /* The thread count applies to this call only (no global OpenMP setting). */
    if (nthreads <= 0)
        nthreads = omp_get_max_threads();
#else
    (void)nthreads;
#endif
    n = (long)nrows * Hq;
#pragma omp parallel for schedule(dynamic, 1) reduction(min : status) num_threads(nthreads)
    for (i = 0; i < n; ++i) {
        int r = (int)(i / Hq);
        int h = (int)(i % Hq);
        int b = rows ? rows[r] : r;
        int rc = attend_row(kv_kind, Hq, Hkv, D, P, max_blocks, num_pages, q,
                            k_pages, v_pages, k_scales, v_scales, block_table,
                            seq_lens, (double)scale, b, h,
                            out + ((size_t)r * Hq + h) * D);
        if (rc < status)
            status = rc;
    }
    return status;
}

/* Number of threads sl_oracle_decode_attn uses for this setting. */
int sl_oracle_max_threads(int nthreads)
{
#ifdef _OPENMP
    return nthreads > 0 ? nthreads : omp_get_max_threads();
#else
    (void)nthreads;
    return 1;
#endif
}
