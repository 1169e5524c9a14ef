/*
 * Reference (oracle) for appending a decode step's new key/value rows to a
 * paged KV cache, including FP8 (E4M3) quantisation on write.
 *
 * TEST INFRASTRUCTURE ONLY, like oracle.c: only the test suite, the smoke
 * check and the benchmark's CPU-baseline leg may load it; the GPU library
 * never links, calls or includes anything from here.
 *
 * What it computes. Each decode step produces one new token per in-flight
 * sample, whose key and value rows join that sample's key-value cache
 * (StreamRL Section 2.1, "Background": decoding reuses the cache of all
 * earlier tokens, so every step must first add its own). Sequence lengths
 * already count the new token, so for every sequence b with L = seq_lens[b]
 * >= 1 the new token is t = L - 1, stored in page block_table[b][t / P] at
 * slot t % P, for every KV head g. L = 0 appends nothing.
 *
 * kv_kind 0 (bf16): the row is copied bit for bit.
 *
 * kv_kind 1 (OCP E4M3 codes with one fp32 scale per (page, KV head), the
 * cached value being decode(code) * scale). The paper says nothing about FP8;
 * the reading taken here keeps every live slot of a page-head tile encoded
 * with the tile's current scale, and lets the scale only grow:
 *   a      = max_d |x_d|                      (fp32; NaN elements ignored)
 *   slot 0 (a fresh page):       s = a / 448, or 1 if a == 0
 *   slot > 0, a <= s_old * 448:  s = s_old                 (no change)
 *   slot > 0, a >  s_old * 448:  s = a / 448, and every earlier slot j of
 *                                the tile is re-encoded:
 *                                c_j <- enc((decode(c_j) * s_old) / s)
 *   the new row:                 c_t <- enc(x_d / s)
 * K and V follow this separately, each with its own scales. All scale and
 * code arithmetic is IEEE binary32 in exactly this order (the code decision
 * depends on it), enc() rounds to nearest with ties to an even mantissa,
 * saturates to +-448 and maps NaN to 0x7F.
 *
 * Status: 0 on success, -1 on an argument the definition cannot be applied to
 * (null pointer, negative or too-long length, page id outside [0, num_pages)).
 * Sequences are processed in order b = 0, 1, ...; callers give every
 * appending sequence a last page of its own.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

double sl_oracle_e4m3_to_double(uint8_t code);   /* oracle.c */

/*
 * binary32 -> OCP E4M3 code, from the format's definition: normal values
 * (1 + k/8) * 2^E for E in [-6, 8] (exponent field E + 7), subnormals
 * k * 2^-9, largest finite 448 = 1.75 * 2^8, the code S.1111.111 is NaN.
 * Round to nearest, ties to the even k; magnitudes >= 448 saturate.
 */
uint8_t sl_oracle_e4m3_encode(float y)
{
    if (isnan(y))
        return 0x7F;
    const uint8_t sign = signbit(y) ? 0x80 : 0x00;
    const double a = fabs((double)y);
    if (a >= 448.0)
        return sign | 0x7E;
    if (a < ldexp(1.0, -6)) {
        /* subnormal range: k * 2^-9 with k in 0..8 (k = 8 is the smallest normal, code 0x08) */
        const double k = nearbyint(a / ldexp(1.0, -9));
        return sign | (uint8_t)k;
    }
    int e;
    frexp(a, &e);                          /* a = f * 2^e, f in [0.5, 1) */
    int E = e - 1;                         /* a in [2^E, 2^(E+1)) */
    const double m = a / ldexp(1.0, E);    /* in [1, 2), exact */
    double k = nearbyint((m - 1.0) * 8.0); /* 0..8, ties to even */
    if (k == 8.0) {
        E += 1;
        k = 0.0;
    }
    return sign | (uint8_t)(((E + 7) << 3) | (int)k);
}

static float bf16_to_float(uint16_t bits)
{
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

/* One page-head tile (P x D codes) gains row x at `slot` (the rules above). */
static void append_e4m3(const uint16_t *x, int D, int slot, uint8_t *tile, float *scale)
{
    float a = 0.0f;
    for (int d = 0; d < D; ++d) {
        const float v = fabsf(bf16_to_float(x[d]));
        if (v > a)                         /* NaN compares false: ignored */
            a = v;
    }
    float s;
    if (slot == 0) {
        s = a > 0.0f ? a / 448.0f : 1.0f;
    } else {
        const float s_old = *scale;
        const float reach = s_old * 448.0f;
        if (a <= reach) {
            s = s_old;
        } else {
            s = a / 448.0f;
            for (int j = 0; j < slot; ++j)
                for (int d = 0; d < D; ++d) {
                    uint8_t *c = &tile[(size_t)j * D + d];
                    const float v = (float)sl_oracle_e4m3_to_double(*c) * s_old;
                    *c = sl_oracle_e4m3_encode(v / s);
                }
        }
    }
    for (int d = 0; d < D; ++d)
        tile[(size_t)slot * D + d] = sl_oracle_e4m3_encode(bf16_to_float(x[d]) / s);
    *scale = s;
}

int sl_oracle_kv_append(int kv_kind, int B, int Hkv, int D, int P, int max_blocks, int num_pages,
                        const uint16_t *k_new, const uint16_t *v_new, const int32_t *block_table,
                        const int32_t *seq_lens, void *k_pages, void *v_pages, float *k_scales,
                        float *v_scales)
{
    if (!k_new || !v_new || !block_table || !seq_lens || !k_pages || !v_pages)
        return -1;
    if (kv_kind == 1 && (!k_scales || !v_scales))
        return -1;
    if (B < 0 || Hkv <= 0 || D <= 0 || P <= 0 || max_blocks < 0 || num_pages < 0)
        return -1;
    for (int b = 0; b < B; ++b) {
        const int L = seq_lens[b];
        if (L == 0)
            continue;
        if (L < 0 || (long long)L > (long long)max_blocks * P)
            return -1;
        const int t = L - 1;
        const int page = block_table[(size_t)b * max_blocks + t / P];
        const int slot = t % P;
        if (page < 0 || page >= num_pages)
            return -1;
        for (int g = 0; g < Hkv; ++g) {
            const size_t tile = ((size_t)page * Hkv + g) * P * D;
            const uint16_t *kx = k_new + ((size_t)b * Hkv + g) * D;
            const uint16_t *vx = v_new + ((size_t)b * Hkv + g) * D;
            if (kv_kind == 0) {
                memcpy((uint16_t *)k_pages + tile + (size_t)slot * D, kx, sizeof(uint16_t) * D);
                memcpy((uint16_t *)v_pages + tile + (size_t)slot * D, vx, sizeof(uint16_t) * D);
            } else {
                append_e4m3(kx, D, slot, (uint8_t *)k_pages + tile, &k_scales[(size_t)page * Hkv + g]);
                append_e4m3(vx, D, slot, (uint8_t *)v_pages + tile, &v_scales[(size_t)page * Hkv + g]);
            }
        }
    }
    return 0;
}
