#ifndef SL_APPEND_UNIT_H
#define SL_APPEND_UNIT_H
// KV append for one decode step: every sequence's new key/value rows join its
// paged cache before the step's attention reads it.
//
// With L = seq_lens[b] already counting the new token, the token t = L - 1
// goes to page block_table[b][t / 16], slot t % 16, for every KV head.
//
// bf16 cache: the row is stored as is.
//
// E4M3 cache (one fp32 scale per (page, KV head) for K and one for V; the
// cached value is decode(code) * scale): the scale of a page-head tile only
// grows. With a = max |x| over the row (NaN elements ignored):
//   slot 0 (fresh page)          s = a / 448 (1 if a == 0)
//   a <= s_old * 448             s = s_old
//   a >  s_old * 448             s = a / 448 and every earlier slot j of the
//                                tile is re-encoded: c = enc(decode(c) * s_old / s)
// and the new row is enc(x / s). enc() rounds to nearest even and saturates
// to +-448 (NaN -> 0x7F). All of it is binary32 arithmetic in that order, so
// the codes are reproducible bit for bit.
//
// One wavefront per (sequence, KV head); lane l holds elements
// [l * D/64, (l + 1) * D/64) of the row. The data per call is a few hundred
// bytes per unit, so the kernel is bound by the latency of its dependent
// loads (length -> block table -> scale -> old codes), not by bandwidth.
#include "sl_internal.h"

namespace sl {
namespace {


typedef short i16x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __builtin_bit_cast(float, (uint32_t)b << 16); }

// One E4M3 code -> binary32, exact (the bf16 conversion covers every code).
__device__ __forceinline__ float e4m3_to_f32(uint32_t code)
{
    const uint32_t w = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(code, 1.0f, false));
    return __builtin_bit_cast(float, w << 16);
}

// Signed-zero code of y if y rounds to zero in E4M3 (|y| <= 2^-10, half the
// smallest subnormal, a tie that goes to the even code 0), else 0xffffffff.
__device__ __forceinline__ uint32_t e4m3_zero_code(float y)
{
    const uint32_t u = __builtin_bit_cast(uint32_t, y);
    return (u & 0x7fffffffu) <= 0x3a800000u ? (u >> 24) & 0x80u : 0xffffffffu;
}

// Two binary32 values -> two E4M3 codes (low byte: a). Clamped to +-448
// first, so the conversion never overflows; NaN maps to 0x7F. Magnitudes up
// to 2^-10 (fp32 denormals among them, which the conversion does not round
// like other inputs) are encoded as signed zero directly.
__device__ __forceinline__ uint32_t f32x2_to_e4m3(float a, float b)
{
    const float ca = __builtin_fminf(__builtin_fmaxf(a, -448.0f), 448.0f);
    const float cb = __builtin_fminf(__builtin_fmaxf(b, -448.0f), 448.0f);
    const i16x2_t r = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(i16x2_t{0, 0}, ca, cb, 1.0f, false);
    uint32_t lo = (uint32_t)(uint16_t)r[0];
    const uint32_t za = e4m3_zero_code(a), zb = e4m3_zero_code(b);
    if (za != 0xffffffffu)
        lo = (lo & 0xff00u) | za;
    if (zb != 0xffffffffu)
        lo = (lo & 0x00ffu) | (zb << 8);
    if (a != a)
        lo = (lo & 0xff00u) | 0x7fu;
    if (b != b)
        lo = (lo & 0x00ffu) | 0x7f00u;
    return lo;
}

__device__ __forceinline__ float wave_absmax(float x)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1)
        x = __builtin_fmaxf(x, __shfl_xor(x, off, kWave));
    return x;
}

// Quantise-on-write of one row into one page-head tile (16 x D codes).
template <int D>
__device__ __forceinline__ void append_e4m3(const uint16_t *x, uint8_t *tile, float *scale, int slot, int lane)
{
    constexpr int E = D / kWave;   // elements per lane (1 or 2)
    float v[E];
    if constexpr (E == 2) {
        const uint32_t w = *reinterpret_cast<const uint32_t *>(x + 2 * lane);
        v[0] = __builtin_bit_cast(float, w << 16);
        v[1] = __builtin_bit_cast(float, w & 0xffff0000u);
    } else {
        v[0] = bf16_to_f32(x[lane]);
    }
    // NaN elements do not count towards the maximum. A comparison skips every
    // NaN (fmax would return a quiet NaN for a signalling one and lose the
    // other operand), so only finite or infinite magnitudes reach the wave max.
    float a = 0.0f;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const float m = __builtin_fabsf(v[e]);
        a = m > a ? m : a;
    }
    a = wave_absmax(a);

    float s;
    if (slot == 0) {
        s = a > 0.0f ? a / 448.0f : 1.0f;
    } else {
        const float s_old = *scale;
        if (a <= s_old * 448.0f) {
            s = s_old;
        } else {
            s = a / 448.0f;
            // Re-encode the earlier rows of the tile with the grown scale.
            uint32_t old[kPageSize - 1];
#pragma unroll
            for (int j = 0; j < kPageSize - 1; ++j)
                if (j < slot)
                    old[j] = E == 2 ? *reinterpret_cast<const uint16_t *>(tile + j * D + 2 * lane)
                                    : tile[j * D + lane];
#pragma unroll
            for (int j = 0; j < kPageSize - 1; ++j) {
                if (j < slot) {
                    const float r0 = (e4m3_to_f32(old[j] & 0xffu) * s_old) / s;
                    if constexpr (E == 2) {
                        const float r1 = (e4m3_to_f32(old[j] >> 8) * s_old) / s;
                        *reinterpret_cast<uint16_t *>(tile + j * D + 2 * lane) = (uint16_t)f32x2_to_e4m3(r0, r1);
                    } else {
                        tile[j * D + lane] = (uint8_t)f32x2_to_e4m3(r0, 0.0f);
                    }
                }
            }
        }
    }
    if constexpr (E == 2)
        *reinterpret_cast<uint16_t *>(tile + slot * D + 2 * lane) = (uint16_t)f32x2_to_e4m3(v[0] / s, v[1] / s);
    else
        tile[slot * D + lane] = (uint8_t)f32x2_to_e4m3(v[0] / s, 0.0f);
    if (lane == 0)
        *scale = s;
}

// The engine's bookkeeping for a step (staged mode only): store the step's
// lengths in set_seq_lens and apply its block-table updates, spread over
// threads [first, first + nthreads) of the launch. Indices were checked by
// the engine.
__device__ __forceinline__ void apply_stage(const AppendParams &p, int first, int nthreads)
{
    for (int i = first; i < p.batch; i += nthreads)
        p.set_seq_lens[i] = p.stage[i];
    for (int i = first; i < p.n_upd; i += nthreads) {
        const int32_t *u = p.stage + 2 * p.batch + 3 * i;
        p.set_block_table[(size_t)u[0] * p.max_blocks + u[1]] = u[2];
    }
}

// Append the new rows of unit `unit` = b * Hkv + g (one wavefront) for a
// sequence of length L (the new token included) whose token L - 1 lives in
// page `page`. An invalid length or page id leaves the cache untouched.
template <int D, bool FP8>
__device__ __forceinline__ void append_row(const AppendParams &p, int unit, int L, int page, int lane)
{
    if (L <= 0 || L > p.max_blocks * kPageSize || page < 0 || page >= p.num_pages)
        return;
    const int g = unit % p.num_kv_heads;
    const int t = L - 1;
    const int slot = t % kPageSize;
    const size_t tile = (size_t)page * p.num_kv_heads + g;   // page-head tile index
    const uint16_t *kx = p.k_new + (size_t)unit * D;
    const uint16_t *vx = p.v_new + (size_t)unit * D;
    if constexpr (!FP8) {
        uint16_t *kd = static_cast<uint16_t *>(p.k_pages) + (tile * kPageSize + slot) * D;
        uint16_t *vd = static_cast<uint16_t *>(p.v_pages) + (tile * kPageSize + slot) * D;
        for (int i = lane; i < D / 2; i += kWave) {
            reinterpret_cast<uint32_t *>(kd)[i] = reinterpret_cast<const uint32_t *>(kx)[i];
            reinterpret_cast<uint32_t *>(vd)[i] = reinterpret_cast<const uint32_t *>(vx)[i];
        }
    } else {
        uint8_t *kt = static_cast<uint8_t *>(p.k_pages) + tile * kPageSize * D;
        uint8_t *vt = static_cast<uint8_t *>(p.v_pages) + tile * kPageSize * D;
        append_e4m3<D>(kx, kt, p.k_scales + tile, slot, lane);
        append_e4m3<D>(vx, vt, p.v_scales + tile, slot, lane);
    }
}

// Append the new rows of unit `unit` = b * Hkv + g (one wavefront), with the
// length from the lengths array and the page from the block table, or, in
// staged mode, both from the staging buffer. Nothing is appended for an
// empty sequence.
template <int D, bool FP8>
__device__ __forceinline__ void append_unit(const AppendParams &p, int unit, int lane)
{
    const int b = unit / p.num_kv_heads;
    const int L = p.stage ? p.stage[b] : p.seq_lens[b];
    if (L <= 0 || L > p.max_blocks * kPageSize)
        return;
    const int page = p.stage ? p.stage[p.batch + b] : p.block_table[(size_t)b * p.max_blocks + (L - 1) / kPageSize];
    append_row<D, FP8>(p, unit, L, page, lane);
}

}  // namespace
}  // namespace sl

#endif  // SL_APPEND_UNIT_H
