#ifndef SL_DECODE_UNIT_H
#define SL_DECODE_UNIT_H
// Split-KV decode attention worker for gfx950.
//
// One wavefront is one worker. It streams its contiguous range of page-head
// tiles (see sl_internal.h) as a flat sequence, keeping an online-softmax
// state for the G query heads of the unit (sequence, KV head) the current tile
// belongs to, and finishing that unit whenever its last tile, or the end of
// the range, is reached. For the shared pages of prefix-shared attention the
// four wavefronts of a workgroup stream the same range, each computing one
// 16-row column block of the shared unit's query rows (kSharedPages).
//
// Per 16-token tile, with lane = n + 16 * quad (n = lane & 15, quad = lane >> 4):
//
//   scores  S^T[t][j] = sum_d K[t][d] Q[j][d]       v_mfma_f32_16x16x32_bf16
//           A = K   (row t = n, 8 consecutive d per lane; the tile is read as
//                    whole 1 KB runs and regrouped through LDS)
//           B = Q^T (column j = n; query rows j >= G are zero padding)
//           -> lane (j, quad) holds the scores of head j for tokens 4 quad + r
//   softmax running max / sum per head j, kept in the lanes of column j: the
//           only cross-lane step is a max over the four quads of a column
//   values  O^T[d][j] += sum_t V[t][d] P[j][t]       v_mfma_f32_16x16x16bf16_1k
//           A = V^T (lane (n, quad) holds V[4 quad + r][d_i(n)] for r = 0..3,
//                    gathered from four 16-byte row loads and repacked)
//           B = P^T exactly as the score MFMA left it (no data movement)
//           -> lane (j, quad) accumulates O[j][d] for D/4 consecutive d
//
// V goes straight from HBM into MFMA operand registers: its loads already
// cover whole 128-byte lines. The K operand layout would read only half a
// line per instruction (each row spread over four lanes), which streams at
// ~6.0 TB/s instead of ~6.85 TB/s on MI355X, so K is read in whole 1 KB runs
// and regrouped through a small per-wave LDS buffer. Both are streamed with
// non-temporal loads. Tiles are software-pipelined (pipeline_depth);
// the block-table entry of a tile (its unit metadata comes from a cursor over
// the units) is fetched one pipeline turn before the tile itself, and the
// query rows of a unit are loaded together with the unit's first tile, so the
// stream never waits on a dependent load, also across unit boundaries.
//
// FP8 pages hold OCP E4M3 codes; they are widened to bf16 exactly
// (v_cvt_scalef32_pk_bf16_fp8 with unit scale), the per-(page, head) key
// scale multiplies the fp32 scores and the value scale multiplies the
// probabilities before they are rounded for the value MFMA.
#include "sl_internal.h"

namespace sl {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

constexpr float kNegInf = -__builtin_inff();
// A partial state l = sum 2^(s - m), acc = sum 2^(s - m) v is exact for any
// reference m. The running maximum is raised only when a score exceeds it by
// more than this slack (base-2 units), which bounds the weights by 2^8 and
// leaves the accumulators untouched on most tiles after a unit's first.
constexpr float kRescaleSlack = 8.0f;
// Tiles in the software pipeline: two for a bf16 cache (three and four
// measured the same); three for E4M3, whose tiles carry half the bytes for
// the same work per tile.
template <bool FP8>
constexpr int pipeline_depth() { return FP8 ? 3 : 2; }
constexpr int kRawBufferWord3 = 0x00020000;  // untyped 32-bit buffer resource (CDNA3/4)

__device__ __forceinline__ u32x4_t ld128(const uint8_t *p) { return *reinterpret_cast<const u32x4_t *>(p); }

// K/V pages are read exactly once per call: stream them with non-temporal loads
// so they do not displace reusable lines in L2 / the Infinity Cache (measured on
// MI355X: random 4 KB tiles reach ~6.8 TB/s this way, ~6.0 TB/s with plain loads).
__device__ __forceinline__ u32x4_t ld128_stream(const uint8_t *p)
{
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(p));
}
__device__ __forceinline__ u32x2_t ld64_stream(const uint8_t *p)
{
    return __builtin_nontemporal_load(reinterpret_cast<const u32x2_t *>(p));
}
__device__ __forceinline__ uint32_t ld32_stream(const uint8_t *p)
{
    return __builtin_nontemporal_load(reinterpret_cast<const uint32_t *>(p));
}

// Two fp32 -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi)
{
    f32x2_t v = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __builtin_bit_cast(float, w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __builtin_bit_cast(float, w & 0xffff0000u); }

// Four E4M3 codes (one dword) -> four bf16 (two dwords), exact.
__device__ __forceinline__ void e4m3x4_to_bf16(uint32_t codes, uint32_t &lo, uint32_t &hi)
{
    lo = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(codes, 1.0f, false));
    hi = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(codes, 1.0f, true));
}

// Max / sum over the lanes n, n + 16, n + 32, n + 48 of a column.
// (The gfx950 lane-swap builtins would avoid the LDS crossbar here, but this
// compiler folds max(h[0], h[1]) of their two results to one of them, so the
// plain shuffles are used.)
__device__ __forceinline__ float quad_max(float x)
{
    x = fmaxf(x, __shfl_xor(x, 16, kWave));
    return fmaxf(x, __shfl_xor(x, 32, kWave));
}
__device__ __forceinline__ float quad_sum(float x)
{
    x += __shfl_xor(x, 16, kWave);
    return x + __shfl_xor(x, 32, kWave);
}

template <int D, bool FP8>
struct Tile {
    // Per-lane dwords of K (score-MFMA A operands) and V (four rows).
    static constexpr int KW = FP8 ? D / 16 : D / 8;
    static constexpr int VW = FP8 ? D / 16 : D / 8;
    uint32_t k[KW];
    uint32_t v[VW];
    u32x4_t q[D / 32];   // the unit's query rows, loaded with a unit's first tile only
    float scl;           // FP8: key scale in lanes 0-31, value scale in lanes 32-63
    uint32_t meta;       // tile metadata (kMeta* bits, wave-uniform)
    bool bad_page;       // the block table named a page outside the pool
};

// Query element index held by (quad, item) in k-step s; must match k_operand.
template <int D, bool FP8>
__device__ __forceinline__ int q_index(int s, int quad)
{
    return FP8 ? quad * (D / 4) + 8 * s : 32 * s + 8 * quad;
}

// Issue every load of one tile. All loads are unconditional. K/V are streamed
// with non-temporal loads (STREAM) unless the tile is read by several
// wavefronts at once (the column blocks of a shared unit), where plain loads
// let the siblings find it in L2. `blk` < 0: a single-unit tile, whose query
// rows are the group's G heads; `blk` >= 0: column block blk of a shared unit
// (rows 16 blk + n, member r / G and head r % G of the group).
template <int D, bool FP8, bool STREAM = true>
__device__ __forceinline__ void issue_tile(Tile<D, FP8> &t, const SplitParams &p, int32_t page,
                                           uint32_t meta, bool with_q, int n, int quad, int lane, int blk = -1)
{
    auto ld128_kv = [](const uint8_t *a) { return STREAM ? ld128_stream(a) : ld128(a); };
    auto ld64_kv = [](const uint8_t *a) {
        return STREAM ? ld64_stream(a) : *reinterpret_cast<const u32x2_t *>(a);
    };
    auto ld32_kv = [](const uint8_t *a) {
        return STREAM ? ld32_stream(a) : *reinterpret_cast<const uint32_t *>(a);
    };
    constexpr size_t kTileBytes = (size_t)kPageSize * D * (FP8 ? 1 : 2);
    t.meta = meta;
    t.bad_page = page < 0;
    const size_t tile = (size_t)(page < 0 ? 0 : page);
    const uint8_t *kt = static_cast<const uint8_t *>(p.k_pages) + tile * kTileBytes;
    const uint8_t *vt = static_cast<const uint8_t *>(p.v_pages) + tile * kTileBytes;
    // K: whole 1 KB runs per instruction (lane l reads bytes 16 l of each
    // run), so every instruction covers complete 128-byte lines; the rows are
    // regrouped into the score-MFMA layout through LDS when the tile is used.
#pragma unroll
    for (int i = 0; i < Tile<D, FP8>::KW / 4; ++i) {
        const u32x4_t x = ld128_kv(kt + 1024 * i + 16 * lane);
#pragma unroll
        for (int c = 0; c < 4; ++c)
            t.k[4 * i + c] = x[c];
    }
    if constexpr (!FP8) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const uint8_t *src = vt + ((4 * quad + r) * D + n * (D / 16)) * 2;
            if constexpr (D == 128) {
                const u32x4_t x = ld128_kv(src);
#pragma unroll
                for (int c = 0; c < 4; ++c)
                    t.v[4 * r + c] = x[c];
            } else {
                const u32x2_t x = ld64_kv(src);
                t.v[2 * r] = x[0];
                t.v[2 * r + 1] = x[1];
            }
        }
    } else {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const uint8_t *src = vt + (4 * quad + r) * D + n * (D / 16);
            if constexpr (D == 128) {
                const u32x2_t x = ld64_kv(src);
                t.v[2 * r] = x[0];
                t.v[2 * r + 1] = x[1];
            } else {
                t.v[r] = ld32_kv(src);
            }
        }
        const float *sp = (lane & 32) ? p.v_scales : p.k_scales;
        t.scl = sp[tile];
    }
    // The query rows of a unit travel with the unit's first tile (or the
    // worker's first tile); lanes past the group read row G - 1 and are zeroed
    // when the operand is formed.
    if (with_q) {
        const int G = p.group;
        int rel = min(n, G - 1);
        if (blk >= 0) {   // rows past the shared unit's read its first row (never written out)
            const int r = 16 * blk + n;
            rel = r < ((int)(meta & 15u) + 1) * G ? (r / G) * p.num_q_heads + r % G : 0;
        }
        const uint16_t *qrow = p.q + ((size_t)(meta >> kMetaRowShift) + (size_t)rel) * D;
#pragma unroll
        for (int s = 0; s < D / 32; ++s)
            t.q[s] = ld128(reinterpret_cast<const uint8_t *>(qrow + q_index<D, FP8>(s, quad)));
    }
}

// Regroup the K tile (loaded as whole 1 KB runs) into the score-MFMA layout
// through this wave's LDS buffer: lane (t, quad) needs row t, and for bf16
// the 16-byte chunks 4 s + quad (s = 0 .. D/32 - 1), for FP8 the D/64 chunks
// starting at quad D/64. A chunk c of row r is stored at position
// c ^ ((r / P) % C) of its row (P rows per 256 bytes, C chunks per row), which
// makes the 16-lane groups of both the writes and the reads hit distinct banks.
template <int D, bool FP8>
__device__ __forceinline__ void regroup_k(const Tile<D, FP8> &t, uint8_t *lds, int lane, int n, int quad,
                                          u32x4_t (&kc)[FP8 ? D / 64 : D / 32])
{
    constexpr int R = D * (FP8 ? 1 : 2);   // bytes per row
    constexpr int C = R / 16;               // 16-byte chunks per row
    constexpr int P = 256 / R;              // rows per 256 bytes
#pragma unroll
    for (int i = 0; i < Tile<D, FP8>::KW / 4; ++i) {
        const int off = 1024 * i + 16 * lane;
        const int r = off / R, c = (off % R) / 16;
        *reinterpret_cast<u32x4_t *>(lds + r * R + 16 * (c ^ ((r / P) % C))) =
            u32x4_t{t.k[4 * i], t.k[4 * i + 1], t.k[4 * i + 2], t.k[4 * i + 3]};
    }
    const int key = (n / P) % C;
#pragma unroll
    for (int s = 0; s < (FP8 ? D / 64 : D / 32); ++s) {
        const int c = FP8 ? quad * (D / 64) + s : 4 * s + quad;
        kc[s] = *reinterpret_cast<const u32x4_t *>(lds + n * R + 16 * (c ^ key));
    }
}

// Score-MFMA A operand for k-step s (8 bf16 values of row t = n).
template <int D, bool FP8>
__device__ __forceinline__ bf16x8_t k_operand(const u32x4_t (&kc)[FP8 ? D / 64 : D / 32], int s)
{
    u32x4_t w;
    if constexpr (!FP8) {
        w = kc[s];
    } else {
        const uint32_t lo = kc[s / 2][2 * (s % 2)], hi = kc[s / 2][2 * (s % 2) + 1];
        uint32_t a, b, c, d;
        e4m3x4_to_bf16(lo, a, b);
        e4m3x4_to_bf16(hi, c, d);
        w = u32x4_t{a, b, c, d};
    }
    return __builtin_bit_cast(bf16x8_t, w);
}

template <int D>
struct Piece {
    f32x4_t acc[D / 16];
    float m;   // running max of this lane's head, base-2 units
    float l;   // this lane's share of the sum of (bf16-rounded) weights
};

template <int D>
__device__ __forceinline__ void reset(Piece<D> &st)
{
#pragma unroll
    for (int i = 0; i < D / 16; ++i)
        st.acc[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    st.m = kNegInf;
    st.l = 0.f;
}

// One tile of the online softmax. `valid` = live tokens in this page (1..16).
template <int D, bool FP8>
__device__ __forceinline__ void compute_tile(Piece<D> &st, const Tile<D, FP8> &t,
                                             const bf16x8_t (&qop)[D / 32], float score_mul,
                                             int valid, uint8_t *lds, int lane, int n, int quad)
{
    u32x4_t kc[FP8 ? D / 64 : D / 32];
    regroup_k<D, FP8>(t, lds, lane, n, quad, kc);
    f32x4_t s4 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < D / 32; ++s)
        s4 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k_operand<D, FP8>(kc, s), qop[s], s4, 0, 0, 0);

    float vmul = 1.0f;
    if constexpr (FP8) {
        const int bits = __builtin_bit_cast(int, t.scl);
        score_mul *= __builtin_bit_cast(float, __builtin_amdgcn_readlane(bits, 0));
        vmul = __builtin_bit_cast(float, __builtin_amdgcn_readlane(bits, 32));
    }
    float sc[4];
#pragma unroll
    for (int r = 0; r < 4; ++r)
        sc[r] = s4[r] * score_mul;
    if (valid < kPageSize) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
            if (4 * quad + r >= valid)
                sc[r] = kNegInf;
    }
    // The head's maximum over the tile (four lanes) is needed only when one of
    // them exceeds the running maximum by the slack: a wave-wide vote skips
    // the cross-lane exchange on the other tiles, with the same result.
    const float lmx = fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3]));
    if (__builtin_amdgcn_ballot_w64(lmx > st.m + kRescaleSlack) != 0) {
        const float mx = quad_max(lmx);
        if (mx > st.m + kRescaleSlack) {
            const float alpha = __builtin_amdgcn_exp2f(st.m - mx);   // 0 on a unit's first tile
            st.l *= alpha;
#pragma unroll
            for (int i = 0; i < D / 16; ++i)
                st.acc[i] *= alpha;
            st.m = mx;
        }
    }
    float pr[4];
#pragma unroll
    for (int r = 0; r < 4; ++r)
        pr[r] = __builtin_amdgcn_exp2f(sc[r] - st.m);
    // The value product takes the weights rounded to bf16, and the sum of
    // weights adds those same rounded values, so the normalisation cancels
    // their rounding: a token that holds all the weight returns its own value
    // row exactly, and the remaining error scales with the spread of the value
    // rows around the output. For E4M3 the weights carry the page's value
    // scale, w = bf16(p s); the sum then adds w / s, the rounded weight without
    // the scale (a zero or non-finite scale, for which that quotient is
    // meaningless, adds the rounded p instead).
    i16x4_t pb;
    if constexpr (FP8) {
        const uint32_t w01 = pack_bf16(pr[0] * vmul, pr[1] * vmul);
        const uint32_t w23 = pack_bf16(pr[2] * vmul, pr[3] * vmul);
        pb = __builtin_bit_cast(i16x4_t, u32x2_t{w01, w23});
        const float vinv = __builtin_amdgcn_rcpf(vmul);   // wave-uniform
        if (__builtin_isfinite(vinv) && vinv != 0.0f) {
            st.l += ((bf16_lo(w01) + bf16_hi(w01)) + (bf16_lo(w23) + bf16_hi(w23))) * vinv;
        } else {
            const uint32_t p01 = pack_bf16(pr[0], pr[1]);
            const uint32_t p23 = pack_bf16(pr[2], pr[3]);
            st.l += (bf16_lo(p01) + bf16_hi(p01)) + (bf16_lo(p23) + bf16_hi(p23));
        }
    } else {
        const uint32_t p01 = pack_bf16(pr[0], pr[1]);
        const uint32_t p23 = pack_bf16(pr[2], pr[3]);
        st.l += (bf16_lo(p01) + bf16_hi(p01)) + (bf16_lo(p23) + bf16_hi(p23));
        pb = __builtin_bit_cast(i16x4_t, u32x2_t{p01, p23});
    }

    // Value operands. Lane (n, quad) holds D/16 consecutive elements of the
    // value rows of tokens 4 quad + r (r = 0..3); value block i takes element i
    // of the four rows, rows 0-1 in its low dword and rows 2-3 in the high one.
    // Byte permutes gather them: bf16 halves directly, E4M3 codes in pairs of
    // rows before one widening per two blocks. Dead slots (only in a
    // sequence's last page) hold arbitrary cache contents and are zeroed first,
    // as 0 * NaN would poison the MFMA.
    constexpr int VR = Tile<D, FP8>::VW / 4;   // dwords per row
    uint32_t vr[4 * VR];
#pragma unroll
    for (int k = 0; k < 4 * VR; ++k)
        vr[k] = t.v[k];
    if (valid < kPageSize) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int c = 0; c < VR; ++c)
                vr[r * VR + c] = 4 * quad + r < valid ? vr[r * VR + c] : 0u;
    }
#pragma unroll
    for (int i = 0; i < D / 16; i += 2) {
        uint32_t lo0, lo1, hi0, hi1;
        if constexpr (FP8) {
            // Bytes (row a, row b) of elements i and i + 1, then one widening per element.
            const int c = i / 4;
            const uint32_t sel = (i % 4) == 0 ? 0x05010400u : 0x07030602u;
            const uint32_t p01 = __builtin_amdgcn_perm(vr[VR + c], vr[c], sel);
            const uint32_t p23 = __builtin_amdgcn_perm(vr[3 * VR + c], vr[2 * VR + c], sel);
            lo0 = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(p01, 1.0f, false));
            lo1 = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(p01, 1.0f, true));
            hi0 = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(p23, 1.0f, false));
            hi1 = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(p23, 1.0f, true));
        } else {
            // Dword w holds elements 2w (low half) and 2w + 1 (high half) of a row.
            const int w = i / 2;
            lo0 = __builtin_amdgcn_perm(vr[VR + w], vr[w], 0x05040100u);
            lo1 = __builtin_amdgcn_perm(vr[VR + w], vr[w], 0x07060302u);
            hi0 = __builtin_amdgcn_perm(vr[3 * VR + w], vr[2 * VR + w], 0x05040100u);
            hi1 = __builtin_amdgcn_perm(vr[3 * VR + w], vr[2 * VR + w], 0x07060302u);
        }
        st.acc[i] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(i16x4_t, u32x2_t{lo0, hi0}), pb,
                                                              st.acc[i], 0, 0, 0);
        st.acc[i + 1] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(i16x4_t, u32x2_t{lo1, hi1}),
                                                                  pb, st.acc[i + 1], 0, 0, 0);
    }
}

// Store this lane's share of a partial state (m, l, acc) as row `row` of
// (part_ml [][2], part_acc [][D]); l is the head's full sum (quad_sum).
template <int D>
__device__ __forceinline__ void store_partial(const Piece<D> &st, float l, bool bad, float *part_ml,
                                              float *part_acc, size_t row, int quad)
{
    const float poison = bad ? __builtin_nanf("") : 0.0f;
    float *dst = part_acc + row * D + quad * (D / 4);
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int i = 0; i < D / 16; i += 4)
            *reinterpret_cast<f32x4_t *>(dst + r * (D / 16) + i) =
                f32x4_t{st.acc[i][r], st.acc[i + 1][r], st.acc[i + 2][r], st.acc[i + 3][r]} + poison;
    if (quad == 0)   // a NaN maximum keeps the poison alive through the merge weights
        *reinterpret_cast<f32x2_t *>(part_ml + row * 2) = f32x2_t{st.m + poison, l};
}

// Finish the current unit: normalise and write its bf16 rows if the whole unit
// was seen and nothing else is merged into it (`full`), else store the partial
// state, G rows, in slot `slot` of (part_ml, part_acc).
template <int D>
__device__ __forceinline__ void finish_unit(const SplitParams &p, Piece<D> &st, uint32_t row0, bool full,
                                            bool bad, float *part_ml, float *part_acc, size_t slot, int n,
                                            int quad)
{
    const int G = p.group;
    const float l = quad_sum(st.l);
    const int d0 = quad * (D / 4);   // this lane holds O[row0 + n][d0 .. d0 + D/4)
    if (n >= G)
        return;
    if (full) {
        const float inv = bad ? __builtin_nanf("") : 1.0f / l;
        uint8_t *dst = reinterpret_cast<uint8_t *>(p.out + ((size_t)row0 + n) * D + d0);
#pragma unroll
        for (int c = 0; c < D / 32; ++c) {
            // output columns d0 + 8c .. 8c + 7 are acc[i][r] with r * D/16 + i = 8c + ...
            uint32_t wv[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int k0 = 8 * c + 2 * e;   // flat index r * (D/16) + i
                const int r0 = k0 / (D / 16), i0 = k0 % (D / 16);
                const int k1 = k0 + 1;
                const int r1 = k1 / (D / 16), i1 = k1 % (D / 16);
                wv[e] = pack_bf16(st.acc[i0][r0] * inv, st.acc[i1][r1] * inv);
            }
            *reinterpret_cast<u32x4_t *>(dst + 16 * c) = u32x4_t{wv[0], wv[1], wv[2], wv[3]};
        }
    } else {
        store_partial<D>(st, l, bad, part_ml, part_acc, slot * G + n, quad);
    }
}

struct ScanSum {
    static constexpr int32_t kIdentity = 0;
    __device__ static int32_t op(int32_t a, int32_t b) { return a + b; }
};
struct ScanMax {
    static constexpr int32_t kIdentity = -2147483647 - 1;
    __device__ static int32_t op(int32_t a, int32_t b) { return a > b ? a : b; }
};

// Output staging for plain attention. Vector-memory stores and loads share
// one completion counter on this part, so a wait for a load issued after a
// store also waits for the store, which under a full read stream takes
// microseconds: writing each finished unit's rows out at once stalled the
// worker at its next tile (measured: ~2.9 us per unit with 256-token
// sequences), and so did the partial state of the range's first, cut unit
// (2.6% of the 7B-like step). Finished rows are therefore normalised into a
// per-wave LDS stage, and the first piece's state kept there too, and both
// are written out only when the stage is full or the worker's range ends,
// where no later load waits on them.
constexpr int kOutStageBytes = 16384;                       // per wave
constexpr int kMaxOutSlots = kOutStageBytes / (1 * 64 * 2); // smallest slot: G = 1, D = 64

// The bf16 rows of a finished unit (this lane's D/4 outputs of row n) into
// its stage slot; l is the head's full sum of weights.
template <int D>
__device__ __forceinline__ void stage_output(const Piece<D> &st, float l, bool bad, uint8_t *slot, int n, int quad)
{
    const float inv = bad ? __builtin_nanf("") : 1.0f / l;
    uint8_t *dst = slot + ((size_t)n * D + quad * (D / 4)) * 2;
#pragma unroll
    for (int c = 0; c < D / 32; ++c) {
        uint32_t wv[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int k0 = 8 * c + 2 * e;   // flat index r * (D/16) + i, as in finish_unit
            const int r0 = k0 / (D / 16), i0 = k0 % (D / 16);
            const int k1 = k0 + 1;
            const int r1 = k1 / (D / 16), i1 = k1 % (D / 16);
            wv[e] = pack_bf16(st.acc[i0][r0] * inv, st.acc[i1][r1] * inv);
        }
        *reinterpret_cast<u32x4_t *>(dst + 16 * c) = u32x4_t{wv[0], wv[1], wv[2], wv[3]};
    }
}

// Write the first `count` staged units out. A unit's G rows are one
// contiguous block of G * D * 2 bytes both in the stage and in `out` (from
// row rows[s]), so every lane copies 16-byte pieces 1 KB apart: each store
// instruction writes whole cache lines. (Stored straight from the
// accumulator layout, each instruction left 16-byte pieces 64 bytes apart,
// over a hundred partial-line writes per unit, which drained slowly enough
// under a full read stream to cost ~20 us per flush of nine units.)
__device__ __forceinline__ void flush_outputs(const SplitParams &p, int head_dim, const uint8_t *stage,
                                              const uint32_t *rows, int count, int slot_bytes, int lane)
{
    for (int s = 0; s < count; ++s) {
        const uint8_t *src = stage + (size_t)s * slot_bytes;
        uint8_t *dst = reinterpret_cast<uint8_t *>(p.out + (size_t)rows[s] * head_dim);
        for (int off = 16 * lane; off < slot_bytes; off += 16 * kWave)
            *reinterpret_cast<u32x4_t *>(dst + off) = *reinterpret_cast<const u32x4_t *>(src + off);
    }
}

// The partial state (m, l, acc) of a cut unit into the stage, laid out as
// in the workspace: G rows of D fp32 (acc), then G pairs (m, l); l is the
// head's full sum of weights.
template <int D>
__device__ __forceinline__ void stage_partial(const Piece<D> &st, float l, bool bad, uint8_t *area, int G, int n,
                                              int quad)
{
    const float poison = bad ? __builtin_nanf("") : 0.0f;
    float *acc = reinterpret_cast<float *>(area) + (size_t)n * D + quad * (D / 4);
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int i = 0; i < D / 16; i += 4)
            *reinterpret_cast<f32x4_t *>(acc + r * (D / 16) + i) =
                f32x4_t{st.acc[i][r], st.acc[i + 1][r], st.acc[i + 2][r], st.acc[i + 3][r]} + poison;
    if (quad == 0)
        *reinterpret_cast<f32x2_t *>(reinterpret_cast<float *>(area) + (size_t)G * D + 2 * n) =
            f32x2_t{st.m + poison, l};
}

// Write a staged partial state to slot `slot` of (part_ml, part_acc) as two
// contiguous blocks.
__device__ __forceinline__ void flush_partial(const SplitParams &p, int head_dim, const uint8_t *area, size_t slot,
                                              int lane)
{
    const int G = p.group;
    const int acc_bytes = G * head_dim * 4;
    uint8_t *dst = reinterpret_cast<uint8_t *>(p.part_acc + slot * G * head_dim);
    for (int off = 16 * lane; off < acc_bytes; off += 16 * kWave)
        *reinterpret_cast<u32x4_t *>(dst + off) = *reinterpret_cast<const u32x4_t *>(area + off);
    if (lane < G)
        *reinterpret_cast<f32x2_t *>(p.part_ml + (slot * G + lane) * 2) =
            *reinterpret_cast<const f32x2_t *>(area + acc_bytes + 8 * lane);
}

// Prefix own pages: the fp32 states of finished own units that the merge
// combines are queued per wave in LDS and written when the queue is full or
// the range ends, for the reason given above for the output stage. The queue
// holds two states at G <= 8 (D = 128) and stays small, so the fused prefix
// kernel keeps two workgroups per CU (a 16 KB queue per wave did not).
constexpr int kOwnStageBytes = 8448;                        // per wave
constexpr int kMaxOwnSlots = kOwnStageBytes / ((1 * (64 + 2) * 4 + 15) & ~15);

// Write `count` queued states: entry s holds G rows of D fp32 (acc) and G
// pairs (m, l) as stage_partial lays them out; dest[s] = slot << 1 | (unit
// area ? 1 : 0), the slot in (part_ml, part_acc) or (unit_ml, unit_acc).
__device__ __forceinline__ void flush_states(const SplitParams &p, int head_dim, const uint8_t *stage,
                                             const uint32_t *dest, int count, int area_bytes, int lane)
{
    const int G = p.group;
    const int acc_bytes = G * head_dim * 4;
    for (int s = 0; s < count; ++s) {
        const uint32_t d = dest[s];
        const size_t slot = d >> 1;
        float *const pml = (d & 1u) ? p.unit_ml : p.part_ml;
        float *const pacc = (d & 1u) ? p.unit_acc : p.part_acc;
        const uint8_t *area = stage + (size_t)s * area_bytes;
        uint8_t *dst = reinterpret_cast<uint8_t *>(pacc + slot * G * head_dim);
        for (int off = 16 * lane; off < acc_bytes; off += 16 * kWave)
            *reinterpret_cast<u32x4_t *>(dst + off) = *reinterpret_cast<const u32x4_t *>(area + off);
        if (lane < G)
            *reinterpret_cast<f32x2_t *>(pml + (slot * G + lane) * 2) =
                *reinterpret_cast<const f32x2_t *>(area + acc_bytes + 8 * lane);
    }
}

// Turns a[0, n) (in LDS, written before a barrier) into its exclusive
// prefix scan under Op (sum or maximum) and stores the total in a[n]. Every
// thread of the workgroup calls it; each scans a contiguous run. Ends with a
// barrier.
template <class Op = ScanSum>
__device__ __forceinline__ void block_exclusive_scan(int32_t *a, int n)
{
    __shared__ int32_t s_wave[kWavesPerBlock];
    constexpr int T = kWave * kWavesPerBlock;
    const int tid = threadIdx.x;
    const int per = (n + T - 1) / T;
    const int lo = min(n, tid * per), hi = min(n, lo + per);
    int local = Op::kIdentity;
    for (int i = lo; i < hi; ++i)
        local = Op::op(local, a[i]);
    const int lane = tid & (kWave - 1), wave = tid / kWave;
    int incl = local;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const int v = __shfl_up(incl, off, kWave);
        if (lane >= off)
            incl = Op::op(incl, v);
    }
    const int excl_in_wave = __shfl_up(incl, 1, kWave);
    if (lane == kWave - 1)
        s_wave[wave] = incl;
    __syncthreads();
    int base = Op::kIdentity, total = Op::kIdentity;
#pragma unroll
    for (int k = 0; k < kWavesPerBlock; ++k) {
        if (k < wave)
            base = Op::op(base, s_wave[k]);
        total = Op::op(total, s_wave[k]);
    }
    int run = Op::op(base, lane > 0 ? excl_in_wave : Op::kIdentity);
    for (int i = lo; i < hi; ++i) {
        const int v = a[i];
        a[i] = run;
        run = Op::op(run, v);
    }
    if (tid == 0)
        a[n] = total;
    __syncthreads();
}

// Two independent exclusive scans, a[0, n) under OpA and b[0, m) under OpB,
// with their totals in a[n] and b[m], sharing the barriers of one scan.
template <class OpA, class OpB>
__device__ __forceinline__ void block_exclusive_scan2(int32_t *a, int n, int32_t *b, int m)
{
    __shared__ int32_t s_wave[2][kWavesPerBlock];
    constexpr int T = kWave * kWavesPerBlock;
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1), wave = tid / kWave;
    const int pa = (n + T - 1) / T, pb = (m + T - 1) / T;
    const int alo = min(n, tid * pa), ahi = min(n, alo + pa);
    const int blo = min(m, tid * pb), bhi = min(m, blo + pb);
    int la = OpA::kIdentity, lb = OpB::kIdentity;
    for (int i = alo; i < ahi; ++i)
        la = OpA::op(la, a[i]);
    for (int i = blo; i < bhi; ++i)
        lb = OpB::op(lb, b[i]);
    int ia = la, ib = lb;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const int va = __shfl_up(ia, off, kWave);
        const int vb = __shfl_up(ib, off, kWave);
        if (lane >= off) {
            ia = OpA::op(ia, va);
            ib = OpB::op(ib, vb);
        }
    }
    const int ea = __shfl_up(ia, 1, kWave), eb = __shfl_up(ib, 1, kWave);
    if (lane == kWave - 1) {
        s_wave[0][wave] = ia;
        s_wave[1][wave] = ib;
    }
    __syncthreads();
    int base_a = OpA::kIdentity, tot_a = OpA::kIdentity, base_b = OpB::kIdentity, tot_b = OpB::kIdentity;
#pragma unroll
    for (int k = 0; k < kWavesPerBlock; ++k) {
        if (k < wave) {
            base_a = OpA::op(base_a, s_wave[0][k]);
            base_b = OpB::op(base_b, s_wave[1][k]);
        }
        tot_a = OpA::op(tot_a, s_wave[0][k]);
        tot_b = OpB::op(tot_b, s_wave[1][k]);
    }
    int ra = OpA::op(base_a, lane > 0 ? ea : OpA::kIdentity);
    for (int i = alo; i < ahi; ++i) {
        const int v = a[i];
        a[i] = ra;
        ra = OpA::op(ra, v);
    }
    int rb = OpB::op(base_b, lane > 0 ? eb : OpB::kIdentity);
    for (int i = blo; i < bhi; ++i) {
        const int v = b[i];
        b[i] = rb;
        rb = OpB::op(rb, v);
    }
    if (tid == 0) {
        a[n] = tot_a;
        b[m] = tot_b;
    }
    __syncthreads();
}

// Pages of a sequence of length L: ceil(clamp(L, 0, max_len) / 16).
__device__ __forceinline__ int pages_of(int L, int max_len)
{
    return L <= 0 ? 0 : (min(L, max_len) + kPageSize - 1) / kPageSize;
}

// Plain attention, run by the whole workgroup before its workers start: the
// pages per sequence, their exclusive prefix sum in s_cum[0 .. B] and the
// lengths in s_len[0 .. B), all in LDS; workgroup 0 also stores the prefix sum
// for the merge.
__device__ __forceinline__ void scan_sequences(const SplitParams &p, int32_t *s_cum, int32_t *s_len)
{
    constexpr int T = kWave * kWavesPerBlock;
    const int B = p.batch;
    const int max_len = p.max_blocks * kPageSize;
    for (int b = threadIdx.x; b < B; b += T) {
        const int L = p.seq_lens[b];
        s_len[b] = L;
        s_cum[b] = pages_of(L, max_len);
    }
    __syncthreads();
    block_exclusive_scan(s_cum, B);
    if (blockIdx.x == 0)
        for (int b = threadIdx.x; b <= B; b += T)
            p.cum_out[b] = s_cum[b];
}

// This wave's staging area for regrouping K tiles (16 tokens x D elements).
// Declared here, keyed only on the tile shape, so that a kernel running the
// worker in several modes (prefix sharing: own and shared pages in different
// workgroups) holds one such array, not one per mode.
template <int D, bool FP8>
__device__ __forceinline__ uint8_t *k_regroup_stage()
{
    __shared__ uint8_t k_stage[kWavesPerBlock][kPageSize * D * (FP8 ? 1 : 2)];
    return k_stage[__builtin_amdgcn_readfirstlane(threadIdx.x / kWave)];
}

// Which tiles a worker streams.
constexpr int kAllPages = 0;      // plain attention: every page of every sequence
constexpr int kOwnPages = 1;      // prefix sharing: the pages after each sequence's shared ones
constexpr int kSharedPages = 2;   // prefix sharing: each group's shared pages once, one column block per wavefront

// LDS view of the unit stream: the exclusive prefix sum of tiles per sequence
// and the lengths; for kOwnPages also each sequence's group and the groups'
// shared-page prefix sum (a sequence's own pages start after its group's
// shared pages). For kSharedPages `cum` is the shared-page prefix sum over the
// groups and `gl` each group's first member and size, packed as
// lead | (members - 1) << 16.
struct StreamLds {
    const int32_t *cum;     // [B + 1], or [NG + 1] for kSharedPages
    const int32_t *len;     // [B]
    const int32_t *group;   // [B], kOwnPages only (-1: no shared pages)
    const int32_t *sh;      // [NG + 1], kOwnPages only
    const int32_t *gl;      // [NG], kSharedPages only
    int32_t num_groups;     // kSharedPages only
};

// Worker w of the split-KV pass over the stream that `sv` describes (in LDS,
// complete: the caller has passed a barrier). A worker is one wavefront, or
// for kSharedPages the four wavefronts of a workgroup, which stream the same
// tiles and compute column blocks blk = 0..3 of each shared unit.
template <int D, bool FP8, int MODE>
__device__ __forceinline__ void split_unit_worker(const SplitParams &p, int w, const StreamLds &sv, int blk = -1)
{
    constexpr bool kShared = MODE == kSharedPages;
    constexpr int kNbuf = pipeline_depth<FP8>();
    if (w >= p.num_workers)
        return;
    const int nseq = kShared ? sv.num_groups : p.batch;   // "sequences" of the stream
    const long long total = (long long)sv.cum[nseq] * p.num_kv_heads;
    const int nw = effective_workers(total, p.num_workers);
    if (w >= nw)
        return;
    const long long s0 = (long long)w * total / nw;
    const long long s1 = (long long)(w + 1) * total / nw;
    if (s0 >= s1)
        return;
    const int ntiles = (int)(s1 - s0);
    const int lane = threadIdx.x & (kWave - 1);
    const int n = lane & 15;
    const int quad = lane >> 4;
    const int G = p.group;
    uint8_t *lds = k_regroup_stage<D, FP8>();
    // Plain attention: a per-wave stage (see stage_output) holding the
    // partial state of the range's first piece, if cut (G * (D + 2) fp32 at
    // the start), then the output rows of finished units, `staged` of them
    // queued, each slot G rows of D bf16.
    constexpr bool kStageOut = MODE == kAllPages;
    __shared__ uint8_t out_stage[kWavesPerBlock][kStageOut ? kOutStageBytes : 16];
    __shared__ uint32_t out_rows[kWavesPerBlock][kStageOut ? kMaxOutSlots : 1];
    uint8_t *const ostage_base = out_stage[__builtin_amdgcn_readfirstlane(threadIdx.x / kWave)];
    uint32_t *const orows = out_rows[__builtin_amdgcn_readfirstlane(threadIdx.x / kWave)];
    const int part_bytes = (G * (D + 2) * 4 + 15) & ~15;   // keeps the output slots 16-byte aligned
    uint8_t *const ostage = ostage_base + part_bytes;
    const int slot_bytes = G * D * 2;
    const int out_slots = (kOutStageBytes - part_bytes) / slot_bytes;   // >= 1 (G <= 16, D <= 128)
    int staged = 0;
    bool part_staged = false;
    // Prefix own pages: the queue of finished own units' states (flush_states).
    constexpr bool kStageOwn = MODE == kOwnPages;
    __shared__ uint8_t own_stage[kWavesPerBlock][kStageOwn ? kOwnStageBytes : 16];
    __shared__ uint32_t own_dest[kWavesPerBlock][kStageOwn ? kMaxOwnSlots : 1];
    uint8_t *const qstage = own_stage[__builtin_amdgcn_readfirstlane(threadIdx.x / kWave)];
    uint32_t *const qdest = own_dest[__builtin_amdgcn_readfirstlane(threadIdx.x / kWave)];
    const int own_slots = kStageOwn ? kOwnStageBytes / part_bytes : 0;   // 1 or more (G <= 16, D <= 128)
    int queued = 0;

    // Tile entries, fetched in tile order (every call below asks for the next
    // tile; past the range the last tile repeats): {block-table entry (loaded
    // through a bounds-checked buffer resource), metadata, KV head}, from a
    // cursor over the units.
    const __amdgpu_buffer_rsrc_t btab = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int32_t *>(p.block_table), 0, p.batch * p.max_blocks * (int)sizeof(int32_t), kRawBufferWord3);
    // Cursor: tile (b, g, j) of the stream, the sequence's tile count n_b and
    // length L_b, and the page index its tiles start at (its group's shared
    // pages for kOwnPages, else 0).
    auto shared_of = [&](int b) -> int {
        if constexpr (MODE == kOwnPages) {
            const int k = sv.group[b];
            return k >= 0 ? sv.sh[k + 1] - sv.sh[k] : 0;
        } else {
            return 0;
        }
    };
    // Largest b with Hkv cum[b] <= s0 (then its n_b > 0).
    int blo = 0, bhi = nseq;
    while (bhi - blo > 1) {
        const int mid = (blo + bhi) >> 1;
        if ((long long)sv.cum[mid] * p.num_kv_heads <= s0)
            blo = mid;
        else
            bhi = mid;
    }
    int cb = blo;
    int cnb = sv.cum[cb + 1] - sv.cum[cb];
    int clen = kShared ? sv.gl[cb] : sv.len[cb];   // kSharedPages: the group's packed lead and size
    int csh = shared_of(cb);
    const int off = (int)(s0 - (long long)sv.cum[cb] * p.num_kv_heads);
    int cg = off / cnb;
    int cj = off - cg * cnb;
    const int max_len = p.max_blocks * kPageSize;
    auto entry = [&](int i) -> u32x4_t {
        uint32_t bt, meta;
        if constexpr (kShared) {
            // Page cj of the group's shared pages, read through its first member's row; the
            // count field holds members - 1 (every shared page is full).
            const int lead = clen & 0xffff;
            bt = __builtin_bit_cast(
                uint32_t, __builtin_amdgcn_raw_buffer_load_b32(btab, 0, (lead * p.max_blocks + cj) * 4, 0));
            meta = (uint32_t)(clen >> 16) | ((uint32_t)(lead * p.num_q_heads + cg * G) << kMetaRowShift);
        } else {
            const int pg = csh + cj;   // page index in the sequence
            bt = __builtin_bit_cast(
                uint32_t, __builtin_amdgcn_raw_buffer_load_b32(btab, 0, (cb * p.max_blocks + pg) * 4, 0));
            const int live = min(kPageSize, clen - pg * kPageSize);
            meta = (uint32_t)(max(live, 1) - 1) | ((uint32_t)(cb * p.num_q_heads + cg * G) << kMetaRowShift);
            if (clen > max_len)
                meta |= kMetaBadLen;
            if (csh > 0)
                meta |= kMetaPrefixed;
        }
        if (cj == 0)
            meta |= kMetaFirst;
        if (cj == cnb - 1)
            meta |= kMetaLast;
        const u32x4_t e = {bt, meta, (uint32_t)cg, 0u};
        if (i < ntiles - 1) {   // advance to the next tile of the stream
            if (++cj == cnb) {
                cj = 0;
                if (++cg == p.num_kv_heads) {
                    cg = 0;
                    do
                        ++cb;
                    while (sv.cum[cb + 1] == sv.cum[cb]);   // tiles remain, so a sequence with tiles follows
                    cnb = sv.cum[cb + 1] - sv.cum[cb];
                    clen = kShared ? sv.gl[cb] : sv.len[cb];
                    csh = shared_of(cb);
                }
            }
        }
        return e;
    };
    auto page_of = [&](u32x4_t e) -> int32_t {
        const uint32_t bt = (uint32_t)__builtin_amdgcn_readfirstlane(e[0]);
        return bt < (uint32_t)p.num_pages ? (int32_t)(bt * (uint32_t)p.num_kv_heads + e[2]) : -1;
    };
    auto meta_of = [](u32x4_t e) { return (uint32_t)__builtin_amdgcn_readfirstlane(e[1]); };

    // Ring of entries: slot k holds the entry of the tile issued at step k (mod
    // kNbuf). The first entries and the ring are fetched together and waited
    // for once here (the empty asm consumes them), so that inside the loop the
    // counter wait for an entry only ever covers the loads of one pipeline turn
    // and never drains the pipeline.
    u32x4_t first[kNbuf - 1];
#pragma unroll
    for (int k = 0; k < kNbuf - 1; ++k)
        first[k] = entry(k);
    u32x4_t ring[kNbuf];
#pragma unroll
    for (int k = 0; k < kNbuf; ++k)
        ring[k] = entry(kNbuf - 1 + k);
#pragma unroll
    for (int k = 0; k < kNbuf; ++k)
        asm volatile("" ::"v"(ring[k]));
    int32_t first_page[kNbuf - 1];
    uint32_t first_meta[kNbuf - 1];
#pragma unroll
    for (int k = 0; k < kNbuf - 1; ++k) {
        first_page[k] = page_of(first[k]);
        first_meta[k] = meta_of(first[k]);
    }

    Tile<D, FP8> buf[kNbuf];
#pragma unroll
    for (int k = 0; k < kNbuf - 1; ++k)
        issue_tile<D, FP8, !kShared>(buf[k], p, first_page[k], first_meta[k],
                                     k == 0 || (first_meta[k] & kMetaFirst) != 0, n, quad, lane, blk);

    Piece<D> st;
    reset(st);
    bf16x8_t qop[D / 32];   // score-MFMA B operands of the current unit (zero columns past its rows)
    bool started = false;   // the current unit's first tile is inside this range
    bool bad = false;
    int slot_sel = 0;
    for (int i0 = 0; i0 < ntiles; i0 += kNbuf) {
#pragma unroll
        for (int k = 0; k < kNbuf; ++k) {
            const int i = i0 + k;
            const uint32_t next_meta = meta_of(ring[k]);
            issue_tile<D, FP8, !kShared>(buf[(k + kNbuf - 1) % kNbuf], p, page_of(ring[k]), next_meta,
                                         (next_meta & kMetaFirst) != 0, n, quad, lane, blk);
            ring[k] = entry(i + 2 * kNbuf - 1);
            if (i < ntiles) {
                const Tile<D, FP8> &t = buf[k];
                const uint32_t meta = t.meta;
                if (i == 0 || (meta & kMetaFirst) != 0) {
#pragma unroll
                    for (int s = 0; s < D / 32; ++s)
                        qop[s] = __builtin_bit_cast(bf16x8_t,
                                                    kShared || n < G ? t.q[s] : u32x4_t{0u, 0u, 0u, 0u});
                }
                started |= (meta & kMetaFirst) != 0;
                bad |= t.bad_page || (meta & kMetaBadLen) != 0;
                compute_tile<D, FP8>(st, t, qop, p.scale_log2, kShared ? kPageSize : (int)(meta & 15u) + 1, lds,
                                     lane, n, quad);
                if (kShared && ((meta & kMetaLast) != 0 || i == ntiles - 1)) {
                    // A shared unit's state is always merged: a whole one goes to the unit area
                    // (indexed by first query row / G), a cut one to the worker's slot; block blk
                    // holds rows 16 blk .. 16 blk + 15 of the unit's kPrefixRows.
                    const uint32_t row0 = meta >> kMetaRowShift;
                    const bool whole = started && (meta & kMetaLast) != 0;
                    const size_t slot = whole ? (size_t)(row0 / (uint32_t)G) : 2 * (size_t)w + slot_sel;
                    const int r = 16 * blk + n;
                    const float l = quad_sum(st.l);
                    if (r < ((int)(meta & 15u) + 1) * G)
                        store_partial<D>(st, l, bad, whole ? p.unit_ml : p.part_ml, whole ? p.unit_acc : p.part_acc,
                                         slot * kPrefixRows + r, quad);
                    reset(st);
                    started = false;
                    bad = false;
                    slot_sel = 1;
                } else if (!kShared && ((meta & kMetaLast) != 0 || i == ntiles - 1)) {
                    // A unit cut by this range leaves its piece in the worker's slot 2w + slot_sel.
                    // A whole unit is written out, unless it still has to be merged (shared pages,
                    // or the own pages of a sequence that has them): then its state goes to its
                    // own slot in the unit area, indexed by (first query row) / G.
                    const uint32_t row0 = meta >> kMetaRowShift;
                    const bool whole = started && (meta & kMetaLast) != 0;
                    const bool to_unit = whole && (meta & kMetaPrefixed) != 0;
                    float *const pml = to_unit ? p.unit_ml : p.part_ml;
                    float *const pacc = to_unit ? p.unit_acc : p.part_acc;
                    const size_t slot = to_unit ? (size_t)(row0 / (uint32_t)G) : 2 * (size_t)w + slot_sel;
                    if (kStageOut && whole) {
                        const float l = quad_sum(st.l);
                        if (n < G)
                            stage_output<D>(st, l, bad, ostage + (size_t)staged * slot_bytes, n, quad);
                        if (lane == 0)
                            orows[staged] = row0;
                        if (++staged == out_slots) {
                            flush_outputs(p, D, ostage, orows, staged, slot_bytes, lane);
                            staged = 0;
                        }
                    } else if (kStageOut && slot_sel == 0) {
                        // the range's first piece, cut: written out with the stage at the end
                        const float l = quad_sum(st.l);
                        if (n < G)
                            stage_partial<D>(st, l, bad, ostage_base, G, n, quad);
                        part_staged = true;
                    } else if (kStageOwn && !(whole && !to_unit)) {
                        // a state the merge combines: queued
                        const float l = quad_sum(st.l);
                        if (queued == own_slots) {
                            flush_states(p, D, qstage, qdest, queued, part_bytes, lane);
                            queued = 0;
                        }
                        if (n < G)
                            stage_partial<D>(st, l, bad, qstage + (size_t)queued * part_bytes, G, n, quad);
                        if (lane == 0)
                            qdest[queued] = (uint32_t)(slot << 1) | (to_unit ? 1u : 0u);
                        ++queued;
                    } else {
                        finish_unit<D>(p, st, row0, whole && !to_unit, bad, pml, pacc, slot, n, quad);
                    }
                    reset(st);
                    started = false;
                    bad = false;
                    slot_sel = 1;
                }
            }
        }
    }
    if (kStageOut && staged > 0)
        flush_outputs(p, D, ostage, orows, staged, slot_bytes, lane);
    if (kStageOut && part_staged)
        flush_partial(p, D, ostage_base, 2 * (size_t)w, lane);
    if (kStageOwn && queued > 0)
        flush_states(p, D, qstage, qdest, queued, part_bytes, lane);
}

}  // namespace
}  // namespace sl

#endif  // SL_DECODE_UNIT_H
