// Split-KV decode attention kernel for gfx950.
//
// One wavefront is one worker; it walks its contiguous range of page-head
// tiles (see sl_internal.h) and, for each (sequence, KV head) unit it touches,
// keeps an online-softmax state for the G query heads that share the KV head.
//
// Per 16-token tile, with lane = n + 16 * quad (n = lane & 15, quad = lane >> 4):
//
//   scores  S^T[t][j] = sum_d K[t][d] Q[j][d]       v_mfma_f32_16x16x32_bf16
//           A = K   (row t = n, 8 consecutive d per lane: one 16-byte load)
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
// K and V go straight from HBM into MFMA operand registers: there is no reuse
// of a tile inside the workgroup, so an LDS round trip would only add
// latency. Tiles are software-pipelined NBUF deep, and the block-table
// entries of a piece are fetched 64 at a time, one per lane, a chunk ahead,
// so a page id never waits on a dependent load.
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
#ifndef SL_NBUF
#define SL_NBUF 2
#endif
constexpr int kNbuf = SL_NBUF;   // tiles in the software pipeline

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

template <int D, bool FP8>
struct Tile {
    // Per-lane dwords of K (score-MFMA A operands) and V (four rows).
    static constexpr int KW = FP8 ? D / 16 : D / 8;
    static constexpr int VW = FP8 ? D / 16 : D / 8;
    uint32_t k[KW];
    uint32_t v[VW];
    float scl;   // FP8: key scale in lanes 0-31, value scale in lanes 32-63
};

// Issue the loads of one page-head tile. kt / vt point at the tile (uniform).
template <int D, bool FP8>
__device__ __forceinline__ void load_tile(Tile<D, FP8> &t, const uint8_t *kt, const uint8_t *vt,
                                          const float *sp, int n, int quad)
{
    if constexpr (!FP8) {
#pragma unroll
        for (int s = 0; s < D / 32; ++s) {
            const u32x4_t x = ld128_stream(kt + (n * D + 32 * s + 8 * quad) * 2);
#pragma unroll
            for (int c = 0; c < 4; ++c)
                t.k[4 * s + c] = x[c];
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const uint8_t *src = vt + ((4 * quad + r) * D + n * (D / 16)) * 2;
            if constexpr (D == 128) {
                const u32x4_t x = ld128_stream(src);
#pragma unroll
                for (int c = 0; c < 4; ++c)
                    t.v[4 * r + c] = x[c];
            } else {
                const u32x2_t x = ld64_stream(src);
                t.v[2 * r] = x[0];
                t.v[2 * r + 1] = x[1];
            }
        }
    } else {
#pragma unroll
        for (int h = 0; h < D / 64; ++h) {
            const u32x4_t x = ld128_stream(kt + n * D + quad * (D / 4) + 16 * h);
#pragma unroll
            for (int c = 0; c < 4; ++c)
                t.k[4 * h + c] = x[c];
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const uint8_t *src = vt + (4 * quad + r) * D + n * (D / 16);
            if constexpr (D == 128) {
                const u32x2_t x = ld64_stream(src);
                t.v[2 * r] = x[0];
                t.v[2 * r + 1] = x[1];
            } else {
                t.v[r] = ld32_stream(src);
            }
        }
        t.scl = *sp;
    }
}

// Score-MFMA A operand for k-step s (8 bf16 values of row t = n).
template <int D, bool FP8>
__device__ __forceinline__ bf16x8_t k_operand(const Tile<D, FP8> &t, int s)
{
    u32x4_t w;
    if constexpr (!FP8) {
        w = u32x4_t{t.k[4 * s], t.k[4 * s + 1], t.k[4 * s + 2], t.k[4 * s + 3]};
    } else {
        uint32_t a, b, c, d;
        e4m3x4_to_bf16(t.k[2 * s], a, b);
        e4m3x4_to_bf16(t.k[2 * s + 1], c, d);
        w = u32x4_t{a, b, c, d};
    }
    return __builtin_bit_cast(bf16x8_t, w);
}

// Query element index held by (quad, item) in k-step s; must match k_operand.
template <int D, bool FP8>
__device__ __forceinline__ int q_index(int s, int quad)
{
    return FP8 ? quad * (D / 4) + 8 * s : 32 * s + 8 * quad;
}

template <int D, bool FP8>
struct Piece {
    bf16x8_t q[D / 32];
    f32x4_t acc[D / 16];
    float m;   // running max of this lane's head, base-2 units
    float l;   // this lane's share of the sum of (bf16-rounded) weights
};

// One tile of the online softmax. `valid` = live tokens in this page (1..16).
template <int D, bool FP8>
__device__ __forceinline__ void compute_tile(Piece<D, FP8> &st, const Tile<D, FP8> &t,
                                             float score_mul, int valid, int quad)
{
    f32x4_t s4 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < D / 32; ++s)
        s4 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k_operand(t, s), st.q[s], s4, 0, 0, 0);

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
    float mx = fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3]));
    mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
    mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
    if (mx > st.m) {
        const float alpha = __builtin_amdgcn_exp2f(st.m - mx);   // 0 on the first tile
        st.l *= alpha;
#pragma unroll
        for (int i = 0; i < D / 16; ++i)
            st.acc[i] *= alpha;
        st.m = mx;
    }
    float p[4];
#pragma unroll
    for (int r = 0; r < 4; ++r)
        p[r] = __builtin_amdgcn_exp2f(sc[r] - st.m);
    const uint32_t p01 = pack_bf16(p[0], p[1]);
    const uint32_t p23 = pack_bf16(p[2], p[3]);
    st.l += (bf16_lo(p01) + bf16_hi(p01)) + (bf16_lo(p23) + bf16_hi(p23));
    i16x4_t pb;
    if constexpr (FP8) {
        const uint32_t w01 = pack_bf16(p[0] * vmul, p[1] * vmul);
        const uint32_t w23 = pack_bf16(p[2] * vmul, p[3] * vmul);
        pb = __builtin_bit_cast(i16x4_t, u32x2_t{w01, w23});
    } else {
        pb = __builtin_bit_cast(i16x4_t, u32x2_t{p01, p23});
    }

    // Value rows as bf16 dwords: row r holds D/16 consecutive elements.
    constexpr int RW = D / 32;   // bf16 dwords per row
    uint32_t vb[4 * RW];
    if constexpr (FP8) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int c = 0; c < D / 64; ++c)
                e4m3x4_to_bf16(t.v[r * (D / 64) + c], vb[r * RW + 2 * c], vb[r * RW + 2 * c + 1]);
    } else {
#pragma unroll
        for (int i = 0; i < 4 * RW; ++i)
            vb[i] = t.v[i];
    }
    uint32_t mlo = 0xffffffffu, mhi = 0xffffffffu;
    if (valid < kPageSize) {   // zero dead rows: their slots may hold NaN
        const int t0 = 4 * quad;
        mlo = (t0 + 0 < valid ? 0x0000ffffu : 0u) | (t0 + 1 < valid ? 0xffff0000u : 0u);
        mhi = (t0 + 2 < valid ? 0x0000ffffu : 0u) | (t0 + 3 < valid ? 0xffff0000u : 0u);
    }
#pragma unroll
    for (int i = 0; i < D / 16; ++i) {
        const int w = i >> 1;
        uint32_t lo, hi;
        if ((i & 1) == 0) {
            lo = (vb[0 * RW + w] & 0xffffu) | (vb[1 * RW + w] << 16);
            hi = (vb[2 * RW + w] & 0xffffu) | (vb[3 * RW + w] << 16);
        } else {
            lo = (vb[0 * RW + w] >> 16) | (vb[1 * RW + w] & 0xffff0000u);
            hi = (vb[2 * RW + w] >> 16) | (vb[3 * RW + w] & 0xffff0000u);
        }
        const i16x4_t va = __builtin_bit_cast(i16x4_t, u32x2_t{lo & mlo, hi & mhi});
        st.acc[i] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(va, pb, st.acc[i], 0, 0, 0);
    }
}

template <int D, bool FP8>
__device__ __forceinline__ void process_piece(const SplitParams &p, int w, int b, int g, int pg0,
                                              int pg1, int nb, int slot_sel, bool full)
{
    constexpr int ES = FP8 ? 1 : 2;                  // bytes per cached element
    constexpr size_t kTileBytes = (size_t)kPageSize * D * ES;
    const int lane = threadIdx.x & (kWave - 1);
    const int n = lane & 15;
    const int quad = lane >> 4;
    const int G = p.group;
    const int Hkv = p.num_kv_heads;
    const int L = p.seq_lens[b];
    bool bad = L < 0 || L > p.max_blocks * kPageSize;
    const int last_valid = L - (nb - 1) * kPageSize;   // live tokens in page nb - 1

    Piece<D, FP8> st;
    const uint16_t *qrow = p.q + ((size_t)b * p.num_q_heads + (size_t)g * G + n) * D;
#pragma unroll
    for (int s = 0; s < D / 32; ++s) {
        u32x4_t x = {0u, 0u, 0u, 0u};
        if (n < G)
            x = ld128(reinterpret_cast<const uint8_t *>(qrow + q_index<D, FP8>(s, quad)));
        st.q[s] = __builtin_bit_cast(bf16x8_t, x);
    }
#pragma unroll
    for (int i = 0; i < D / 16; ++i)
        st.acc[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    st.m = kNegInf;
    st.l = 0.f;

    const uint8_t *kbase = static_cast<const uint8_t *>(p.k_pages) + (size_t)g * kTileBytes;
    const uint8_t *vbase = static_cast<const uint8_t *>(p.v_pages) + (size_t)g * kTileBytes;
    const size_t page_stride = (size_t)Hkv * kTileBytes;
    const float *scale_src = (lane & 32) ? p.v_scales : p.k_scales;
    const int32_t *bt_row = p.block_table + (size_t)b * p.max_blocks;

    // Block-table entries for pages [c0, c0 + 64) (btc) and the next 64 (btn).
    int c0 = pg0;
    int btc = (c0 + lane < pg1) ? bt_row[c0 + lane] : 0;
    int btn = (c0 + 64 + lane < pg1) ? bt_row[c0 + 64 + lane] : 0;

    auto issue = [&](Tile<D, FP8> &t, int pg) {
        if (pg - c0 >= 64) {
            c0 += 64;
            btc = btn;
            btn = (c0 + 64 + lane < pg1) ? bt_row[c0 + 64 + lane] : 0;
        }
        int pid = __builtin_amdgcn_readlane(btc, pg - c0);
        if ((unsigned)pid >= (unsigned)p.num_pages) {
            bad = true;
            pid = 0;
        }
        const size_t off = (size_t)pid * page_stride;
        load_tile<D, FP8>(t, kbase + off, vbase + off,
                          FP8 ? scale_src + (size_t)pid * Hkv + g : nullptr, n, quad);
    };

    Tile<D, FP8> buf[kNbuf];
    const int np = pg1 - pg0;
#pragma unroll
    for (int k = 0; k < kNbuf - 1; ++k)
        issue(buf[k], pg0 + min(k, np - 1));
    for (int i0 = 0; i0 < np; i0 += kNbuf) {
#pragma unroll
        for (int k = 0; k < kNbuf; ++k) {
            const int i = i0 + k;
            issue(buf[(k + kNbuf - 1) % kNbuf], pg0 + min(i + kNbuf - 1, np - 1));
            if (i < np) {
                const int pg = pg0 + i;
                compute_tile<D, FP8>(st, buf[k], p.scale_log2,
                                     pg == nb - 1 ? last_valid : kPageSize, quad);
            }
        }
    }

    // Total weight of head n: sum the four quads' shares.
    st.l += __shfl_xor(st.l, 16, kWave);
    st.l += __shfl_xor(st.l, 32, kWave);
    if (n >= G)
        return;
    const int h = g * G + n;
    const int d0 = quad * (D / 4);   // this lane holds O[h][d0 .. d0 + D/4)
    if (full) {
        const float inv = bad ? __builtin_nanf("") : 1.0f / st.l;
        uint32_t packed[D / 8];
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int i = 0; i < D / 16; i += 2)
                packed[(r * (D / 16) + i) / 2] = pack_bf16(st.acc[i][r] * inv, st.acc[i + 1][r] * inv);
        uint8_t *dst = reinterpret_cast<uint8_t *>(p.out + ((size_t)b * p.num_q_heads + h) * D + d0);
#pragma unroll
        for (int c = 0; c < D / 32; ++c)
            *reinterpret_cast<u32x4_t *>(dst + 16 * c) =
                u32x4_t{packed[4 * c], packed[4 * c + 1], packed[4 * c + 2], packed[4 * c + 3]};
    } else {
        const size_t slot = 2 * (size_t)w + slot_sel;
        const float poison = bad ? __builtin_nanf("") : 0.0f;
        float *dst = p.part_acc + (slot * G + n) * D + d0;
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int i = 0; i < D / 16; i += 4)
                *reinterpret_cast<f32x4_t *>(dst + r * (D / 16) + i) =
                    f32x4_t{st.acc[i][r], st.acc[i + 1][r], st.acc[i + 2][r], st.acc[i + 3][r]} + poison;
        if (quad == 0)
            *reinterpret_cast<f32x2_t *>(p.part_ml + (slot * G + n) * 2) = f32x2_t{st.m, st.l};
    }
}

template <int D, bool FP8>
__global__ __launch_bounds__(kWave * kWavesPerBlock) void split_kv_kernel(SplitParams p)
{
    const int w = blockIdx.x * kWavesPerBlock + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    if (w >= p.num_workers)
        return;
    const int Hkv = p.num_kv_heads;
    const long long total = (long long)p.cum_pages[p.batch] * Hkv;
    const long long s0 = (long long)w * total / p.num_workers;
    const long long s1 = (long long)(w + 1) * total / p.num_workers;
    if (s0 >= s1)
        return;
    const int u = p.worker_unit[w];
    if (u < 0)
        return;
    int b = u / Hkv;
    int g = u - b * Hkv;
    int cb = p.cum_pages[b];
    int nb = p.cum_pages[b + 1] - cb;
    int pg = (int)(s0 - ((long long)Hkv * cb + (long long)g * nb));
    long long pos = s0;
    int slot_sel = 0;
    while (pos < s1) {
        const int take = (int)min((long long)(nb - pg), s1 - pos);
        if (take <= 0 || pg < 0)
            break;   // inconsistent partition: stop rather than loop
        process_piece<D, FP8>(p, w, b, g, pg, pg + take, nb, slot_sel, pg == 0 && take == nb);
        pos += take;
        slot_sel = 1;
        if (pos >= s1)
            break;
        pg = 0;
        if (++g == Hkv) {
            g = 0;
            do {
                if (b + 1 >= p.batch)
                    return;   // inconsistent partition: no later unit exists
                ++b;
                cb = p.cum_pages[b];
                nb = p.cum_pages[b + 1] - cb;
            } while (nb == 0);
        }
    }
}

}  // namespace

hipError_t launch_split(const SplitParams &p, int head_dim, bool fp8, hipStream_t stream)
{
    const dim3 grid((p.num_workers + kWavesPerBlock - 1) / kWavesPerBlock);
    const dim3 block(kWave * kWavesPerBlock);
    if (head_dim == 128 && !fp8)
        hipLaunchKernelGGL((split_kv_kernel<128, false>), grid, block, 0, stream, p);
    else if (head_dim == 64 && !fp8)
        hipLaunchKernelGGL((split_kv_kernel<64, false>), grid, block, 0, stream, p);
    else if (head_dim == 128 && fp8)
        hipLaunchKernelGGL((split_kv_kernel<128, true>), grid, block, 0, stream, p);
    else if (head_dim == 64 && fp8)
        hipLaunchKernelGGL((split_kv_kernel<64, true>), grid, block, 0, stream, p);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t split_blocks_per_cu(int head_dim, bool fp8, int *blocks)
{
    const int threads = kWave * kWavesPerBlock;
    if (head_dim == 128 && !fp8)
        return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, split_kv_kernel<128, false>, threads, 0);
    if (head_dim == 64 && !fp8)
        return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, split_kv_kernel<64, false>, threads, 0);
    if (head_dim == 128 && fp8)
        return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, split_kv_kernel<128, true>, threads, 0);
    if (head_dim == 64 && fp8)
        return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, split_kv_kernel<64, true>, threads, 0);
    return hipErrorInvalidValue;
}

}  // namespace sl
