// Device code of the decode engine (engine.cpp): filling newly admitted
// prompts' pages with synthetic key/value data, and the one-launch step for
// steps with little attention work. (Otherwise a step's bookkeeping is
// applied by the KV-append launch, append.hip, or by the merge launch.)
#include "append_unit.h"
#include "decode_unit.h"
#include "engine_internal.h"

namespace sl {
namespace {

constexpr int kEngineThreads = 256;

// 32-bit integer mixer ("lowbias32": xorshift-multiply rounds).
__device__ __forceinline__ uint32_t mix32(uint32_t x)
{
    x ^= x >> 16;
    x *= 0x7feb352du;
    x ^= x >> 15;
    x *= 0x846ca68bu;
    x ^= x >> 16;
    return x;
}

// One workgroup per (prompt page, KV head) tile: 16 x D synthetic values for
// K and V. bf16: uniform in [-2, 2). E4M3: codes of magnitude below 2 (exponent
// field <= 7) with a random sign, and scale 1.
template <int D, bool FP8>
__global__ __launch_bounds__(kEngineThreads) void engine_fill_kernel(const int32_t *pages, int32_t hkv,
                                                                     uint32_t seed, void *k_pages, void *v_pages,
                                                                     float *k_scales, float *v_scales)
{
    const int page = pages[blockIdx.x / hkv];
    const int g = blockIdx.x % hkv;
    const size_t tile = (size_t)page * hkv + g;
    const uint32_t base = seed ^ ((uint32_t)tile * 0x9e3779b1u);
    for (int e = threadIdx.x; e < kPageSize * D; e += kEngineThreads) {
        const uint32_t hk = mix32(base ^ ((uint32_t)e * 0x85ebca77u));
        const uint32_t hv = mix32(hk ^ 0xc2b2ae3du);
        if constexpr (FP8) {
            static_cast<uint8_t *>(k_pages)[tile * kPageSize * D + e] = (uint8_t)((hk & 0x3fu) | ((hk >> 24) & 0x80u));
            static_cast<uint8_t *>(v_pages)[tile * kPageSize * D + e] = (uint8_t)((hv & 0x3fu) | ((hv >> 24) & 0x80u));
        } else {
            const float fk = ((float)(hk >> 8) * (1.0f / 16777216.0f) - 0.5f) * 4.0f;
            const float fv = ((float)(hv >> 8) * (1.0f / 16777216.0f) - 0.5f) * 4.0f;
            static_cast<__bf16 *>(k_pages)[tile * kPageSize * D + e] = (__bf16)fk;
            static_cast<__bf16 *>(v_pages)[tile * kPageSize * D + e] = (__bf16)fv;
        }
    }
    if constexpr (FP8) {
        if (threadIdx.x == 0) {
            k_scales[tile] = 1.0f;
            v_scales[tile] = 1.0f;
        }
    }
}

// ---------------------------------------------------------------------------
// One-launch step (UnitStepParams). Workgroups, in this order:
//   unit_blocks  attention: K_e workgroups per unit (sequence e, KV head g);
//                the unit's tiles are split evenly over its K_e * kUnitWaves
//                waves, each running the split kernel's tile pipeline and
//                online softmax over its range;
//   zero_blocks  one per listed empty slot: its output rows set to zero;
//   next_blocks  the next step's staged bookkeeping and KV append.
// The append writes nothing this step's attention reads: the lengths come
// from the kernel arguments, the new token of a sequence of length L goes to
// position L (its last tile's rows past L are zeroed before the value
// product, whatever they hold), its table entries are past the ones read,
// and the host keeps the append in a launch of its own when it would reuse a
// page this step reads (a page freed by a sequence that finished in it).
// An E4M3 append may also re-encode the earlier rows of that page and raise
// its scale; there the unit's own workgroup appends the unit's row once all
// of the unit's reads are done (units_append), and next_blocks only apply
// the bookkeeping.

constexpr int kUnitThreads = kUnitWaves * kWave;
template <bool FP8>
constexpr int unit_depth() { return FP8 ? 3 : 2; }   // tiles in flight per wave (as the split kernel)

// LDS of an attention workgroup: the waves' K regroup stages (sized for
// bf16 tiles, which E4M3 tiles fit), then every wave's final state,
// lane-major (D / 4 accumulator values, m and l per lane): 100 KB for D = 128, which gfx950's 160 KB of LDS per CU holds (the
// kernel's registers allow one such workgroup per CU anyway).
template <int D>
constexpr int unit_state_floats() { return D / 4 + 2; }
template <int D>
constexpr int unit_stage_bytes() { return kUnitWaves * kPageSize * D * 2; }
template <int D>
constexpr int unit_smem_bytes() { return unit_stage_bytes<D>() + kUnitWaves * unit_state_floats<D>() * kWave * 4; }

// Device-scope (cross-XCD coherent) accesses to the piece slots: buffer
// loads and stores with the SC1 cache-policy bit. Unlike atomic accesses
// they are ordinary memory operations for the compiler, so many can be in
// flight at once.
constexpr int kCachePolicyDevice = 16;   // SC1
__device__ __forceinline__ __amdgpu_buffer_rsrc_t piece_rsrc(const float *base, size_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(base), 0, (int)bytes, kRawBufferWord3);
}
__device__ __forceinline__ void store4_device(__amdgpu_buffer_rsrc_t r, int off, f32x4_t v)
{
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, v), r, off, 0, kCachePolicyDevice);
}
__device__ __forceinline__ void store2_device(__amdgpu_buffer_rsrc_t r, int off, f32x2_t v)
{
    __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2_t, v), r, off, 0, kCachePolicyDevice);
}
__device__ __forceinline__ f32x4_t load4_device(__amdgpu_buffer_rsrc_t r, int off)
{
    return __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kCachePolicyDevice));
}
__device__ __forceinline__ f32x2_t load2_device(__amdgpu_buffer_rsrc_t r, int off)
{
    return __builtin_bit_cast(f32x2_t, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, kCachePolicyDevice));
}

template <int D, bool FP8>
__device__ __forceinline__ void unit_attention(const UnitStepParams &up, int blk, uint8_t *smem, int32_t *s_last)
{
    const SplitParams &p = up.cur;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int lane = threadIdx.x & (kWave - 1);
    const int n = lane & 15, quad = lane >> 4;
    const int G = p.group, Hkv = p.num_kv_heads;

    // Entry e with first[e] <= blk < first[e + 1], head g and piece k.
    int lo = 0, hi = up.n_entries;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (up.first[mid] <= blk)
            lo = mid;
        else
            hi = mid;
    }
    const int e = lo;
    const int K = (up.first[e + 1] - up.first[e]) / Hkv;
    const int local = blk - up.first[e];
    const int g = local / K, k = local - g * K;
    const int b = up.seq[e];
    const int L = up.len[e];
    const int max_len = p.max_blocks * kPageSize;
    const int Lc = min(L, max_len);
    const int nb = pages_of(L, max_len);
    const uint32_t row0 = (uint32_t)(b * p.num_q_heads + g * G);
    if (nb == 0) {   // the host lists sequences of length >= 1 only; defined anyway: zero rows
        if (k == 0)
            for (int i = threadIdx.x; i < G * D / 8; i += kUnitThreads)
                reinterpret_cast<u32x4_t *>(p.out + (size_t)row0 * D)[i] = u32x4_t{0u, 0u, 0u, 0u};
        return;
    }

    // This wave's tiles [t0, t1) of the unit.
    const long long waves = (long long)K * kUnitWaves;
    const int gw = k * kUnitWaves + wave;
    const int t0 = (int)((long long)gw * nb / waves);
    const int nt = (int)((long long)(gw + 1) * nb / waves) - t0;

    Piece<D> st;
    reset(st);
    bool bad = L > max_len;
    if (nt > 0) {
        uint8_t *lds = smem + wave * (kPageSize * D * 2);
        const int32_t *bt_row = p.block_table + (size_t)b * p.max_blocks + t0;
        // The query rows (lanes past the group read row G - 1 and use zeros)
        // and the first 64 block-table entries of the range, issued together.
        bf16x8_t qop[D / 32];
        {
            const uint16_t *qrow = p.q + ((size_t)row0 + (size_t)min(n, G - 1)) * D;
#pragma unroll
            for (int s = 0; s < D / 32; ++s) {
                const u32x4_t x = ld128(reinterpret_cast<const uint8_t *>(qrow + q_index<D, FP8>(s, quad)));
                qop[s] = __builtin_bit_cast(bf16x8_t, n < G ? x : u32x4_t{0u, 0u, 0u, 0u});
            }
        }
        int32_t ids = lane < nt ? bt_row[lane] : 0;
        auto page_at = [&](int i) -> int32_t {   // tile i of the range; its entry is in `ids`
            const uint32_t v = (uint32_t)__builtin_amdgcn_readlane(ids, i & (kWave - 1));
            return v < (uint32_t)p.num_pages ? (int32_t)(v * (uint32_t)Hkv + (uint32_t)g) : -1;
        };
        auto meta_at = [&](int i) -> uint32_t {
            const int live = min(kPageSize, Lc - (t0 + i) * kPageSize);   // >= 1: t0 + i < nb
            return (uint32_t)(live - 1) | (row0 << kMetaRowShift);
        };
        // kDepth tiles in flight.
        constexpr int kDepth = unit_depth<FP8>();
        Tile<D, FP8> buf[kDepth];
#pragma unroll
        for (int k0 = 0; k0 < kDepth - 1; ++k0)
            if (k0 < nt)
                issue_tile<D, FP8>(buf[k0], p, page_at(k0), meta_at(k0), false, n, quad, lane);
        for (int i0 = 0; i0 < nt; i0 += kDepth) {
#pragma unroll
            for (int kk = 0; kk < kDepth; ++kk) {
                const int i = i0 + kk;
                if (i < nt) {
                    const int ia = i + kDepth - 1;   // the tile issued now
                    if (ia < nt) {
                        if ((ia & (kWave - 1)) == 0)     // the next 64 entries
                            ids = lane < nt - ia ? bt_row[ia + lane] : 0;
                        issue_tile<D, FP8>(buf[(kk + kDepth - 1) % kDepth], p, page_at(ia), meta_at(ia), false, n,
                                           quad, lane);
                    }
                    const Tile<D, FP8> &t = buf[kk];
                    bad |= t.bad_page;
                    compute_tile<D, FP8>(st, t, qop, p.scale_log2, (int)(t.meta & 15u) + 1, lds, lane, n, quad);
                }
            }
        }
    }

    // Every wave leaves its state in its own LDS area (past the regroup
    // stages, so nothing needs to wait for them), then one barrier.
    constexpr int SF = unit_state_floats<D>();
    float *const states = reinterpret_cast<float *>(smem + unit_stage_bytes<D>());
    {
        float *dst = states + (size_t)wave * SF * kWave + lane;
#pragma unroll
        for (int i = 0; i < D / 16; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                dst[(4 * i + r) * kWave] = st.acc[i][r];
        dst[(D / 4) * kWave] = st.m;
        dst[(D / 4 + 1) * kWave] = st.l;
    }
    const bool bad_any = __syncthreads_or(bad ? 1 : 0) != 0;
    const float poison = bad_any ? __builtin_nanf("") : 0.0f;

    // Combine the kUnitWaves states, in wave order (so the result does not
    // depend on timing): thread t = (16 n + 4 quad + r) takes lane
    // (n, quad)'s accumulator values 4 i + r, i = 0 .. D/16 - 1, which are
    // the D/16 consecutive columns quad D/4 + r D/16 + i of row n.
    const int unit = e * Hkv + g;
    const int mls = unit_ml_stride(G);
    const __amdgpu_buffer_rsrc_t ml_rsrc = piece_rsrc(p.part_ml, sizeof(float) * kMaxUnitBlocks * mls);
    const __amdgpu_buffer_rsrc_t acc_rsrc = piece_rsrc(p.part_acc, sizeof(float) * kMaxUnitBlocks * G * D);
    const int t = threadIdx.x;
    if (t < 16 * G) {
        const int cn = t >> 4, cq = (t >> 2) & 3, cr = t & 3;
        const int cl = cn + 16 * cq;   // source lane
        float m[kUnitWaves], ls[kUnitWaves];
        float M = kNegInf;
#pragma unroll
        for (int w = 0; w < kUnitWaves; ++w) {
            const float *src = states + (size_t)w * SF * kWave;
            m[w] = src[(D / 4) * kWave + cl];
            ls[w] = (src[(D / 4 + 1) * kWave + cn] + src[(D / 4 + 1) * kWave + cn + 16]) +
                    (src[(D / 4 + 1) * kWave + cn + 32] + src[(D / 4 + 1) * kWave + cn + 48]);
            M = fmaxf(M, m[w]);
        }
        float L = 0.0f;
        float a[D / 16];
#pragma unroll
        for (int i = 0; i < D / 16; ++i)
            a[i] = 0.0f;
#pragma unroll
        for (int w = 0; w < kUnitWaves; ++w) {
            const float c = m[w] == kNegInf ? 0.0f : __builtin_amdgcn_exp2f(m[w] - M);
            const float *src = states + (size_t)w * SF * kWave + cl;
            L += c * ls[w];
#pragma unroll
            for (int i = 0; i < D / 16; ++i)
                a[i] += c * src[(4 * i + cr) * kWave];
        }
        const int col = cq * (D / 4) + cr * (D / 16);
        if (K == 1) {   // the whole unit: normalise and write the row's D/16 columns
            const float inv = bad_any ? __builtin_nanf("") : 1.0f / L;
            uint32_t wv[D / 32];
#pragma unroll
            for (int h = 0; h < D / 32; ++h)
                wv[h] = pack_bf16(a[2 * h] * inv, a[2 * h + 1] * inv);
            uint16_t *dst = p.out + ((size_t)row0 + cn) * D + col;
            if constexpr (D == 128)
                *reinterpret_cast<u32x4_t *>(dst) = u32x4_t{wv[0], wv[1], wv[2], wv[3]};
            else
                *reinterpret_cast<u32x2_t *>(dst) = u32x2_t{wv[0], wv[1]};
        } else {
            // A piece goes to slot blk; the last of the unit's K workgroups
            // to arrive merges them. The pieces cross XCDs, whose L2 caches
            // are not coherent with each other, so they are written and read
            // with device-scope accesses (each goes to the coherent level
            // itself), and the writers' stores complete before the count. An
            // agent-scope fence would do the same by writing back, or
            // invalidating, the whole L2 of the XCD, at several microseconds
            // per workgroup.
            const int off = (blk * G + cn) * D + col;
#pragma unroll
            for (int i = 0; i < D / 16; i += 4)
                store4_device(acc_rsrc, 4 * (off + i),
                              f32x4_t{a[i], a[i + 1], a[i + 2], a[i + 3]} + poison);
            if (cq == 0 && cr == 0)
                store2_device(ml_rsrc, 4 * (blk * mls + 2 * cn), f32x2_t{M + poison, L});
        }
    }
    // The unit's next-step row, by the last wave (which has no combine work
    // for any G <= 16: the combine takes threads below 16 G): with one
    // workgroup per unit, every wave's reads of the unit's pages are done
    // once the barrier above has passed.
    const bool tail_append = up.units_append && wave == kUnitWaves - 1;
    if (K == 1) {
        if (tail_append)
            append_row<D, FP8>(up.next, b * Hkv + g, L + 1, up.next_page[e], lane);
        return;
    }
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0);   // this wave's part of the piece has reached the coherent level
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __syncthreads();
    if (threadIdx.x == 0)
        *s_last = __hip_atomic_fetch_add(up.counters + unit, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == K - 1;
    __syncthreads();
    if (*s_last == 0)
        return;
    // Every workgroup of the unit has counted its arrival after its loads
    // returned, so none reads the unit's pages any more.
    if (tail_append)
        append_row<D, FP8>(up.next, b * Hkv + g, L + 1, up.next_page[e], lane);
    // The last arrival merges the unit's K pieces (slots first[e] + g K ..),
    // in slot order, row j and four columns per thread. Up to eight pieces:
    // every load at once; more: the (m, l) pairs through LDS first, then
    // eight pieces' columns at a time.
    const int slot0 = up.first[e] + g * K;
    if (K <= 8) {
        for (int idx = threadIdx.x; idx < G * (D / 4); idx += kUnitThreads) {
            const int j = idx / (D / 4), c = (idx - j * (D / 4)) * 4;
            f32x2_t ml[8];
            f32x4_t a[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                if (u < K) {
                    ml[u] = load2_device(ml_rsrc, 4 * ((slot0 + u) * mls + 2 * j));
                    a[u] = load4_device(acc_rsrc, 4 * (((slot0 + u) * G + j) * D + c));
                }
            }
            float M = kNegInf;
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if (u < K)
                    M = fmaxf(M, ml[u][0]);
            float l = 0.0f;
            f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                if (u < K) {
                    const float w = ml[u][0] == kNegInf ? 0.0f : __builtin_amdgcn_exp2f(ml[u][0] - M);
                    l += w * ml[u][1];
                    acc += w * a[u];
                }
            }
            const float inv = 1.0f / l;
            *reinterpret_cast<u32x2_t *>(p.out + ((size_t)row0 + j) * D + c) =
                u32x2_t{pack_bf16(acc[0] * inv, acc[1] * inv), pack_bf16(acc[2] * inv, acc[3] * inv)};
        }
    } else {
        f32x2_t *const s_ml = reinterpret_cast<f32x2_t *>(smem);   // [K][G], in the regroup stages
        for (int q = threadIdx.x; q < K * G; q += kUnitThreads) {
            const int pq = q / G, j = q - pq * G;
            s_ml[q] = load2_device(ml_rsrc, 4 * ((slot0 + pq) * mls + 2 * j));
        }
        __syncthreads();
        for (int idx = threadIdx.x; idx < G * (D / 4); idx += kUnitThreads) {
            const int j = idx / (D / 4), c = (idx - j * (D / 4)) * 4;
            float M = kNegInf;
            for (int q = 0; q < K; ++q)
                M = fmaxf(M, s_ml[q * G + j][0]);
            float l = 0.0f;
            f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
            for (int q0 = 0; q0 < K; q0 += 8) {
                f32x4_t a[8];
#pragma unroll
                for (int u = 0; u < 8; ++u)
                    if (q0 + u < K)
                        a[u] = load4_device(acc_rsrc, 4 * (((slot0 + q0 + u) * G + j) * D + c));
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    if (q0 + u < K) {
                        const f32x2_t ml = s_ml[(q0 + u) * G + j];
                        const float w = ml[0] == kNegInf ? 0.0f : __builtin_amdgcn_exp2f(ml[0] - M);
                        l += w * ml[1];
                        acc += w * a[u];
                    }
                }
            }
            const float inv = 1.0f / l;
            *reinterpret_cast<u32x2_t *>(p.out + ((size_t)row0 + j) * D + c) =
                u32x2_t{pack_bf16(acc[0] * inv, acc[1] * inv), pack_bf16(acc[2] * inv, acc[3] * inv)};
        }
    }
    if (threadIdx.x == 0)   // for the next launch (ordered by the kernel boundary)
        __hip_atomic_store(up.counters + unit, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <int D, bool FP8>
__global__ __launch_bounds__(kUnitThreads) void engine_unit_step_kernel(UnitStepParams up)
{
    __shared__ __attribute__((aligned(16))) uint8_t smem[unit_smem_bytes<D>()];
    __shared__ int32_t s_last;
    int blk = (int)blockIdx.x;
    if (blk < up.unit_blocks) {
        unit_attention<D, FP8>(up, blk, smem, &s_last);
        return;
    }
    blk -= up.unit_blocks;
    if (blk < up.zero_blocks) {
        u32x4_t *dst = reinterpret_cast<u32x4_t *>(up.cur.out + (size_t)up.zero[blk] * up.cur.num_q_heads * D);
        for (int i = threadIdx.x; i < up.cur.num_q_heads * D / 8; i += kUnitThreads)
            dst[i] = u32x4_t{0u, 0u, 0u, 0u};
        return;
    }
    blk -= up.zero_blocks;
    apply_stage(up.next, blk * kUnitThreads + (int)threadIdx.x, up.next_blocks * kUnitThreads);
    if (up.units_append)
        return;
    const int unit = blk * kUnitWaves + (int)(threadIdx.x / kWave);
    if (unit < up.next.batch * up.next.num_kv_heads)
        append_unit<D, FP8>(up.next, unit, threadIdx.x & (kWave - 1));
}

}  // namespace

hipError_t launch_unit_step(const UnitStepParams &up, int head_dim, bool fp8, hipStream_t stream)
{
    const dim3 grid((unsigned)(up.unit_blocks + up.zero_blocks + up.next_blocks)), block(kUnitThreads);
    if (grid.x == 0)
        return hipSuccess;
    if (head_dim == 128 && !fp8)
        hipLaunchKernelGGL((engine_unit_step_kernel<128, false>), grid, block, 0, stream, up);
    else if (head_dim == 64 && !fp8)
        hipLaunchKernelGGL((engine_unit_step_kernel<64, false>), grid, block, 0, stream, up);
    else if (head_dim == 128 && fp8)
        hipLaunchKernelGGL((engine_unit_step_kernel<128, true>), grid, block, 0, stream, up);
    else if (head_dim == 64 && fp8)
        hipLaunchKernelGGL((engine_unit_step_kernel<64, true>), grid, block, 0, stream, up);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t launch_engine_fill(const int32_t *pages, int n_pages, int hkv, int head_dim, bool fp8, uint32_t seed,
                              void *k_pages, void *v_pages, float *k_scales, float *v_scales, hipStream_t stream)
{
    const dim3 grid((unsigned)(n_pages * hkv)), block(kEngineThreads);
    if (head_dim == 128 && !fp8)
        hipLaunchKernelGGL((engine_fill_kernel<128, false>), grid, block, 0, stream, pages, hkv, seed, k_pages,
                           v_pages, k_scales, v_scales);
    else if (head_dim == 64 && !fp8)
        hipLaunchKernelGGL((engine_fill_kernel<64, false>), grid, block, 0, stream, pages, hkv, seed, k_pages,
                           v_pages, k_scales, v_scales);
    else if (head_dim == 128 && fp8)
        hipLaunchKernelGGL((engine_fill_kernel<128, true>), grid, block, 0, stream, pages, hkv, seed, k_pages,
                           v_pages, k_scales, v_scales);
    else if (head_dim == 64 && fp8)
        hipLaunchKernelGGL((engine_fill_kernel<64, true>), grid, block, 0, stream, pages, hkv, seed, k_pages,
                           v_pages, k_scales, v_scales);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

}  // namespace sl
