// Log-sum-exp merge of split-KV partial states.
//
// A unit (sequence b, KV head g) whose tiles were cut across workers
// w_first..w_last left, per worker, a partial state (m_i, l_i, acc_i) for each
// of its G query heads: m_i the largest score (base-2 units), l_i the sum of
// 2^(s - m_i) and acc_i the matching un-normalised sum of value rows. With
// M = max_i m_i the exact softmax result is
//     out = sum_i 2^(m_i - M) acc_i / sum_i 2^(m_i - M) l_i
// in fp32, rounded to bf16.
//
// One wavefront per (unit, query head). Lane i first fetches (m_i, l_i) of
// piece i, so the maximum, the weights c_i = 2^(m_i - M) and their weighted
// sum come out of two wave reductions instead of a serial walk; then every
// lane accumulates its D/64 output columns over the pieces with independent
// loads. Units finished by a single worker were already written and are
// skipped. Sequences without pages get zero rows (NaN rows for an invalid
// negative length), which no split-KV worker visits.
#include "append_unit.h"

namespace sl {
namespace {

typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float wave_max(float x)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1)
        x = fmaxf(x, __shfl_xor(x, off, kWave));
    return x;
}

__device__ __forceinline__ float wave_sum(float x)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1)
        x += __shfl_xor(x, off, kWave);
    return x;
}

// floor(x / y) for 0 <= x < 2^53, 0 < y < 2^31: a double quotient corrected by
// one step (64-bit integer division is a long software sequence on the GPU).
__device__ __forceinline__ long long div_floor(long long x, long long y)
{
    long long q = (long long)((double)x / (double)y);
    if (q * y > x)
        --q;
    else if ((q + 1) * y <= x)
        ++q;
    return q;
}

// NEXT: the decode engine's next-step append in the same launch (0 none,
// 1 bf16 cache, 2 E4M3 cache), in the workgroups after the merge's.
template <int D, int NEXT>
__global__ __launch_bounds__(kMergeThreads) void merge_kernel(MergeParams p, int merge_blocks)
{
    constexpr int E = D / kWave;   // output columns per lane (1 or 2)
    constexpr int kBatch = 8;      // pieces whose rows are fetched together with the weights
    if constexpr (NEXT != 0) {
        if ((int)blockIdx.x >= merge_blocks) {
            const int ab = (int)blockIdx.x - merge_blocks;
            apply_stage(p.next, ab * kMergeThreads + threadIdx.x, ((int)gridDim.x - merge_blocks) * kMergeThreads);
            const int unit = ab * (kMergeThreads / kWave) + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
            if (unit < p.next.batch * p.next.num_kv_heads)
                append_unit<D, NEXT == 2>(p.next, unit, threadIdx.x & (kWave - 1));
            return;
        }
    }
    const int Hkv = p.num_kv_heads;
    const int G = p.group;
    const int item = blockIdx.x * (kMergeThreads / kWave) +
                     __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    if (item >= p.batch * Hkv * G)
        return;
    const int u = item / G;
    const int j = item - u * G;
    const int b = u / Hkv;
    const int g = u - b * Hkv;
    const int lane = threadIdx.x & (kWave - 1);
    uint16_t *dst = p.out + ((size_t)b * p.num_q_heads + (size_t)g * G + j) * D + E * lane;
    // First round trip: the unit's place in the tile stream.
    const int cb = p.cum_pages[b];
    const int nb = p.cum_pages[b + 1] - cb;
    const int len = p.seq_lens[b];
    const long long total = (long long)p.cum_pages[p.batch] * Hkv;

    if (nb == 0) {
        const uint16_t fill = len < 0 ? 0x7fc0 : 0x0000;   // bf16 NaN / +0
#pragma unroll
        for (int e = 0; e < E; ++e)
            dst[e] = fill;
        return;
    }
    const long long NW = effective_workers(total, p.num_workers);
    const long long a = (long long)Hkv * cb + (long long)g * nb;   // first tile of the unit
    const long long e = a + nb;                                    // one past its last tile
    // Worker holding tile x: the largest w with floor(w * total / NW) <= x.
    const int wf = (int)div_floor((a + 1) * NW - 1, total);
    const int wl = (int)div_floor(e * NW - 1, total);
    if (wf == wl)
        return;
    const int np = wl - wf + 1;

    // Piece i (lane i, i < 64) comes from worker wf + i. Its slot is 2w, except
    // for the unit's first worker when the unit began after that worker's first
    // tile (then it was the worker's trailing piece, slot 2w + 1). A worker with
    // an empty range has no piece (slot -1).
    auto slot_of = [&](int i) -> int {
        const long long w = wf + i;
        const long long s = div_floor(w * total, NW);
        if (s == div_floor((w + 1) * total, NW))
            return -1;
        return (int)(2 * w + ((i == 0 && s < a) ? 1 : 0));
    };
    // Second round trip: the weights of up to 64 pieces and the rows of the
    // first kBatch pieces, all loads issued together.
    const int my_slot = lane < np ? slot_of(lane) : -1;
    f32x2_t ml = {-__builtin_inff(), 0.0f};
    if (my_slot >= 0)
        ml = *reinterpret_cast<const f32x2_t *>(p.part_ml + ((size_t)my_slot * G + j) * 2);
    float row[kBatch][E];
#pragma unroll
    for (int i = 0; i < kBatch; ++i) {
        const int si = __builtin_amdgcn_readlane(my_slot, i);
#pragma unroll
        for (int k = 0; k < E; ++k)
            row[i][k] = 0.0f;
        if (i < np && si >= 0) {
            const float *src = p.part_acc + ((size_t)si * G + j) * D + E * lane;
            if constexpr (E == 2) {
                const f32x2_t v = *reinterpret_cast<const f32x2_t *>(src);
                row[i][0] = v[0];
                row[i][1] = v[1];
            } else {
                row[i][0] = src[0];
            }
        }
    }
    float M = wave_max(ml[0]);
    for (int c0 = kWave; c0 < np; c0 += kWave) {   // units spread over more than 64 workers
        const int s2 = lane + c0 < np ? slot_of(lane + c0) : -1;
        M = fmaxf(M, wave_max(s2 >= 0 ? p.part_ml[((size_t)s2 * G + j) * 2] : -__builtin_inff()));
    }
    // Weights c_i = 2^(m_i - M); a zero weight (empty worker, underflow) drops its row.
    float c = my_slot >= 0 ? __builtin_amdgcn_exp2f(ml[0] - M) : 0.0f;
    float Lsum = wave_sum(c * ml[1]);
    float acc[E];
#pragma unroll
    for (int k = 0; k < E; ++k)
        acc[k] = 0.0f;
#pragma unroll
    for (int i = 0; i < kBatch; ++i) {
        const float ci = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, c), i));
#pragma unroll
        for (int k = 0; k < E; ++k)
            acc[k] += ci != 0.0f ? ci * row[i][k] : 0.0f;
    }
    // Pieces past the first kBatch (long units cut across many workers).
    for (int c0 = 0; c0 < np; c0 += kWave) {
        int sl = my_slot;
        float cl = c;
        if (c0 > 0) {
            sl = lane + c0 < np ? slot_of(lane + c0) : -1;
            float ml0 = -__builtin_inff(), ml1 = 0.0f;
            if (sl >= 0) {
                const f32x2_t v = *reinterpret_cast<const f32x2_t *>(p.part_ml + ((size_t)sl * G + j) * 2);
                ml0 = v[0];
                ml1 = v[1];
            }
            cl = sl >= 0 ? __builtin_amdgcn_exp2f(ml0 - M) : 0.0f;
            Lsum += wave_sum(cl * ml1);
        }
        const int lo = c0 == 0 ? kBatch : 0;
        const int cnt = min(kWave, np - c0);
        for (int i = lo; i < cnt; ++i) {
            const float ci = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, cl), i));
            const int si = __builtin_amdgcn_readlane(sl, i);
            if (ci == 0.0f || si < 0)
                continue;
            const float *src = p.part_acc + ((size_t)si * G + j) * D + E * lane;
#pragma unroll
            for (int k = 0; k < E; ++k)
                acc[k] += ci * src[k];
        }
    }
    const float inv = 1.0f / Lsum;
    if constexpr (E == 2) {
        const f32x2_t o = {acc[0] * inv, acc[1] * inv};
        *reinterpret_cast<bf16x2_t *>(dst) = __builtin_convertvector(o, bf16x2_t);
    } else {
        *reinterpret_cast<__bf16 *>(dst) = (__bf16)(acc[0] * inv);
    }
}

// Prefix-sharing mode: every (sequence, head) row with shared pages, or whose
// own pages were cut across workers, combines the pieces of its sub-group's
// shared unit (row member * G + head of the shared partial states) with the
// pieces of its own unit. A unit cut across workers left one piece per worker
// in the worker slots; a unit that one worker saw whole left its state in the
// unit area, at (first query row) / G. Rows finished by one worker with no
// shared pages were written by the split kernel. A sequence shorter than its
// group's shared prefix, or with an invalid length, gets a NaN row.
template <int D>
__global__ __launch_bounds__(kMergeThreads) void merge_prefix_kernel(PrefixMergeParams p)
{
    constexpr int E = D / kWave;
    constexpr int kBatch = 8;   // pieces whose rows are fetched together with the weights
    const int Hkv = p.num_kv_heads, G = p.group, Hq = p.num_q_heads;
    const int item = blockIdx.x * (kMergeThreads / kWave) + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    if (item >= p.batch * Hq)
        return;
    const int b = item / Hq;
    const int h = item - b * Hq;
    const int g = h / G;
    const int hl = h - g * G;
    const int lane = threadIdx.x & (kWave - 1);
    uint16_t *dst = p.out + ((size_t)b * Hq + h) * D + E * lane;
    // First round trip: the sequence's place in both tile streams.
    const int32_t *info = p.seq_shared + 4 * (size_t)b;   // shared-page start, count, lead, group
    const int s_start = info[0], sk = info[1], lead = info[2];
    const int L = p.seq_lens[b];
    const int co = p.cum_own[b];
    const int ob = p.cum_own[b + 1] - co;
    const long long tot_o = (long long)p.cum_own[p.batch] * Hkv;
    const long long tot_s = (long long)p.cum_shared[p.max_sub] * Hkv;
    const bool bad = L < 0 || L > p.max_blocks * kPageSize || L < sk * kPageSize;
    if (sk == 0 && ob == 0) {
        const uint16_t fill = L < 0 ? 0x7fc0 : 0x0000;   // bf16 NaN / +0
#pragma unroll
        for (int e = 0; e < E; ++e)
            dst[e] = fill;
        return;
    }
    const long long nw_o = effective_workers(tot_o, p.num_workers);
    const long long a_o = (long long)Hkv * co + (long long)g * ob;
    int wf_o = 0, n_o = 0;
    if (ob > 0) {
        wf_o = (int)div_floor((a_o + 1) * nw_o - 1, tot_o);
        n_o = (int)div_floor((a_o + ob) * nw_o - 1, tot_o) - wf_o + 1;
    }
    if (sk == 0 && n_o == 1)
        return;   // finished by a single worker
    const long long nw_s =
        tot_s > 0 ? effective_workers(tot_s, effective_shared_workers(tot_o, p.num_workers, p.num_shared_workers,
                                                                      p.max_shared_workers))
                  : 1;
    long long a_s = 0;
    int wf_s = 0, n_s = 0, row = 0;
    if (sk > 0) {
        a_s = (long long)Hkv * s_start + (long long)g * sk;
        wf_s = (int)div_floor((a_s + 1) * nw_s - 1, tot_s);
        n_s = (int)div_floor((a_s + sk) * nw_s - 1, tot_s) - wf_s + 1;
        row = (b - lead) * G + hl;
    }
    const int np = n_s + n_o;
    // Piece i: code = shared (bit 31) | unit area (bit 30) | slot << 6 | row, or -1 if
    // the worker's range is empty. Slots stay below 2^17 (workers) and unit indices
    // below B Hkv < 2^24, so no code is -1.
    auto piece = [&](int i) -> int {
        if (i < n_s) {
            if (n_s == 1)
                return (int)(0xC0000000u | ((uint32_t)(lead * Hkv + g) << 6) | (uint32_t)row);
            const long long w = wf_s + i;
            const long long s = div_floor(w * tot_s, nw_s);
            if (s == div_floor((w + 1) * tot_s, nw_s))
                return -1;
            const long long slot = 2 * w + ((w == wf_s && s < a_s) ? 1 : 0);
            return (int)(0x80000000u | (uint32_t)(slot << 6) | (uint32_t)row);
        }
        if (n_o == 1)   // sk > 0 here: a whole own unit of an unshared sequence was written out
            return (int)(0x40000000u | ((uint32_t)(b * Hkv + g) << 6) | (uint32_t)hl);
        const long long w = wf_o + (i - n_s);
        const long long s = div_floor(w * tot_o, nw_o);
        if (s == div_floor((w + 1) * tot_o, nw_o))
            return -1;
        const long long slot = 2 * w + ((w == wf_o && s < a_o) ? 1 : 0);
        return (int)((uint32_t)(slot << 6) | (uint32_t)hl);
    };
    auto ml_of = [&](int code) -> const float * {
        const size_t slot = (size_t)((uint32_t)code & 0x3fffffffu) >> 6;
        const size_t r = (size_t)(code & 63);
        const bool unit = ((uint32_t)code & 0x40000000u) != 0;
        if (code < 0)
            return (unit ? p.shared_unit_ml : p.shared_ml) + (slot * kPrefixRows + r) * 2;
        return (unit ? p.own_unit_ml : p.own_ml) + (slot * G + r) * 2;
    };
    auto acc_of = [&](int code) -> const float * {
        const size_t slot = (size_t)((uint32_t)code & 0x3fffffffu) >> 6;
        const size_t r = (size_t)(code & 63);
        const bool unit = ((uint32_t)code & 0x40000000u) != 0;
        if (code < 0)
            return (unit ? p.shared_unit_acc : p.shared_acc) + (slot * kPrefixRows + r) * D;
        return (unit ? p.own_unit_acc : p.own_acc) + (slot * G + r) * D;
    };
    // Second round trip: the weights of up to 64 pieces and the rows of the
    // first kBatch pieces, all loads issued together.
    const int my_code = lane < np ? piece(lane) : -1;
    f32x2_t ml = {-__builtin_inff(), 0.0f};
    if (my_code != -1)
        ml = *reinterpret_cast<const f32x2_t *>(ml_of(my_code));
    float rowv[kBatch][E];
#pragma unroll
    for (int i = 0; i < kBatch; ++i) {
        const int ci = __builtin_amdgcn_readlane(my_code, i);
#pragma unroll
        for (int e = 0; e < E; ++e)
            rowv[i][e] = 0.0f;
        if (i < np && ci != -1) {
            const float *src = acc_of(ci) + E * lane;
#pragma unroll
            for (int e = 0; e < E; ++e)
                rowv[i][e] = src[e];
        }
    }
    float M = wave_max(ml[0]);
    for (int c0 = kWave; c0 < np; c0 += kWave) {   // more than 64 pieces
        const int c2 = lane + c0 < np ? piece(lane + c0) : -1;
        M = fmaxf(M, wave_max(c2 != -1 ? ml_of(c2)[0] : -__builtin_inff()));
    }
    // Weights c_i = 2^(m_i - M); a zero weight (empty worker, underflow) drops its row.
    const float c = my_code != -1 ? __builtin_amdgcn_exp2f(ml[0] - M) : 0.0f;
    float Lsum = wave_sum(c * ml[1]);
    float acc[E];
#pragma unroll
    for (int e = 0; e < E; ++e)
        acc[e] = 0.0f;
#pragma unroll
    for (int i = 0; i < kBatch; ++i) {
        const float ci = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, c), i));
#pragma unroll
        for (int e = 0; e < E; ++e)
            acc[e] += ci != 0.0f ? ci * rowv[i][e] : 0.0f;
    }
    // Pieces past the first kBatch.
    for (int c0 = 0; c0 < np; c0 += kWave) {
        int cl = my_code;
        float wl = c;
        if (c0 > 0) {
            cl = lane + c0 < np ? piece(lane + c0) : -1;
            float m0 = -__builtin_inff(), l0 = 0.0f;
            if (cl != -1) {
                const f32x2_t v = *reinterpret_cast<const f32x2_t *>(ml_of(cl));
                m0 = v[0];
                l0 = v[1];
            }
            wl = cl != -1 ? __builtin_amdgcn_exp2f(m0 - M) : 0.0f;
            Lsum += wave_sum(wl * l0);
        }
        const int lo = c0 == 0 ? kBatch : 0;
        const int cnt = min(kWave, np - c0);
        for (int i = lo; i < cnt; ++i) {
            const float ci = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, wl), i));
            const int ki = __builtin_amdgcn_readlane(cl, i);
            if (ki == -1 || ci == 0.0f)
                continue;
            const float *src = acc_of(ki) + E * lane;
#pragma unroll
            for (int e = 0; e < E; ++e)
                acc[e] += ci * src[e];
        }
    }
    const float inv = bad ? __builtin_nanf("") : 1.0f / Lsum;
    if constexpr (E == 2) {
        const f32x2_t o = {acc[0] * inv, acc[1] * inv};
        *reinterpret_cast<bf16x2_t *>(dst) = __builtin_convertvector(o, bf16x2_t);
    } else {
        *reinterpret_cast<__bf16 *>(dst) = (__bf16)(acc[0] * inv);
    }
}

}  // namespace

hipError_t launch_merge(const MergeParams &p, int head_dim, hipStream_t stream)
{
    const long long items = (long long)p.batch * p.num_kv_heads * p.group;
    const int per_block = kMergeThreads / kWave;
    const int merge_blocks = (int)((items + per_block - 1) / per_block);
    const int next_blocks =
        p.next_kind != 0 ? (int)(((long long)p.next.batch * p.next.num_kv_heads + per_block - 1) / per_block) : 0;
    const dim3 grid((unsigned)(merge_blocks + next_blocks));
    const dim3 block(kMergeThreads);
#define SL_MERGE(DD, NN) hipLaunchKernelGGL((merge_kernel<DD, NN>), grid, block, 0, stream, p, merge_blocks)
    if (head_dim == 128 && p.next_kind == 0)
        SL_MERGE(128, 0);
    else if (head_dim == 128 && p.next_kind == 1)
        SL_MERGE(128, 1);
    else if (head_dim == 128 && p.next_kind == 2)
        SL_MERGE(128, 2);
    else if (head_dim == 64 && p.next_kind == 0)
        SL_MERGE(64, 0);
    else if (head_dim == 64 && p.next_kind == 1)
        SL_MERGE(64, 1);
    else if (head_dim == 64 && p.next_kind == 2)
        SL_MERGE(64, 2);
    else
        return hipErrorInvalidValue;
#undef SL_MERGE
    return hipGetLastError();
}

}  // namespace sl

namespace sl {

hipError_t launch_merge_prefix(const PrefixMergeParams &p, int head_dim, hipStream_t stream)
{
    const long long items = (long long)p.batch * p.num_q_heads;
    const int per_block = kMergeThreads / kWave;
    const dim3 grid((unsigned)((items + per_block - 1) / per_block));
    if (head_dim == 128)
        hipLaunchKernelGGL(merge_prefix_kernel<128>, grid, dim3(kMergeThreads), 0, stream, p);
    else if (head_dim == 64)
        hipLaunchKernelGGL(merge_prefix_kernel<64>, grid, dim3(kMergeThreads), 0, stream, p);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

}  // namespace sl
