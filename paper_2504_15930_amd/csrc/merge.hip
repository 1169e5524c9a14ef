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
#include "sl_internal.h"

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

template <int D>
__global__ __launch_bounds__(kMergeThreads) void merge_kernel(MergeParams p)
{
    constexpr int E = D / kWave;   // output columns per lane (1 or 2)
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
    const int cb = p.cum_pages[b];
    const int nb = p.cum_pages[b + 1] - cb;

    if (nb == 0) {
        const uint16_t fill = p.seq_lens[b] < 0 ? 0x7fc0 : 0x0000;   // bf16 NaN / +0
#pragma unroll
        for (int e = 0; e < E; ++e)
            dst[e] = fill;
        return;
    }
    const long long total = (long long)p.cum_pages[p.batch] * Hkv;
    const long long NW = effective_workers(total, p.num_workers);
    const long long a = (long long)Hkv * cb + (long long)g * nb;   // first tile of the unit
    const long long e = a + nb;                                    // one past its last tile
    // Worker holding tile x: the largest w with floor(w * total / NW) <= x.
    const int wf = (int)(((a + 1) * NW - 1) / total);
    const int wl = (int)((e * NW - 1) / total);
    if (wf == wl)
        return;

    // Pass 1: lane i owns piece wf + c0 + i. The slot of worker w is 2w, except
    // for the unit's first worker when the unit began after that worker's
    // first tile (then it was the worker's trailing piece, slot 2w + 1).
    float M = -__builtin_inff();
    for (int c0 = 0; c0 <= wl - wf; c0 += kWave) {
        const int w = wf + c0 + lane;
        float m = -__builtin_inff();
        if (w <= wl) {
            const long long s = (long long)w * total / NW;
            if (s != (long long)(w + 1) * total / NW) {
                const long long slot = 2LL * w + ((w == wf && s < a) ? 1 : 0);
                m = p.part_ml[(slot * G + j) * 2];
            }
        }
        M = fmaxf(M, wave_max(m));
    }
    // Pass 2: weights per piece (in their lanes), then the weighted sums.
    float Lsum = 0.0f;
    float acc[E];
#pragma unroll
    for (int k = 0; k < E; ++k)
        acc[k] = 0.0f;
    for (int c0 = 0; c0 <= wl - wf; c0 += kWave) {
        const int w = wf + c0 + lane;
        float c = 0.0f, l = 0.0f;
        long long slot = 0;
        if (w <= wl) {
            const long long s = (long long)w * total / NW;
            if (s != (long long)(w + 1) * total / NW) {
                slot = 2LL * w + ((w == wf && s < a) ? 1 : 0);
                const f32x2_t ml = *reinterpret_cast<const f32x2_t *>(p.part_ml + (slot * G + j) * 2);
                c = __builtin_amdgcn_exp2f(ml[0] - M);
                l = ml[1];
            }
        }
        Lsum += wave_sum(c * l);
        const int cnt = min(kWave, wl - wf - c0 + 1);
        const int slot_lo = (int)slot;   // slots < 2^17, exchanged as 32-bit lanes
#pragma unroll 4
        for (int i = 0; i < cnt; ++i) {
            const float ci = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, c), i));
            const int si = __builtin_amdgcn_readlane(slot_lo, i);
            if (ci == 0.0f)
                continue;   // empty worker (or a weight that underflowed)
            const float *src = p.part_acc + ((size_t)si * G + j) * D + E * lane;
            if constexpr (E == 2) {
                const f32x2_t v = *reinterpret_cast<const f32x2_t *>(src);
                acc[0] += ci * v[0];
                acc[1] += ci * v[1];
            } else {
                acc[0] += ci * src[0];
            }
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

}  // namespace

hipError_t launch_merge(const MergeParams &p, int head_dim, hipStream_t stream)
{
    const long long items = (long long)p.batch * p.num_kv_heads * p.group;
    const int per_block = kMergeThreads / kWave;
    const dim3 grid((unsigned)((items + per_block - 1) / per_block));
    if (head_dim == 128)
        hipLaunchKernelGGL(merge_kernel<128>, grid, dim3(kMergeThreads), 0, stream, p);
    else if (head_dim == 64)
        hipLaunchKernelGGL(merge_kernel<64>, grid, dim3(kMergeThreads), 0, stream, p);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

}  // namespace sl
