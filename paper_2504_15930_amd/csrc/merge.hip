// Log-sum-exp merge of split-KV partial states.
//
// A unit (sequence b, KV head g) whose tiles were cut across workers
// w_first..w_last left, per worker, a partial state (m_i, l_i, acc_i) for each
// of its G query heads: m_i the largest score (base-2 units), l_i the sum of
// 2^(s - m_i) and acc_i the matching un-normalised sum of value rows. With
// M = max_i m_i the exact softmax result is
//     out = sum_i 2^(m_i - M) acc_i / sum_i 2^(m_i - M) l_i,
// evaluated here as a running (online) combination in fp32 and rounded to
// bf16. One workgroup per unit; units finished by a single worker were
// already written and are skipped. Units with no page write zero rows (or NaN
// rows for an invalid negative length).
#include "sl_internal.h"

namespace sl {
namespace {

typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

__global__ __launch_bounds__(kMergeThreads) void merge_kernel(MergeParams p)
{
    const int Hkv = p.num_kv_heads;
    const int b = blockIdx.x / Hkv;
    const int g = blockIdx.x - b * Hkv;
    const int G = p.group;
    const int D = p.head_dim;
    const int per_head = D / 4;   // threads per head, 4 outputs each
    const int L = p.seq_lens[b];
    const int cb = p.cum_pages[b];
    const int nb = p.cum_pages[b + 1] - cb;
    uint16_t *out = p.out + ((size_t)b * p.num_q_heads + (size_t)g * G) * D;

    if (nb == 0) {
        const float fill = L < 0 ? __builtin_nanf("") : 0.0f;
        const bf16x4_t f = {(__bf16)fill, (__bf16)fill, (__bf16)fill, (__bf16)fill};
        for (int idx = threadIdx.x; idx < G * per_head; idx += blockDim.x)
            *reinterpret_cast<u32x2_t *>(out + (size_t)idx * 4) = __builtin_bit_cast(u32x2_t, f);
        return;
    }
    const long long total = (long long)p.cum_pages[p.batch] * Hkv;
    const long long NW = p.num_workers;
    const long long a = (long long)Hkv * cb + (long long)g * nb;   // first tile of the unit
    const long long e = a + nb;                                    // one past its last tile
    // Worker holding tile x: the largest w with floor(w * total / NW) <= x.
    const int wf = (int)(((a + 1) * NW - 1) / total);
    const int wl = (int)((e * NW - 1) / total);
    if (wf == wl)
        return;

    for (int idx = threadIdx.x; idx < G * per_head; idx += blockDim.x) {
        const int j = idx / per_head;
        const int d = (idx - j * per_head) * 4;
        float M = -__builtin_inff();
        float Lsum = 0.0f;
        f32x4_t A = {0.f, 0.f, 0.f, 0.f};
        for (int w = wf; w <= wl; ++w) {
            const long long s = (long long)w * total / NW;
            const long long s1 = (long long)(w + 1) * total / NW;
            if (s == s1)
                continue;   // worker with an empty range
            const long long slot = 2LL * w + ((w == wf && s < a) ? 1 : 0);
            const f32x2_t ml = *reinterpret_cast<const f32x2_t *>(p.part_ml + (slot * G + j) * 2);
            const f32x4_t acc = *reinterpret_cast<const f32x4_t *>(p.part_acc + (slot * G + j) * D + d);
            const float Mn = fmaxf(M, ml[0]);
            const float c_old = M == -__builtin_inff() ? 0.0f : __builtin_amdgcn_exp2f(M - Mn);
            const float c_new = __builtin_amdgcn_exp2f(ml[0] - Mn);
            A = A * c_old + acc * c_new;
            Lsum = Lsum * c_old + ml[1] * c_new;
            M = Mn;
        }
        const f32x4_t o = A / Lsum;
        const bf16x4_t ob = __builtin_convertvector(o, bf16x4_t);
        *reinterpret_cast<u32x2_t *>(out + (size_t)j * D + d) = __builtin_bit_cast(u32x2_t, ob);
    }
}

}  // namespace

hipError_t launch_merge(const MergeParams &p, hipStream_t stream)
{
    const dim3 grid((unsigned)p.batch * (unsigned)p.num_kv_heads);
    hipLaunchKernelGGL(merge_kernel, grid, dim3(kMergeThreads), 0, stream, p);
    return hipGetLastError();
}

}  // namespace sl
