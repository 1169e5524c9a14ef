// Device helpers of the decode engine (engine.cpp): applying one step's
// bookkeeping (sequence lengths, new block-table entries) and filling newly
// admitted prompts' pages with synthetic key/value data.
#include "sl_internal.h"

namespace sl {
namespace {

constexpr int kEngineThreads = 256;

// stage = [seq_lens: bs][updates: n_upd x (slot, block, page)]. Every index was
// checked on the host (slot < bs, block < max_blocks).
__global__ __launch_bounds__(kEngineThreads) void engine_apply_kernel(const int32_t *stage, int32_t bs,
                                                                      int32_t n_upd, int32_t max_blocks,
                                                                      int32_t *seq_lens, int32_t *block_table)
{
    const int i = blockIdx.x * kEngineThreads + threadIdx.x;
    if (i < bs)
        seq_lens[i] = stage[i];
    if (i < n_upd) {
        const int32_t *u = stage + bs + 3 * i;
        block_table[(size_t)u[0] * max_blocks + u[1]] = u[2];
    }
}

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

}  // namespace

hipError_t launch_engine_apply(const int32_t *stage, int bs, int n_upd, int max_blocks, int32_t *seq_lens,
                               int32_t *block_table, hipStream_t stream)
{
    const int n = bs > n_upd ? bs : n_upd;
    hipLaunchKernelGGL(engine_apply_kernel, dim3((n + kEngineThreads - 1) / kEngineThreads), dim3(kEngineThreads),
                       0, stream, stage, bs, n_upd, max_blocks, seq_lens, block_table);
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
