// Device helper of the decode engine (engine.cpp): filling newly admitted
// prompts' pages with synthetic key/value data. (A step's bookkeeping is
// applied by the KV-append launch, append.hip.)
#include "sl_internal.h"

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

}  // namespace

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
