// KV append kernel: one wavefront per (sequence, KV head) runs append_unit
// (append_unit.h, which states the rules); in the engine's staged mode the
// launch also applies the step's lengths and block-table updates.
#include "append_unit.h"

namespace sl {
namespace {

template <int D, bool FP8>
__global__ __launch_bounds__(kWave * kWavesPerBlock) void append_kernel(AppendParams p)
{
    if (p.stage)   // nothing in this launch reads the lengths or the block table from memory in this mode
        apply_stage(p, blockIdx.x * blockDim.x + threadIdx.x, gridDim.x * blockDim.x);
    const int unit = blockIdx.x * kWavesPerBlock + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    if (unit < p.batch * p.num_kv_heads)
        append_unit<D, FP8>(p, unit, threadIdx.x & (kWave - 1));
}

}  // namespace

hipError_t launch_append(const AppendParams &p, int head_dim, bool fp8, hipStream_t stream)
{
    const long long units = (long long)p.batch * p.num_kv_heads;
    const dim3 grid((unsigned)((units + kWavesPerBlock - 1) / kWavesPerBlock));
    const dim3 block(kWave * kWavesPerBlock);
    if (head_dim == 128 && !fp8)
        hipLaunchKernelGGL((append_kernel<128, false>), grid, block, 0, stream, p);
    else if (head_dim == 64 && !fp8)
        hipLaunchKernelGGL((append_kernel<64, false>), grid, block, 0, stream, p);
    else if (head_dim == 128 && fp8)
        hipLaunchKernelGGL((append_kernel<128, true>), grid, block, 0, stream, p);
    else if (head_dim == 64 && fp8)
        hipLaunchKernelGGL((append_kernel<64, true>), grid, block, 0, stream, p);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

}  // namespace sl
