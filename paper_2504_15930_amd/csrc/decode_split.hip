// Split-KV decode attention kernel for gfx950: one wavefront per worker, the
// worker itself (tile pipeline, MFMA layout, online softmax, epilogue) is in
// decode_unit.h.
#include "decode_unit.h"

namespace sl {
namespace {

// Every workgroup derives the tile stream from the lengths and the block
// table (its dynamic LDS holds the page prefix sum and the lengths).
//
// Worker w = wave * gridDim.x + block: the four wavefronts of a workgroup take
// ranges a quarter of the stream apart, so a CU streams four unrelated
// sequences or heads at once rather than four neighbouring ranges of one
// unit (whose tiles all sit at the same offset inside their pages), and a
// stream too small for every worker still spreads over as many CUs as it
// has workers.
template <int D, bool FP8>
__global__ __launch_bounds__(kWave * kWavesPerBlock) void split_kv_kernel(SplitParams p)
{
    extern __shared__ int32_t s_dyn[];
    int32_t *const s_cum = s_dyn;                // [B + 1]
    int32_t *const s_len = s_dyn + p.batch + 1;  // [B]
    scan_sequences(p, s_cum, s_len);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    split_unit_worker<D, FP8, kAllPages>(p, wave * (int)gridDim.x + (int)blockIdx.x,
                                         StreamLds{s_cum, s_len, nullptr, nullptr});
}

}  // namespace

hipError_t launch_split(const SplitParams &p, int head_dim, bool fp8, hipStream_t stream)
{
    const dim3 grid((p.num_workers + kWavesPerBlock - 1) / kWavesPerBlock);
    const dim3 block(kWave * kWavesPerBlock);
    const size_t lds = split_dynamic_lds(p.batch);
    if (head_dim == 128 && !fp8)
        hipLaunchKernelGGL((split_kv_kernel<128, false>), grid, block, lds, stream, p);
    else if (head_dim == 64 && !fp8)
        hipLaunchKernelGGL((split_kv_kernel<64, false>), grid, block, lds, stream, p);
    else if (head_dim == 128 && fp8)
        hipLaunchKernelGGL((split_kv_kernel<128, true>), grid, block, lds, stream, p);
    else if (head_dim == 64 && fp8)
        hipLaunchKernelGGL((split_kv_kernel<64, true>), grid, block, lds, stream, p);
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
