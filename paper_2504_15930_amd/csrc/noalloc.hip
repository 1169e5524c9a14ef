// sl_decode_attn_noalloc: decode attention with a bf16 cache for callers that
// cannot allocate device memory (code under HIP graph capture, tight serving
// loops, harnesses that forbid hipMalloc). It runs exactly the kernels of
// sl_decode_attn; their scratch (the page prefix sum and the split-KV partial
// states) lives in a fixed array of this library instead of a caller
// workspace.
//
// The array is a file-scope __device__ variable: every GPU the library runs
// on holds its own copy, at its own address, until the process ends. In host
// code its name is only a host-side stand-in, so the device address is taken
// once per device with hipGetSymbolAddress (on the first call on that device,
// with that device current) and only that address is ever passed to kernels.
// Nothing in the array needs to start at zero: the split kernel writes the
// prefix sum and every partial state the merge then reads. Calls that overlap
// in time on one GPU share the array and race.
#include <mutex>

#include "../../include/sl.h"
#include "sl_internal.h"

namespace sl {
namespace {

// SL_NOALLOC_SCRATCH_BYTES (16 MiB) covers the default worker count for every
// supported shape (the largest, head_dim 128 with 16 query heads per KV head
// and 8192 sequences, needs about 12.8 MB).
constexpr size_t kScratchBytes = SL_NOALLOC_SCRATCH_BYTES;

static __device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;

struct ScratchAddress {
    std::once_flag once;
    hipError_t err = hipSuccess;
    void *ptr = nullptr;
};
ScratchAddress g_scratch[kMaxDevices];

// Device address of this device's copy of `scratch` (looked up once per device).
hipError_t scratch_address(void **out)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return e;
    if (dev < 0 || dev >= kMaxDevices)
        return hipErrorInvalidDevice;
    ScratchAddress &s = g_scratch[dev];
    std::call_once(s.once, [&s] {
        void *p = nullptr;
        s.err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (s.err == hipSuccess && p == nullptr)
            s.err = hipErrorInvalidSymbol;
        s.ptr = p;
    });
    *out = s.ptr;
    return s.err;
}

}  // namespace
}  // namespace sl

extern "C" sl_status sl_decode_attn_noalloc(const sl_attn_desc *desc, const uint16_t *q, const uint16_t *k_pages,
                                            const uint16_t *v_pages, const int32_t *block_table,
                                            const int32_t *seq_lens, float scale, uint16_t *out)
{
    if (!desc)
        return SL_ERR_NULL;
    // Validates the sizes and resolves the worker count, as the call itself will.
    int32_t nw = 0;
    sl_status st = sl_decode_attn_num_workers(desc, 0, &nw);
    if (st != SL_OK)
        return st;
    if (desc->batch == 0)
        return SL_OK;
    const size_t need = sl::workspace_layout(nullptr, desc->batch, desc->max_blocks_per_seq, desc->num_kv_heads,
                                             desc->num_q_heads / desc->num_kv_heads, desc->head_dim, nw, nullptr);
    if (need > sl::kScratchBytes)
        return SL_ERR_SCRATCH_LIMIT;
    void *ptr = nullptr;
    if (sl::scratch_address(&ptr) != hipSuccess)
        return SL_ERR_HIP;
    sl_attn_desc d = *desc;
    d.workspace = ptr;
    d.workspace_bytes = sl::kScratchBytes;
    return sl_decode_attn(&d, q, k_pages, v_pages, block_table, seq_lens, scale, out);
}
