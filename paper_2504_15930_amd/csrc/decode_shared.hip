// Prefix-shared decode attention for gfx950: the fused split kernel that
// streams the own pages and the shared pages of a batch in one launch.
//
// A shared unit is (group of samples, KV head): its tiles are the group's
// shared pages, read through the first member's block-table row, and its
// query rows are the members x G query heads of that KV head, at most
// kPrefixRows = 64, as four 16-row MFMA column blocks (row r = 16 c + n is
// member r / G, head r % G of the group).
//
// Workgroups [0, own_blocks) run the single-unit workers of the own pages
// (decode_unit.h, four per workgroup). The others are shared-page workers,
// one per workgroup: the workgroup's four wavefronts stream the same range of
// shared tiles with the single-unit pipeline, and wavefront c computes column
// block c of every unit in it. They read each tile at the same time with
// plain (not streaming) loads, so the tile comes from HBM once and the
// siblings find it in L2; no wavefront waits for another. Each wavefront
// keeps one block's registers.
//
// The kernel is instantiated for bf16 and E4M3 pages. For E4M3 every
// wavefront widens the whole shared tile itself (its block needs all keys and
// values) and scales it by the page's own per-(page, KV head) scales.
//
// The own-page workgroups come first, so each CU holds one of them beside a
// shared-page workgroup: the memory-bound and the MFMA-heavy pass share the
// CUs instead of running one after the other.
//
// Partial states: a unit cut by a worker's range leaves its piece in slot 2w
// (first piece) or 2w + 1 (trailing piece) of the worker; a unit seen whole
// goes to its own slot of the unit area, at (first query row) / G. Every
// shared state still has to be merged with the members' own pages, and so do
// the own units of sequences that have shared pages.
#include "decode_unit.h"

namespace sl {
namespace {

// Prologue of the fused prefix kernel, run by the whole workgroup: builds in
// LDS the group of every sequence (-1: none), the lengths, the exclusive
// prefix sums of own pages per sequence and of shared pages per group, and
// each group's packed first member and size; workgroup 0 also stores the sums
// and every sequence's sharing descriptor for the merge. A group that is
// empty, has more than min(16, kPrefixRows / G) members, or whose range or
// page count is out of bounds gets no shared pages: its members are attended
// like unshared sequences, so the result stays exact, only without the saving.
__device__ __forceinline__ void scan_prefix_groups(const SplitParams &p, const PrefixParams &pp, int32_t *s_own,
                                                   int32_t *s_len, int32_t *s_group, int32_t *s_sh, int32_t *s_gl)
{
    constexpr int T = kWave * kWavesPerBlock;
    const int B = p.batch, NG = pp.num_groups;
    const int tid = threadIdx.x;
    const int max_members = min(16, kPrefixRows / p.group);
    for (int b = tid; b < B; b += T)
        s_group[b] = -1;
    __syncthreads();
    for (int k = tid; k < NG; k += T) {
        const int lo = pp.group_start[k], hi = pp.group_start[k + 1];
        const int sp = pp.shared_pages[k];
        const bool ok = lo >= 0 && hi <= B && hi - lo >= 1 && hi - lo <= max_members && sp > 0 &&
                        sp <= p.max_blocks;
        s_sh[k] = ok ? sp : 0;
        s_gl[k] = ok ? lo | (hi - lo - 1) << 16 : 0;
        if (ok)
            for (int b = lo; b < hi; ++b)
                atomicMax(&s_group[b], k);   // ascending groups never overlap; otherwise every workgroup agrees
    }
    __syncthreads();
    const int max_len = p.max_blocks * kPageSize;
    for (int b = tid; b < B; b += T) {
        const int L = p.seq_lens[b];
        const int k = s_group[b];
        const int n = pages_of(L, max_len);
        const int sh = k >= 0 ? s_sh[k] : 0;
        s_len[b] = L;
        s_own[b] = n > sh ? n - sh : 0;
    }
    __syncthreads();
    block_exclusive_scan(s_own, B);
    block_exclusive_scan(s_sh, NG);
    if (blockIdx.x == 0) {
        for (int i = tid; i <= B; i += T)
            pp.cum_own[i] = s_own[i];
        for (int i = tid; i <= NG; i += T)
            pp.cum_shared[i] = s_sh[i];
        typedef int32_t i32x4_t __attribute__((ext_vector_type(4)));
        for (int i = tid; i < B; i += T) {
            const int k = s_group[i];
            *reinterpret_cast<i32x4_t *>(pp.seq_shared + 4 * (size_t)i) =
                k >= 0 ? i32x4_t{s_sh[k], s_sh[k + 1] - s_sh[k], s_gl[k] & 0xffff, k} : i32x4_t{0, 0, 0, -1};
        }
    }
}

// Both passes of prefix-shared attention in one launch (see the top of this
// file). Every workgroup first derives both streams in its dynamic LDS
// (3 B + 2 NG + 2 ints); the number of shared-page workers that take part is
// effective_shared_workers of the own-page total, as in the merge.
template <int D, bool FP8>
__global__ __launch_bounds__(kWave * kWavesPerBlock) void prefix_split_kernel(SplitParams own, SplitParams shared,
                                                                               PrefixParams pp, int own_blocks,
                                                                               int max_shared)
{
    extern __shared__ int32_t s_dyn[];
    const int B = own.batch, NG = pp.num_groups;
    int32_t *const s_own = s_dyn;            // [B + 1]
    int32_t *const s_len = s_own + B + 1;    // [B]
    int32_t *const s_group = s_len + B;      // [B]
    int32_t *const s_sh = s_group + B;       // [NG + 1]
    int32_t *const s_gl = s_sh + NG + 1;     // [NG]
    scan_prefix_groups(own, pp, s_own, s_len, s_group, s_sh, s_gl);
    if ((int)blockIdx.x < own_blocks)
        split_unit_worker<D, FP8, kOwnPages>(
            own, blockIdx.x * kWavesPerBlock + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave),
            StreamLds{s_own, s_len, s_group, s_sh});
    else {
        SplitParams sh = shared;
        sh.num_workers = effective_shared_workers((long long)s_own[B] * own.num_kv_heads, own.num_workers,
                                                  shared.num_workers, max_shared);
        split_unit_worker<D, FP8, kSharedPages>(sh, (int)blockIdx.x - own_blocks,
                                                  StreamLds{s_sh, nullptr, nullptr, nullptr, s_gl, NG},
                                                  __builtin_amdgcn_readfirstlane(threadIdx.x / kWave));
    }
}

}  // namespace

hipError_t launch_prefix_split(const SplitParams &own, const SplitParams &shared, int max_shared,
                               const PrefixParams &pp, int head_dim, bool fp8, hipStream_t stream)
{
    const int own_blocks = (own.num_workers + kWavesPerBlock - 1) / kWavesPerBlock;
    const dim3 grid(own_blocks + max_shared);
    const dim3 block(kWave * kWavesPerBlock);
    const size_t lds = prefix_dynamic_lds(own.batch, pp.num_groups);
#define SL_PREFIX(DD, FF) \
    hipLaunchKernelGGL((prefix_split_kernel<DD, FF>), grid, block, lds, stream, own, shared, pp, own_blocks, max_shared)
    if (head_dim == 128 && !fp8)
        SL_PREFIX(128, false);
    else if (head_dim == 64 && !fp8)
        SL_PREFIX(64, false);
    else if (head_dim == 128 && fp8)
        SL_PREFIX(128, true);
    else if (head_dim == 64 && fp8)
        SL_PREFIX(64, true);
    else
        return hipErrorInvalidValue;
#undef SL_PREFIX
    return hipGetLastError();
}

}  // namespace sl
