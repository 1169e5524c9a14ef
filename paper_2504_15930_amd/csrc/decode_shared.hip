// Prefix-shared decode attention for gfx950: the fused split kernel that
// streams the own pages and the shared pages of a batch in one launch.
//
// A shared unit is (sub-group of samples, KV head): its tiles are the
// group's shared pages, read through the sub-group's first member's
// block-table row, and its query rows are the members x G query heads of that
// KV head, at most kPrefixRows = 64, as four 16-row MFMA column blocks (row
// r = 16 c + n is member r / G, head r % G of the sub-group). A group larger
// than that is cut into sub-groups, each reading the shared pages once.
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

// Prologue of the fused prefix kernel, run by the whole workgroup. A group k
// is shared if its range [group_start[k], group_start[k+1]) is non-empty,
// inside the batch and starts at or after the end of every earlier group's
// range (so the groups that are shared never overlap, whatever the order of
// group_start), and its page count is in 1 .. max_blocks. Others are attended
// like unshared sequences: exact, only without the saving. A shared group of
// m members is cut into ns = ceil(m / M) sub-groups of ceil(m / ns) members
// (the last may be smaller), M = min(16, kPrefixRows / G), each of which
// reads the shared pages once: the shared stream has one "sequence" per
// sub-group. Builds in LDS, with every pass parallel over groups,
// sub-groups or sequences:
//   s_group[b]  the sub-group of sequence b (-1: none; B + 1 entries, the
//               last one scratch),
//   s_len[b]    the lengths,
//   s_own[0..B] the exclusive prefix sum of own (unshared) pages per sequence,
//   s_sh[0..S]  the exclusive prefix sum of shared pages per sub-group, and
//   s_gl[s]     each sub-group's first member and size, lead | (members - 1) << 16,
// where S = max_sub bounds the sub-group count (sub-groups past the real
// count have no pages). Workgroup 0 also stores the sums and every
// sequence's sharing descriptor for the merge.
__device__ __forceinline__ void scan_prefix_groups(const SplitParams &p, const PrefixParams &pp, int32_t *s_own,
                                                   int32_t *s_len, int32_t *s_group, int32_t *s_sh, int32_t *s_gl,
                                                   int32_t *s_gs, int32_t *s_sp)
{
    constexpr int T = kWave * kWavesPerBlock;
    const int B = p.batch, NG = pp.num_groups, S = pp.max_sub;
    const int tid = threadIdx.x;
    const int M = prefix_max_members(p.group);
    const int32_t *gs = s_gs;   // group_start and shared_pages, read from memory once
    // Scratch for the group passes, in arrays filled only later: s_len (B
    // entries, followed by s_sh, whose first entry takes the scan's total when
    // NG == B) and s_own (B + 1 entries).
    int32_t *const s_prev_end = s_len;   // [NG + 1]: largest end of the earlier groups
    int32_t *const s_base = s_own;       // [NG + 1]: first sub-group of each group
    // 1. Each group's earlier ends; every sequence starts unmarked. With
    //    group_start ascending (the usual case) the largest earlier end of
    //    group k is its own start, and the scan is skipped.
    bool descends = false;
    for (int k = tid; k < NG; k += T) {
        const int lo = pp.group_start[k], hi = pp.group_start[k + 1];
        s_gs[k] = lo;
        s_sp[k] = pp.shared_pages[k];
        if (k == NG - 1)
            s_gs[NG] = hi;
        descends |= lo > hi;
    }
    for (int b = tid; b < B; b += T)
        s_group[b] = -1;
    const bool ascending = !__syncthreads_or(descends);
    if (!ascending) {
        for (int k = tid; k < NG; k += T)
            s_prev_end[k] = gs[k + 1];
        __syncthreads();
        block_exclusive_scan<ScanMax>(s_prev_end, NG);
    }
    // 2. Which groups are shared, how many sub-groups each has, and a mark at
    //    each shared group's first member (shared groups never overlap, so no
    //    two marks collide).
    for (int k = tid; k < NG; k += T) {
        const int lo = gs[k], hi = gs[k + 1], sp = s_sp[k];
        const bool ok = lo >= 0 && hi <= B && hi > lo && (ascending || lo >= s_prev_end[k]) && sp > 0 &&
                        sp <= p.max_blocks;
        s_base[k] = ok ? (hi - lo + M - 1) / M : 0;
        if (ok)
            s_group[lo] = k;
    }
    __syncthreads();
    // s_base: first sub-group of each group; s_group[b + 1]: the latest mark at or before b.
    block_exclusive_scan2<ScanSum, ScanMax>(s_base, NG, s_group, B);
    // 3. The sub-groups: shared pages and packed first member and size.
    const int NS = s_base[NG];
    for (int sg = tid; sg < S; sg += T) {
        int sp = 0, gl = 0;
        if (sg < NS) {
            int klo = 0, khi = NG;   // largest k with s_base[k] <= sg (a group with sub-groups)
            while (khi - klo > 1) {
                const int mid = (klo + khi) >> 1;
                if (s_base[mid] <= sg)
                    klo = mid;
                else
                    khi = mid;
            }
            const int lo = gs[klo], m = gs[klo + 1] - lo;
            const int ns = (m + M - 1) / M, cm = (m + ns - 1) / ns;
            const int slo = lo + (sg - s_base[klo]) * cm;
            sp = s_sp[klo];
            gl = slo | (min(cm, lo + m - slo) - 1) << 16;
        }
        s_sh[sg] = sp;
        s_gl[sg] = gl;
    }
    // 4. The sub-group of every sequence: the group of the latest mark at or
    //    before b (the exclusive scan's entry b + 1; entry B holds the
    //    maximum), if b lies inside that group's range.
    constexpr int kPer = (kMaxPrefixBatch + T - 1) / T;
    int32_t sub[kPer];
#pragma unroll
    for (int r = 0; r < kPer; ++r) {
        const int b = tid + r * T;
        sub[r] = -1;
        if (b < B) {
            const int k = s_group[b + 1];
            if (k >= 0 && b < gs[k + 1]) {
                const int lo = gs[k], m = gs[k + 1] - lo;
                const int ns = (m + M - 1) / M, cm = (m + ns - 1) / ns;
                const int sg = s_base[k] + (b - lo) / cm;
                sub[r] = sg < S ? sg : -1;   // always below S (prefix_max_sub bounds the count)
            }
        }
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kPer; ++r) {
        const int b = tid + r * T;
        if (b < B)
            s_group[b] = sub[r];
    }
    __syncthreads();
    // 5. Lengths and own pages (the pages after the sub-group's shared ones).
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
    block_exclusive_scan2<ScanSum, ScanSum>(s_own, B, s_sh, S);
    if (blockIdx.x == 0) {
        for (int i = tid; i <= B; i += T)
            pp.cum_own[i] = s_own[i];
        for (int i = tid; i <= S; i += T)
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
// (prefix_dynamic_lds: 3 B + 2 S + 2 NG + 4 ints, S = pp.max_sub); the number of
// shared-page workers that take part is effective_shared_workers of the
// own-page total, as in the merge.
template <int D, bool FP8>
__global__ __launch_bounds__(kWave * kWavesPerBlock) void prefix_split_kernel(SplitParams own, SplitParams shared,
                                                                               PrefixParams pp, int own_blocks,
                                                                               int max_shared)
{
    extern __shared__ int32_t s_dyn[];
    const int B = own.batch, S = pp.max_sub;
    int32_t *const s_own = s_dyn;             // [B + 1]
    int32_t *const s_group = s_own + B + 1;   // [B + 1]
    int32_t *const s_len = s_group + B + 1;   // [B]
    int32_t *const s_sh = s_len + B;          // [S + 1]
    int32_t *const s_gl = s_sh + S + 1;       // [S]
    int32_t *const s_gs = s_gl + S;           // [NG + 1]
    int32_t *const s_sp = s_gs + pp.num_groups + 1;   // [NG]
    scan_prefix_groups(own, pp, s_own, s_len, s_group, s_sh, s_gl, s_gs, s_sp);
    if ((int)blockIdx.x < own_blocks)
        split_unit_worker<D, FP8, kOwnPages>(
            own, blockIdx.x * kWavesPerBlock + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave),
            StreamLds{s_own, s_len, s_group, s_sh});
    else {
        SplitParams sh = shared;
        sh.num_workers = effective_shared_workers((long long)s_own[B] * own.num_kv_heads, own.num_workers,
                                                  shared.num_workers, max_shared);
        split_unit_worker<D, FP8, kSharedPages>(sh, (int)blockIdx.x - own_blocks,
                                                  StreamLds{s_sh, nullptr, nullptr, nullptr, s_gl, S},
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
    const size_t lds = prefix_dynamic_lds(own.batch, pp.max_sub, pp.num_groups);
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
