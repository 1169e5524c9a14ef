// Work partitioner of prefix-shared decode attention: turns device-resident
// sequence lengths, block tables and group descriptions into the two flat
// tile lists (own pages, shared pages) that the split-KV workers stream, with
// no host synchronisation. (Plain decode attention partitions inside the
// split kernel, from the lengths and the block table directly.)
#include "sl_internal.h"

namespace sl {

// ---- prefix-sharing mode ----------------------------------------------------
//
// Groups are runs of consecutive sequences [group_start[k], group_start[k+1])
// whose first shared_pages[k] pages are the same (the group's first member's
// block-table entries are read). Each workgroup builds in LDS: the group of
// every sequence, the exclusive prefix sum of every sequence's own (unshared)
// pages and of every group's shared pages; workgroup 0 also stores them for
// the merge. Then the grid walks both page sets: own pages give entries like
// the plain partitioner's (first / last relative to the own pages, flagged
// kMetaPrefixed when the sequence has shared pages), shared pages give one
// entry per (group, KV head, page) with members - 1 in bits [3:0].
//
// A group that is empty, has more than 16 members or more members than
// kPrefixRows / G, or whose range or page count is out of bounds, is treated
// as unshared; so the result stays exact, only without the saving.

namespace {

__device__ __forceinline__ int block_exclusive_scan(int local, int32_t *s_part, int tid, int *total)
{
    const int lane = tid & (kWave - 1);
    const int wave = tid / kWave;
    int incl = local;
    for (int off = 1; off < kWave; off <<= 1) {
        const int v = __shfl_up(incl, off, kWave);
        if (lane >= off)
            incl += v;
    }
    if (lane == kWave - 1)
        s_part[wave] = incl;
    __syncthreads();
    if (wave == 0) {
        int t = lane < kPartitionThreads / kWave ? s_part[lane] : 0;
        for (int off = 1; off < kWave; off <<= 1) {
            const int v = __shfl_up(t, off, kWave);
            if (lane >= off)
                t += v;
        }
        if (lane < kPartitionThreads / kWave)
            s_part[lane] = t;
    }
    __syncthreads();
    const int excl = incl - local + (wave > 0 ? s_part[wave - 1] : 0);
    *total = s_part[kPartitionThreads / kWave - 1];
    __syncthreads();
    return excl;
}

}  // namespace

__global__ __launch_bounds__(kPartitionThreads) void partition_prefix_kernel(PrefixPartitionParams p)
{
    extern __shared__ int32_t s_mem[];
    __shared__ int32_t s_part[kPartitionThreads / kWave];
    const int B = p.batch, NG = p.num_groups;
    int32_t *s_group = s_mem;              // [B]   group of each sequence (-1: unshared)
    int32_t *s_own = s_mem + B;            // [B+1] own pages, then their exclusive prefix sum
    int32_t *s_sh = s_own + B + 1;         // [NG+1] shared pages per group, then the prefix sum
    const int tid = threadIdx.x;
    const int G = p.num_q_heads / p.num_kv_heads;
    const int max_members = min(16, kPrefixRows / G);

    for (int b = tid; b < B; b += kPartitionThreads)
        s_group[b] = -1;
    __syncthreads();
    // Effective shared pages per group, and the group of each member.
    for (int k = tid; k < NG; k += kPartitionThreads) {
        const int lo = p.group_start[k], hi = p.group_start[k + 1];
        const int sp = p.shared_pages[k];
        const bool ok = lo >= 0 && hi <= B && hi - lo >= 1 && hi - lo <= max_members && sp > 0 &&
                        sp <= p.max_blocks;
        s_sh[k] = ok ? sp : 0;
        if (ok)
            for (int b = lo; b < hi; ++b)
                s_group[b] = k;
    }
    __syncthreads();
    const int max_len = p.max_blocks * kPageSize;
    for (int b = tid; b < B; b += kPartitionThreads) {
        const int L = p.seq_lens[b];
        const int n = L <= 0 ? 0 : (min(L, max_len) + kPageSize - 1) / kPageSize;
        const int k = s_group[b];
        const int sh = k >= 0 ? s_sh[k] : 0;
        s_own[b] = n > sh ? n - sh : 0;
    }
    __syncthreads();
    // Exclusive prefix sums (each thread scans a contiguous run).
    {
        const int per = (B + kPartitionThreads - 1) / kPartitionThreads;
        const int lo = min(B, tid * per), hi = min(B, lo + per);
        int local = 0;
        for (int i = lo; i < hi; ++i)
            local += s_own[i];
        int total;
        int run = block_exclusive_scan(local, s_part, tid, &total);
        for (int i = lo; i < hi; ++i) {
            const int v = s_own[i];
            s_own[i] = run;
            run += v;
        }
        if (tid == 0)
            s_own[B] = total;
    }
    {
        const int per = (NG + kPartitionThreads - 1) / kPartitionThreads;
        const int lo = min(NG, tid * per), hi = min(NG, lo + per);
        int local = 0;
        for (int i = lo; i < hi; ++i)
            local += s_sh[i];
        int total;
        int run = block_exclusive_scan(local, s_part, tid, &total);
        for (int i = lo; i < hi; ++i) {
            const int v = s_sh[i];
            s_sh[i] = run;
            run += v;
        }
        if (tid == 0)
            s_sh[NG] = total;
    }
    __syncthreads();
    if (blockIdx.x == 0) {
        for (int i = tid; i <= B; i += kPartitionThreads)
            p.cum_own[i] = s_own[i];
        for (int i = tid; i <= NG; i += kPartitionThreads)
            p.cum_shared[i] = s_sh[i];
        for (int i = tid; i < B; i += kPartitionThreads) {
            const int k = s_group[i];
            typedef int32_t i32x4_t __attribute__((ext_vector_type(4)));
            *reinterpret_cast<i32x4_t *>(p.seq_shared + 4 * (size_t)i) =
                k >= 0 ? i32x4_t{s_sh[k], s_sh[k + 1] - s_sh[k], p.group_start[k], k} : i32x4_t{0, 0, 0, -1};
        }
    }

    const int Hkv = p.num_kv_heads;
    // Own pages.
    const int own_total = s_own[B];
    for (int x = blockIdx.x * kPartitionThreads + tid; x < own_total; x += gridDim.x * kPartitionThreads) {
        int blo = 0, bhi = B;
        while (bhi - blo > 1) {
            const int mid = (blo + bhi) >> 1;
            if (s_own[mid] <= x)
                blo = mid;
            else
                bhi = mid;
        }
        const int b = blo;
        const int ob = s_own[b + 1] - s_own[b];
        const int j = x - s_own[b];                      // own page index
        const int k = s_group[b];
        const int sh = k >= 0 ? s_sh[k + 1] - s_sh[k] : 0;
        const int pg = sh + j;                           // page index in the sequence
        const int L = p.seq_lens[b];
        const int pid = p.block_table[(size_t)b * p.max_blocks + pg];
        const bool page_ok = (unsigned)pid < (unsigned)p.num_pages;
        const int live = min(kPageSize, L - pg * kPageSize);
        uint32_t meta = (uint32_t)(max(live, 1) - 1);
        if (j == ob - 1)
            meta |= kMetaLast;
        if (j == 0)
            meta |= kMetaFirst;
        if (L > max_len)
            meta |= kMetaBadLen;
        if (sh > 0)
            meta |= kMetaPrefixed;
        const long long base = (long long)Hkv * s_own[b] + j;
        for (int g = 0; g < Hkv; ++g) {
            TileEntry e;
            e.page = page_ok ? pid * Hkv + g : -1;
            e.meta = meta | ((uint32_t)(b * p.num_q_heads + g * G) << kMetaRowShift);
            p.own_tiles[base + (long long)g * ob] = e;
        }
    }
    // Shared pages, read through the group's first member.
    const int sh_total = s_sh[NG];
    for (int x = blockIdx.x * kPartitionThreads + tid; x < sh_total; x += gridDim.x * kPartitionThreads) {
        int klo = 0, khi = NG;
        while (khi - klo > 1) {
            const int mid = (klo + khi) >> 1;
            if (s_sh[mid] <= x)
                klo = mid;
            else
                khi = mid;
        }
        const int k = klo;
        const int sk = s_sh[k + 1] - s_sh[k];
        const int pg = x - s_sh[k];
        const int lead = p.group_start[k];
        const int members = p.group_start[k + 1] - lead;
        const int pid = p.block_table[(size_t)lead * p.max_blocks + pg];
        const bool page_ok = (unsigned)pid < (unsigned)p.num_pages;
        uint32_t meta = (uint32_t)(members - 1);
        if (pg == sk - 1)
            meta |= kMetaLast;
        if (pg == 0)
            meta |= kMetaFirst;
        const long long base = (long long)Hkv * s_sh[k] + pg;
        for (int g = 0; g < Hkv; ++g) {
            TileEntry e;
            e.page = page_ok ? pid * Hkv + g : -1;
            e.meta = meta | ((uint32_t)(lead * p.num_q_heads + g * G) << kMetaRowShift);
            p.shared_tiles[base + (long long)g * sk] = e;
        }
    }
}

hipError_t launch_partition_prefix(const PrefixPartitionParams &p, hipStream_t stream)
{
    const long long max_pages = (long long)p.batch * p.max_blocks;
    int grid = (int)((max_pages + kPartitionThreads - 1) / kPartitionThreads);
    grid = grid < 1 ? 1 : (grid > 256 ? 256 : grid);
    const size_t lds = sizeof(int32_t) * (2 * (size_t)p.batch + 1 + (size_t)p.num_groups + 1);
    hipLaunchKernelGGL(partition_prefix_kernel, dim3(grid), dim3(kPartitionThreads), lds, stream, p);
    return hipGetLastError();
}

}  // namespace sl
