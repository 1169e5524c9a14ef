// CU-level work partitioner: turns device-resident sequence lengths and block
// tables into the flat tile list the split-KV workers stream, with no host
// synchronisation.
//
// Every workgroup (1024 threads) first recomputes, in LDS, the pages per
// sequence n_b = ceil(clamp(L_b, 0, max_blocks * 16) / 16) and their exclusive
// prefix sum; workgroup 0 also stores that sum (cum_pages) for the other
// kernels. Then the grid walks the live pages: page p of sequence b yields one
// entry per KV head g at tile index Hkv * cum[b] + g * n_b + p, holding the
// page-head tile index (page id * Hkv + g, or -1 for an id outside the pool)
// and the unit's metadata (live tokens, first/last-tile flags, invalid-length
// flag, first query row). Consecutive threads take consecutive pages of a
// row, so block-table reads and entry writes are coalesced.
// Cost: B prefix-sum work per workgroup plus 8 bytes written per tile.
#include "sl_internal.h"

namespace sl {

__global__ __launch_bounds__(kPartitionThreads) void partition_kernel(PartitionParams p)
{
    extern __shared__ int32_t s_cum[];   // B + 1
    __shared__ int32_t s_part[kPartitionThreads / kWave];

    const int tid = threadIdx.x;
    const int B = p.batch;
    const int max_len = p.max_blocks * kPageSize;
    const int per = (B + kPartitionThreads - 1) / kPartitionThreads;
    const int lo = min(B, tid * per);
    const int hi = min(B, lo + per);

    int local = 0;
    for (int i = lo; i < hi; ++i) {
        const int L = p.seq_lens[i];
        const int n = L <= 0 ? 0 : (min(L, max_len) + kPageSize - 1) / kPageSize;
        s_cum[i] = n;
        local += n;
    }

    // Block-wide exclusive scan of `local`: inclusive scan inside each wave,
    // then a scan of the per-wave totals.
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
            s_part[lane] = t;  // inclusive over waves
    }
    __syncthreads();
    int run = incl - local + (wave > 0 ? s_part[wave - 1] : 0);
    for (int i = lo; i < hi; ++i) {
        const int n = s_cum[i];
        s_cum[i] = run;
        run += n;
    }
    if (tid == 0)
        s_cum[B] = s_part[kPartitionThreads / kWave - 1];
    __syncthreads();

    if (blockIdx.x == 0)
        for (int i = tid; i <= B; i += kPartitionThreads)
            p.cum_pages[i] = s_cum[i];

    const int Hkv = p.num_kv_heads;
    const int G = p.num_q_heads / Hkv;
    const int total_pages = s_cum[B];
    for (int x = blockIdx.x * kPartitionThreads + tid; x < total_pages;
         x += gridDim.x * kPartitionThreads) {
        // Largest b with cum[b] <= x; then cum[b + 1] > x, so n_b >= 1.
        int blo = 0, bhi = B;
        while (bhi - blo > 1) {
            const int mid = (blo + bhi) >> 1;
            if (s_cum[mid] <= x)
                blo = mid;
            else
                bhi = mid;
        }
        const int b = blo;
        const int nb = s_cum[b + 1] - s_cum[b];
        const int pg = x - s_cum[b];
        const int L = p.seq_lens[b];
        const int pid = p.block_table[(size_t)b * p.max_blocks + pg];
        const bool page_ok = (unsigned)pid < (unsigned)p.num_pages;
        const int live = min(kPageSize, L - pg * kPageSize);   // >= 1 for a valid length
        uint32_t meta = (uint32_t)(max(live, 1) - 1);
        if (pg == nb - 1)
            meta |= kMetaLast;
        if (pg == 0)
            meta |= kMetaFirst;
        if (L > max_len)
            meta |= kMetaBadLen;
        const long long base = (long long)Hkv * s_cum[b] + pg;
        for (int g = 0; g < Hkv; ++g) {
            TileEntry e;
            e.page = page_ok ? pid * Hkv + g : -1;
            e.meta = meta | ((uint32_t)(b * p.num_q_heads + g * G) << kMetaRowShift);
            p.tiles[base + (long long)g * nb] = e;
        }
    }
}

hipError_t launch_partition(const PartitionParams &p, hipStream_t stream)
{
    // Enough workgroups to give each thread about one page of the largest
    // possible batch; the prefix sum is recomputed by every workgroup.
    const long long max_pages = (long long)p.batch * p.max_blocks;
    int grid = (int)((max_pages + kPartitionThreads - 1) / kPartitionThreads);
    grid = grid < 1 ? 1 : (grid > 256 ? 256 : grid);
    const size_t lds = sizeof(int32_t) * ((size_t)p.batch + 1);
    hipLaunchKernelGGL(partition_kernel, dim3(grid), dim3(kPartitionThreads), lds, stream, p);
    return hipGetLastError();
}

}  // namespace sl
