// CU-level work partitioner: turns device-resident sequence lengths into the
// tile ranges of the split-KV workers without any host synchronisation.
//
// One workgroup of 1024 threads:
//   1. pages per sequence, n_b = ceil(clamp(L_b, 0, max_blocks * 16) / 16),
//      and their exclusive prefix sum (kept in LDS, copied to cum_pages);
//   2. for each worker w, the unit (b, g) holding tile floor(w W / NW),
//      found by binary search over the prefix sum.
// Cost: O(B + NW log B) integer work, a few microseconds.
#include "sl_internal.h"

namespace sl {

__global__ __launch_bounds__(kPartitionThreads) void partition_kernel(PartitionParams p)
{
    __shared__ int32_t s_cum[kMaxBatch + 1];
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

    for (int i = tid; i <= B; i += kPartitionThreads)
        p.cum_pages[i] = s_cum[i];

    const int Hkv = p.num_kv_heads;
    const long long total = (long long)s_cum[B] * Hkv;
    const int NW = p.num_workers;
    for (int w = tid; w < NW; w += kPartitionThreads) {
        const long long s = (long long)w * total / NW;
        const long long e = (long long)(w + 1) * total / NW;
        if (s >= e) {
            p.worker_unit[w] = -1;
            continue;
        }
        // Largest b with Hkv * cum[b] <= s; then cum[b + 1] > s / Hkv, so n_b >= 1.
        int blo = 0, bhi = B;
        while (bhi - blo > 1) {
            const int mid = (blo + bhi) >> 1;
            if ((long long)Hkv * s_cum[mid] <= s)
                blo = mid;
            else
                bhi = mid;
        }
        const long long nb = s_cum[blo + 1] - s_cum[blo];
        const int g = (int)((s - (long long)Hkv * s_cum[blo]) / nb);
        p.worker_unit[w] = blo * Hkv + g;
    }
}

hipError_t launch_partition(const PartitionParams &p, hipStream_t stream)
{
    hipLaunchKernelGGL(partition_kernel, dim3(1), dim3(kPartitionThreads), 0, stream, p);
    return hipGetLastError();
}

}  // namespace sl
