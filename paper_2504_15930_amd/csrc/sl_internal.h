// Internal interface between the host-side entry points (api.cpp) and the
// gfx950 kernels (decode_split.hip and decode_shared.hip with the worker in
// decode_unit.h; append.hip and merge.hip with the append worker in
// append_unit.h; engine.hip), and the decode engine (engine.cpp).
//
// Work decomposition. A "unit" is one (sequence b, KV head g) pair and owns
// n_b = ceil(L_b / 16) page-head tiles (16 tokens x head_dim of one KV head).
// Units are laid out b-major, g-minor, and their tiles are numbered
// consecutively, giving W = Hkv * sum_b n_b tiles in total. Worker w (one
// wavefront) owns tiles [floor(w W / NW), floor((w + 1) W / NW)): every worker
// reads the same number of tiles (+-1) whatever the length skew, so a few very
// long sequences are spread over many workers instead of leaving most of the
// chip idle (the on-chip analogue of StreamRL's skewness bubbles, Section 2.4
// and Section 5.1).
//
// A worker streams its range as one flat sequence of tiles, which every
// workgroup derives itself: it scans the lengths (and, with prefix sharing,
// the group descriptions) into LDS, locates its workers' first tiles by
// binary search and walks the block table with a cursor. There is no
// partitioning launch and no tile list in memory. The block-table entry of a
// tile is fetched a pipeline turn ahead, so unit boundaries inside the range
// cost no dependent load and do not drain the load pipeline.
//
// (For the shared pages of prefix-shared attention a worker is a workgroup
// whose four wavefronts stream the same range, one query block each.)
//
// A unit that lies inside one worker's range is finished by that worker; a
// unit cut by a range boundary leaves one partial softmax state per worker
// that touched it, combined afterwards by the merge kernel. Worker w writes
// the piece its range starts with to slot 2w and, if its range ends inside a
// later unit, that trailing piece to slot 2w + 1.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime.h>

namespace sl {

constexpr int kPageSize = 16;
constexpr int kWave = 64;
constexpr int kWavesPerBlock = 4;          // split kernel: 4 independent workers per block
constexpr int kMaxGroup = 16;              // query heads per KV head (one MFMA column block)
constexpr int kMaxBatch = 8192;            // the split kernel keeps two ints per sequence in LDS
constexpr int kMergeThreads = 256;         // one wave per unit, four units per block
constexpr int kMaxWorkers = 1 << 16;       // keeps partial-state offsets below 2^31 bytes
#ifndef SL_MIN_TILES_PER_WORKER
#define SL_MIN_TILES_PER_WORKER 8
#endif
// A worker is given at least this many tiles: a small stream (a small batch, a
// short context) is split over fewer workers rather than cut into pieces of
// one or two tiles, each of which would cost a partial state and a merge step.
constexpr int kMinTilesPerWorker = SL_MIN_TILES_PER_WORKER;

// Workers that take part in a stream of `total` tiles (the others exit at
// once); both the split kernel and the merge derive it from the same total.
__host__ __device__ inline int effective_workers(long long total, int num_workers)
{
    const long long want = (total + kMinTilesPerWorker - 1) / kMinTilesPerWorker;
    return want < 1 ? 1 : (want < num_workers ? (int)want : num_workers);
}
// Prefix sharing: shared-page workgroups that take part in a call. The launch
// holds the own-page workgroups and up to twice `base` shared ones, and a CU
// holds two such workgroups; own-page workgroups without work exit at once,
// and a shared workgroup beyond `base` takes such an idle slot, so a batch with
// few own pages still streams its shared pages with two workgroups per CU.
// The split kernel and the merge derive it from the same totals (own tiles).
__host__ __device__ inline int effective_shared_workers(long long own_total, int own_workers, int base,
                                                        int max_workers)
{
    const int own_blocks = (own_workers + kWavesPerBlock - 1) / kWavesPerBlock;
    const int active =
        own_total > 0 ? (effective_workers(own_total, own_workers) + kWavesPerBlock - 1) / kWavesPerBlock : 0;
    const int idle = own_blocks - active;
    const int n = base + (idle < base ? idle : base);
    return n < max_workers ? n : max_workers;
}
constexpr size_t kAlign = 256;

// Tile metadata, one wave-uniform word per tile, from bit 0:
//   [3:0] live tokens in the tile minus one, [4] last tile of its unit,
//   [5] first tile of its unit, [6] the sequence length is invalid,
//   [7] see kMetaPrefixed, [31:8] first query row of the unit, b * Hq + g * G.
// A tile's KV data is page-head tile page_id * Hkv + g of the
// [num_pages][Hkv] grid (-1: the block table named a page outside the pool).
constexpr uint32_t kMetaLast = 1u << 4;
constexpr uint32_t kMetaFirst = 1u << 5;
constexpr uint32_t kMetaBadLen = 1u << 6;
constexpr uint32_t kMetaPrefixed = 1u << 7;   // own-page unit of a sequence whose first pages are shared
// Prefix-sharing mode: the shared-page stream holds, per (group, KV head),
// the group's shared pages once; their metadata keeps members - 1 in bits [3:0]
// (every shared page is full) and the first query row of the group's first
// member in [31:8]. The query rows of a shared unit are (member j, head h) ->
// row0 + j * Hq + h, at most kPrefixRows of them (kPrefixBlocks MFMA column
// blocks of 16).
constexpr int kPrefixBlocks = 4;
constexpr int kPrefixRows = 16 * kPrefixBlocks;
constexpr int kMetaRowShift = 8;

struct Workspace {
    int32_t *cum_pages;   // [B + 1] exclusive prefix sum of pages per sequence (written by the split kernel)
    float *part_ml;       // [2 NW][G][2]  (running max in log2 units, sum of weights)
    float *part_acc;      // [2 NW][G][D]  un-normalised weighted value sums
};

struct SplitParams {
    const uint16_t *q;
    const void *k_pages;
    const void *v_pages;
    const float *k_scales;
    const float *v_scales;
    uint16_t *out;
    float *part_ml;
    float *part_acc;
    int32_t batch, num_kv_heads, group, num_workers;
    int32_t num_q_heads;   // query-row stride of one sequence (prefix mode)
    float scale_log2;      // scale * log2(e): scores are kept in base-2 units
    // Prefix mode: a unit seen whole by one worker that still has to be merged
    // (a shared unit, or the own pages of a sequence with shared pages) keeps
    // its partial state here, at unit index (first query row) / G, with the
    // row stride of part_ml / part_acc; null otherwise.
    float *unit_ml;
    float *unit_acc;
    // The kernel derives every tile from the lengths and the block table
    // itself; workgroup 0 stores the page prefix sum in cum_out for the merge
    // (plain attention; prefix sharing stores its sums through PrefixParams).
    const int32_t *seq_lens;
    const int32_t *block_table;
    int32_t *cum_out;
    int32_t max_blocks, num_pages;
};

// Prefix-sharing mode. Groups are runs of consecutive sequences
// [group_start[k], group_start[k+1]) whose first shared_pages[k] block-table
// entries are the same; the group's first member's entries are used. Every
// workgroup of the fused split kernel derives both page streams from these;
// workgroup 0 stores the sums below for the merge.
struct PrefixParams {
    const int32_t *group_start;   // [num_groups + 1]
    const int32_t *shared_pages;  // [num_groups]
    int32_t *cum_own;             // [B + 1] prefix sum of own (unshared) pages
    int32_t *cum_shared;          // [max_sub + 1] prefix sum of shared pages per sub-group
    int32_t *seq_shared;          // [B][4] per sequence: first shared page of its sub-group in the shared
                                  // stream, shared pages, sub-group's first member, sub-group (-1, zeros if
                                  // unshared)
    int32_t num_groups;
    int32_t max_sub;              // prefix_max_sub: bound on the sub-groups (shared-stream "sequences")
};

// Members of one shared unit: as many samples as fit kPrefixRows query rows,
// at most 16 (the tile metadata keeps members - 1 in four bits).
__host__ __device__ inline int prefix_max_members(int group) { return 16 < kPrefixRows / group ? 16 : kPrefixRows / group; }
// Bound on the sub-groups of a call: shared groups are disjoint ranges of the
// batch and a group of m members is cut into ceil(m / M) sub-groups, so there
// are at most num_groups + batch / M of them, and never more than batch.
__host__ __device__ inline int prefix_max_sub(int batch, int num_groups, int group)
{
    if (num_groups <= 0)
        return 0;
    const int bound = num_groups + batch / prefix_max_members(group);
    return bound < batch ? bound : batch;
}

struct PrefixMergeParams {
    const int32_t *seq_lens;
    const int32_t *group_start;
    const int32_t *shared_pages;
    const int32_t *cum_own;
    const int32_t *cum_shared;
    const int32_t *seq_shared;   // [B][4], as written by the split kernel
    const float *own_ml, *own_acc;        // [2 NW][G][2], [2 NW][G][D]
    const float *shared_ml, *shared_acc;  // [2 NW][kPrefixRows][2], [2 NW][kPrefixRows][D]
    const float *own_unit_ml, *own_unit_acc;        // [B Hkv][G][2 | D]: whole own units
    const float *shared_unit_ml, *shared_unit_acc;  // [B Hkv][kPrefixRows][2 | D]: whole shared units
    uint16_t *out;
    int32_t batch, max_sub, num_q_heads, num_kv_heads, group, num_workers, max_blocks;
    int32_t num_shared_workers;   // base and largest count of shared-page workgroups
    int32_t max_shared_workers;   // (effective_shared_workers)
};

struct AppendParams {
    const uint16_t *k_new;      // [B][Hkv][D] bf16 rows of the step's new token
    const uint16_t *v_new;
    const int32_t *block_table;
    const int32_t *seq_lens;    // already counting the new token
    void *k_pages;              // bf16 or E4M3 pool [num_pages][Hkv][16][D]
    void *v_pages;
    float *k_scales;            // E4M3 only: [num_pages][Hkv]
    float *v_scales;
    int32_t batch, num_kv_heads, max_blocks, num_pages;
    // Decode-engine mode (null otherwise): the step's lengths and the page of
    // every sequence's new token are read from a staging buffer laid out as
    // [lengths: B][token pages: B][block-table updates: n_upd x (slot, block,
    // page)], and the same launch also stores the lengths in set_seq_lens and
    // applies the updates to set_block_table for the attention that follows
    // (seq_lens and block_table are not read).
    const int32_t *stage;
    int32_t n_upd;
    int32_t *set_seq_lens;
    int32_t *set_block_table;
};

struct MergeParams {
    const int32_t *seq_lens;
    const int32_t *cum_pages;
    const float *part_ml;
    const float *part_acc;
    uint16_t *out;
    int32_t batch, num_q_heads, num_kv_heads, group, num_workers;
    // Decode engine: the next step's staged append (and its bookkeeping) runs
    // in the same launch, in workgroups after the merge's; 0 none, 1 bf16
    // cache, 2 E4M3 cache. The merge never reads what it writes: it reads the
    // lengths only for sequences without pages, whose rows are zero whatever
    // the step (the engine's lengths are never negative).
    AppendParams next;
    int32_t next_kind;
};


constexpr int kMaxPrefixBatch = 4096;      // the fused prefix kernel keeps three ints per sequence in LDS

struct PrefixWorkspace {
    int32_t *cum_own, *seq_shared, *cum_shared;
    float *own_ml, *own_acc, *shared_ml, *shared_acc;
    float *own_unit_ml, *own_unit_acc, *shared_unit_ml, *shared_unit_acc;
};
size_t prefix_workspace_layout(void *base, int batch, int max_blocks, int num_kv_heads, int group, int head_dim,
                               int num_workers, int num_groups, PrefixWorkspace *ws);

// Layout of the workspace for the given sizes; `base` may be null to size it.
size_t workspace_layout(void *base, int batch, int max_blocks, int num_kv_heads, int group,
                        int head_dim, int num_workers, Workspace *ws);

// The split kernel's dynamic LDS: the page prefix sum (B + 1 ints) and the
// lengths (B ints).
inline size_t split_dynamic_lds(int batch) { return sizeof(int32_t) * (2 * (size_t)batch + 1); }
// The fused prefix kernel's: for the sequences the own-page prefix sum, the
// sub-groups and the lengths (3 B + 2 ints), for the sub-groups the
// shared-page prefix sum and the packed first member and size (2 S + 1 ints),
// and the groups' starts and page counts (2 NG + 1 ints).
inline size_t prefix_dynamic_lds(int batch, int max_sub, int num_groups)
{
    return sizeof(int32_t) * (3 * (size_t)batch + 2 * (size_t)max_sub + 2 * (size_t)num_groups + 4);
}
hipError_t launch_split(const SplitParams &p, int head_dim, bool fp8, hipStream_t stream);
// Prefix mode: the own-page pass (single-unit workers) and the shared-page
// pass (one workgroup of kPrefixBlocks wavefronts per worker, one 16-row
// column block each, partial states only) in one launch, followed by the
// merge. shared.num_workers is the base count of shared workgroups and
// max_shared the largest (effective_shared_workers).
hipError_t launch_prefix_split(const SplitParams &own, const SplitParams &shared, int max_shared,
                               const PrefixParams &pp, int head_dim, bool fp8, hipStream_t stream);
hipError_t launch_merge_prefix(const PrefixMergeParams &p, int head_dim, hipStream_t stream);
hipError_t launch_merge(const MergeParams &p, int head_dim, hipStream_t stream);
hipError_t launch_append(const AppendParams &p, int head_dim, bool fp8, hipStream_t stream);
// Decode engine helper (engine.hip): fill prompt pages with synthetic data.
hipError_t launch_engine_fill(const int32_t *pages, int n_pages, int hkv, int head_dim, bool fp8, uint32_t seed,
                              void *k_pages, void *v_pages, float *k_scales, float *v_scales, hipStream_t stream);
// Resident split-kernel workgroups per CU (occupancy query), for the default worker count.
hipError_t split_blocks_per_cu(int head_dim, bool fp8, int *blocks);

}  // namespace sl
