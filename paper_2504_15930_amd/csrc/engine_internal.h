#ifndef SL_ENGINE_INTERNAL_H
#define SL_ENGINE_INTERNAL_H
// Device-side interface of the decode engine's one-launch step, shared by
// engine.cpp (the host plan) and engine.hip (the kernel).
#include "sl_internal.h"

namespace sl {

// Decode engine, one-launch step (engine.hip): a step's whole attention and
// the next step's staged append. The host lists the step's sequences with
// their lengths and how many workgroups of kUnitWaves waves each of its
// units (sequence, KV head) gets; a unit's waves split its tiles evenly. A
// workgroup combines its waves' states in LDS; with one workgroup per unit it
// writes the rows, else it stores its state in its piece slot (workgroup
// index) and the last of the unit's workgroups to arrive merges the pieces.
// With an E4M3 cache the next step's append of a unit's row may re-encode the
// page the unit reads, so that workgroup (the single one, or the last to
// arrive) appends it once the unit's reads are done (units_append).
constexpr int kUnitWaves = 8;
constexpr int kMaxUnitEntries = 128;   // sequences per launch (kernel arguments)
constexpr int kMaxUnitBlocks = 2048;   // attention workgroups per launch (piece slots)
constexpr int kMaxUnitSplit = 32;      // workgroups per unit
// Floats per piece slot of (m, l) pairs: G pairs on whole 128-byte lines, so
// no two slots share a cache line.
__host__ __device__ inline int unit_ml_stride(int group) { return (2 * group + 31) / 32 * 32; }

struct UnitStepParams {
    // q, k/v pages (and their scales for E4M3), out, group, num_kv_heads,
    // num_q_heads, scale_log2, block_table, max_blocks, num_pages; part_ml /
    // part_acc are the piece slots (kMaxUnitBlocks of unit_ml_stride(G)
    // floats, and of G * D floats). seq_lens is not read.
    SplitParams cur;
    AppendParams next;            // the next step's staged append (next_blocks > 0)
    int32_t *counters;            // [kMaxUnitEntries * Hkv] arrivals per unit; zero between launches
    int32_t n_entries, unit_blocks, zero_blocks, next_blocks;
    // 1: each unit's workgroup appends that unit's next-step row (every slot
    // the next step appends to is one of this step's entries, whose next
    // length is len + 1 and whose new token goes to next_page) and the
    // next_blocks workgroups apply only the staged bookkeeping.
    int32_t units_append;
    int32_t seq[kMaxUnitEntries];        // slot of entry e (length >= 1)
    int32_t len[kMaxUnitEntries];        // its length
    int32_t next_page[kMaxUnitEntries];  // units_append: page of its next token (-1: it finished)
    int32_t first[kMaxUnitEntries + 1];  // its first workgroup; Hkv * K_e workgroups, head-major
    int32_t zero[kMaxUnitEntries];       // slots whose output rows are cleared (zero_blocks of them)
};
hipError_t launch_unit_step(const UnitStepParams &up, int head_dim, bool fp8, hipStream_t stream);

}  // namespace sl

#endif  // SL_ENGINE_INTERNAL_H
