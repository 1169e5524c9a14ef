/*
 * libsl decode engine: a multi-step generation loop on one GPU, driving the
 * KV append and decode-attention kernels of sl.h for a whole set of samples.
 *
 * What it runs (StreamRL Section 5.3, "Scheduling Order", and Section 6). An
 * instance holds more samples than its batch size BS, so generation runs in
 * rounds: the batch is BS slots, each decode step every occupied slot
 * generates one token, a sample occupies its slot for as many steps as it
 * has output tokens, and a finished sample is released at once (continuous
 * batching). Samples are admitted longest-first by their estimated output
 * length (LPT); whenever a sample finishes, the next sample in that order
 * takes the freed slot. Readings where the paper is silent: ties keep index
 * order; freed slots are refilled before the next step, lowest slot first;
 * a sample's prompt of p tokens is present in the cache when it is admitted
 * (prefill is not part of this engine; the prompt pages are filled with
 * synthetic values); while generating its k-th token (k = 1..o) the sample's
 * sequence length is p + k.
 *
 * KV pages: one pool of num_pages pages of 16 tokens, handed out from a LIFO
 * free stack that initially yields 0, 1, 2, ...; a sample takes ceil(p / 16)
 * pages on admission and one more page in each step whose new token starts a
 * page; a finished sample's pages return to the stack last block first.
 *
 * Every step, on desc.stream and in this order: new prompt pages are filled;
 * the step's new K/V rows are stored (a set of the caller's k_new / v_new
 * rows: one set every step, or the sets in turn with row_sets > 1; with the
 * quantise-on-write of sl_kv_append_fp8 for an E4M3 cache) and the step's sequence lengths and new block-table entries are
 * written into seq_lens and block_table, all read by the device from a mapped
 * pinned staging buffer; the step's attention output (sl_decode_attn or
 * _fp8) is computed into `out` with the caller's q. Slots without a sample
 * have length 0 (zero output rows). Within one sl_engine_run call the next
 * step's rows and bookkeeping are written by the launch that finishes this
 * step's attention (after, or beside, its reads of the cache), unless that
 * step admits prompts. A step whose attention fits the chip in one pass of
 * workgroups (at most one workgroup of 8 waves per CU, counting one per
 * (sequence, KV head), and no wave range much longer than a split worker's
 * share) is a single launch: its whole attention, computed in workgroups
 * that combine their own partial states, and the next step's append (kept in
 * a launch of its own when it would reuse a page freed in this step). With a
 * bf16 cache the append runs beside the attention; with an E4M3 cache, whose
 * append may re-encode a page and raise its scale, each unit's workgroup
 * appends that unit's row once the unit's reads are done. Other steps run
 * the split kernel, then the merge carrying the next step's append. Every
 * step's output is complete when its launches are.
 * When the call's work has completed on desc.stream, the buffers hold the
 * state after its last step.
 *
 * The schedule is fixed by the lengths given at creation, so the host never
 * waits for the device during a run: steps are enqueued asynchronously, and
 * the host only waits for the kernels that read a staging buffer it is about
 * to reuse.
 *
 * Memory: all buffers in sl_engine_buffers are the caller's; the engine keeps
 * their pointers until sl_engine_destroy. The engine allocates, at creation
 * only, a small ring of mapped pinned host buffers for its staging and, with
 * launch_mode 0, one device buffer (hipMalloc) for the single-launch step: 2048 partial-state slots of G * D accumulator floats
 * and G (m, l) pairs (padded to whole 128-byte lines), and 128 * Hkv
 * arrival counters (7.6 MB for G = 7, D = 128). Both are released by
 * sl_engine_destroy.
 * desc.workspace is used by the steps that run the split kernel and merge.
 */
#ifndef SL_ENGINE_H
#define SL_ENGINE_H

#include "sl.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct sl_engine sl_engine;

typedef struct sl_engine_config {
    int32_t num_samples;        /* M >= 1 */
    int32_t admission;          /* 1: longest estimated output first (LPT); 0: index order (FIFO) */
    int32_t kv_fp8;             /* 0: bf16 cache; 1: E4M3 cache with per-(page, head) scales */
    uint32_t fill_seed;         /* seed of the synthetic prompt KV values */
    float attn_scale;           /* softmax scale of the attention calls */
    const int32_t *prompt_len;  /* host [M], >= 0; read during sl_engine_create only */
    const int32_t *output_len;  /* host [M], >= 1; tokens each sample generates */
    const int32_t *est_len;     /* host [M]; admission key for LPT */
    int32_t launch_mode;        /* 0 (default): a step with little attention work runs in one launch
                                   (attention and the next step's append); 1: every step runs the split
                                   kernel and the merge. Either cache type. */
} sl_engine_config;

typedef struct sl_engine_buffers {
    /* batch = BS slots; heads, head_dim, page_size 16, max_blocks_per_seq,
       num_pages, num_workers, stream and workspace as for sl_decode_attn. */
    sl_attn_desc desc;
    const uint16_t *q;          /* bf16 [BS][Hq][D], used every step */
    const uint16_t *k_new;      /* bf16 [R][BS][Hkv][D], R = max(1, row_sets): step s appends set s % R */
    const uint16_t *v_new;
    void *k_pages;              /* bf16 or E4M3 [num_pages][Hkv][16][D] */
    void *v_pages;
    float *k_scales;            /* E4M3 only: fp32 [num_pages][Hkv] */
    float *v_scales;
    int32_t *block_table;       /* [BS][max_blocks_per_seq], written by the engine */
    int32_t *seq_lens;          /* [BS], written by the engine */
    uint16_t *out;              /* bf16 [BS][Hq][D], the latest step's attention output */
    uint16_t *out_history;      /* optional (NULL): bf16 [history_steps][BS][Hq][D]; step s's output is
                                   copied to entry s (s < history_steps), one device copy per step */
    int32_t history_steps;      /* >= 0; entries of out_history */
    int32_t row_sets;           /* >= 0; sets of new rows in k_new / v_new (0 and 1: one set, appended
                                   every step) */
} sl_engine_buffers;

/*
 * Validate and build an engine: admission order, free stack, empty slots.
 * Requires max_blocks_per_seq >= ceil((p_i + o_i) / 16) for every sample and
 * num_pages >= BS * max_blocks_per_seq (so a page is always available).
 * Errors: SL_ERR_NULL, SL_ERR_SHAPE (lengths, sizes), SL_ERR_UNSUPPORTED (as
 * sl_decode_attn), SL_ERR_WORKSPACE, SL_ERR_ALIGNMENT, SL_ERR_HIP (allocation).
 */
sl_status sl_engine_create(const sl_engine_config *config, const sl_engine_buffers *buffers,
                           sl_engine **engine);

/*
 * Enqueue up to max_steps further decode steps (fewer if every sample
 * finishes); *steps_run receives the number enqueued (0 once done).
 * Asynchronous: synchronise desc.stream before reading device buffers.
 * Errors: SL_ERR_NULL, SL_ERR_SHAPE (max_steps < 0), SL_ERR_HIP or the
 * status of a failing append / attention call (the engine then stops).
 */
sl_status sl_engine_run(sl_engine *engine, int32_t max_steps, int32_t *steps_run);

/*
 * The schedule so far (host arrays, caller-owned): per sample its slot,
 * first and last step (-1 while not admitted / not finished); *steps the
 * number of steps enqueued; active[s] (for s < min(*steps, active_cap), may
 * be NULL) the number of occupied slots in step s.
 */
sl_status sl_engine_schedule(const sl_engine *engine, int32_t *slot, int32_t *admit_step,
                             int32_t *finish_step, int32_t *steps, int32_t *active,
                             int32_t active_cap);

/* Wait for the engine's stream, then release its staging memory. NULL is a no-op.
 * (Calls on one engine must not overlap: one host thread at a time. Separate
 * engines share nothing.) */
sl_status sl_engine_destroy(sl_engine *engine);

#ifdef __cplusplus
}
#endif

#endif /* SL_ENGINE_H */
