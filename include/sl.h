/*
 * libsl: batched GQA decode attention over a paged KV cache, for AMD
 * Instinct MI355X (gfx950).
 *
 * One call performs the attention part of one decode step of a batch of
 * in-flight samples, each attending over its own growing context (StreamRL,
 * Section 2.1: in the decoding phase every sample computes only its newest
 * token and reuses the key-value cache of all earlier tokens; Section 2.4: the
 * decode batch holds hundreds of samples whose output lengths are
 * long-tailed; Section 6: continuous batching releases finished samples
 * early, so lengths in one batch are ragged, and prefix sharing lets samples
 * reference the same cache pages). The cache is paged as in PagedAttention
 * (cited in Section 8): page `block_table[b][i]` of the pool holds tokens
 * [i * page_size, (i + 1) * page_size) of sequence b.
 *
 * For every sequence b and query head h (G = num_q_heads / num_kv_heads,
 * KV head g = h / G, L = seq_lens[b]):
 *
 *   out[b][h][:] = sum_t softmax_t(scale * q[b][h] . K_t) * V_t,  t < L
 *
 * and out[b][h][:] = 0 when L == 0. Arithmetic: bf16 inputs, fp32 scores and
 * accumulators (softmax probabilities enter the value product rounded to
 * bf16), bf16 output rounded to nearest even.
 *
 * Conventions shared by every entry point:
 *  - All array pointers are device memory of the current HIP device, owned by
 *    the caller; the library keeps no pointer after the call returns and
 *    allocates nothing.
 *  - Calls are asynchronous: work is enqueued on desc->stream and the call
 *    returns; the caller synchronises. No host<->device copy and no host
 *    synchronisation happen inside a call.
 *  - Errors are reported by the returned sl_status; nothing throws across the
 *    ABI. Argument checks happen before any work is enqueued, so an error
 *    status means nothing was enqueued (SL_ERR_HIP excepted: a launch may
 *    have failed part-way).
 *  - Device-side data errors cannot be reported by status (the host never
 *    reads seq_lens or block_table). They never cause an out-of-bounds
 *    access: a sequence with seq_lens[b] < 0 or > max_blocks_per_seq *
 *    page_size, or whose live block-table entries name a page outside
 *    [0, num_pages), gets NaN in all its output rows.
 *  - Calls sharing one workspace must not overlap in time (e.g. run them on
 *    one stream).
 */
#ifndef SL_H
#define SL_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum sl_status {
    SL_OK = 0,
    SL_ERR_NULL = -1,        /* a required pointer is NULL */
    SL_ERR_SHAPE = -2,       /* a size is negative, zero where it must not be, or inconsistent */
    SL_ERR_UNSUPPORTED = -3, /* valid but not implemented: head_dim, page_size, group size, batch */
    SL_ERR_WORKSPACE = -4,   /* workspace NULL, too small or not 256-byte aligned */
    SL_ERR_HIP = -5,         /* a HIP runtime call or kernel launch failed */
    SL_ERR_ALIGNMENT = -6,   /* q, out or a page pool not 16-byte aligned; block_table,
                                seq_lens or a scale array not 4-byte aligned */
    SL_ERR_SCRATCH_LIMIT = -7 /* sl_decode_attn_noalloc: the call needs more scratch than
                                 SL_NOALLOC_SCRATCH_BYTES (use fewer workers) */
} sl_status;

/*
 * Sizes of one decode step. Layouts (row-major, innermost last):
 *   q, out          [batch][num_q_heads][head_dim]                 bf16
 *   k_pages,v_pages [num_pages][num_kv_heads][page_size][head_dim] bf16 or e4m3
 *   k_scales,...    [num_pages][num_kv_heads]                      fp32 (fp8 only)
 *   block_table     [batch][max_blocks_per_seq]                    int32
 *   seq_lens        [batch]                                        int32
 * Supported: head_dim 64 or 128; page_size 16; 1 <= num_q_heads /
 * num_kv_heads <= 16; batch <= 8192; batch * max_blocks_per_seq *
 * num_kv_heads < 2^31.
 */
typedef struct sl_attn_desc {
    int32_t batch;              /* sequences in the step; 0 makes every call a no-op */
    int32_t num_q_heads;        /* Hq */
    int32_t num_kv_heads;       /* Hkv; divides Hq; query head h reads KV head h / (Hq / Hkv) */
    int32_t head_dim;           /* D */
    int32_t page_size;          /* tokens per page */
    int32_t max_blocks_per_seq; /* row length of block_table */
    int32_t num_pages;          /* pages in each pool; valid page ids are [0, num_pages) */
    int32_t num_workers;        /* split-KV workers (wavefronts). 0: library default
                                   (three per CU for bf16, four per CU for FP8 and for
                                   prefix-shared attention); 1..65536: exactly this
                                   many. The result does not depend on it beyond fp32
                                   rounding; tests vary it to exercise the merge. */
    hipStream_t stream;         /* stream the work is enqueued on (0: null stream) */
    void *workspace;            /* device scratch, >= sl_decode_attn_workspace_size bytes,
                                   256-byte aligned; contents need no initialisation */
    size_t workspace_bytes;
    hipEvent_t timing_start;    /* optional (may be NULL): recorded on `stream` right */
    hipEvent_t timing_stop;     /* before and after the split-KV kernel, for profiling */
} sl_attn_desc;

/*
 * Bytes of workspace the calls need for `desc` (sizes and num_workers; no
 * pointer is read). With num_workers == 0 this queries the current device.
 * Errors: SL_ERR_NULL, SL_ERR_SHAPE, SL_ERR_UNSUPPORTED, SL_ERR_HIP.
 */
sl_status sl_decode_attn_workspace_size(const sl_attn_desc *desc, size_t *bytes);

/*
 * Number of workers (wavefronts of the split-KV kernel) a call with `desc`
 * would use: desc->num_workers when positive, else the device default for the
 * bf16 (kv_fp8 == 0) or FP8 (kv_fp8 != 0) kernel. Errors as
 * sl_decode_attn_workspace_size.
 */
sl_status sl_decode_attn_num_workers(const sl_attn_desc *desc, int32_t kv_fp8,
                                     int32_t *num_workers);

/*
 * Decode attention with a bf16 KV cache (formula above).
 *   q            bf16 bits [batch][Hq][D]
 *   k_pages      bf16 bits [num_pages][Hkv][page_size][D]
 *   v_pages      bf16 bits, same shape
 *   block_table  [batch][max_blocks_per_seq]; only the first
 *                ceil(seq_lens[b] / page_size) entries of row b are read;
 *                rows may name the same pages (prefix sharing)
 *   seq_lens     [batch] cached tokens per sequence, the newest included
 *   scale        multiplies q . k (usually 1 / sqrt(D))
 *   out          bf16 bits [batch][Hq][D], written entirely
 * Slots of a page past a sequence's end may hold anything (NaN included).
 * Errors: SL_ERR_NULL, SL_ERR_SHAPE, SL_ERR_UNSUPPORTED, SL_ERR_WORKSPACE,
 * SL_ERR_ALIGNMENT, SL_ERR_HIP.
 */
sl_status sl_decode_attn(const sl_attn_desc *desc, const uint16_t *q,
                         const uint16_t *k_pages, const uint16_t *v_pages,
                         const int32_t *block_table, const int32_t *seq_lens,
                         float scale, uint16_t *out);

/*
 * Decode attention with an FP8 KV cache: pages hold OCP FP8 E4M3 codes
 * (exponent bias 7, largest finite 448, 0x7F / 0xFF are NaN) and the cached
 * value of element d of token t in (page, KV head g) is
 * e4m3(code) * k_scales[page][g] for keys and * v_scales[page][g] for values.
 * Everything else is as sl_decode_attn. Errors: as sl_decode_attn.
 */
sl_status sl_decode_attn_fp8(const sl_attn_desc *desc, const uint16_t *q,
                             const uint8_t *k_pages, const uint8_t *v_pages,
                             const float *k_scales, const float *v_scales,
                             const int32_t *block_table, const int32_t *seq_lens,
                             float scale, uint16_t *out);

/*
 * Decode attention with prefix sharing (bf16 cache): the same result as
 * sl_decode_attn, reading each page that several sequences share only once
 * per sub-group of at most min(16, 64 / (Hq / Hkv)) samples.
 * StreamRL's engine shares key-value cache between samples of one prompt
 * (Section 6, prefix sharing); here the samples of a group are run together
 * over the group's shared pages.
 *
 * Groups are runs of consecutive sequences: group k is sequences
 * [group_start[k], group_start[k+1]), and their first shared_pages[k] pages
 * are the same, i.e. block_table[b][i] == block_table[group_start[k]][i] for
 * i < shared_pages[k] and every member b (only the first member's entries of
 * each sub-group are read), and seq_lens[b] >= 16 * shared_pages[k].
 * Sequences in no group, or in a group with shared_pages 0, are attended as
 * by sl_decode_attn.
 *   group_start   device int32 [num_groups + 1], ascending, within [0, batch]
 *   shared_pages  device int32 [num_groups]
 *   num_groups    0 .. batch (0: plain attention, in two passes)
 * A group of m members with M = min(16, 64 / (Hq / Hkv)) is read as
 * ceil(m / M) consecutive sub-groups of ceil(m / ceil(m / M)) members (the
 * last may be smaller), each of which reads the shared pages once. A group
 * that is empty, lies outside [0, batch], starts before the end of an earlier
 * group's range (group_start not ascending), or whose page count lies outside
 * 1 .. max_blocks_per_seq is treated as unshared (exact, without the saving).
 * A member shorter than its group's shared pages gets NaN rows.
 * Everything else is as sl_decode_attn; batch is at most 4096, and the
 * workspace is sized by sl_decode_attn_prefix_workspace_size.
 * Errors: as sl_decode_attn (SL_ERR_SHAPE also for num_groups outside
 * [0, batch]; SL_ERR_UNSUPPORTED for batch > 4096).
 */
sl_status sl_decode_attn_prefix(const sl_attn_desc *desc, const uint16_t *q,
                                const uint16_t *k_pages, const uint16_t *v_pages,
                                const int32_t *block_table, const int32_t *seq_lens,
                                const int32_t *group_start, const int32_t *shared_pages,
                                int32_t num_groups, float scale, uint16_t *out);

/*
 * Prefix sharing over an FP8 E4M3 cache: the pages, codes and per-(page, KV
 * head) scales of sl_decode_attn_fp8, the groups of sl_decode_attn_prefix,
 * and the same result as sl_decode_attn_fp8 on the same arguments (a shared
 * page's scales are read once, from its own entry). k_scales and v_scales
 * are device float [num_pages][Hkv], 4-byte aligned. Everything else, the
 * workspace and the errors are as sl_decode_attn_prefix.
 */
sl_status sl_decode_attn_prefix_fp8(const sl_attn_desc *desc, const uint16_t *q,
                                    const uint8_t *k_pages, const uint8_t *v_pages,
                                    const float *k_scales, const float *v_scales,
                                    const int32_t *block_table, const int32_t *seq_lens,
                                    const int32_t *group_start, const int32_t *shared_pages,
                                    int32_t num_groups, float scale, uint16_t *out);

/* Workspace bytes sl_decode_attn_prefix and sl_decode_attn_prefix_fp8 need
 * for desc and num_groups (one size serves both). */
sl_status sl_decode_attn_prefix_workspace_size(const sl_attn_desc *desc, int32_t num_groups,
                                               size_t *bytes);

/*
 * KV append: stores one decode step's new key and value rows in the paged
 * cache, the step that precedes attention in every decode step (StreamRL,
 * Section 2.1: each decoding step computes the newest token and keeps its
 * per-token state in the key-value cache that later steps reuse).
 *
 * seq_lens already counts the new token (the same array the step's attention
 * call takes): for every sequence b with L = seq_lens[b] >= 1 the row of the
 * token t = L - 1 goes to page block_table[b][t / page_size], slot
 * t % page_size, for every KV head g. L == 0 appends nothing.
 *   k_new, v_new  bf16 bits [batch][Hkv][D], read only
 *   block_table   [batch][max_blocks_per_seq]; only entry (L - 1) / page_size
 *                 of row b is read
 *   seq_lens      [batch]
 *   k_pages, v_pages  the cache, written only in the new tokens' slots
 * The page receiving a sequence's new token must not be the receiving page of
 * another sequence in the same call (copy a shared last page first);
 * otherwise the result for those sequences is unspecified (no fault).
 * A sequence with seq_lens[b] < 0 or > max_blocks_per_seq * page_size, or
 * whose receiving page id lies outside [0, num_pages), is left untouched.
 * Uses desc fields batch, num_kv_heads, head_dim, page_size,
 * max_blocks_per_seq, num_pages, stream, timing_start/timing_stop (optional
 * events recorded around the kernel); num_q_heads must be valid as for
 * attention; the workspace is not used.
 * Errors: SL_ERR_NULL, SL_ERR_SHAPE, SL_ERR_UNSUPPORTED, SL_ERR_ALIGNMENT
 * (k_new, v_new, block_table, seq_lens need 4-byte, pages 16-byte alignment),
 * SL_ERR_HIP.
 */
sl_status sl_kv_append(const sl_attn_desc *desc, const uint16_t *k_new, const uint16_t *v_new,
                       const int32_t *block_table, const int32_t *seq_lens,
                       uint16_t *k_pages, uint16_t *v_pages);

/*
 * KV append into an FP8 (E4M3) cache with one fp32 scale per (page, KV head)
 * for keys and another for values, quantising on write. The scale of a
 * page-head tile only grows; with a = max_d |x_d| of the new row (NaN
 * elements ignored):
 *   slot 0 (the row opens the page):  scale = a / 448, or 1 if a == 0
 *   a <= scale * 448:                 scale unchanged
 *   a >  scale * 448:                 scale' = a / 448, and every earlier slot
 *                                     j of the tile is re-encoded as
 *                                     enc(e4m3(code) * scale / scale')
 * and the new row is stored as enc(x_d / scale). enc rounds to nearest with
 * ties to even, saturates to +-448 and maps NaN to 0x7F. All of this is
 * binary32 arithmetic in the order written, so codes and scales are exact and
 * reproducible. Keys and values are handled separately. The paper does not
 * describe FP8 storage; this rule keeps every live slot of a tile encoded
 * with the tile's current scale, which is what sl_decode_attn_fp8 reads.
 *   k_pages, v_pages    E4M3 codes [num_pages][Hkv][page_size][D]
 *   k_scales, v_scales  fp32 [num_pages][Hkv], read and written
 * Everything else is as sl_kv_append (scales need 4-byte alignment).
 */
sl_status sl_kv_append_fp8(const sl_attn_desc *desc, const uint16_t *k_new, const uint16_t *v_new,
                           const int32_t *block_table, const int32_t *seq_lens,
                           uint8_t *k_pages, uint8_t *v_pages, float *k_scales,
                           float *v_scales);

/*
 * Decode attention with a bf16 cache that allocates nothing, for callers that
 * cannot allocate device memory: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc. Same arguments, kernels and result
 * as sl_decode_attn (bit for bit, for the same worker count), except that
 * desc->workspace and desc->workspace_bytes are ignored: the scratch lives in
 * a fixed array of SL_NOALLOC_SCRATCH_BYTES inside the library, one per GPU,
 * held until the process ends. The call makes no hipMalloc, hipFree or other
 * allocating call. Calls on one GPU share that array: calls that overlap in
 * time on one GPU (two streams, two threads) race and give undefined results;
 * serialise them, e.g. on one stream. A call whose scratch (as
 * sl_decode_attn_workspace_size would count it for its worker count) exceeds
 * the array returns SL_ERR_SCRATCH_LIMIT before enqueuing anything; with the
 * default worker count every supported shape fits.
 * Errors: as sl_decode_attn, SL_ERR_WORKSPACE excepted, plus
 * SL_ERR_SCRATCH_LIMIT.
 */
#define SL_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)
sl_status sl_decode_attn_noalloc(const sl_attn_desc *desc, const uint16_t *q,
                                 const uint16_t *k_pages, const uint16_t *v_pages,
                                 const int32_t *block_table, const int32_t *seq_lens,
                                 float scale, uint16_t *out);

/* Static English description of a status code (never NULL). Takes any
 * integer: a value that is no sl_status gives "unknown status". */
const char *sl_status_string(int32_t status);

#ifdef __cplusplus
}
#endif

#endif /* SL_H */
