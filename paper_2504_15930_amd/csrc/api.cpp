// Host side of libsl: argument checks, workspace layout, launch geometry and
// the launches of one decode-attention call (split-KV, which partitions the
// work itself -> merge; prefix sharing: fused own- and shared-page split ->
// merge), all enqueued on the caller's stream with no host synchronisation.
#include <mutex>

#include "../../include/sl.h"
#include "api_internal.h"
#include "sl_internal.h"

namespace sl {

static size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

size_t workspace_layout(void *base, int batch, int max_blocks, int num_kv_heads, int group,
                        int head_dim, int num_workers, Workspace *ws)
{
    char *p = static_cast<char *>(base);
    size_t off = 0;
    auto take = [&](size_t bytes) {
        char *r = p ? p + off : nullptr;
        off += align_up(bytes);
        return r;
    };
    Workspace w;
    w.cum_pages = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * ((size_t)batch + 1)));
    w.part_ml = reinterpret_cast<float *>(take(sizeof(float) * 2 * (size_t)num_workers * group * 2));
    w.part_acc = reinterpret_cast<float *>(
        take(sizeof(float) * 2 * (size_t)num_workers * group * head_dim));
    if (ws)
        *ws = w;
    return off;
}

size_t prefix_workspace_layout(void *base, int batch, int max_blocks, int num_kv_heads, int group,
                               int head_dim, int num_workers, int num_groups, PrefixWorkspace *ws)
{
    char *p = static_cast<char *>(base);
    size_t off = 0;
    auto take = [&](size_t bytes) {
        char *r = p ? p + off : nullptr;
        off += align_up(bytes);
        return r;
    };
    PrefixWorkspace w;
    w.cum_own = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * ((size_t)batch + 1)));
    w.seq_shared = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * 4 * (size_t)batch));
    w.cum_shared = reinterpret_cast<int32_t *>(
        take(sizeof(int32_t) * ((size_t)prefix_max_sub(batch, num_groups, group) + 1)));
    w.own_ml = reinterpret_cast<float *>(take(sizeof(float) * 2 * (size_t)num_workers * group * 2));
    w.own_acc = reinterpret_cast<float *>(take(sizeof(float) * 2 * (size_t)num_workers * group * head_dim));
    w.shared_ml = reinterpret_cast<float *>(take(sizeof(float) * 2 * (size_t)num_workers * kPrefixRows * 2));
    w.shared_acc = reinterpret_cast<float *>(take(sizeof(float) * 2 * (size_t)num_workers * kPrefixRows * head_dim));
    const size_t units = (size_t)batch * num_kv_heads;
    w.own_unit_ml = reinterpret_cast<float *>(take(sizeof(float) * units * group * 2));
    w.own_unit_acc = reinterpret_cast<float *>(take(sizeof(float) * units * group * head_dim));
    w.shared_unit_ml = reinterpret_cast<float *>(take(sizeof(float) * units * kPrefixRows * 2));
    w.shared_unit_acc = reinterpret_cast<float *>(take(sizeof(float) * units * kPrefixRows * head_dim));
    if (ws)
        *ws = w;
    return off;
}

namespace {

constexpr int kMaxDevices = 64;

struct DeviceInfo {
    std::once_flag once;
    hipError_t err = hipSuccess;
    int cus = 0;
    int blocks[2][2] = {{0, 0}, {0, 0}};   // [head_dim == 128][fp8]
};
DeviceInfo g_devices[kMaxDevices];

hipError_t device_info(DeviceInfo **out)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return e;
    if (dev < 0 || dev >= kMaxDevices)
        return hipErrorInvalidDevice;
    DeviceInfo &d = g_devices[dev];
    std::call_once(d.once, [&d, dev] {
        d.err = hipDeviceGetAttribute(&d.cus, hipDeviceAttributeMultiprocessorCount, dev);
        for (int hd = 0; hd < 2 && d.err == hipSuccess; ++hd)
            for (int f = 0; f < 2 && d.err == hipSuccess; ++f)
                d.err = split_blocks_per_cu(hd ? 128 : 64, f != 0, &d.blocks[hd][f]);
    });
    *out = &d;
    return d.err;
}

sl_status check_desc(const sl_attn_desc *d)
{
    if (!d)
        return SL_ERR_NULL;
    if (d->batch < 0 || d->num_q_heads <= 0 || d->num_kv_heads <= 0 || d->head_dim <= 0 ||
        d->page_size <= 0 || d->max_blocks_per_seq <= 0 || d->num_pages <= 0 ||
        d->num_workers < 0)
        return SL_ERR_SHAPE;
    if (d->num_q_heads % d->num_kv_heads != 0)
        return SL_ERR_SHAPE;
    if (d->num_q_heads / d->num_kv_heads > kMaxGroup)
        return SL_ERR_UNSUPPORTED;
    if (d->head_dim != 64 && d->head_dim != 128)
        return SL_ERR_UNSUPPORTED;
    if (d->page_size != kPageSize)
        return SL_ERR_UNSUPPORTED;
    if (d->batch > kMaxBatch)
        return SL_ERR_UNSUPPORTED;
    // Tile-list entries: at most 2^28 tiles (8-byte entries addressed with
    // 32-bit byte offsets), page-head tile indices and query-row numbers that
    // fit their fields.
    if ((long long)d->batch * d->max_blocks_per_seq * d->num_kv_heads >= (1LL << 28) ||
        (long long)d->max_blocks_per_seq * kPageSize >= (1LL << 31) ||
        (long long)d->num_pages * d->num_kv_heads >= (1LL << 31) ||
        (long long)d->batch * d->num_q_heads >= (1LL << (32 - kMetaRowShift)))
        return SL_ERR_UNSUPPORTED;
    if (d->num_workers > kMaxWorkers)
        return SL_ERR_UNSUPPORTED;
    return SL_OK;
}

sl_status resolve_workers(const sl_attn_desc *d, bool fp8, int *nw, bool prefix = false)
{
    if (d->num_workers > 0) {
        *nw = d->num_workers;
        return SL_OK;
    }
    DeviceInfo *info = nullptr;
    if (device_info(&info) != hipSuccess)
        return SL_ERR_HIP;
    // Split-KV workgroups of four workers (one per SIMD), measured on
    // MI355X: the E4M3 cache streams best with one per CU; the bf16 cache,
    // whose tiles carry twice the bytes, already saturates HBM with three
    // workgroups per four CUs (1.5-2.5% faster than one per CU, as fewer
    // streams compete for the memory; 640 or fewer workers, or 1280 and more,
    // were slower). Two waves per SIMD were slower for both. Prefix-shared
    // attention keeps one own-page workgroup per CU beside its shared-page
    // workgroups (three per four CUs was 12% slower).
    const int blocks = info->blocks[d->head_dim == 128][fp8 ? 1 : 0];
    const int per_cu4 = fp8 || prefix ? 4 : 3;   // workgroups per four CUs
    *nw = (blocks > 0 ? info->cus * per_cu4 / 4 : info->cus) * kWavesPerBlock;
    if (*nw > kMaxWorkers)
        *nw = kMaxWorkers;
    return SL_OK;
}

// Workgroups of the shared-page pass. They run in the same launch as the
// own-page workers (four per workgroup, nw / 4 workgroups): one shared-page
// workgroup per own-page workgroup puts one of each on every CU by default,
// the best ratio measured on MI355X (an eighth or three eighths of nw were
// both about 12% slower). Never more than nw, for which the partial-state
// slots are sized.
int shared_workers(int nw) { return nw / 4 > 0 ? nw / 4 : 1; }

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

sl_status run(const sl_attn_desc *d, const uint16_t *q, const void *k_pages, const void *v_pages,
              const float *k_scales, const float *v_scales, const int32_t *block_table,
              const int32_t *seq_lens, float scale, uint16_t *out, bool fp8, const AppendParams *next = nullptr)
{
    sl_status st = check_desc(d);
    if (st != SL_OK)
        return st;
    if (d->batch == 0)
        return SL_OK;
    if (!q || !k_pages || !v_pages || !block_table || !seq_lens || !out)
        return SL_ERR_NULL;
    if (fp8 && (!k_scales || !v_scales))
        return SL_ERR_NULL;
    if (!aligned16(q) || !aligned16(out) || !aligned16(k_pages) || !aligned16(v_pages))
        return SL_ERR_ALIGNMENT;
    if (!aligned4(block_table) || !aligned4(seq_lens) ||
        (fp8 && (!aligned4(k_scales) || !aligned4(v_scales))))
        return SL_ERR_ALIGNMENT;
    int nw = 0;
    st = resolve_workers(d, fp8, &nw);
    if (st != SL_OK)
        return st;
    const int G = d->num_q_heads / d->num_kv_heads;
    Workspace ws;
    const size_t need = workspace_layout(d->workspace, d->batch, d->max_blocks_per_seq,
                                         d->num_kv_heads, G, d->head_dim, nw, &ws);
    if (!d->workspace || d->workspace_bytes < need ||
        (reinterpret_cast<uintptr_t>(d->workspace) & (kAlign - 1)) != 0)
        return SL_ERR_WORKSPACE;

    // The split kernel partitions the work itself: each workgroup scans the
    // lengths into LDS and walks the block table.
    SplitParams sp;
    sp.q = q;
    sp.k_pages = k_pages;
    sp.v_pages = v_pages;
    sp.k_scales = k_scales;
    sp.v_scales = v_scales;
    sp.out = out;
    sp.part_ml = ws.part_ml;
    sp.part_acc = ws.part_acc;
    sp.batch = d->batch;
    sp.num_kv_heads = d->num_kv_heads;
    sp.group = G;
    sp.num_workers = nw;
    sp.scale_log2 = scale * 1.4426950408889634f;
    sp.num_q_heads = d->num_q_heads;
    sp.unit_ml = nullptr;
    sp.unit_acc = nullptr;
    sp.seq_lens = seq_lens;
    sp.block_table = block_table;
    sp.cum_out = ws.cum_pages;
    sp.max_blocks = d->max_blocks_per_seq;
    sp.num_pages = d->num_pages;
    if (d->timing_start && hipEventRecord(d->timing_start, d->stream) != hipSuccess)
        return SL_ERR_HIP;
    if (launch_split(sp, d->head_dim, fp8, d->stream) != hipSuccess)
        return SL_ERR_HIP;
    if (d->timing_stop && hipEventRecord(d->timing_stop, d->stream) != hipSuccess)
        return SL_ERR_HIP;

    MergeParams mp;
    mp.seq_lens = seq_lens;
    mp.cum_pages = ws.cum_pages;
    mp.part_ml = ws.part_ml;
    mp.part_acc = ws.part_acc;
    mp.out = out;
    mp.batch = d->batch;
    mp.num_q_heads = d->num_q_heads;
    mp.num_kv_heads = d->num_kv_heads;
    mp.group = G;
    mp.num_workers = nw;
    mp.next_kind = 0;
    if (next) {
        mp.next = *next;
        mp.next_kind = fp8 ? 2 : 1;
    }
    if (launch_merge(mp, d->head_dim, d->stream) != hipSuccess)
        return SL_ERR_HIP;
    return SL_OK;
}

sl_status run_append(const sl_attn_desc *d, const uint16_t *k_new, const uint16_t *v_new,
                     const int32_t *block_table, const int32_t *seq_lens, void *k_pages, void *v_pages,
                     float *k_scales, float *v_scales, bool fp8)
{
    sl_status st = check_desc(d);
    if (st != SL_OK)
        return st;
    if (d->batch == 0)
        return SL_OK;
    if (!k_new || !v_new || !block_table || !seq_lens || !k_pages || !v_pages)
        return SL_ERR_NULL;
    if (fp8 && (!k_scales || !v_scales))
        return SL_ERR_NULL;
    if (!aligned4(k_new) || !aligned4(v_new) || !aligned4(block_table) || !aligned4(seq_lens) ||
        !aligned16(k_pages) || !aligned16(v_pages) ||
        (fp8 && (!aligned4(k_scales) || !aligned4(v_scales))))
        return SL_ERR_ALIGNMENT;
    AppendParams ap;
    ap.k_new = k_new;
    ap.v_new = v_new;
    ap.block_table = block_table;
    ap.seq_lens = seq_lens;
    ap.k_pages = k_pages;
    ap.v_pages = v_pages;
    ap.k_scales = k_scales;
    ap.v_scales = v_scales;
    ap.batch = d->batch;
    ap.num_kv_heads = d->num_kv_heads;
    ap.max_blocks = d->max_blocks_per_seq;
    ap.num_pages = d->num_pages;
    ap.stage = nullptr;
    ap.n_upd = 0;
    ap.set_seq_lens = nullptr;
    ap.set_block_table = nullptr;
    if (d->timing_start && hipEventRecord(d->timing_start, d->stream) != hipSuccess)
        return SL_ERR_HIP;
    if (launch_append(ap, d->head_dim, fp8, d->stream) != hipSuccess)
        return SL_ERR_HIP;
    if (d->timing_stop && hipEventRecord(d->timing_stop, d->stream) != hipSuccess)
        return SL_ERR_HIP;
    return SL_OK;
}

sl_status check_prefix(const sl_attn_desc *d, int32_t num_groups)
{
    sl_status st = check_desc(d);
    if (st != SL_OK)
        return st;
    if (num_groups < 0 || num_groups > d->batch)
        return SL_ERR_SHAPE;
    if (d->batch > kMaxPrefixBatch)
        return SL_ERR_UNSUPPORTED;
    return SL_OK;
}

sl_status run_prefix(const sl_attn_desc *d, const uint16_t *q, const void *k_pages, const void *v_pages,
                     const float *k_scales, const float *v_scales, const int32_t *block_table,
                     const int32_t *seq_lens, const int32_t *group_start, const int32_t *shared_pages,
                     int32_t num_groups, float scale, uint16_t *out, bool fp8)
{
    sl_status st = check_prefix(d, num_groups);
    if (st != SL_OK)
        return st;
    if (d->batch == 0)
        return SL_OK;
    if (!q || !k_pages || !v_pages || !block_table || !seq_lens || !out ||
        (num_groups > 0 && (!group_start || !shared_pages)) || (fp8 && (!k_scales || !v_scales)))
        return SL_ERR_NULL;
    if (!aligned16(q) || !aligned16(out) || !aligned16(k_pages) || !aligned16(v_pages) || !aligned4(block_table) ||
        !aligned4(seq_lens) || (num_groups > 0 && (!aligned4(group_start) || !aligned4(shared_pages))) ||
        (fp8 && (!aligned4(k_scales) || !aligned4(v_scales))))
        return SL_ERR_ALIGNMENT;
    int nw = 0;
    st = resolve_workers(d, fp8, &nw, true);
    if (st != SL_OK)
        return st;
    const int G = d->num_q_heads / d->num_kv_heads;
    PrefixWorkspace ws;
    const size_t need = prefix_workspace_layout(d->workspace, d->batch, d->max_blocks_per_seq, d->num_kv_heads, G,
                                                d->head_dim, nw, num_groups, &ws);
    if (!d->workspace || d->workspace_bytes < need || (reinterpret_cast<uintptr_t>(d->workspace) & (kAlign - 1)) != 0)
        return SL_ERR_WORKSPACE;
    // With no groups the group arrays are never read; point them at the workspace.
    const int32_t *gs = num_groups > 0 ? group_start : ws.cum_shared;
    const int32_t *sp = num_groups > 0 ? shared_pages : ws.cum_shared;

    // Both page streams are derived inside the fused split kernel, whose
    // workgroup 0 stores the sums the merge reads.
    PrefixParams pp;
    pp.group_start = gs;
    pp.shared_pages = sp;
    pp.cum_own = ws.cum_own;
    pp.cum_shared = ws.cum_shared;
    pp.seq_shared = ws.seq_shared;
    pp.num_groups = num_groups;
    pp.max_sub = prefix_max_sub(d->batch, num_groups, G);

    SplitParams sp_;
    sp_.q = q;
    sp_.k_pages = k_pages;
    sp_.v_pages = v_pages;
    sp_.k_scales = fp8 ? k_scales : nullptr;
    sp_.v_scales = fp8 ? v_scales : nullptr;
    sp_.out = out;
    sp_.batch = d->batch;
    sp_.num_kv_heads = d->num_kv_heads;
    sp_.group = G;
    sp_.num_workers = nw;
    sp_.num_q_heads = d->num_q_heads;
    sp_.scale_log2 = scale * 1.4426950408889634f;
    sp_.seq_lens = seq_lens;
    sp_.block_table = block_table;
    sp_.cum_out = nullptr;   // the sums go through pp
    sp_.max_blocks = d->max_blocks_per_seq;
    sp_.num_pages = d->num_pages;
    // Shared-page pass: one workgroup of four wavefronts per worker; up to
    // twice the base count when own-page workgroups are idle.
    const int nws = shared_workers(nw);
    const int nws_max = nw > 2 * nws ? 2 * nws : (nw > nws ? nw : nws);   // slots are sized for nw workers
    SplitParams shp = sp_;
    shp.num_workers = nws;
    shp.part_ml = ws.shared_ml;
    shp.part_acc = ws.shared_acc;
    shp.unit_ml = ws.shared_unit_ml;
    shp.unit_acc = ws.shared_unit_acc;
    // Own-page pass: the single-unit workers.
    sp_.num_workers = nw;
    sp_.part_ml = ws.own_ml;
    sp_.part_acc = ws.own_acc;
    sp_.unit_ml = ws.own_unit_ml;
    sp_.unit_acc = ws.own_unit_acc;
    if (d->timing_start && hipEventRecord(d->timing_start, d->stream) != hipSuccess)
        return SL_ERR_HIP;
    if (launch_prefix_split(sp_, shp, nws_max, pp, d->head_dim, fp8, d->stream) != hipSuccess)
        return SL_ERR_HIP;
    if (d->timing_stop && hipEventRecord(d->timing_stop, d->stream) != hipSuccess)
        return SL_ERR_HIP;

    PrefixMergeParams mp;
    mp.seq_lens = seq_lens;
    mp.group_start = gs;
    mp.shared_pages = sp;
    mp.cum_own = ws.cum_own;
    mp.cum_shared = ws.cum_shared;
    mp.seq_shared = ws.seq_shared;
    mp.own_ml = ws.own_ml;
    mp.own_acc = ws.own_acc;
    mp.shared_ml = ws.shared_ml;
    mp.shared_acc = ws.shared_acc;
    mp.own_unit_ml = ws.own_unit_ml;
    mp.own_unit_acc = ws.own_unit_acc;
    mp.shared_unit_ml = ws.shared_unit_ml;
    mp.shared_unit_acc = ws.shared_unit_acc;
    mp.out = out;
    mp.batch = d->batch;
    mp.max_sub = pp.max_sub;
    mp.num_q_heads = d->num_q_heads;
    mp.num_kv_heads = d->num_kv_heads;
    mp.group = G;
    mp.num_workers = nw;
    mp.num_shared_workers = nws;
    mp.max_shared_workers = nws_max;
    mp.max_blocks = d->max_blocks_per_seq;
    if (launch_merge_prefix(mp, d->head_dim, d->stream) != hipSuccess)
        return SL_ERR_HIP;
    return SL_OK;
}

}  // namespace

sl_status decode_attn_then_append(const sl_attn_desc *d, const uint16_t *q, const void *k_pages, const void *v_pages,
                                  const float *k_scales, const float *v_scales, const int32_t *block_table,
                                  const int32_t *seq_lens, float scale, uint16_t *out, bool fp8,
                                  const AppendParams *next)
{
    return run(d, q, k_pages, v_pages, k_scales, v_scales, block_table, seq_lens, scale, out, fp8, next);
}

}  // namespace sl

extern "C" {

sl_status sl_kv_append(const sl_attn_desc *desc, const uint16_t *k_new, const uint16_t *v_new,
                       const int32_t *block_table, const int32_t *seq_lens, uint16_t *k_pages,
                       uint16_t *v_pages)
{
    return sl::run_append(desc, k_new, v_new, block_table, seq_lens, k_pages, v_pages, nullptr, nullptr,
                          false);
}

sl_status sl_kv_append_fp8(const sl_attn_desc *desc, const uint16_t *k_new, const uint16_t *v_new,
                           const int32_t *block_table, const int32_t *seq_lens, uint8_t *k_pages,
                           uint8_t *v_pages, float *k_scales, float *v_scales)
{
    return sl::run_append(desc, k_new, v_new, block_table, seq_lens, k_pages, v_pages, k_scales, v_scales,
                          true);
}


sl_status sl_decode_attn_num_workers(const sl_attn_desc *desc, int32_t kv_fp8,
                                     int32_t *num_workers)
{
    sl_status st = sl::check_desc(desc);
    if (st != SL_OK)
        return st;
    if (!num_workers)
        return SL_ERR_NULL;
    int nw = 0;
    st = sl::resolve_workers(desc, kv_fp8 != 0, &nw);
    if (st == SL_OK)
        *num_workers = nw;
    return st;
}

sl_status sl_decode_attn_workspace_size(const sl_attn_desc *desc, size_t *bytes)
{
    sl_status st = sl::check_desc(desc);
    if (st != SL_OK)
        return st;
    if (!bytes)
        return SL_ERR_NULL;
    // Size for the larger of the bf16 and fp8 worker counts, so one workspace serves both.
    int nw_bf16 = 0, nw_fp8 = 0;
    st = sl::resolve_workers(desc, false, &nw_bf16);
    if (st == SL_OK)
        st = sl::resolve_workers(desc, true, &nw_fp8);
    if (st != SL_OK)
        return st;
    const int nw = nw_bf16 > nw_fp8 ? nw_bf16 : nw_fp8;
    *bytes = sl::workspace_layout(nullptr, desc->batch, desc->max_blocks_per_seq,
                                  desc->num_kv_heads, desc->num_q_heads / desc->num_kv_heads,
                                  desc->head_dim, nw, nullptr);
    return SL_OK;
}

sl_status sl_decode_attn(const sl_attn_desc *desc, const uint16_t *q, const uint16_t *k_pages,
                         const uint16_t *v_pages, const int32_t *block_table,
                         const int32_t *seq_lens, float scale, uint16_t *out)
{
    return sl::run(desc, q, k_pages, v_pages, nullptr, nullptr, block_table, seq_lens, scale, out,
                   false);
}

sl_status sl_decode_attn_fp8(const sl_attn_desc *desc, const uint16_t *q, const uint8_t *k_pages,
                             const uint8_t *v_pages, const float *k_scales, const float *v_scales,
                             const int32_t *block_table, const int32_t *seq_lens, float scale,
                             uint16_t *out)
{
    return sl::run(desc, q, k_pages, v_pages, k_scales, v_scales, block_table, seq_lens, scale,
                   out, true);
}

const char *sl_status_string(int32_t status)
{
    switch (status) {
    case SL_OK: return "success";
    case SL_ERR_NULL: return "a required pointer is NULL";
    case SL_ERR_SHAPE: return "a size is negative, zero or inconsistent";
    case SL_ERR_UNSUPPORTED: return "unsupported head_dim, page_size, group size or batch";
    case SL_ERR_WORKSPACE: return "workspace missing, too small or not 256-byte aligned";
    case SL_ERR_HIP: return "HIP runtime call or kernel launch failed";
    case SL_ERR_ALIGNMENT: return "q, out or a page pool not 16-byte aligned, or an int/scale array not 4-byte aligned";
    case SL_ERR_SCRATCH_LIMIT: return "the call needs more scratch than the allocation-free entry point's fixed array holds";
    }
    return "unknown status";
}

}  // extern "C"

extern "C" {

sl_status sl_decode_attn_prefix_workspace_size(const sl_attn_desc *desc, int32_t num_groups, size_t *bytes)
{
    sl_status st = sl::check_prefix(desc, num_groups);
    if (st != SL_OK)
        return st;
    if (!bytes)
        return SL_ERR_NULL;
    // Sized for the larger of the bf16 and E4M3 worker counts, so one
    // workspace serves both entry points.
    int nw = 0, nw_fp8 = 0;
    st = sl::resolve_workers(desc, false, &nw, true);
    if (st == SL_OK)
        st = sl::resolve_workers(desc, true, &nw_fp8, true);
    if (st != SL_OK)
        return st;
    if (nw_fp8 > nw)
        nw = nw_fp8;
    *bytes = sl::prefix_workspace_layout(nullptr, desc->batch, desc->max_blocks_per_seq, desc->num_kv_heads,
                                         desc->num_q_heads / desc->num_kv_heads, desc->head_dim, nw, num_groups,
                                         nullptr);
    return SL_OK;
}

sl_status sl_decode_attn_prefix(const sl_attn_desc *desc, const uint16_t *q, const uint16_t *k_pages,
                                const uint16_t *v_pages, const int32_t *block_table, const int32_t *seq_lens,
                                const int32_t *group_start, const int32_t *shared_pages, int32_t num_groups,
                                float scale, uint16_t *out)
{
    return sl::run_prefix(desc, q, k_pages, v_pages, nullptr, nullptr, block_table, seq_lens, group_start,
                          shared_pages, num_groups, scale, out, false);
}

sl_status sl_decode_attn_prefix_fp8(const sl_attn_desc *desc, const uint16_t *q, const uint8_t *k_pages,
                                    const uint8_t *v_pages, const float *k_scales, const float *v_scales,
                                    const int32_t *block_table, const int32_t *seq_lens, const int32_t *group_start,
                                    const int32_t *shared_pages, int32_t num_groups, float scale, uint16_t *out)
{
    return sl::run_prefix(desc, q, k_pages, v_pages, k_scales, v_scales, block_table, seq_lens, group_start,
                          shared_pages, num_groups, scale, out, true);
}

}  // extern "C"
