// Decode engine: the multi-step generation loop of include/sl_engine.h.
//
// The host owns the schedule. Samples are admitted in LPT (or index) order
// into BS slots, pages come from a LIFO free stack, and the lengths given at
// creation fix every step in advance. Each step is packed into a pinned
// staging buffer ([seq_lens][page of each new token][block-table updates]
// [prompt pages to fill]). On the caller's stream a step is: its
// bookkeeping and KV append (the lengths and block-table updates applied,
// the new K/V rows stored), then decode attention (split kernel and merge).
// Since the host knows the next step before the GPU has run this one, the
// next step's bookkeeping and append run in this step's merge launch, after
// the attention has read the cache: a step costs two launches. A step that
// admits prompts fills their pages first (fill kernel) and runs its own
// append launch, and so does the first step of each sl_engine_run call. The
// kernels read the staging buffer in place (mapped pinned memory), which
// saves a copy command per step; a ring of such buffers, each reused only
// once the kernels that read it have completed, lets the host run ahead of
// the GPU.
//
// A bf16 step whose attention fits the chip in one pass of workgroups runs
// in a single launch instead (engine_unit_step_kernel): the host passes the
// step's sequences and lengths as kernel arguments, gives each (sequence, KV
// head) unit a share of the CUs in whole workgroups, and the unit's
// workgroups combine their states themselves; the next step's append rides
// in the same launch unless it would reuse a page freed in this step, which
// this step's attention may still be reading. Empty slots' rows are cleared
// once per run call and whenever a slot empties.
#include <algorithm>
#include <cstring>
#include <new>
#include <vector>

#include "sl.h"
#include "sl_engine.h"
#include "api_internal.h"
#include "engine_internal.h"

namespace {

using sl::kPageSize;
// Staging ring: kRing mapped pinned buffers, taken in order. The host may
// rewrite a buffer only after the kernels that read it have finished. An
// event is recorded after the launch that reads the last buffer of each
// group of kRingGroup (launches read the buffers in ring order, on one
// stream), so one event covers the whole group and the host still runs at
// least kRing - kRingGroup steps ahead: recording one after every launch
// left the device idle for ~5 us before each step's first kernel.
constexpr int kRing = 8;
constexpr int kRingGroup = 4;
constexpr int kRingEvents = kRing / kRingGroup;
// One-launch step: a wave gets at least this many tiles of its unit, and the
// step takes the one-launch path only while its longest wave range is within
// kUnitSlackTiles tiles of a split-kernel worker's share (the two-launch
// step spreads tiles over all workers but pays a second launch).
constexpr int kUnitMinTiles = 1;
constexpr int kUnitThreads = sl::kUnitWaves * sl::kWave;
constexpr int kUnitSlackTiles = 8;

bool aligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

}  // namespace

struct sl_engine {
    sl_engine_buffers buf{};
    sl_attn_desc step_desc{};          // buf.desc without timing events
    int M = 0, BS = 0, max_blocks = 0, num_pages = 0, Hkv = 0, D = 0, row_sets = 1;
    bool fp8 = false;
    uint32_t seed = 0;
    float attn_scale = 0.f;
    std::vector<int32_t> prompt, outlen;
    std::vector<int32_t> queue;        // admission order
    size_t head = 0;
    std::vector<int32_t> free_stack;   // back() is popped next
    std::vector<int32_t> occupant, made;
    std::vector<std::vector<int32_t>> pages;
    std::vector<int32_t> slot, admit, finish, active;
    int step = 0;
    bool done = false;
    sl_status failed = SL_OK;
    size_t stage_ints = 0;
    int32_t *h_stage[kRing] = {};   // mapped pinned staging buffers
    int32_t *d_stage[kRing] = {};   // their device addresses
    hipEvent_t ev[kRingEvents] = {};    // one per group of kRingGroup buffers
    bool ev_pending[kRingEvents] = {};
    int ring = 0;

    // One-launch step: device memory for the pieces and the arrival
    // counters, the CU and split-worker counts, which slots' rows are known
    // to be zero, and whether a sample finished in the current step.
    void *unit_mem = nullptr;
    int cus = 0, nw = 0;
    sl::UnitStepParams up{};
    std::vector<uint8_t> zeroed;
    bool freed_now = false;

    void release()
    {
        for (int k = 0; k < kRingEvents; ++k)
            if (ev[k])
                (void)hipEventDestroy(ev[k]);
        for (int r = 0; r < kRing; ++r)
            if (h_stage[r])
                (void)hipHostFree(h_stage[r]);
        if (unit_mem)
            (void)hipFree(unit_mem);
    }

    // A step's staging: ring slot, update and fill counts, active samples.
    struct Staged {
        int ring = 0, n_upd = 0, n_fill = 0, n_active = 0, step = 0;
    };
    // The next step's staging: not prepared yet, prepared but not launched
    // (it admits prompts), or applied and appended by the last merge launch.
    enum { kNone, kPrepared, kLaunched } next_state = kNone;
    Staged next;

    sl_status prepare(Staged &out);
    sl_status staged_launched(int r, hipStream_t s);
    sl::AppendParams append_params(const Staged &sg) const;
    sl_status launch_staged(const Staged &sg);
    bool plan_unit_step(const Staged &sg);
    sl_status one_step(bool chain);
};

sl_status sl_engine::prepare(Staged &out)
{
    // Refill free slots, lowest first, taking prompt pages in block order.
    std::vector<int32_t> upd;    // (slot, block, page) triples
    std::vector<int32_t> fills;  // prompt pages to fill
    for (int b = 0; b < BS; ++b) {
        if (occupant[b] >= 0 || head >= queue.size())
            continue;
        const int i = queue[head++];
        occupant[b] = i;
        made[b] = 0;
        slot[i] = b;
        admit[i] = step;
        const int n = (prompt[i] + kPageSize - 1) / kPageSize;
        pages[b].clear();
        for (int k = 0; k < n; ++k) {
            const int32_t pg = free_stack.back();
            free_stack.pop_back();
            pages[b].push_back(pg);
            upd.insert(upd.end(), {b, k, pg});
            fills.push_back(pg);
        }
    }
    out.n_active = 0;
    for (int b = 0; b < BS; ++b)
        out.n_active += occupant[b] >= 0;
    if (out.n_active == 0)
        return SL_OK;

    // This step's lengths, the page of every slot's new token, and a new page
    // for every token that opens one.
    const int r = ring;
    ring = (ring + 1) % kRing;
    const int grp = r / kRingGroup;   // its group's event, recorded a lap ago, covers its last use
    if (ev_pending[grp] && hipEventSynchronize(ev[grp]) != hipSuccess)
        return SL_ERR_HIP;
    ev_pending[grp] = false;
    int32_t *h = h_stage[r];
    for (int b = 0; b < BS; ++b) {
        const int i = occupant[b];
        if (i < 0) {
            h[b] = 0;
            h[BS + b] = -1;
            continue;
        }
        const int t = prompt[i] + made[b];   // position of this step's token
        if (t % kPageSize == 0) {
            const int32_t pg = free_stack.back();
            free_stack.pop_back();
            pages[b].push_back(pg);
            upd.insert(upd.end(), {b, t / kPageSize, pg});
        }
        h[b] = t + 1;
        h[BS + b] = pages[b][t / kPageSize];
    }
    out.ring = r;
    out.step = step;   // the step these rows belong to (prepare runs after the previous step's ++step)
    out.n_upd = (int)upd.size() / 3;
    out.n_fill = (int)fills.size();
    if (!upd.empty())   // (an empty vector's data() may be null, which memcpy must not get)
        std::memcpy(h + 2 * BS, upd.data(), sizeof(int32_t) * upd.size());
    if (!fills.empty())
        std::memcpy(h + 2 * BS + upd.size(), fills.data(), sizeof(int32_t) * fills.size());
    return SL_OK;
}

sl::AppendParams sl_engine::append_params(const Staged &sg) const
{
    sl::AppendParams ap;
    const size_t set = (size_t)(sg.step % row_sets) * BS * Hkv * D;   // this step's set of new rows
    ap.k_new = buf.k_new + set;
    ap.v_new = buf.v_new + set;
    ap.block_table = nullptr;   // the lengths and token pages come from the staging buffer
    ap.seq_lens = nullptr;
    ap.k_pages = buf.k_pages;
    ap.v_pages = buf.v_pages;
    ap.k_scales = fp8 ? buf.k_scales : nullptr;
    ap.v_scales = fp8 ? buf.v_scales : nullptr;
    ap.batch = BS;
    ap.num_kv_heads = Hkv;
    ap.max_blocks = max_blocks;
    ap.num_pages = num_pages;
    ap.stage = d_stage[sg.ring];
    ap.n_upd = sg.n_upd;
    ap.set_seq_lens = buf.seq_lens;
    ap.set_block_table = buf.block_table;
    return ap;
}

sl_status sl_engine::launch_staged(const Staged &sg)
{
    hipStream_t s = step_desc.stream;
    const int32_t *ds = d_stage[sg.ring];
    // Prompt data first: the new token of an admitted sample may land in its last prompt page.
    if (sg.n_fill > 0 &&
        sl::launch_engine_fill(ds + 2 * BS + 3 * sg.n_upd, sg.n_fill, Hkv, D, fp8, seed, buf.k_pages, buf.v_pages,
                               buf.k_scales, buf.v_scales, s) != hipSuccess)
        return SL_ERR_HIP;
    if (sl::launch_append(append_params(sg), D, fp8, s) != hipSuccess)
        return SL_ERR_HIP;
    return staged_launched(sg.ring, s);
}

// The launch that reads staging buffer r has been enqueued on s: after the
// last buffer of a group, record the group's event.
sl_status sl_engine::staged_launched(int r, hipStream_t s)
{
    if (r % kRingGroup != kRingGroup - 1)
        return SL_OK;
    if (hipEventRecord(ev[r / kRingGroup], s) != hipSuccess)
        return SL_ERR_HIP;
    ev_pending[r / kRingGroup] = true;
    return SL_OK;
}

// Fill `up` for a one-launch step over the lengths staged in `sg`, or
// return false if the step should take the two-launch path.
bool sl_engine::plan_unit_step(const Staged &sg)
{
    if (!unit_mem)
        return false;
    const int32_t *h = h_stage[sg.ring];
    int n = 0, z = 0;
    long long tiles = 0;   // per KV head
    for (int b = 0; b < BS; ++b) {
        if (h[b] > 0) {
            if (n == sl::kMaxUnitEntries)
                return false;
            up.seq[n] = b;
            up.len[n] = h[b];
            ++n;
            tiles += (h[b] + kPageSize - 1) / kPageSize;
        } else if (!zeroed[b]) {
            if (z == sl::kMaxUnitEntries)
                return false;
            up.zero[z++] = b;
        }
    }
    if (n == 0 || (long long)n * Hkv > cus)
        return false;
    // Workgroups per unit: its share of the CUs by tiles, at least one, and
    // at most enough to give every wave kUnitMinTiles tiles.
    int blocks = 0, wave_tiles = 0;
    for (int e = 0; e < n; ++e) {
        const int nb = (up.len[e] + kPageSize - 1) / kPageSize;
        long long k = (long long)cus * nb / (tiles * Hkv);
        const long long kmax = (nb + sl::kUnitWaves * kUnitMinTiles - 1) / (sl::kUnitWaves * kUnitMinTiles);
        k = std::max(1LL, std::min(std::min(k, kmax), (long long)sl::kMaxUnitSplit));
        up.first[e] = blocks;
        blocks += Hkv * (int)k;
        wave_tiles = std::max(wave_tiles, (int)((nb + sl::kUnitWaves * k - 1) / (sl::kUnitWaves * k)));
    }
    up.first[n] = blocks;
    const long long worker_tiles = (tiles * Hkv + nw - 1) / nw;
    if (blocks > sl::kMaxUnitBlocks || wave_tiles > worker_tiles + kUnitSlackTiles)
        return false;
    up.n_entries = n;
    up.unit_blocks = blocks;
    up.zero_blocks = z;
    return true;
}

sl_status sl_engine::one_step(bool chain)
{
    // This step's bookkeeping and KV append: launched now, unless the previous
    // step's merge already ran them.
    sl_status st;
    Staged cur = next;
    if (next_state == kNone) {
        st = prepare(cur);
        if (st != SL_OK)
            return st;
        if (cur.n_active == 0) {
            done = true;
            return SL_OK;
        }
    }
    if (next_state != kLaunched) {
        st = launch_staged(cur);
        if (st != SL_OK)
            return st;
    }
    next_state = kNone;

    const int this_step = step;
    // The step's tokens are decided: every occupied slot makes one; finished
    // samples leave and give their pages back, last block first.
    active.push_back(cur.n_active);
    freed_now = false;
    for (int b = 0; b < BS; ++b) {
        const int i = occupant[b];
        if (i < 0)
            continue;
        if (++made[b] == outlen[i]) {
            freed_now = true;
            finish[i] = step;
            for (auto it = pages[b].rbegin(); it != pages[b].rend(); ++it)
                free_stack.push_back(*it);
            pages[b].clear();
            occupant[b] = -1;
        }
    }
    ++step;

    // With more steps to run, stage the next one now. Its bookkeeping and KV
    // append then run in this step's last launch, after (or, in the
    // one-launch step, beside) the attention, unless it admits prompts: their
    // pages must be filled before the append, so that step launches them
    // itself. Beside the attention it also must not reuse a page freed in
    // this step: the free stack hands those out first.
    const sl::AppendParams *fused = nullptr;
    sl::AppendParams nap;
    bool last = false, fuse = false;
    if (chain) {
        st = prepare(next);
        if (st != SL_OK)
            return st;
        if (next.n_active == 0)
            last = true;
        else
            fuse = next.n_fill == 0;
    }
    const bool one_launch = plan_unit_step(cur);
    if (one_launch && freed_now && next.n_upd > 0)
        fuse = false;
    // E4M3: the units append their own next-step rows after their reads, so
    // every slot the next step appends to must be one of this step's (a
    // prompt of length 0 admits a sample without filling pages).
    if (one_launch && fp8 && fuse) {
        const int32_t *hc = h_stage[cur.ring], *hn = h_stage[next.ring];
        for (int b = 0; b < BS && fuse; ++b)
            fuse = hn[b] <= 0 || (hc[b] > 0 && hn[b] == hc[b] + 1);
        for (int e = 0; e < up.n_entries; ++e)
            up.next_page[e] = hn[up.seq[e]] > 0 ? hn[BS + up.seq[e]] : -1;
    }
    if (chain && !last) {
        next_state = fuse ? kLaunched : kPrepared;
        if (fuse) {
            nap = append_params(next);
            fused = &nap;
        }
    }
    if (one_launch) {
        up.next = fused ? *fused : sl::AppendParams{};
        up.units_append = fused && fp8;
        if (!fused)
            up.next_blocks = 0;
        else if (fp8)   // the bookkeeping only: BS lengths and the table updates
            up.next_blocks = (std::max(BS, next.n_upd) + kUnitThreads - 1) / kUnitThreads;
        else            // and a wave per (slot, KV head) append
            up.next_blocks = (BS * Hkv + sl::kUnitWaves - 1) / sl::kUnitWaves;
        if (sl::launch_unit_step(up, D, fp8, step_desc.stream) != hipSuccess)
            return SL_ERR_HIP;
        for (int e = 0; e < up.n_entries; ++e)
            zeroed[up.seq[e]] = 0;
        for (int z = 0; z < up.zero_blocks; ++z)
            zeroed[up.zero[z]] = 1;
    } else {
        if (fp8)
            st = sl::decode_attn_then_append(&step_desc, buf.q, buf.k_pages, buf.v_pages, buf.k_scales,
                                             buf.v_scales, buf.block_table, buf.seq_lens, attn_scale, buf.out, true,
                                             fused);
        else
            st = sl::decode_attn_then_append(&step_desc, buf.q, buf.k_pages, buf.v_pages, nullptr, nullptr,
                                             buf.block_table, buf.seq_lens, attn_scale, buf.out, false, fused);
        if (st != SL_OK)
            return st;
        const int32_t *h = h_stage[cur.ring];   // the merge writes every empty slot's rows
        for (int b = 0; b < BS; ++b)
            zeroed[b] = h[b] <= 0;
    }
    if (buf.out_history && this_step < buf.history_steps) {
        const size_t bytes = sizeof(uint16_t) * BS * step_desc.num_q_heads * D;
        if (hipMemcpyAsync(buf.out_history + (size_t)this_step * (bytes / sizeof(uint16_t)), buf.out, bytes,
                           hipMemcpyDeviceToDevice, step_desc.stream) != hipSuccess)
            return SL_ERR_HIP;
    }
    if (fused && (st = staged_launched(next.ring, step_desc.stream)) != SL_OK)
        return st;
    if (last)
        done = true;
    return SL_OK;
}

extern "C" {

sl_status sl_engine_create(const sl_engine_config *cfg, const sl_engine_buffers *bufs, sl_engine **out)
{
    if (!cfg || !bufs || !out)
        return SL_ERR_NULL;
    *out = nullptr;
    const sl_attn_desc &d = bufs->desc;
    size_t need = 0;
    sl_status st = sl_decode_attn_workspace_size(&d, &need);   // validates the descriptor
    if (st != SL_OK)
        return st;
    if (!d.workspace || d.workspace_bytes < need || !aligned(d.workspace, 256))
        return SL_ERR_WORKSPACE;
    const int M = cfg->num_samples, BS = d.batch;
    if (M < 1 || BS < 1 || (cfg->admission != 0 && cfg->admission != 1) ||
        (cfg->launch_mode != 0 && cfg->launch_mode != 1) || bufs->history_steps < 0 || bufs->row_sets < 0)
        return SL_ERR_SHAPE;
    if (bufs->history_steps > 0 && !bufs->out_history)
        return SL_ERR_NULL;
    if (!cfg->prompt_len || !cfg->output_len || !cfg->est_len)
        return SL_ERR_NULL;
    if (!bufs->q || !bufs->k_new || !bufs->v_new || !bufs->k_pages || !bufs->v_pages || !bufs->block_table ||
        !bufs->seq_lens || !bufs->out)
        return SL_ERR_NULL;
    const bool fp8 = cfg->kv_fp8 != 0;
    if (fp8 && (!bufs->k_scales || !bufs->v_scales))
        return SL_ERR_NULL;
    if (!aligned(bufs->q, 16) || !aligned(bufs->out, 16) || !aligned(bufs->k_pages, 16) ||
        !aligned(bufs->v_pages, 16) || !aligned(bufs->k_new, 4) || !aligned(bufs->v_new, 4) ||
        !aligned(bufs->block_table, 4) || !aligned(bufs->seq_lens, 4) || !aligned(bufs->out_history, 16) ||
        (fp8 && (!aligned(bufs->k_scales, 4) || !aligned(bufs->v_scales, 4))))
        return SL_ERR_ALIGNMENT;
    int max_prompt_blocks = 0;
    for (int i = 0; i < M; ++i) {
        const long long p = cfg->prompt_len[i], o = cfg->output_len[i];
        if (p < 0 || o < 1 || (p + o + kPageSize - 1) / kPageSize > d.max_blocks_per_seq)
            return SL_ERR_SHAPE;
        max_prompt_blocks = std::max(max_prompt_blocks, (int)((p + kPageSize - 1) / kPageSize));
    }
    if ((long long)d.num_pages < (long long)BS * d.max_blocks_per_seq)
        return SL_ERR_SHAPE;

    sl_engine *e = new (std::nothrow) sl_engine;
    if (!e)
        return SL_ERR_HIP;
    e->buf = *bufs;
    e->step_desc = d;
    e->step_desc.timing_start = nullptr;
    e->step_desc.timing_stop = nullptr;
    e->M = M;
    e->BS = BS;
    e->max_blocks = d.max_blocks_per_seq;
    e->num_pages = d.num_pages;
    e->Hkv = d.num_kv_heads;
    e->D = d.head_dim;
    e->fp8 = fp8;
    e->row_sets = std::max(1, (int)bufs->row_sets);
    e->seed = cfg->fill_seed;
    e->attn_scale = cfg->attn_scale;
    e->prompt.assign(cfg->prompt_len, cfg->prompt_len + M);
    e->outlen.assign(cfg->output_len, cfg->output_len + M);
    e->queue.resize(M);
    for (int i = 0; i < M; ++i)
        e->queue[i] = i;
    if (cfg->admission == 1) {
        const int32_t *est = cfg->est_len;
        std::stable_sort(e->queue.begin(), e->queue.end(), [est](int a, int b) { return est[a] > est[b]; });
    }
    e->free_stack.resize(d.num_pages);
    for (int k = 0; k < d.num_pages; ++k)
        e->free_stack[k] = d.num_pages - 1 - k;   // pops 0, 1, 2, ...
    e->occupant.assign(BS, -1);
    e->made.assign(BS, 0);
    e->pages.assign(BS, {});
    e->slot.assign(M, -1);
    e->admit.assign(M, -1);
    e->finish.assign(M, -1);
    // staging: lengths, token pages, at most BS * (prompt blocks + 1) updates, BS * prompt blocks fills
    e->stage_ints = 2 * (size_t)BS + 3 * (size_t)BS * (max_prompt_blocks + 1) + (size_t)BS * max_prompt_blocks;
    e->zeroed.assign(BS, 0);
    // One-launch step: piece slots (kMaxUnitBlocks workgroups, each G pairs
    // (m, l) on whole cache lines and G rows of D accumulators) and the
    // arrival counters, zeroed.
    if (cfg->launch_mode == 0) {
        const int G = d.num_q_heads / d.num_kv_heads;
        int dev = 0, nw = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&e->cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) {
            delete e;
            return SL_ERR_HIP;
        }
        st = sl_decode_attn_num_workers(&d, fp8 ? 1 : 0, &nw);
        if (st != SL_OK) {
            delete e;
            return st;
        }
        e->nw = nw;
        const size_t rows = (size_t)sl::kMaxUnitBlocks * G;
        const size_t ml_bytes = (size_t)sl::kMaxUnitBlocks * sl::unit_ml_stride(G) * sizeof(float);
        const size_t acc_bytes = (rows * d.head_dim * sizeof(float) + 255) / 256 * 256;
        const size_t cnt_bytes = sizeof(int32_t) * sl::kMaxUnitEntries * d.num_kv_heads;
        if (hipMalloc(&e->unit_mem, ml_bytes + acc_bytes + cnt_bytes) != hipSuccess) {
            e->unit_mem = nullptr;
            delete e;
            return SL_ERR_HIP;
        }
        char *base = static_cast<char *>(e->unit_mem);
        if (hipMemset(base + ml_bytes + acc_bytes, 0, cnt_bytes) != hipSuccess) {
            e->release();
            delete e;
            return SL_ERR_HIP;
        }
        sl::SplitParams &sp = e->up.cur;
        sp.q = bufs->q;
        sp.k_pages = bufs->k_pages;
        sp.v_pages = bufs->v_pages;
        sp.k_scales = fp8 ? bufs->k_scales : nullptr;
        sp.v_scales = fp8 ? bufs->v_scales : nullptr;
        sp.out = bufs->out;
        sp.part_ml = reinterpret_cast<float *>(base);
        sp.part_acc = reinterpret_cast<float *>(base + ml_bytes);
        sp.batch = BS;
        sp.num_kv_heads = d.num_kv_heads;
        sp.group = G;
        sp.num_workers = 0;
        sp.num_q_heads = d.num_q_heads;
        sp.scale_log2 = cfg->attn_scale * 1.4426950408889634f;
        sp.unit_ml = nullptr;
        sp.unit_acc = nullptr;
        sp.seq_lens = nullptr;
        sp.block_table = bufs->block_table;
        sp.cum_out = nullptr;
        sp.max_blocks = d.max_blocks_per_seq;
        sp.num_pages = d.num_pages;
        e->up.counters = reinterpret_cast<int32_t *>(base + ml_bytes + acc_bytes);
    }
    bool ok = true;
    for (int r = 0; ok && r < kRing; ++r)
        ok = hipHostMalloc(reinterpret_cast<void **>(&e->h_stage[r]), sizeof(int32_t) * e->stage_ints,
                           hipHostMallocMapped) == hipSuccess &&
             hipHostGetDevicePointer(reinterpret_cast<void **>(&e->d_stage[r]), e->h_stage[r], 0) == hipSuccess;
    for (int k = 0; ok && k < kRingEvents; ++k)
        ok = hipEventCreateWithFlags(&e->ev[k], hipEventDisableTiming) == hipSuccess;
    if (!ok) {
        e->release();
        delete e;
        return SL_ERR_HIP;
    }
    *out = e;
    return SL_OK;
}

sl_status sl_engine_run(sl_engine *e, int32_t max_steps, int32_t *steps_run)
{
    if (!e || !steps_run)
        return SL_ERR_NULL;
    if (max_steps < 0)
        return SL_ERR_SHAPE;
    *steps_run = 0;
    if (e->failed != SL_OK)
        return e->failed;
    // The caller may have written `out` between calls: clear empty slots' rows again.
    std::fill(e->zeroed.begin(), e->zeroed.end(), 0);
    for (int k = 0; k < max_steps && !e->done; ++k) {
        const int before = e->step;
        const sl_status st = e->one_step(k + 1 < max_steps);
        if (st != SL_OK) {
            e->failed = st;
            return st;
        }
        *steps_run += e->step - before;
    }
    return SL_OK;
}

sl_status sl_engine_schedule(const sl_engine *e, int32_t *slot, int32_t *admit_step, int32_t *finish_step,
                             int32_t *steps, int32_t *active, int32_t active_cap)
{
    if (!e)
        return SL_ERR_NULL;
    if (slot)
        std::copy(e->slot.begin(), e->slot.end(), slot);
    if (admit_step)
        std::copy(e->admit.begin(), e->admit.end(), admit_step);
    if (finish_step)
        std::copy(e->finish.begin(), e->finish.end(), finish_step);
    if (steps)
        *steps = e->step;
    if (active && active_cap > 0) {
        const size_t n = std::min((size_t)active_cap, e->active.size());
        std::copy(e->active.begin(), e->active.begin() + n, active);
    }
    return SL_OK;
}

sl_status sl_engine_destroy(sl_engine *e)
{
    if (!e)
        return SL_OK;
    const sl_status st = hipStreamSynchronize(e->step_desc.stream) == hipSuccess ? SL_OK : SL_ERR_HIP;
    e->release();
    delete e;
    return st;
}

}  // extern "C"
