// Shared-page pass of prefix-shared decode attention, for gfx950.
//
// A shared unit is (group of samples, KV head): its tiles are the group's
// shared pages, and its query rows are the members x G query heads of that
// KV head, at most kPrefixRows = 64, as four 16-row MFMA column blocks
// (row r = 16 c + n is member r / G, head r % G of the group).
//
// One workgroup of four wavefronts is one worker; it streams a contiguous
// range of shared tiles. Each wavefront loads a quarter of every K and V tile
// into registers, writes it to an LDS stage, and after one barrier per tile
// all four read the whole tile from LDS: wavefront c then computes the scores,
// online softmax and value accumulation of column block c with the same MFMA
// layout as the single-unit kernel (scores K.Q^T on v_mfma_f32_16x16x32_bf16,
// values V^T.P^T on v_mfma_f32_16x16x16bf16_1k). A shared page is therefore
// read from HBM once per workgroup, and each wavefront carries one block's
// registers. K and V rows are stored in LDS with 16-byte chunk c of row r at
// position c ^ ((r / P) % C) (P rows per 256 bytes, C chunks per row), so the
// 16 lanes that read one operand at a time hit distinct banks.
//
// Tiles are software-pipelined: while tile i is computed from one LDS stage,
// the loads of tiles i+1 .. i+kAhead+1 are in flight, and tile i+1 is written
// to the other stage. The query block of a unit is loaded with the unit's
// first tile. Every iteration issues the same loads (a load that is not needed
// goes through an empty buffer resource and touches no memory), so the
// compiler's counter waits stay exact and never drain the pipeline.
//
// The pass runs in the same launch as the own-page pass (prefix_split_kernel):
// its workgroups share the CUs with the memory-bound single-unit workers, so
// its latency- and MFMA-bound tiles are hidden under their streaming instead
// of adding to it.
//
// Partial states: a unit cut by the range leaves its piece in worker slot
// 2w (first piece) or 2w + 1 (trailing piece); a unit seen whole goes to its
// own slot of the unit area, at (first query row) / G. Every state still has
// to be merged with the members' own pages.
#include "decode_unit.h"

namespace sl {
namespace {

constexpr int kSharedWaves = kPrefixBlocks;   // one wavefront per 16-row column block
static_assert(kSharedWaves == kWavesPerBlock, "the fused prefix kernel runs both passes in one block shape");
// Tiles in flight beyond the one computed. One is enough: the pass shares its
// CUs with the memory-bound own-page workers, and a deeper ring (3) was
// slower for the registers it took.
constexpr int kAhead = 1;
constexpr int kNonTemporal = 2;                // buffer cache policy: non-temporal (streamed once)

// Bytes of one K (or V) tile, of the quarter one wavefront loads, and the
// per-lane load width.
template <int D>
struct Geo {
    static constexpr int kTile = kPageSize * D * 2;
    static constexpr int kQuarter = kTile / kSharedWaves;
    static constexpr int kLane = kQuarter / kWave;          // 16 (D = 128) or 8 (D = 64)
    static constexpr int kRow = D * 2;                       // bytes per row
    static constexpr int kChunks = kRow / 16;                // 16-byte chunks per row
    static constexpr int kRowsPer256 = 256 / kRow;
};

// Offset in an LDS tile of byte `c16 * 16 + within` of row r.
template <int D>
__device__ __forceinline__ int lds_offset(int r, int c16)
{
    using g = Geo<D>;
    return r * g::kRow + 16 * (c16 ^ ((r / g::kRowsPer256) % g::kChunks));
}

// One wavefront's quarter of a K and a V tile, in registers.
template <int D>
struct Quarter {
    uint32_t k[Geo<D>::kLane / 4];
    uint32_t v[Geo<D>::kLane / 4];
};

// Loads go through a buffer resource covering one tile: a tile past the
// range gets an empty resource, whose loads return zeros without touching
// memory, so every iteration issues the same loads and the counter waits
// stay exact.
template <int D>
__device__ __forceinline__ void load_quarter(Quarter<D> &qt, const SplitParams &p, int32_t page, bool live, int wave,
                                             int lane)
{
    using g = Geo<D>;
    const size_t tile = (size_t)(page < 0 ? 0 : page);
    const int bytes = live ? g::kTile : 0;
    const __amdgpu_buffer_rsrc_t kr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint8_t *>(static_cast<const uint8_t *>(p.k_pages)) + tile * g::kTile, 0, bytes, kRawBufferWord3);
    const __amdgpu_buffer_rsrc_t vr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint8_t *>(static_cast<const uint8_t *>(p.v_pages)) + tile * g::kTile, 0, bytes, kRawBufferWord3);
    const int off = wave * g::kQuarter + lane * g::kLane;
    if constexpr (g::kLane == 16) {
        const u32x4_t a = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(kr, off, 0, kNonTemporal));
        const u32x4_t b = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(vr, off, 0, kNonTemporal));
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            qt.k[c] = a[c];
            qt.v[c] = b[c];
        }
    } else {
        const u32x2_t a = __builtin_bit_cast(u32x2_t, __builtin_amdgcn_raw_buffer_load_b64(kr, off, 0, kNonTemporal));
        const u32x2_t b = __builtin_bit_cast(u32x2_t, __builtin_amdgcn_raw_buffer_load_b64(vr, off, 0, kNonTemporal));
        qt.k[0] = a[0];
        qt.k[1] = a[1];
        qt.v[0] = b[0];
        qt.v[1] = b[1];
    }
}

// Write a wavefront's quarter into an LDS stage (K then V, D * 32 bytes each).
template <int D>
__device__ __forceinline__ void store_quarter(const Quarter<D> &qt, uint8_t *stage, int wave, int lane)
{
    using g = Geo<D>;
    const int byte = wave * g::kQuarter + lane * g::kLane;   // offset in the tile
    const int r = byte / g::kRow;
    const int c16 = (byte % g::kRow) / 16;
    const int within = byte % 16;
    const int o = lds_offset<D>(r, c16) + within;
    if constexpr (g::kLane == 16) {
        *reinterpret_cast<u32x4_t *>(stage + o) = u32x4_t{qt.k[0], qt.k[1], qt.k[2], qt.k[3]};
        *reinterpret_cast<u32x4_t *>(stage + g::kTile + o) = u32x4_t{qt.v[0], qt.v[1], qt.v[2], qt.v[3]};
    } else {
        *reinterpret_cast<u32x2_t *>(stage + o) = u32x2_t{qt.k[0], qt.k[1]};
        *reinterpret_cast<u32x2_t *>(stage + g::kTile + o) = u32x2_t{qt.v[0], qt.v[1]};
    }
}

template <int D>
struct State {
    f32x4_t acc[D / 16];
    float m, l;
};

// One tile of one column block: scores, online softmax, value accumulation.
// Every token of a shared page is live.
template <int D>
__device__ __forceinline__ void compute(State<D> &st, const uint8_t *stage, const bf16x8_t (&qop)[D / 32],
                                        float score_mul, int n, int quad)
{
    using g = Geo<D>;
    f32x4_t s4 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < D / 32; ++s) {   // A = K rows t = n, dims 32 s + 8 quad .. + 7
        const bf16x8_t kv = *reinterpret_cast<const bf16x8_t *>(stage + lds_offset<D>(n, 4 * s + quad));
        s4 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kv, qop[s], s4, 0, 0, 0);
    }
    float sc[4];
#pragma unroll
    for (int r = 0; r < 4; ++r)
        sc[r] = s4[r] * score_mul;
    // Cross-lane maximum only when a lane exceeds the running maximum by the
    // slack (a wave-wide vote), as in the single-unit worker.
    const float lmx = fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3]));
    if (__builtin_amdgcn_ballot_w64(lmx > st.m + kRescaleSlack) != 0) {
        const float mx = quad_max(lmx);
        if (mx > st.m + kRescaleSlack) {
            const float alpha = __builtin_amdgcn_exp2f(st.m - mx);   // 0 on a piece's first tile
            st.l *= alpha;
#pragma unroll
            for (int i = 0; i < D / 16; ++i)
                st.acc[i] *= alpha;
            st.m = mx;
        }
    }
    float pr[4];
#pragma unroll
    for (int r = 0; r < 4; ++r)
        pr[r] = __builtin_amdgcn_exp2f(sc[r] - st.m);
    const uint32_t p01 = pack_bf16(pr[0], pr[1]);
    const uint32_t p23 = pack_bf16(pr[2], pr[3]);
    st.l += (bf16_lo(p01) + bf16_hi(p01)) + (bf16_lo(p23) + bf16_hi(p23));
    const i16x4_t pb = __builtin_bit_cast(i16x4_t, u32x2_t{p01, p23});

    // Value rows 4 quad + r, elements n D/16 .. + D/16 - 1, as bf16 dwords.
    constexpr int RW = D / 32;
    uint32_t vb[4 * RW];
    const uint8_t *vs = stage + g::kTile;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int row = 4 * quad + r;
        const int byte = n * (D / 16) * 2;   // 16 (D = 128) or 8 (D = 64) bytes per lane
        const int o = lds_offset<D>(row, byte / 16) + byte % 16;
        if constexpr (D == 128) {
            const u32x4_t x = *reinterpret_cast<const u32x4_t *>(vs + o);
#pragma unroll
            for (int c = 0; c < 4; ++c)
                vb[r * RW + c] = x[c];
        } else {
            const u32x2_t x = *reinterpret_cast<const u32x2_t *>(vs + o);
            vb[r * RW] = x[0];
            vb[r * RW + 1] = x[1];
        }
    }
#pragma unroll
    for (int i = 0; i < D / 16; ++i) {
        // Element i % 2 of dword i / 2 of rows 0 and 1 (lo) and rows 2 and 3
        // (hi): one byte permute each (v_perm_b32 selects bytes of {a, b},
        // selector bytes 4..7 from a, 0..3 from b).
        const int w = i >> 1;
        const uint32_t sel = (i & 1) == 0 ? 0x05040100u : 0x07060302u;
        const uint32_t lo = __builtin_amdgcn_perm(vb[1 * RW + w], vb[0 * RW + w], sel);
        const uint32_t hi = __builtin_amdgcn_perm(vb[3 * RW + w], vb[2 * RW + w], sel);
        const i16x4_t va = __builtin_bit_cast(i16x4_t, u32x2_t{lo, hi});
        st.acc[i] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(va, pb, st.acc[i], 0, 0, 0);
    }
}

// Store the partial state of row r (this lane's column n of block `wave`) in
// slot `slot` (kPrefixRows rows per slot) when r is one of the unit's rows.
template <int D>
__device__ __forceinline__ void finish(State<D> &st, int r, int rows, bool bad, float *part_ml, float *part_acc,
                                       size_t slot, int quad)
{
    const float l = quad_sum(st.l);
    if (r >= rows)
        return;
    const float poison = bad ? __builtin_nanf("") : 0.0f;
    const int d0 = quad * (D / 4);
    float *dst = part_acc + (slot * kPrefixRows + r) * D + d0;
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4)
#pragma unroll
        for (int i = 0; i < D / 16; i += 4)
            *reinterpret_cast<f32x4_t *>(dst + q4 * (D / 16) + i) =
                f32x4_t{st.acc[i][q4], st.acc[i + 1][q4], st.acc[i + 2][q4], st.acc[i + 3][q4]} + poison;
    if (quad == 0)
        *reinterpret_cast<f32x2_t *>(part_ml + (slot * kPrefixRows + r) * 2) = f32x2_t{st.m + poison, l};
}

template <int D>
__device__ __forceinline__ void reset(State<D> &st)
{
#pragma unroll
    for (int i = 0; i < D / 16; ++i)
        st.acc[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    st.m = kNegInf;
    st.l = 0.f;
}

// Query operands of column block `wave` of the unit whose first query row is
// meta's row0: rows past the unit's read its first row (their columns are
// never written out). With `live` false the loads are empty (zeros, no memory
// access), so they can be issued on every tile.
template <int D>
__device__ __forceinline__ void load_q(bf16x8_t (&qop)[D / 32], const SplitParams &p, uint32_t meta, bool live,
                                       int wave, int n, int quad)
{
    const int G = p.group;
    const int members = (int)(meta & 15u) + 1;
    const int rows = members * G;
    const int r = 16 * wave + n;
    const int rel = r < rows ? (r / G) * p.num_q_heads + r % G : 0;   // row offset from row0
    const int span = ((members - 1) * p.num_q_heads + G) * D * 2;     // bytes from row0 to the last row's end
    const __amdgpu_buffer_rsrc_t qr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t *>(p.q) + (size_t)(meta >> kMetaRowShift) * D, 0, live ? span : 0, kRawBufferWord3);
#pragma unroll
    for (int s = 0; s < D / 32; ++s)
        qop[s] = __builtin_bit_cast(
            bf16x8_t, __builtin_amdgcn_raw_buffer_load_b128(qr, rel * D * 2 + 2 * (32 * s + 8 * quad), 0, 0));
}

// LDS view of the shared-page stream: the exclusive prefix sum of shared
// pages per group, and each group's first member and size packed as
// lead | (members - 1) << 16 (a group without shared pages has no tiles).
struct SharedLds {
    const int32_t *sh;   // [NG + 1]
    const int32_t *gl;   // [NG]
    int32_t num_groups;
};

// Worker w (one workgroup) of the shared-page pass over the stream that `sv`
// describes (complete in LDS). Stream tile s = Hkv sh[k] + g s_k + j is page j
// of group k's shared pages (s_k of them, read through the group's first
// member's block-table row) for KV head g.
template <int D>
__device__ __forceinline__ void split_shared_worker(const SplitParams &p, int w, const SharedLds &sv)
{
    const long long total = (long long)sv.sh[sv.num_groups] * p.num_kv_heads;
    const int nw = effective_workers(total, p.num_workers);
    if (w >= nw)
        return;
    const long long s0 = (long long)w * total / nw;
    const long long s1 = (long long)(w + 1) * total / nw;
    if (s0 >= s1)
        return;
    const int ntiles = (int)(s1 - s0);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int lane = threadIdx.x & (kWave - 1);
    const int n = lane & 15;
    const int quad = lane >> 4;
    const int G = p.group;

    __shared__ __attribute__((aligned(16))) uint8_t stage[2][2 * Geo<D>::kTile];

    // Tile entries {block-table entry, metadata, KV head}, fetched in tile
    // order (every call asks for the next tile; past the range the last tile
    // repeats) from a cursor (k, g, j) over the stream; the block-table entry
    // is loaded through a bounds-checked buffer resource, by every lane.
    const __amdgpu_buffer_rsrc_t btab = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int32_t *>(p.block_table), 0, p.batch * p.max_blocks * (int)sizeof(int32_t), kRawBufferWord3);
    // Largest k with Hkv sh[k] <= s0 (then group k has shared pages).
    int klo = 0, khi = sv.num_groups;
    while (khi - klo > 1) {
        const int mid = (klo + khi) >> 1;
        if ((long long)sv.sh[mid] * p.num_kv_heads <= s0)
            klo = mid;
        else
            khi = mid;
    }
    int ck = klo;
    int csk = sv.sh[ck + 1] - sv.sh[ck];
    int cgl = sv.gl[ck];
    const int off = (int)(s0 - (long long)sv.sh[ck] * p.num_kv_heads);
    int cg = off / csk;
    int cj = off - cg * csk;
    auto entry = [&](int i) -> u32x4_t {
        const int lead = cgl & 0xffff;
        const uint32_t bt = __builtin_bit_cast(
            uint32_t, __builtin_amdgcn_raw_buffer_load_b32(btab, 0, (lead * p.max_blocks + cj) * 4, 0));
        uint32_t meta = (uint32_t)(cgl >> 16) | ((uint32_t)(lead * p.num_q_heads + cg * G) << kMetaRowShift);
        if (cj == 0)
            meta |= kMetaFirst;
        if (cj == csk - 1)
            meta |= kMetaLast;
        const u32x4_t e = {bt, meta, (uint32_t)cg, 0u};
        if (i < ntiles - 1) {   // advance to the next tile of the stream
            if (++cj == csk) {
                cj = 0;
                if (++cg == p.num_kv_heads) {
                    cg = 0;
                    do
                        ++ck;
                    while (sv.sh[ck + 1] == sv.sh[ck]);   // tiles remain, so a group with tiles follows
                    csk = sv.sh[ck + 1] - sv.sh[ck];
                    cgl = sv.gl[ck];
                }
            }
        }
        return e;
    };
    auto page_of = [&](u32x4_t e) -> int32_t {
        const uint32_t bt = (uint32_t)__builtin_amdgcn_readfirstlane(e[0]);
        return bt < (uint32_t)p.num_pages ? (int32_t)(bt * (uint32_t)p.num_kv_heads + e[2]) : -1;
    };
    auto meta_of = [](u32x4_t e) { return (uint32_t)__builtin_amdgcn_readfirstlane(e[1]); };

    // Every iteration issues the same loads: tile i + R (its K/V quarters and,
    // when it starts a unit, the unit's query block; empty loads otherwise)
    // and the entry of tile i + 2R. Ring slot k = i % R holds tile i's data,
    // metadata and query block; the entry ring holds the entries of the tiles
    // to issue next. The prologue fetches the first 2R entries and waits once.
    constexpr int R = kAhead + 1;
    static_assert(R % 2 == 0, "a ring turn must cover whole stage pairs");
    u32x4_t first_e[R], ering[R];
#pragma unroll
    for (int k = 0; k < R; ++k)
        first_e[k] = entry(k);
#pragma unroll
    for (int k = 0; k < R; ++k)
        ering[k] = entry(R + k);
#pragma unroll
    for (int k = 0; k < R; ++k)
        asm volatile("" ::"v"(first_e[k]), "v"(ering[k]));

    Quarter<D> ring[R];
    uint32_t ring_meta[R];
    bf16x8_t qring[R][D / 32];
#pragma unroll
    for (int k = 0; k < R; ++k) {
        const int32_t pg = page_of(first_e[k]);
        const uint32_t mt = meta_of(first_e[k]);
        load_quarter<D>(ring[k], p, pg, k < ntiles, wave, lane);
        ring_meta[k] = pg < 0 ? (mt | kMetaBadLen) : mt;   // a page outside the pool poisons its unit
        load_q<D>(qring[k], p, mt, k == 0 || (k < ntiles && (mt & kMetaFirst) != 0), wave, n, quad);
    }
    store_quarter<D>(ring[0], stage[0], wave, lane);
    __syncthreads();

    bf16x8_t qop[D / 32];
    State<D> st;
    reset(st);
    bool started = false, bad = false;
    int slot_sel = 0;
    for (int i0 = 0; i0 < ntiles; i0 += R) {
#pragma unroll
        for (int k = 0; k < R; ++k) {
            const int i = i0 + k;
            const bool act = i < ntiles;   // the last turn may run past the range: loads only
            const uint32_t meta = ring_meta[k];
            if (i == 0 || (meta & kMetaFirst) != 0) {   // a unit starts: its query block
#pragma unroll
                for (int s = 0; s < D / 32; ++s)
                    qop[s] = qring[k][s];
            }
            // Issue tile t = i + R into slot k (tile i is already in LDS).
            {
                const int t = i + R;
                const int32_t pg = page_of(ering[k]);
                const uint32_t mt = meta_of(ering[k]);
                load_quarter<D>(ring[k], p, pg, t < ntiles, wave, lane);
                ring_meta[k] = pg < 0 ? (mt | kMetaBadLen) : mt;
                load_q<D>(qring[k], p, mt, t < ntiles && (mt & kMetaFirst) != 0, wave, n, quad);
                ering[k] = entry(t + R);
            }
            if (!act)
                continue;
            started |= (meta & kMetaFirst) != 0;
            bad |= (meta & kMetaBadLen) != 0;
            compute<D>(st, stage[k & 1], qop, p.scale_log2, n, quad);
            if ((meta & kMetaLast) != 0 || i == ntiles - 1) {
                const uint32_t row0 = meta >> kMetaRowShift;
                const bool whole = started && (meta & kMetaLast) != 0;
                float *const pml = whole ? p.unit_ml : p.part_ml;
                float *const pacc = whole ? p.unit_acc : p.part_acc;
                const size_t slot = whole ? (size_t)(row0 / (uint32_t)G) : 2 * (size_t)w + slot_sel;
                finish<D>(st, 16 * wave + n, ((int)(meta & 15u) + 1) * G, bad, pml, pacc, slot, quad);
                reset(st);
                started = false;
                bad = false;
                slot_sel = 1;
            }
            if (i + 1 < ntiles) {   // tile i + 1 into the other stage, published by the barrier
                store_quarter<D>(ring[(k + 1) % R], stage[(k + 1) & 1], wave, lane);
                __syncthreads();
            }
        }
    }
}

// Prologue of the fused prefix kernel, run by the whole workgroup: builds in
// LDS the group of every sequence (-1: none), the lengths, the exclusive
// prefix sums of own pages per sequence and of shared pages per group, and
// each group's packed first member and size; workgroup 0 also stores the sums
// and every sequence's sharing descriptor for the merge. A group that is
// empty, has more than min(16, kPrefixRows / G) members, or whose range or
// page count is out of bounds gets no shared pages: its members are attended
// like unshared sequences, so the result stays exact, only without the saving.
__device__ __forceinline__ void scan_prefix_groups(const SplitParams &p, const PrefixParams &pp, int32_t *s_own,
                                                   int32_t *s_len, int32_t *s_group, int32_t *s_sh, int32_t *s_gl)
{
    constexpr int T = kWave * kWavesPerBlock;
    const int B = p.batch, NG = pp.num_groups;
    const int tid = threadIdx.x;
    const int max_members = min(16, kPrefixRows / p.group);
    for (int b = tid; b < B; b += T)
        s_group[b] = -1;
    __syncthreads();
    for (int k = tid; k < NG; k += T) {
        const int lo = pp.group_start[k], hi = pp.group_start[k + 1];
        const int sp = pp.shared_pages[k];
        const bool ok = lo >= 0 && hi <= B && hi - lo >= 1 && hi - lo <= max_members && sp > 0 &&
                        sp <= p.max_blocks;
        s_sh[k] = ok ? sp : 0;
        s_gl[k] = ok ? lo | (hi - lo - 1) << 16 : 0;
        if (ok)
            for (int b = lo; b < hi; ++b)
                atomicMax(&s_group[b], k);   // ascending groups never overlap; otherwise every workgroup agrees
    }
    __syncthreads();
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
    block_exclusive_scan(s_own, B);
    block_exclusive_scan(s_sh, NG);
    if (blockIdx.x == 0) {
        for (int i = tid; i <= B; i += T)
            pp.cum_own[i] = s_own[i];
        for (int i = tid; i <= NG; i += T)
            pp.cum_shared[i] = s_sh[i];
        typedef int32_t i32x4_t __attribute__((ext_vector_type(4)));
        for (int i = tid; i < B; i += T) {
            const int k = s_group[i];
            *reinterpret_cast<i32x4_t *>(pp.seq_shared + 4 * (size_t)i) =
                k >= 0 ? i32x4_t{s_sh[k], s_sh[k + 1] - s_sh[k], s_gl[k] & 0xffff, k} : i32x4_t{0, 0, 0, -1};
        }
    }
}

// Both passes of prefix-shared attention in one launch: workgroups
// [0, own_blocks) run the single-unit workers of the own pages (four per
// workgroup), the rest run shared-page workers. The own-page workgroups come
// first, so each CU holds one of them beside a shared-page workgroup: the
// memory-bound and the MFMA-heavy pass share the CUs instead of running one
// after the other. Every workgroup first derives both streams in its dynamic
// LDS (3 B + 2 NG + 2 ints).
template <int D>
__global__ __launch_bounds__(kWave * kWavesPerBlock) void prefix_split_kernel(SplitParams own, SplitParams shared,
                                                                               PrefixParams pp, int own_blocks,
                                                                               int max_shared)
{
    extern __shared__ int32_t s_dyn[];
    const int B = own.batch, NG = pp.num_groups;
    int32_t *const s_own = s_dyn;            // [B + 1]
    int32_t *const s_len = s_own + B + 1;    // [B]
    int32_t *const s_group = s_len + B;      // [B]
    int32_t *const s_sh = s_group + B;       // [NG + 1]
    int32_t *const s_gl = s_sh + NG + 1;     // [NG]
    scan_prefix_groups(own, pp, s_own, s_len, s_group, s_sh, s_gl);
    if ((int)blockIdx.x < own_blocks)
        split_unit_worker<D, false, kOwnPages>(
            own, blockIdx.x * kWavesPerBlock + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave),
            StreamLds{s_own, s_len, s_group, s_sh});
    else {
        SplitParams sh = shared;
        sh.num_workers = effective_shared_workers((long long)s_own[B] * own.num_kv_heads, own.num_workers,
                                                  shared.num_workers, max_shared);
        split_shared_worker<D>(sh, (int)blockIdx.x - own_blocks, SharedLds{s_sh, s_gl, NG});
    }
}

}  // namespace

hipError_t launch_prefix_split(const SplitParams &own, const SplitParams &shared, int max_shared,
                               const PrefixParams &pp, int head_dim, hipStream_t stream)
{
    const int own_blocks = (own.num_workers + kWavesPerBlock - 1) / kWavesPerBlock;
    const dim3 grid(own_blocks + max_shared);
    const dim3 block(kWave * kWavesPerBlock);
    const size_t lds = prefix_dynamic_lds(own.batch, pp.num_groups);
    if (head_dim == 128)
        hipLaunchKernelGGL(prefix_split_kernel<128>, grid, block, lds, stream, own, shared, pp, own_blocks,
                           max_shared);
    else if (head_dim == 64)
        hipLaunchKernelGGL(prefix_split_kernel<64>, grid, block, lds, stream, own, shared, pp, own_blocks,
                           max_shared);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

}  // namespace sl
