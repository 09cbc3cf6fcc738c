/*
 * parason.hip -- C-ABI of the Parason accounting/reward path for gfx950.
 * The kernels are in parason_kernels.h; this file validates arguments, lays
 * out the caller's workspace and enqueues the launches on the caller's stream.
 * The policy-gradient step (pg.hip) and the decode step (decode.hip) are
 * further entry points of the same library.
 *
 * Launches are written with HIP's hipLaunchKernelGGL rather than the triple
 * chevron, so that this file also compiles as plain C++ against the CPU
 * emulation of the HIP runtime that the tests run the kernels on.
 */
#include <algorithm>
#include <cstring>
#include <new>

#include "abi_common.h"
#include "parason_kernels.h"

using abi::ALIGN;
using abi::align_up;
using abi::cu_count;
using abi::is_finite;

namespace {

#ifndef PARASON_SCAN_BLOCKS_PER_CU
#define PARASON_SCAN_BLOCKS_PER_CU 4
#endif
constexpr int SCAN_BLOCKS_PER_CU = PARASON_SCAN_BLOCKS_PER_CU; /* persistent grid of 4-wave blocks */
/* slot indices are 32-bit: GATHER_SLOTS + POOL_PER_SEG slots per segment and
 * POOL_MIN more must stay below 2^32 (about 3.6e11 tokens, far beyond what
 * one GPU holds) */
constexpr int64_t MAX_SEGMENTS =
    (((int64_t)1 << 32) - 1 - pk::POOL_MIN) / (pk::GATHER_SLOTS + pk::POOL_PER_SEG);
constexpr int MID_BLOCKS_PER_CU = 2; /* rows_mid blocks hold 64 KB of LDS frames each */
constexpr int GATHER_BLOCKS_PER_CU = 8; /* 4-wave blocks of gather_rows */
constexpr int ROWS_WAVES_PER_CU = 20;   /* rows_fast waves a CU holds (8 KB of LDS frames each) */

/* Byte offsets of the workspace sections for n rows. */
struct Layout {
    size_t seg_off, tile_sum, tile_off, counters, mode, mid_rows, deep_rows, split_rows;
    size_t red_d, red_i, stats;
    size_t fixed;  /* bytes before the per-segment sections */
    int64_t n_tiles;
};

Layout layout_for(int64_t n)
{
    Layout L;
    L.n_tiles = n > 0 ? (n + pk::PLAN_TILE - 1) / pk::PLAN_TILE : 1;
    size_t o = 0;
    L.seg_off = o;
    o = align_up(o + (size_t)(n + 1) * sizeof(int64_t));
    L.tile_sum = o;
    o = align_up(o + (size_t)L.n_tiles * sizeof(int64_t));
    L.tile_off = o;
    o = align_up(o + (size_t)L.n_tiles * sizeof(int64_t));
    L.counters = o;
    o = align_up(o + 4 * sizeof(int32_t));
    L.mode = o;
    o = align_up(o + (size_t)(n > 0 ? n : 1));
    L.mid_rows = o;
    o = align_up(o + (size_t)(n > 0 ? n : 1) * sizeof(int32_t));
    L.deep_rows = o;
    o = align_up(o + (size_t)(n > 0 ? n : 1) * sizeof(int32_t));
    L.split_rows = o;
    o = align_up(o + (size_t)(n > 0 ? n : 1) * sizeof(int32_t));
    /* partial sums of the batch reductions (one record per 4096 rows) */
    L.red_d = o;
    o = align_up(o + (size_t)L.n_tiles * 3 * sizeof(double));
    L.red_i = o;
    o = align_up(o + (size_t)L.n_tiles * pk::NMI * sizeof(int64_t));
    L.stats = o;
    o = align_up(o + sizeof(pk::BatchStats));
    L.fixed = o;
    return L;
}

/* The sections after the fixed ones, for a capacity of cap segments: the
 * deep tier's frames and entry bits (sized for any row that fits in cap
 * segments), one SegRec per segment, then the event slots: GATHER_SLOTS per
 * segment, then the pool (POOL_PER_SEG slots per segment, at least
 * POOL_MIN).  About 56 bytes per 1024-token segment once the deep store
 * reaches its maximum (2^20 frames, 32 MiB, from about 6,100 segments on). */
struct CapSections {
    size_t frames, bits, seg, slots, end;            /* byte offsets; end = bytes needed */
    int64_t n_frames, n_bits, pool_base, pool_slots; /* the pool in slots */
};

CapSections cap_sections(const Layout &L, int64_t cap)
{
    CapSections q;
    q.n_frames = std::min(pk::DEEP_FRAMES, pk::DEEP_FRAMES_PER_SEG * cap + 1);
    q.n_bits = std::min(pk::DEEP_ENTRY_BITS, (pk::DEEP_BITS_PER_SEG * cap + 32 + 31) / 32 * 32);
    q.pool_slots = std::max((int64_t)pk::POOL_PER_SEG * cap, pk::POOL_MIN);
    size_t o = L.fixed;
    q.frames = o;
    o = align_up(o + (size_t)q.n_frames * pk::FRAME_WORDS * sizeof(int32_t));
    q.bits = o;
    o = align_up(o + (size_t)(q.n_bits / 32) * sizeof(uint32_t));
    q.seg = o;
    o = align_up(o + (size_t)cap * sizeof(pk::SegRec));
    q.slots = o;
    q.pool_base = (int64_t)pk::GATHER_SLOTS * cap;
    q.end = o + (size_t)(q.pool_base + q.pool_slots) * sizeof(uint32_t);
    return q;
}

/* Segments a workspace of `bytes` can hold for n rows (the bytes needed grow
 * with the capacity, so the largest one that fits is found by bisection). */
int64_t capacity_for(int64_t n, size_t bytes)
{
    const Layout L = layout_for(n);
    if (cap_sections(L, 1).end > bytes) return 0;
    int64_t lo = 1, hi = MAX_SEGMENTS + 1; /* cap_sections(lo) fits, hi does not (or is past the maximum) */
    while (hi - lo > 1) {
        const int64_t mid = lo + (hi - lo) / 2;
        if (cap_sections(L, mid).end <= bytes) lo = mid;
        else hi = mid;
    }
    return lo;
}

/* Upper bound of the number of segments of rows whose lengths add up to total. */
int64_t segment_bound(int64_t n, int64_t total)
{
    /* a row of len tokens covers at most (len + 6) / 4 + 1 vectors */
    return (total + 7 * n) / (4 * pk::SEG_VEC) + 2 * n + 1;
}


/* The first shift pair (a < b) whose slot function separates the twelve ids;
 * tm.hashed stays 0 when none does (the scan then compares with all twelve). */
void find_tag_hash(pk::TagMatch &tm)
{
    for (int a = 0; a < 32; ++a) {
        for (int b = a + 1; b < 32; ++b) {
            uint64_t used = 0;
            int32_t slot[12];
            bool ok = true;
            for (int i = 0; i < 12 && ok; ++i) {
                const uint32_t u = (uint32_t)tm.ids[i];
                slot[i] = (int32_t)(((u >> a) ^ (u >> b)) & (uint32_t)(pk::TAG_SLOTS - 1));
                ok = !((used >> slot[i]) & 1u);
                used |= (uint64_t)1 << slot[i];
            }
            if (!ok) continue;
            tm.hashed = 1;
            tm.hash_a = a;
            tm.hash_b = b;
            /* an empty slot holds an id of another slot: no token of this slot equals it */
            for (int s = 0; s < pk::TAG_SLOTS; ++s) tm.slot_id[s] = s == slot[0] ? tm.ids[1] : tm.ids[0];
            for (int i = 0; i < 12; ++i) tm.slot_id[slot[i]] = tm.ids[i];
            return;
        }
    }
}

/* The tiers of the row automaton, in the grammar's strict or lenient form.
 * The deep tier is a launch of its own only when deep_launch is set (the
 * batch-wide statistics need every row first); otherwise group_reward runs
 * it. */
/* A small batch (fewer rows than ROWS_WAVES_PER_CU waves on every CU, with
 * two rows per wave) takes rows_par, one wave per row. */
bool rows_par_batch(int64_t n, int cus) { return n / 2 < (int64_t)cus * ROWS_WAVES_PER_CU; }

template <bool LENIENT>
void launch_rows(const pk::RowArgs &ra, const pk::GatherArgs &ga, int cus, uint8_t *mode, int32_t *counters,
                 int32_t *mid_rows, int32_t *deep_rows, int32_t *deep_frames, uint32_t *deep_bits, bool deep_launch,
                 hipStream_t stream)
{
    /* A small batch (fewer rows than ROWS_WAVES_PER_CU waves on every CU):
     * rows_par, one wave per row, its lanes over the row's events.  A larger
     * one: rows_fast, one row per lane, with as many rows per wave as keep
     * ROWS_WAVES_PER_CU waves on every CU (64 once the batch is large). */
    int64_t per_wave = 1;
    int32_t lane_shift = 6; /* log2(64 / per_wave) */
    /* per_wave stays 1 exactly when rows_par_batch(ra.n, cus) */
    while (per_wave < 64 && ra.n / (per_wave * 2) >= (int64_t)cus * ROWS_WAVES_PER_CU) {
        per_wave *= 2;
        --lane_shift;
    }
    const unsigned row_blocks = (unsigned)((ra.n + per_wave - 1) / per_wave);
    if (per_wave == 1) {
        /* rows_par runs the rows it does not hold through the automaton
         * itself (the second tier), so rows_mid has nothing to do */
        hipLaunchKernelGGL(pk::rows_par<LENIENT>, dim3(row_blocks), dim3(64), 0, stream, ra, mode, counters, deep_rows);
    } else {
        /* the per-lane automaton reads split rows best as compact lists */
        hipLaunchKernelGGL(pk::gather_rows, dim3((unsigned)(cus * GATHER_BLOCKS_PER_CU)), dim3(256), 0, stream, ga);
        hipLaunchKernelGGL(pk::rows_fast<LENIENT>, dim3(row_blocks), dim3(64), 0, stream, ra, mode, counters, mid_rows,
                           lane_shift);
        hipLaunchKernelGGL(pk::rows_mid<LENIENT>, dim3((unsigned)(cus * MID_BLOCKS_PER_CU)), dim3(64), 0, stream, ra,
                           mode, counters, mid_rows, deep_rows);
    }
    if (deep_launch)
        hipLaunchKernelGGL(pk::rows_deep<LENIENT>, dim3(1), dim3(64), 0, stream, ra, mode, counters, deep_rows,
                           deep_frames, deep_bits);
}

/* The scan's persistent grid: SCAN_BLOCKS_PER_CU blocks of SCAN_WAVES waves
 * per CU, or the same waves in blocks of scan_waves<PLAN>(). */
template <bool PLAN>
void launch_scan(const pk::TagMatch &tm, const pk::ScanArgs &sa, int cus, hipStream_t stream)
{
    constexpr int NW = pk::scan_waves<PLAN>();
    static_assert(SCAN_BLOCKS_PER_CU * pk::SCAN_WAVES % NW == 0, "whole blocks per CU");
    const dim3 grid((unsigned)(cus * (SCAN_BLOCKS_PER_CU * pk::SCAN_WAVES / NW))), block(pk::WAVE * NW);
    if (tm.contiguous)
        hipLaunchKernelGGL((pk::scan_rows<pk::TM_CONTIG, PLAN>), grid, block, 0, stream, sa);
    else if (tm.hashed)
        hipLaunchKernelGGL((pk::scan_rows<pk::TM_HASH, PLAN>), grid, block, 0, stream, sa);
    else
        hipLaunchKernelGGL((pk::scan_rows<pk::TM_LINEAR, PLAN>), grid, block, 0, stream, sa);
}

}  // namespace

void abi::launch_plan(const int64_t *starts, const int32_t *lengths, int64_t n, int64_t mis, int64_t n_tiles,
                      int64_t *tile_sum, int64_t *tile_off, int64_t *seg_off, int32_t *counters, uint8_t *mode,
                      hipStream_t stream)
{
    const unsigned tiles = (unsigned)n_tiles;
    if (n_tiles == 1) {
        hipLaunchKernelGGL(pk::plan_rows<true>, dim3(1), dim3(pk::PLAN_THREADS), 0, stream, starts, lengths, n, mis,
                           nullptr, seg_off, mode, counters);
        return;
    }
    hipLaunchKernelGGL(pk::plan_tiles, dim3(tiles), dim3(pk::PLAN_THREADS), 0, stream, starts, lengths, n, mis,
                       tile_sum);
    hipLaunchKernelGGL(pk::plan_top, dim3(1), dim3(1024), 0, stream, tile_sum, n_tiles, tile_off, seg_off, n, counters);
    hipLaunchKernelGGL(pk::plan_rows<false>, dim3(tiles), dim3(pk::PLAN_THREADS), 0, stream, starts, lengths, n, mis,
                       tile_off, seg_off, mode, counters);
}

extern "C" {

const char *parason_strerror(int status)
{
    switch (status) {
    case PARASON_OK: return "ok";
    case PARASON_ERR_NULL: return "a required pointer argument is NULL";
    case PARASON_ERR_SIZE: return "negative or too large size argument";
    case PARASON_ERR_GROUP: return "group_size < 1 or n_traj is not a multiple of group_size";
    case PARASON_ERR_WORKSPACE: return "workspace smaller than parason_workspace_size";
    case PARASON_ERR_TAGS: return "tag ids must be distinct and non-negative";
    case PARASON_ERR_PARAM: return "a reward parameter is not finite";
    case PARASON_ERR_ALIGN: return "tokens must be 4-byte aligned and the workspace 256-byte aligned";
    case PARASON_ERR_HIP: return "a HIP call or kernel launch failed";
    case PARASON_ERR_DEVICE: return "the current HIP device is not a gfx950 GPU or cannot be queried";
    case PARASON_ERR_SCRATCH:
        return "the batch needs more scratch than parason_run_noalloc's static buffer holds "
               "(PARASON_NOALLOC_SCRATCH_BYTES); use parason_run with a workspace";
    default: return "unknown status";
    }
}

int parason_create(const parason_config *cfg, parason_handle **out)
{
    if (!cfg || !out) return PARASON_ERR_NULL;
    *out = nullptr;
    if (cfg->group_size < 1) return PARASON_ERR_GROUP;
    for (int i = 0; i < 12; ++i) {
        if (cfg->tag_ids[i] < 0) return PARASON_ERR_TAGS;
        for (int j = 0; j < i; ++j)
            if (cfg->tag_ids[i] == cfg->tag_ids[j]) return PARASON_ERR_TAGS;
    }
    if (!is_finite(cfg->alpha) || !is_finite(cfg->beta_subtask) || !is_finite(cfg->beta_trial) || !is_finite(cfg->rho) ||
        !is_finite(cfg->rho_clip))
        return PARASON_ERR_PARAM;

    parason_handle *h = new (std::nothrow) parason_handle;
    if (!h) return PARASON_ERR_NULL;
    h->cfg = *cfg;
    std::memset(&h->tm, 0, sizeof(h->tm));
    int32_t lo = cfg->tag_ids[0], hi = cfg->tag_ids[0];
    for (int i = 0; i < 12; ++i) {
        h->tm.ids[i] = cfg->tag_ids[i];
        lo = cfg->tag_ids[i] < lo ? cfg->tag_ids[i] : lo;
        hi = cfg->tag_ids[i] > hi ? cfg->tag_ids[i] : hi;
    }
    /* twelve distinct ids spanning 12 values: a permutation of [lo, lo + 12) */
    h->tm.contiguous = (int64_t)hi - (int64_t)lo == 11;
    h->tm.base = lo;
    if (h->tm.contiguous) {
        for (int i = 0; i < 12; ++i) {
            uint32_t o = (uint32_t)(cfg->tag_ids[i] - lo), c = (uint32_t)(i + 1);
            if (o < 8) h->tm.lut_lo |= c << (4 * o);
            else h->tm.lut_hi |= c << (4 * (o - 8));
        }
    } else if (!(cfg->flags & PARASON_CFG_TAG_COMPARE)) {
        find_tag_hash(h->tm);
    }
    *out = h;
    return PARASON_OK;
}

void parason_destroy(parason_handle *h) { delete h; }

int parason_workspace_size(const parason_handle *h, int64_t n_traj, int64_t total_tokens, size_t *bytes)
{
    if (!h || !bytes) return PARASON_ERR_NULL;
    if (n_traj < 0 || total_tokens < 0 || n_traj > INT32_MAX) return PARASON_ERR_SIZE;
    int64_t segs = segment_bound(n_traj, total_tokens);
    if (segs > MAX_SEGMENTS) return PARASON_ERR_SIZE;
    *bytes = cap_sections(layout_for(n_traj), segs).end;
    return PARASON_OK;
}

int parason_run_timed(const parason_handle *h, const int32_t *tokens, const int64_t *starts, const int32_t *lengths,
                      const uint8_t *correct, int64_t n_traj, const parason_outputs *out, void *workspace,
                      size_t workspace_bytes, void *stream_ptr, void *const *scan_events)
{
    if (!h || !out) return PARASON_ERR_NULL;
    if (n_traj < 0 || n_traj > INT32_MAX) return PARASON_ERR_SIZE;
    const int32_t G = h->cfg.group_size;
    if (n_traj % G != 0) return PARASON_ERR_GROUP;
    if (n_traj == 0) return PARASON_OK;
    if (!tokens || !starts || !lengths || !correct || !workspace) return PARASON_ERR_NULL;
    if (!out->total || !out->latency || !out->n_subtask || !out->n_trial || !out->n_blocks || !out->max_depth ||
        !out->first_error_pos || !out->flags || !out->reward)
        return PARASON_ERR_NULL;
    if (((uintptr_t)tokens & 3u) != 0 || ((uintptr_t)workspace & (ALIGN - 1)) != 0) return PARASON_ERR_ALIGN;
    const int64_t cap = capacity_for(n_traj, workspace_bytes);
    if (cap < 1) return PARASON_ERR_WORKSPACE;

    const int cus = cu_count();
    if (cus <= 0) return PARASON_ERR_DEVICE;
    hipStream_t stream = (hipStream_t)stream_ptr;

    /* The scan reads 16-byte vectors on the 16-byte grid below `tokens`. */
    const int64_t mis = (int64_t)(((uintptr_t)tokens & 15u) >> 2);
    const int32_t *tok_base = tokens - mis;

    Layout L = layout_for(n_traj);
    char *ws = (char *)workspace;
    int64_t *seg_off = (int64_t *)(ws + L.seg_off);
    int64_t *tile_sum = (int64_t *)(ws + L.tile_sum);
    int64_t *tile_off = (int64_t *)(ws + L.tile_off);
    int32_t *counters = (int32_t *)(ws + L.counters);
    uint8_t *mode = (uint8_t *)(ws + L.mode);
    int32_t *mid_rows = (int32_t *)(ws + L.mid_rows);
    int32_t *deep_rows = (int32_t *)(ws + L.deep_rows);
    int32_t *split_rows = (int32_t *)(ws + L.split_rows);
    double *red_d = (double *)(ws + L.red_d);
    int64_t *red_i = (int64_t *)(ws + L.red_i);
    pk::BatchStats *stats = (pk::BatchStats *)(ws + L.stats);
    const CapSections q = cap_sections(L, cap);
    int32_t *deep_frames = (int32_t *)(ws + q.frames);
    uint32_t *deep_bits = (uint32_t *)(ws + q.bits);
    pk::SegRec *seg = (pk::SegRec *)(ws + q.seg);
    uint32_t *slots = (uint32_t *)(ws + q.slots);

    const unsigned tiles = (unsigned)L.n_tiles;
    /* a batch that takes rows_par and fits one scan block's plan is planned
     * by the scan blocks themselves (one launch less, and the scan waves find
     * their rows in LDS) */
    const bool plan_in_scan = n_traj <= pk::SCAN_PLAN_ROWS && rows_par_batch(n_traj, cus);
    if (!plan_in_scan)
        abi::launch_plan(starts, lengths, n_traj, mis, L.n_tiles, tile_sum, tile_off, seg_off, counters, mode, stream);

    const pk::RowOut row_out{out->total,    out->latency,   out->n_subtask,       out->n_trial,
                             out->n_blocks, out->max_depth, out->first_error_pos, out->flags};
    pk::ScanArgs sa;
    sa.tok_base = tok_base;
    sa.mis = mis;
    sa.starts = starts;
    sa.lengths = lengths;
    sa.n = n_traj;
    sa.seg_off = seg_off;
    sa.seg_cap = cap;
    sa.seg = seg;
    sa.slots = slots;
    sa.pool_base = (uint32_t)q.pool_base;
    sa.pool_slots = (uint32_t)q.pool_slots;
    sa.mode = mode;
    sa.tm = h->tm;
    sa.split_count = counters + 2;
    sa.split_rows = split_rows;
    sa.counters = counters;
    if (scan_events && hipEventRecord((hipEvent_t)scan_events[0], stream) != hipSuccess) return PARASON_ERR_HIP;
    if (plan_in_scan)
        launch_scan<true>(h->tm, sa, cus, stream);
    else
        launch_scan<false>(h->tm, sa, cus, stream);
    if (scan_events && hipEventRecord((hipEvent_t)scan_events[1], stream) != hipSuccess) return PARASON_ERR_HIP;

    pk::RowArgs ra;
    ra.tok_base = tok_base;
    ra.mis = mis;
    ra.starts = starts;
    ra.lengths = lengths;
    ra.n = n_traj;
    ra.seg_off = seg_off;
    ra.seg_cap = cap;
    ra.seg = seg;
    ra.slots = slots;
    ra.deep_frames = q.n_frames;
    ra.deep_bits = q.n_bits;
    ra.tm = h->tm;
    ra.out = row_out;
    const pk::GatherArgs ga{starts, n_traj, mis, seg_off, cap, seg, slots, mode, counters + 2, split_rows};
    const bool lenient = (h->cfg.flags & PARASON_CFG_LENIENT_GAPS) != 0;
    const bool batch_stats = (h->cfg.flags & PARASON_CFG_BATCH_STATS) != 0;
    if (lenient)
        launch_rows<true>(ra, ga, cus, mode, counters, mid_rows, deep_rows, deep_frames, deep_bits, batch_stats,
                          stream);
    else
        launch_rows<false>(ra, ga, cus, mode, counters, mid_rows, deep_rows, deep_frames, deep_bits, batch_stats,
                           stream);

    pk::RewardArgs rw;
    rw.total = out->total;
    rw.latency = out->latency;
    rw.n_subtask = out->n_subtask;
    rw.n_trial = out->n_trial;
    rw.flags = out->flags;
    rw.correct = correct;
    rw.n_groups = n_traj / G;
    rw.G = G;
    rw.alpha = h->cfg.alpha;
    rw.beta_s = h->cfg.beta_subtask;
    rw.beta_r = h->cfg.beta_trial;
    rw.rho = h->cfg.rho;
    rw.rho_clip = h->cfg.rho_clip;
    rw.cfg_flags = h->cfg.flags;
    rw.reward = out->reward;
    rw.r_subtask = out->r_subtask;
    rw.r_trial = out->r_trial;
    rw.eta = out->eta;
    rw.accel = out->accel;
    rw.saved = out->saved;
    rw.batch = nullptr;
    rw.n = n_traj;
    if (batch_stats) {
        pk::StatsArgs st{out->total, out->latency, out->n_subtask, out->n_trial, out->flags, n_traj, red_d, red_i, stats};
        hipLaunchKernelGGL(pk::batch_stats_tiles<1>, dim3(tiles), dim3(pk::RED_THREADS), 0, stream, st);
        hipLaunchKernelGGL(pk::batch_stats_final<1>, dim3(1), dim3(pk::RED_THREADS), 0, stream, st, L.n_tiles);
        hipLaunchKernelGGL(pk::batch_stats_tiles<2>, dim3(tiles), dim3(pk::RED_THREADS), 0, stream, st);
        hipLaunchKernelGGL(pk::batch_stats_final<2>, dim3(1), dim3(pk::RED_THREADS), 0, stream, st, L.n_tiles);
        rw.batch = stats;
        hipLaunchKernelGGL(pk::batch_reward, dim3((unsigned)((n_traj + 255) / 256)), dim3(256), 0, stream, rw);
    } else {
        const pk::DeepArgs da{ra, mode, counters, deep_rows, deep_frames, deep_bits};
        const dim3 grid((unsigned)((n_traj + 255) / 256));
        if (lenient) hipLaunchKernelGGL(pk::group_reward<true>, grid, dim3(256), 0, stream, rw, da);
        else hipLaunchKernelGGL(pk::group_reward<false>, grid, dim3(256), 0, stream, rw, da);
    }
    if (out->metrics) {
        pk::MetricsArgs ma{out->total, out->latency, out->n_subtask, out->n_trial, out->flags, correct,
                           out->reward, n_traj, red_i, red_d, out->metrics};
        hipLaunchKernelGGL(pk::metrics_tiles, dim3(tiles), dim3(pk::RED_THREADS), 0, stream, ma);
        hipLaunchKernelGGL(pk::metrics_final, dim3(1), dim3(pk::RED_THREADS), 0, stream, ma, L.n_tiles);
    }

    return hipGetLastError() == hipSuccess ? PARASON_OK : PARASON_ERR_HIP;
}

int parason_run(const parason_handle *h, const int32_t *tokens, const int64_t *starts, const int32_t *lengths,
                const uint8_t *correct, int64_t n_traj, const parason_outputs *out, void *workspace,
                size_t workspace_bytes, void *stream)
{
    return parason_run_timed(h, tokens, starts, lengths, correct, n_traj, out, workspace, workspace_bytes, stream,
                             nullptr);
}

/* The scratch of parason_run_noalloc: one static array per GPU the library
 * runs on, held until the process ends.  Host code never uses its name as an
 * address (on the host it is a stand-in symbol); each device's address comes
 * from hipGetSymbolAddress, once per device, with that device current. */
static __device__ __align__(256) unsigned char scratch[PARASON_NOALLOC_SCRATCH_BYTES];

namespace {
std::atomic<void *> scratch_ptr[64];

/* This device's address of `scratch`, or nullptr if it cannot be had. */
void *scratch_for_current_device()
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
    void *p = scratch_ptr[dev].load(std::memory_order_acquire);
    if (p) return p;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
    scratch_ptr[dev].store(p, std::memory_order_release);
    return p;
}

/* The chunk counter of parason_read_probe, one per GPU (probes on one GPU
 * must not overlap); its address is had as the scratch's is. */
static __device__ int32_t probe_next;
std::atomic<int32_t *> probe_ptr[64];

int32_t *probe_counter_for_current_device()
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
    int32_t *p = probe_ptr[dev].load(std::memory_order_acquire);
    if (p) return p;
    void *q = nullptr;
    if (hipGetSymbolAddress(&q, HIP_SYMBOL(probe_next)) != hipSuccess || !q) return nullptr;
    probe_ptr[dev].store((int32_t *)q, std::memory_order_release);
    return (int32_t *)q;
}
}  // namespace

int parason_run_noalloc(const parason_handle *h, const int32_t *tokens, const int64_t *starts, const int32_t *lengths,
                        const uint8_t *correct, int64_t n_traj, int64_t total_tokens, const parason_outputs *out,
                        void *stream)
{
    if (!h || !out) return PARASON_ERR_NULL;
    if (n_traj < 0 || n_traj > INT32_MAX || total_tokens < 0) return PARASON_ERR_SIZE;
    if (n_traj % h->cfg.group_size != 0) return PARASON_ERR_GROUP;
    if (n_traj == 0) return PARASON_OK;
    size_t need = 0;
    const int rc = parason_workspace_size(h, n_traj, total_tokens, &need);
    if (rc != PARASON_OK) return rc;
    if (need > (size_t)PARASON_NOALLOC_SCRATCH_BYTES) return PARASON_ERR_SCRATCH;
    if (cu_count() <= 0) return PARASON_ERR_DEVICE;
    void *ws = scratch_for_current_device();
    if (!ws) return PARASON_ERR_HIP;
    /* parason_run needs no initialised workspace: its first launch clears
     * what must start at zero, so nothing here writes to the scratch */
    return parason_run_timed(h, tokens, starts, lengths, correct, n_traj, out, ws,
                             (size_t)PARASON_NOALLOC_SCRATCH_BYTES, stream, nullptr);
}

int parason_read_probe(const void *data, size_t bytes, uint32_t *sink, int64_t sink_len, void *stream_ptr)
{
    if (bytes == 0) return PARASON_OK;
    if (!data || !sink) return PARASON_ERR_NULL;
    if (sink_len < 1 || (bytes & 3u) != 0) return PARASON_ERR_SIZE;
    if (((uintptr_t)data & 15u) != 0 || ((uintptr_t)sink & 3u) != 0) return PARASON_ERR_ALIGN;
    const int cus = cu_count();
    if (cus <= 0) return PARASON_ERR_DEVICE;
    const int64_t n_vec = (int64_t)(bytes / 16);
    const int32_t n_tail = (int32_t)((bytes % 16) / 4);
    const int32_t *tail = (const int32_t *)((const char *)data + (size_t)n_vec * 16);
    int32_t *next = probe_counter_for_current_device();
    if (!next) return PARASON_ERR_HIP;
    hipLaunchKernelGGL(pk::probe_reset, dim3(1), dim3(1), 0, (hipStream_t)stream_ptr, next);
    hipLaunchKernelGGL(pk::read_probe, dim3((unsigned)(cus * SCAN_BLOCKS_PER_CU)), dim3(pk::WAVE * pk::SCAN_WAVES), 0,
                       (hipStream_t)stream_ptr, (const int4 *)data, n_vec, tail, n_tail, sink, sink_len, next);
    return hipGetLastError() == hipSuccess ? PARASON_OK : PARASON_ERR_HIP;
}

}  // extern "C"
