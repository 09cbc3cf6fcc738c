/*
 * parason.hip -- C-ABI of the Parason accounting/reward path for gfx950.
 * The kernels are in parason_kernels.h; this file validates arguments, lays
 * out the caller's workspace and enqueues the launches on the caller's stream.
 */
#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>
#include <cstring>
#include <new>

#include "parason.h"
#include "parason_kernels.h"
#include "pg_kernels.h"
#include "decode_kernels.h"

struct parason_handle {
    parason_config cfg;
    pk::TagMatch tm;
};

namespace {

constexpr size_t ALIGN = 256;
#ifndef PARASON_SCAN_BLOCKS_PER_CU
#define PARASON_SCAN_BLOCKS_PER_CU 4
#endif
constexpr int SCAN_BLOCKS_PER_CU = PARASON_SCAN_BLOCKS_PER_CU; /* persistent grid of 4-wave blocks */
constexpr int64_t MAX_SEGMENTS = (int64_t)1 << 40;

size_t align_up(size_t x) { return (x + ALIGN - 1) / ALIGN * ALIGN; }

/* Byte offsets of the workspace sections for n rows. */
struct Layout {
    size_t seg_off, tile_sum, tile_off, counters, mode, deep_rows, deep_frames, deep_bits, seg_count, events;
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
    L.deep_rows = o;
    o = align_up(o + (size_t)(n > 0 ? n : 1) * sizeof(int32_t));
    L.deep_frames = o;
    o = align_up(o + (size_t)pk::DEEP_FRAMES * pk::FRAME_WORDS * sizeof(int32_t));
    L.deep_bits = o;
    o = align_up(o + (size_t)(pk::DEEP_ENTRY_BITS / 32) * sizeof(uint32_t));
    /* partial sums of the batch reductions (one record per 4096 rows) */
    L.red_d = o;
    o = align_up(o + (size_t)L.n_tiles * 3 * sizeof(double));
    L.red_i = o;
    o = align_up(o + (size_t)L.n_tiles * pk::NMI * sizeof(int64_t));
    L.stats = o;
    o = align_up(o + sizeof(pk::BatchStats));
    L.fixed = o;
    L.seg_count = o;
    L.events = 0; /* depends on the capacity */
    return L;
}

constexpr size_t PER_SEGMENT = sizeof(int32_t) + (size_t)pk::EV_CAP * sizeof(uint32_t);

/* Segments a workspace of `bytes` can hold for n rows. */
int64_t capacity_for(int64_t n, size_t bytes)
{
    Layout L = layout_for(n);
    if (bytes < L.fixed + 2 * ALIGN) return 0;
    int64_t cap = (int64_t)((bytes - L.fixed - 2 * ALIGN) / PER_SEGMENT);
    return cap < MAX_SEGMENTS ? cap : MAX_SEGMENTS;
}

/* Upper bound of the number of segments of rows whose lengths add up to total. */
int64_t segment_bound(int64_t n, int64_t total)
{
    /* a row of len tokens covers at most (len + 6) / 4 + 1 vectors */
    return (total + 7 * n) / (4 * pk::SEG_VEC) + 2 * n + 1;
}

int cu_count()
{
    static std::atomic<int> cached[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return -1;
    if (dev >= 0 && dev < 64) {
        int c = cached[dev].load(std::memory_order_relaxed);
        if (c > 0) return c;
    }
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) return -1;
    if (dev >= 0 && dev < 64) cached[dev].store(cus, std::memory_order_relaxed);
    return cus;
}

bool is_finite(double x) { return std::isfinite(x); }

}  // namespace

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
    case PARASON_ERR_DEVICE: return "no usable HIP device";
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
    Layout L = layout_for(n_traj);
    *bytes = L.fixed + 2 * ALIGN + (size_t)segs * PER_SEGMENT;
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
    int32_t *deep_rows = (int32_t *)(ws + L.deep_rows);
    int32_t *deep_frames = (int32_t *)(ws + L.deep_frames);
    uint32_t *deep_bits = (uint32_t *)(ws + L.deep_bits);
    int32_t *seg_count = (int32_t *)(ws + L.seg_count);
    double *red_d = (double *)(ws + L.red_d);
    int64_t *red_i = (int64_t *)(ws + L.red_i);
    pk::BatchStats *stats = (pk::BatchStats *)(ws + L.stats);
    uint32_t *events = (uint32_t *)(ws + align_up(L.seg_count + (size_t)cap * sizeof(int32_t)));

    const unsigned tiles = (unsigned)L.n_tiles;
    pk::plan_tiles<<<dim3(tiles), dim3(pk::PLAN_THREADS), 0, stream>>>(starts, lengths, n_traj, mis, tile_sum);
    pk::plan_top<<<dim3(1), dim3(1024), 0, stream>>>(tile_sum, L.n_tiles, tile_off, seg_off, n_traj, counters);
    pk::plan_rows<<<dim3(tiles), dim3(pk::PLAN_THREADS), 0, stream>>>(starts, lengths, n_traj, mis, tile_off,
                                                                        seg_off, mode);

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
    sa.seg_count = seg_count;
    sa.events = events;
    sa.mode = mode;
    sa.tm = h->tm;
    const unsigned scan_blocks = (unsigned)(cus * SCAN_BLOCKS_PER_CU);
    if (scan_events && hipEventRecord((hipEvent_t)scan_events[0], stream) != hipSuccess) return PARASON_ERR_HIP;
    if (h->tm.contiguous)
        pk::scan_rows<true><<<dim3(scan_blocks), dim3(pk::WAVE * pk::SCAN_WAVES), 0, stream>>>(sa);
    else
        pk::scan_rows<false><<<dim3(scan_blocks), dim3(pk::WAVE * pk::SCAN_WAVES), 0, stream>>>(sa);
    if (scan_events && hipEventRecord((hipEvent_t)scan_events[1], stream) != hipSuccess) return PARASON_ERR_HIP;

    pk::RowArgs ra;
    ra.tok_base = tok_base;
    ra.mis = mis;
    ra.starts = starts;
    ra.lengths = lengths;
    ra.n = n_traj;
    ra.seg_off = seg_off;
    ra.seg_cap = cap;
    ra.seg_count = seg_count;
    ra.events = events;
    ra.tm = h->tm;
    ra.out = row_out;
    const unsigned row_blocks = (unsigned)((n_traj + 63) / 64);
    pk::rows_fast<<<dim3(row_blocks), dim3(64), 0, stream>>>(ra, mode, counters, deep_rows);
    pk::rows_deep<<<dim3(1), dim3(64), 0, stream>>>(ra, mode, counters, deep_rows, deep_frames, deep_bits);

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
    rw.batch = nullptr;
    rw.n = n_traj;
    if (h->cfg.flags & PARASON_CFG_BATCH_STATS) {
        pk::StatsArgs st{out->total, out->latency, out->n_subtask, out->n_trial, out->flags, n_traj, red_d, red_i, stats};
        pk::batch_stats_tiles<1><<<dim3(tiles), dim3(pk::RED_THREADS), 0, stream>>>(st);
        pk::batch_stats_final<1><<<dim3(1), dim3(pk::RED_THREADS), 0, stream>>>(st, L.n_tiles);
        pk::batch_stats_tiles<2><<<dim3(tiles), dim3(pk::RED_THREADS), 0, stream>>>(st);
        pk::batch_stats_final<2><<<dim3(1), dim3(pk::RED_THREADS), 0, stream>>>(st, L.n_tiles);
        rw.batch = stats;
        pk::batch_reward<<<dim3((unsigned)((n_traj + 255) / 256)), dim3(256), 0, stream>>>(rw);
    } else {
        const unsigned reward_blocks = (unsigned)((rw.n_groups + 255) / 256);
        pk::group_reward<<<dim3(reward_blocks), dim3(256), 0, stream>>>(rw);
    }
    if (out->metrics) {
        pk::MetricsArgs ma{out->total, out->latency, out->n_subtask, out->n_trial, out->flags, correct,
                           out->reward, n_traj, red_i, red_d, out->metrics};
        pk::metrics_tiles<<<dim3(tiles), dim3(pk::RED_THREADS), 0, stream>>>(ma);
        pk::metrics_final<<<dim3(1), dim3(pk::RED_THREADS), 0, stream>>>(ma, L.n_tiles);
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

/* ---- policy-gradient step ---------------------------------------------- */

namespace {

constexpr int PG_BLOCKS_PER_CU = 4;
constexpr int64_t PG_MAX_WAVES = 1 << 16;

struct PgLayout {
    size_t seg_off, tile_sum, tile_off, counters, mode, len_part, n_tokens, wsum, wcnt, end;
    int64_t n_tiles;
};

PgLayout pg_layout_for(int64_t n)
{
    PgLayout L;
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
    L.len_part = o;
    o = align_up(o + (size_t)L.n_tiles * sizeof(int64_t));
    L.n_tokens = o;
    o = align_up(o + sizeof(int64_t));
    L.wsum = o;
    o = align_up(o + (size_t)PG_MAX_WAVES * sizeof(double));
    L.wcnt = o;
    o = align_up(o + (size_t)PG_MAX_WAVES * 2 * sizeof(int64_t));
    L.end = o;
    return L;
}

}  // namespace

int parason_pg_workspace_size(int64_t n_traj, size_t *bytes)
{
    if (!bytes) return PARASON_ERR_NULL;
    if (n_traj < 0 || n_traj > INT32_MAX) return PARASON_ERR_SIZE;
    *bytes = pg_layout_for(n_traj).end;
    return PARASON_OK;
}

int parason_pg_run(const parason_pg_config *cfg, const float *reward, const float *logp, const float *logp_old,
                   const int64_t *starts, const int32_t *lengths, int64_t n_traj, float *advantage, float *grad,
                   double *stats, void *workspace, size_t workspace_bytes, void *stream_ptr)
{
    if (!cfg) return PARASON_ERR_NULL;
    if (n_traj < 0 || n_traj > INT32_MAX) return PARASON_ERR_SIZE;
    if (cfg->group_size < 1 || n_traj % cfg->group_size != 0) return PARASON_ERR_GROUP;
    if (!is_finite(cfg->clip_low) || !is_finite(cfg->clip_high) || cfg->clip_low < 0.0 || cfg->clip_low >= 1.0 ||
        cfg->clip_high < 0.0)
        return PARASON_ERR_PARAM;
    if (n_traj == 0) return PARASON_OK;
    if (!reward || !logp || !logp_old || !starts || !lengths || !advantage || !grad || !stats || !workspace)
        return PARASON_ERR_NULL;
    const uintptr_t a0 = (uintptr_t)logp, a1 = (uintptr_t)logp_old, a2 = (uintptr_t)grad;
    if (((a0 | a1 | a2) & 3u) != 0 || (a0 & 15u) != (a1 & 15u) || (a0 & 15u) != (a2 & 15u) ||
        ((uintptr_t)workspace & (ALIGN - 1)) != 0)
        return PARASON_ERR_ALIGN;
    const PgLayout L = pg_layout_for(n_traj);
    if (workspace_bytes < L.end) return PARASON_ERR_WORKSPACE;
    const int cus = cu_count();
    if (cus <= 0) return PARASON_ERR_DEVICE;
    const int64_t waves = (int64_t)cus * PG_BLOCKS_PER_CU * 4;
    if (waves > PG_MAX_WAVES) return PARASON_ERR_DEVICE;
    hipStream_t stream = (hipStream_t)stream_ptr;

    const int64_t mis = (int64_t)((a0 & 15u) >> 2);
    char *ws = (char *)workspace;
    int64_t *seg_off = (int64_t *)(ws + L.seg_off);
    int64_t *tile_sum = (int64_t *)(ws + L.tile_sum);
    int64_t *tile_off = (int64_t *)(ws + L.tile_off);
    int32_t *counters = (int32_t *)(ws + L.counters);
    uint8_t *mode = (uint8_t *)(ws + L.mode);
    int64_t *len_part = (int64_t *)(ws + L.len_part);
    int64_t *n_tokens = (int64_t *)(ws + L.n_tokens);
    double *wsum = (double *)(ws + L.wsum);
    int64_t *wcnt = (int64_t *)(ws + L.wcnt);

    const unsigned tiles = (unsigned)L.n_tiles;
    pk::plan_tiles<<<dim3(tiles), dim3(pk::PLAN_THREADS), 0, stream>>>(starts, lengths, n_traj, mis, tile_sum);
    pk::plan_top<<<dim3(1), dim3(1024), 0, stream>>>(tile_sum, L.n_tiles, tile_off, seg_off, n_traj, counters);
    pk::plan_rows<<<dim3(tiles), dim3(pk::PLAN_THREADS), 0, stream>>>(starts, lengths, n_traj, mis, tile_off,
                                                                        seg_off, mode);
    pk::sum_lengths_tiles<<<dim3(tiles), dim3(pk::RED_THREADS), 0, stream>>>(lengths, n_traj, len_part);
    pk::sum_lengths_final<<<dim3(1), dim3(pk::RED_THREADS), 0, stream>>>(len_part, L.n_tiles, n_tokens);
    const int64_t n_groups = n_traj / cfg->group_size;
    pk::pg_advantage<<<dim3((unsigned)((n_groups + 255) / 256)), dim3(256), 0, stream>>>(reward, n_groups,
                                                                                          cfg->group_size, advantage);
    pk::PgArgs pa;
    pa.logp_base = logp - mis;
    pa.old_base = logp_old - mis;
    pa.grad_base = grad - mis;
    pa.mis = mis;
    pa.starts = starts;
    pa.lengths = lengths;
    pa.n = n_traj;
    pa.seg_off = seg_off;
    pa.adv = advantage;
    pa.thr_low = (float)std::log1p(-cfg->clip_low);
    pa.thr_high = (float)std::log1p(cfg->clip_high);
    pa.lo_val = (float)(1.0 - cfg->clip_low);
    pa.hi_val = (float)(1.0 + cfg->clip_high);
    pa.n_tokens = n_tokens;
    pa.wsum = wsum;
    pa.wcnt = wcnt;
    pk::pg_surrogate<<<dim3((unsigned)(cus * PG_BLOCKS_PER_CU)), dim3(256), 0, stream>>>(pa);
    pk::pg_final<<<dim3(1), dim3(pk::RED_THREADS), 0, stream>>>(wsum, wcnt, waves, n_tokens, stats);
    return hipGetLastError() == hipSuccess ? PARASON_OK : PARASON_ERR_HIP;
}

/* ---- grammar-constrained decode step ----------------------------------- */

static_assert(sizeof(parason_decode_state) == sizeof(pk::DecodeState), "decode state layout");
static_assert(sizeof(parason_decode_state) == 16, "decode state is 16 bytes");

namespace {
constexpr int DECODE_BLOCKS_PER_CU = 8;
}  // namespace

int parason_decode_init(parason_decode_state *states, int64_t batch, void *stream_ptr)
{
    if (batch < 0 || batch > INT32_MAX) return PARASON_ERR_SIZE;
    if (batch == 0) return PARASON_OK;
    if (!states) return PARASON_ERR_NULL;
    if (((uintptr_t)states & 15u) != 0) return PARASON_ERR_ALIGN;
    hipStream_t stream = (hipStream_t)stream_ptr;
    pk::decode_init<<<dim3((unsigned)((batch + 255) / 256)), dim3(256), 0, stream>>>(
        reinterpret_cast<pk::DecodeState *>(states), batch);
    return hipGetLastError() == hipSuccess ? PARASON_OK : PARASON_ERR_HIP;
}

int parason_decode_step(const parason_handle *h, parason_decode_state *states, const int32_t *tokens, int64_t batch,
                        void *logits, int64_t vocab, int64_t row_stride, int32_t dtype, int32_t eos_id,
                        void *stream_ptr)
{
    if (!h) return PARASON_ERR_NULL;
    if (batch < 0 || batch > INT32_MAX || vocab < 1 || vocab > INT32_MAX || row_stride < vocab) return PARASON_ERR_SIZE;
    int32_t elem = 0;
    uint32_t ninf = 0;
    switch (dtype) {
    case PARASON_DTYPE_F32: elem = 4, ninf = 0xFF800000u; break;
    case PARASON_DTYPE_BF16: elem = 2, ninf = 0xFF80u; break;
    case PARASON_DTYPE_F16: elem = 2, ninf = 0xFC00u; break;
    default: return PARASON_ERR_PARAM;
    }
    for (int i = 0; i < 12; ++i)
        if (h->tm.ids[i] >= vocab || h->tm.ids[i] == eos_id) return PARASON_ERR_TAGS;
    if (eos_id < -1 || eos_id >= vocab) return PARASON_ERR_TAGS;
    if (row_stride > INT64_MAX / 4 / (batch > 0 ? batch : 1)) return PARASON_ERR_SIZE;
    if (batch == 0) return PARASON_OK;
    if (!states || !logits) return PARASON_ERR_NULL;
    if (((uintptr_t)states & 15u) != 0 || ((uintptr_t)logits & (uintptr_t)(elem - 1)) != 0 ||
        (tokens && ((uintptr_t)tokens & 3u) != 0))
        return PARASON_ERR_ALIGN;
    const int cus = cu_count();
    if (cus <= 0) return PARASON_ERR_DEVICE;
    hipStream_t stream = (hipStream_t)stream_ptr;

    pk::DecodeArgs da;
    da.states = reinterpret_cast<pk::DecodeState *>(states);
    da.tokens = tokens;
    da.batch = batch;
    da.logits = (char *)logits;
    da.vocab = vocab;
    da.row_bytes = row_stride * elem;
    da.elem = elem;
    da.ninf = ninf;
    da.eos_id = eos_id;
    da.tm = h->tm;
    const int64_t max_blocks = (int64_t)cus * DECODE_BLOCKS_PER_CU;
    const unsigned blocks = (unsigned)(batch < max_blocks ? batch : max_blocks);
    pk::decode_step<<<dim3(blocks), dim3(256), 0, stream>>>(da);
    return hipGetLastError() == hipSuccess ? PARASON_OK : PARASON_ERR_HIP;
}

}  // extern "C"
