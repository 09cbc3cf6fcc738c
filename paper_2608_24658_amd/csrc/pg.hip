/*
 * pg.hip -- C-ABI of the policy-gradient step (kernels in pg_kernels.h).
 */
#include "abi_common.h"
#include "pg_kernels.h"

using abi::ALIGN;
using abi::align_up;
using abi::cu_count;
using abi::is_finite;

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

extern "C" {

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
    abi::launch_plan(starts, lengths, n_traj, mis, L.n_tiles, tile_sum, tile_off, seg_off, counters, mode, stream);
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

}  // extern "C"
