/*
 * fork.hip -- C-ABI of fork/join packing for tool-call execution (kernels in
 * fork_kernels.h).
 *
 * Launches use hipLaunchKernelGGL, as in parason.hip, so that the same source
 * also compiles against a host-side stand-in for the HIP runtime.
 */
#include <algorithm>

#include "abi_common.h"
#include "fork_kernels.h"

using abi::align_up;
using abi::cu_count;

namespace {

constexpr int COPY_BLOCKS_PER_CU = 8;

/* Workspace of fork (K = 3 counts per row: workers, context tokens, copy
 * units) or join (K = 1). */
struct PackLayout {
    size_t counts, outl, tile_sum, tile_off, tok_off, unit_off, summ, over, end;
    int64_t tiles;
};

PackLayout pack_layout(int64_t n, int K)
{
    PackLayout L;
    L.tiles = n > 0 ? (n + pk::PACK_TILE - 1) / pk::PACK_TILE : 1;
    size_t o = 0;
    L.counts = o;
    o = align_up(o + (size_t)(n > 0 ? n : 1) * K * sizeof(int64_t));
    L.outl = o;
    o = align_up(o + (size_t)(n > 0 ? n : 1) * sizeof(int32_t));
    L.tile_sum = o;
    o = align_up(o + (size_t)L.tiles * K * sizeof(int64_t));
    L.tile_off = o;
    o = align_up(o + (size_t)L.tiles * K * sizeof(int64_t));
    L.tok_off = o;
    o = align_up(o + (size_t)(n + 1) * sizeof(int64_t));
    L.unit_off = o;
    if (K == 3) o = align_up(o + (size_t)(n + 1) * sizeof(int64_t));
    L.summ = o;
    if (K == 3) o = align_up(o + (size_t)(n > 0 ? n : 1) * pk::SUMM_ENTRIES * sizeof(uint64_t));
    L.over = o;
    o = align_up(o + sizeof(int32_t));
    L.end = o;
    return L;
}

bool aligned(const void *p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

/* Exclusive scans of the per-row counts: one block when the rows fit one tile
 * (pack_single; also n = 0, which only writes the zero totals), otherwise tile
 * sums, their scan and the per-row offsets. */
template <int K>
void launch_pack(const pk::PackScan<K> &ps, int64_t tiles, hipStream_t stream)
{
    if (ps.n <= pk::PACK_TILE) {
        hipLaunchKernelGGL(pk::pack_single<K>, dim3(1), dim3(pk::PACK_THREADS), 0, stream, ps);
        return;
    }
    hipLaunchKernelGGL(pk::pack_tiles<K>, dim3((unsigned)tiles), dim3(pk::PACK_THREADS), 0, stream, ps);
    hipLaunchKernelGGL(pk::pack_top<K>, dim3(1), dim3(1024), 0, stream, ps, tiles);
    hipLaunchKernelGGL(pk::pack_rows<K>, dim3((unsigned)tiles), dim3(pk::PACK_THREADS), 0, stream, ps);
}

}  // namespace

extern "C" {

int parason_fork_workspace_size(int64_t n_rows, size_t *bytes)
{
    if (!bytes) return PARASON_ERR_NULL;
    if (n_rows < 0 || n_rows > INT32_MAX) return PARASON_ERR_SIZE;
    *bytes = pack_layout(n_rows, 3).end;
    return PARASON_OK;
}

int parason_join_workspace_size(int64_t n_rows, size_t *bytes)
{
    if (!bytes) return PARASON_ERR_NULL;
    if (n_rows < 0 || n_rows > INT32_MAX) return PARASON_ERR_SIZE;
    *bytes = pack_layout(n_rows, 1).end;
    return PARASON_OK;
}

int parason_fork(const parason_handle *h, const int32_t *tokens, const int64_t *starts, const int32_t *lengths,
                 int64_t n_rows, uint32_t flags, const parason_fork_outputs *out, void *workspace,
                 size_t workspace_bytes, void *stream_ptr)
{
    if (!h || !out) return PARASON_ERR_NULL;
    if (n_rows < 0 || n_rows > INT32_MAX || out->max_workers < 0 || out->ctx_capacity < 0) return PARASON_ERR_SIZE;
    if (flags & ~(uint32_t)PARASON_FORK_SEED_ENTRY) return PARASON_ERR_PARAM;
    if (!out->worker_off || !out->totals || !workspace) return PARASON_ERR_NULL;
    if (n_rows > 0 && (!tokens || !starts || !lengths || !out->row_status)) return PARASON_ERR_NULL;
    if (out->max_workers > 0 &&
        (!out->ctx_starts || !out->ctx_lengths || !out->ctx_row || !out->ctx_entry || !out->ctx_kind))
        return PARASON_ERR_NULL;
    if (out->ctx_capacity > 0 && !out->ctx_tokens) return PARASON_ERR_NULL;
    if ((tokens && !aligned(tokens, 4)) || !aligned(workspace, abi::ALIGN)) return PARASON_ERR_ALIGN;
    const PackLayout L = pack_layout(n_rows, 3);
    if (workspace_bytes < L.end) return PARASON_ERR_WORKSPACE;
    const int cus = cu_count();
    if (cus <= 0) return PARASON_ERR_DEVICE;
    hipStream_t stream = (hipStream_t)stream_ptr;
    char *ws = (char *)workspace;

    pk::ForkArgs fa;
    fa.tokens = tokens;
    fa.starts = starts;
    fa.lengths = lengths;
    fa.n = n_rows;
    fa.tm = h->tm;
    fa.seed = (flags & PARASON_FORK_SEED_ENTRY) != 0;
    fa.lenient = (h->cfg.flags & PARASON_CFG_LENIENT_GAPS) != 0;
    fa.thread_id = h->cfg.tag_ids[pk::C_THR - 1];
    fa.status = out->row_status;
    fa.counts = (int64_t *)(ws + L.counts);
    fa.outl = (int32_t *)(ws + L.outl);
    fa.worker_off = out->worker_off;
    fa.tok_off = (const int64_t *)(ws + L.tok_off);
    fa.unit_off = (const int64_t *)(ws + L.unit_off);
    fa.summ = (uint64_t *)(ws + L.summ);
    fa.over = (const int32_t *)(ws + L.over);
    fa.ctx_starts = out->ctx_starts;
    fa.ctx_lengths = out->ctx_lengths;
    fa.ctx_row = out->ctx_row;
    fa.ctx_entry = out->ctx_entry;
    fa.ctx_kind = out->ctx_kind;
    fa.ctx_tokens = out->ctx_tokens;

    pk::PackScan<3> ps;
    ps.vals = fa.counts;
    ps.n = n_rows;
    ps.tile_sum = (int64_t *)(ws + L.tile_sum);
    ps.tile_off = (int64_t *)(ws + L.tile_off);
    ps.out[0] = out->worker_off;
    ps.out[1] = (int64_t *)(ws + L.tok_off);
    ps.out[2] = (int64_t *)(ws + L.unit_off);
    ps.cap[0] = out->max_workers;
    ps.cap[1] = out->ctx_capacity;
    ps.cap[2] = INT64_MAX; /* internal: never over */
    ps.totals = out->totals;
    ps.report = 2; /* totals = workers, context tokens, over */
    ps.over = (int32_t *)(ws + L.over);

    const unsigned wave_blocks = (unsigned)std::min<int64_t>((n_rows + pk::OUTLINE_WAVES - 1) / pk::OUTLINE_WAVES,
                                                             (int64_t)cus * (32 / pk::OUTLINE_WAVES));
    if (n_rows > 0) hipLaunchKernelGGL(pk::fork_outline<false>, dim3(wave_blocks), dim3(pk::OUTLINE_WAVES * pk::WAVE), 0, stream, fa);
    if (n_rows <= pk::FORK_SINGLE) {
        /* scans and records in one launch (at least one block: it writes the totals) */
        const unsigned blocks = (unsigned)std::max<int64_t>(1, (n_rows + pk::FORK_REC_WAVES - 1) / pk::FORK_REC_WAVES);
        hipLaunchKernelGGL(pk::fork_records, dim3(blocks), dim3(pk::FORK_REC_THREADS), 0, stream, fa, ps);
    } else {
        launch_pack(ps, L.tiles, stream);
        hipLaunchKernelGGL(pk::fork_outline<true>, dim3(wave_blocks), dim3(pk::OUTLINE_WAVES * pk::WAVE), 0, stream, fa);
    }
    if (n_rows > 0) {
        const unsigned copy_blocks = (unsigned)(cus * COPY_BLOCKS_PER_CU); /* persistent, tiled over the output */
        hipLaunchKernelGGL(pk::fork_copy, dim3(copy_blocks), dim3(pk::PACK_THREADS), 0, stream, fa);
    }
    return hipGetLastError() == hipSuccess ? PARASON_OK : PARASON_ERR_HIP;
}

int parason_join(const parason_handle *h, const int32_t *tokens, const int64_t *starts, const int32_t *lengths,
                 int64_t n_rows, const int64_t *worker_off, const int32_t *wtokens, const int64_t *wstarts,
                 const int32_t *wlengths, int64_t n_workers, uint32_t flags, const parason_join_outputs *out,
                 void *workspace, size_t workspace_bytes, void *stream_ptr)
{
    if (!h || !out) return PARASON_ERR_NULL;
    if (n_rows < 0 || n_rows > INT32_MAX || n_workers < 0 || out->capacity < 0) return PARASON_ERR_SIZE;
    if (flags & ~(uint32_t)(PARASON_JOIN_CLOSE_PARALLEL | PARASON_JOIN_APPEND_ONLY)) return PARASON_ERR_PARAM;
    if (!out->starts || !out->totals || !workspace) return PARASON_ERR_NULL;
    if (n_rows > 0 && (!tokens || !starts || !lengths || !worker_off || !out->lengths || !out->row_status))
        return PARASON_ERR_NULL;
    if (n_workers > 0 && (!wtokens || !wstarts || !wlengths)) return PARASON_ERR_NULL;
    if (out->capacity > 0 && !out->tokens) return PARASON_ERR_NULL;
    if ((tokens && !aligned(tokens, 4)) || (wtokens && !aligned(wtokens, 4)) || !aligned(workspace, abi::ALIGN))
        return PARASON_ERR_ALIGN;
    const PackLayout L = pack_layout(n_rows, 1);
    if (workspace_bytes < L.end) return PARASON_ERR_WORKSPACE;
    const int cus = cu_count();
    if (cus <= 0) return PARASON_ERR_DEVICE;
    hipStream_t stream = (hipStream_t)stream_ptr;
    char *ws = (char *)workspace;

    pk::JoinArgs ja;
    ja.tokens = tokens;
    ja.starts = starts;
    ja.lengths = lengths;
    ja.n = n_rows;
    ja.worker_off = worker_off;
    ja.n_workers = n_workers;
    ja.wtokens = wtokens;
    ja.wstarts = wstarts;
    ja.wlengths = wlengths;
    ja.thread_id = h->cfg.tag_ids[pk::C_THR - 1];
    ja.end_thread_id = h->cfg.tag_ids[pk::C_END_THR - 1];
    ja.end_par_id = h->cfg.tag_ids[pk::C_END_PAR - 1];
    ja.close = (flags & PARASON_JOIN_CLOSE_PARALLEL) != 0;
    ja.append_only = (flags & PARASON_JOIN_APPEND_ONLY) != 0;
    ja.status = out->row_status;
    ja.out_len64 = (int64_t *)(ws + L.counts);
    ja.out_lengths = out->lengths;
    ja.out_starts = out->starts;
    ja.over = (const int32_t *)(ws + L.over);
    ja.out_tokens = out->tokens;

    pk::PackScan<1> ps;
    ps.vals = ja.out_len64;
    ps.n = n_rows;
    ps.tile_sum = (int64_t *)(ws + L.tile_sum);
    ps.tile_off = (int64_t *)(ws + L.tile_off);
    ps.out[0] = out->starts;
    ps.cap[0] = out->capacity;
    ps.totals = out->totals;
    ps.report = 1;
    ps.over = (int32_t *)(ws + L.over);

    if (n_rows > 0) hipLaunchKernelGGL(pk::join_size, dim3((unsigned)((n_rows + pk::JOIN_SIZE_THREADS - 1) / pk::JOIN_SIZE_THREADS)),
                                       dim3(pk::JOIN_SIZE_THREADS), 0, stream, ja);
    const unsigned copy_blocks = n_rows > 0 ? (unsigned)(cus * COPY_BLOCKS_PER_CU) : 1u;
    if (n_rows <= pk::JOIN_SINGLE) {
        /* the scan inside the copy (no rows: one block, which writes the zero totals) */
        hipLaunchKernelGGL(pk::join_copy<true>, dim3(copy_blocks), dim3(pk::PACK_THREADS), 0, stream, ja, ps);
    } else {
        launch_pack(ps, L.tiles, stream);
        hipLaunchKernelGGL(pk::join_copy<false>, dim3(copy_blocks), dim3(pk::PACK_THREADS), 0, stream, ja, ps);
    }
    return hipGetLastError() == hipSuccess ? PARASON_OK : PARASON_ERR_HIP;
}

}  // extern "C"
