/*
 * fork_kernels.h -- gfx950 kernels of fork/join packing for tool-call
 * execution (Sec. 3.4 "Inference": the runtime decodes until an outline is
 * complete, dispatches each <Subtask> / <Trial> entry as a worker and returns
 * the workers' <Thread> outputs to the main trajectory; format of Figure 4).
 *
 * fork
 *   fork_outline<false>  one wave per row: checks that the row ends with
 *                        </Outlines>, searches backwards for the outline's
 *                        <Outlines> (512 tokens a step), then walks the
 *                        outline forwards in 256-token chunks (the next
 *                        chunk's loads in flight), compacting its tags in order with
 *                        ballots and checking each against the one before it
 *                        (entries open, hold text, close, back to back).
 *                        Writes the row's worker and token counts.
 *   pack_single, or      exclusive scans of those counts (worker_off, the
 *   pack_tiles/top/rows  context token offsets and the copy units), totals
 *                        and the capacity check: one block up to 4096 rows.
 *   fork_outline<true>   the same walk again, now writing each worker's record
 *                        (row, entry, kind, context start and length).
 *   fork_copy            tiled over copy units (row tokens times groups of
 *                        up to eight workers) by waves: every wave step loads
 *                        1024 row tokens once and stores them into the
 *                        contexts of the group's workers, then their <Thread>
 *                        and seeds; it finds its row by a 64-way search over
 *                        the unit offsets.
 * join
 *   join_size            one thread per row: joined length and thread checks.
 *   pack_*               exclusive scan of the joined lengths.
 *   join_copy            tiled the same way over the joined tokens: the row,
 *                        each worker's <Thread> ... </Thread> span (positions
 *                        of 64 workers from one wave scan), and </Parallel>;
 *                        16-byte stores aligned on the output, 16-byte loads
 *                        at dword alignment.
 *
 * With PARASON_CFG_LENIENT_GAPS Text may stand between <Parallel> and
 * <Outlines>, after <Outlines>, between entries and before </Outlines>: the
 * walk then checks only the order of the tags, takes the entry text lengths
 * from the tag positions (a wave prefix scan gives each worker's seed offset,
 * in both modes), and fork_copy finds the texts of a group's entries by one
 * ballot scan of the outline.
 *
 * Rows, contexts and joined rows start at any element offset.  fork_copy
 * moves dwords (the contexts of a group start at unrelated alignments, and
 * the loads are shared between them); join_copy moves 16-byte vectors.
 * Tiling keeps every wave step's work bounded however long the rows are: 1024
 * positions and, in fork_copy, eight stores of each.
 */
#pragma once
#include "device_common.h"

namespace pk {

constexpr int PACK_THREADS = 256;
constexpr int PACK_ROWS_PER_THREAD = 16;
constexpr int PACK_TILE = PACK_THREADS * PACK_ROWS_PER_THREAD;
#ifndef PARASON_OUTLINE_LOADS
#define PARASON_OUTLINE_LOADS 4
#endif
constexpr int CHUNK_J = PARASON_OUTLINE_LOADS; /* loads per lane per step of the outline walk */
constexpr int CHUNK = CHUNK_J * WAVE;          /* tokens per wave step of the outline walk */
#ifndef PARASON_BACK_LOADS
#define PARASON_BACK_LOADS 8
#endif
/* The backward search for the outline's start looks for two tags only, so its
 * steps are longer: one round of loads covers most outlines. */
constexpr int BACK_J = PARASON_BACK_LOADS; /* loads per lane per step of the backward search */
constexpr int BACK = BACK_J * WAVE;
constexpr int COPY_GROUP = 8;   /* worker contexts fork_copy writes from one read of a row tile */
constexpr int SUMM_ENTRIES = 8; /* outline entries per row the first walk keeps for the second */
#ifndef PARASON_OUTLINE_WAVES
#define PARASON_OUTLINE_WAVES 4
#endif
constexpr int OUTLINE_WAVES = PARASON_OUTLINE_WAVES; /* waves (rows at a time) per fork_outline block */
constexpr int JOIN_UNROLL = 4;  /* workers of a row whose records join_size loads together */
constexpr int JOIN_SINGLE = 1024; /* rows up to which join_copy scans the joined lengths itself */
/* join_size: small blocks spread its scattered loads of worker tokens over
 * many compute units (256-thread blocks measured 0.9 us slower at 1,024 rows) */
constexpr int JOIN_SIZE_THREADS = 64;

/* Orders the LDS accesses of a wave's lanes: what one lane wrote before it is
 * visible to every lane of the wave after it. */
__device__ __forceinline__ void wave_lds_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

/* ---- exclusive scans of K int64 values per row -------------------------- */

template <int K>
struct PackScan {
    const int64_t *vals;   /* [n][K] */
    int64_t n;
    int64_t *tile_sum;     /* [tiles][K] */
    int64_t *tile_off;     /* [tiles][K] */
    int64_t *out[K];       /* [n + 1] each: exclusive offsets, out[k][n] = total */
    int64_t cap[K];        /* totals above these set *over */
    int64_t *totals;       /* optional: totals[0 .. report) and then the over flag, for the caller */
    int report;            /* totals reported (the first `report` of the K) */
    int32_t *over;         /* workspace copy of the over flag */
};

template <int K>
__global__ void __launch_bounds__(PACK_THREADS) pack_tiles(PackScan<K> a)
{
    __shared__ int64_t lds[K * PACK_THREADS];
    const int64_t r0 = (int64_t)blockIdx.x * PACK_TILE + (int64_t)threadIdx.x * PACK_ROWS_PER_THREAD;
    int64_t v[K];
#pragma unroll
    for (int k = 0; k < K; ++k) v[k] = 0;
    for (int j = 0; j < PACK_ROWS_PER_THREAD; ++j) {
        const int64_t r = r0 + j;
        if (r < a.n) {
#pragma unroll
            for (int k = 0; k < K; ++k) v[k] += a.vals[r * K + k];
        }
    }
    block_tree_sum<int64_t, K>(v, lds);
    if (threadIdx.x == 0) {
#pragma unroll
        for (int k = 0; k < K; ++k) a.tile_sum[blockIdx.x * K + k] = v[k];
    }
}

template <int K>
__global__ void __launch_bounds__(1024) pack_top(PackScan<K> a, int64_t tiles)
{
    __shared__ int64_t part[K][1024 / WAVE];
    __shared__ int64_t carry[K];
    if (threadIdx.x < K) carry[threadIdx.x] = 0;
    __syncthreads();
    for (int64_t base = 0; base < tiles; base += 1024) {
        const int64_t i = base + threadIdx.x;
        int64_t v[K], inc[K];
#pragma unroll
        for (int k = 0; k < K; ++k) {
            v[k] = i < tiles ? a.tile_sum[i * K + k] : 0;
            inc[k] = wave_inclusive_scan(v[k]);
            if ((threadIdx.x & (WAVE - 1)) == WAVE - 1) part[k][threadIdx.x / WAVE] = inc[k];
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < K; ++k) {
            int64_t before = carry[k];
            for (int w = 0; w < (int)(threadIdx.x / WAVE); ++w) before += part[k][w];
            if (i < tiles) a.tile_off[i * K + k] = before + inc[k] - v[k];
        }
        __syncthreads();
        if (threadIdx.x < K) {
            int64_t t = 0;
            for (int w = 0; w < 1024 / WAVE; ++w) t += part[threadIdx.x][w];
            carry[threadIdx.x] += t;
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        int32_t over = 0;
#pragma unroll
        for (int k = 0; k < K; ++k) {
            a.out[k][a.n] = carry[k];
            over |= carry[k] > a.cap[k] ? 1 : 0;
            if (a.totals && k < a.report) a.totals[k] = carry[k];
        }
        if (a.totals) a.totals[a.report] = over;
        a.over[0] = over;
    }
}

template <int K>
__global__ void __launch_bounds__(PACK_THREADS) pack_rows(PackScan<K> a)
{
    __shared__ int64_t part[K][PACK_THREADS / WAVE];
    const int64_t r0 = (int64_t)blockIdx.x * PACK_TILE + (int64_t)threadIdx.x * PACK_ROWS_PER_THREAD;
    int64_t s[K], off[K];
#pragma unroll
    for (int k = 0; k < K; ++k) {
        s[k] = 0;
        for (int j = 0; j < PACK_ROWS_PER_THREAD; ++j) {
            const int64_t r = r0 + j;
            s[k] += r < a.n ? a.vals[r * K + k] : 0;
        }
        const int64_t inc = wave_inclusive_scan(s[k]);
        if ((threadIdx.x & (WAVE - 1)) == WAVE - 1) part[k][threadIdx.x / WAVE] = inc;
        off[k] = inc - s[k];
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < K; ++k) {
        off[k] += a.tile_off[blockIdx.x * K + k];
        for (int w = 0; w < (int)(threadIdx.x / WAVE); ++w) off[k] += part[k][w];
        for (int j = 0; j < PACK_ROWS_PER_THREAD; ++j) {
            const int64_t r = r0 + j;
            if (r < a.n) {
                a.out[k][r] = off[k];
                off[k] += a.vals[r * K + k];
            }
        }
    }
}

/* The three passes in one block when the rows fit one tile (n <= PACK_TILE):
 * every thread loads its rows' values once, then offsets, totals and the
 * capacity check as above. */
template <int K>
__global__ void __launch_bounds__(PACK_THREADS) pack_single(PackScan<K> a)
{
    __shared__ int64_t part[K][PACK_THREADS / WAVE];
    const int wv = threadIdx.x / WAVE;
    const int64_t r0 = (int64_t)threadIdx.x * PACK_ROWS_PER_THREAD;
    int64_t v[PACK_ROWS_PER_THREAD][K];
#pragma unroll
    for (int j = 0; j < PACK_ROWS_PER_THREAD; ++j) {
#pragma unroll
        for (int k = 0; k < K; ++k) v[j][k] = r0 + j < a.n ? a.vals[(r0 + j) * K + k] : 0;
    }
    int64_t off[K];
#pragma unroll
    for (int k = 0; k < K; ++k) {
        int64_t s = 0;
#pragma unroll
        for (int j = 0; j < PACK_ROWS_PER_THREAD; ++j) s += v[j][k];
        const int64_t inc = wave_inclusive_scan(s);
        if ((threadIdx.x & (WAVE - 1)) == WAVE - 1) part[k][wv] = inc;
        off[k] = inc - s;
    }
    __syncthreads();
    int32_t over = 0;
#pragma unroll
    for (int k = 0; k < K; ++k) {
        int64_t total = 0;
        for (int w = 0; w < PACK_THREADS / WAVE; ++w) {
            if (w < wv) off[k] += part[k][w];
            total += part[k][w];
        }
#pragma unroll
        for (int j = 0; j < PACK_ROWS_PER_THREAD; ++j) {
            if (r0 + j < a.n) a.out[k][r0 + j] = off[k];
            off[k] += v[j][k];
        }
        over |= total > a.cap[k] ? 1 : 0;
        if (threadIdx.x == 0) {
            a.out[k][a.n] = total;
            if (a.totals && k < a.report) a.totals[k] = total;
        }
    }
    if (threadIdx.x == 0) {
        if (a.totals) a.totals[a.report] = over;
        a.over[0] = over;
    }
}

/* ---- fork --------------------------------------------------------------- */

struct ForkArgs {
    const int32_t *tokens;
    const int64_t *starts;
    const int32_t *lengths;
    int64_t n;
    TagMatch tm;
    bool seed;              /* contexts end with the entry's text */
    bool lenient;           /* PARASON_CFG_LENIENT_GAPS */
    int32_t thread_id;      /* token id of <Thread> */
    uint32_t *status;       /* [n] PARASON_PACK_* */
    int64_t *counts;        /* [n][3]: workers, context tokens, copy units */
    int32_t *outl;          /* [n]: position of the outline's <Outlines> */
    /* filled in by the scan, read by the write pass and the copy */
    const int64_t *worker_off;
    const int64_t *tok_off;
    const int64_t *unit_off; /* [n + 1]: scan of the copy units (fork_copy) */
    uint64_t *summ;          /* [n][SUMM_ENTRIES]: the row's first entries, text start | length << 32 |
                                (Trial) << 63, written by the first walk */
    const int32_t *over;
    int64_t *ctx_starts;
    int32_t *ctx_lengths, *ctx_row, *ctx_entry, *ctx_kind;
    int32_t *ctx_tokens;
};

/* Largest value over the wave (positions, so int32), in every lane. */
__device__ __forceinline__ int32_t wave_max_pos(int32_t v, int lane) { return lane63(dpp_incl_scan<OpMax>(v, lane)); }

/* Inclusive prefix sum over the wave's lanes (every lane must call it). */
__device__ __forceinline__ int64_t wave_incl_scan(int64_t v, int lane)
{
#pragma unroll
    for (int d = 1; d < WAVE; d <<= 1) {
        const int64_t o = __shfl_up(v, (unsigned)d, WAVE);
        v += lane >= d ? o : 0;
    }
    return v;
}

/* Token p of the row at g for p < end, else 0 (end >= 1).  The load is
 * unconditional, at min(p, end - 1), and the value selected after it: a load
 * under a condition is a branch, and the wave waits for it before the next
 * one, so J conditional loads cost J round trips instead of one. */
__device__ __forceinline__ int32_t row_token(const ForkArgs &a, int64_t g, int64_t p, int64_t end)
{
    const int32_t t = a.tokens[g + min(p, end - 1)];
    return p < end ? t : 0;
}

/* Position of the last tag before position o of the row at g (-1 if none);
 * called by a whole wave. */
__device__ __forceinline__ int64_t last_tag_before(const ForkArgs &a, int64_t g, int64_t o, int lane, bool contig)
{
    for (int64_t e = o; e > 0; e -= CHUNK) {
        const int64_t lo = e > CHUNK ? e - CHUNK : 0;
        int32_t best = -1, tk[CHUNK_J];
#pragma unroll
        for (int j = 0; j < CHUNK_J; ++j) tk[j] = row_token(a, g, lo + lane + WAVE * j, e);
#pragma unroll
        for (int j = 0; j < CHUNK_J; ++j) {
            const int64_t p = lo + lane + WAVE * j;
            if (p < e && classify(a.tm, tk[j], contig) != C_TEXT) best = (int32_t)p > best ? (int32_t)p : best;
        }
        best = wave_max_pos(best, lane);
        if (best >= 0) return best;
    }
    return -1;
}

/* Tokens lo + lane + WAVE * j of the row at g below end (0 beyond), end >= 1. */
__device__ __forceinline__ void outline_tokens(const ForkArgs &a, int64_t g, int64_t lo, int64_t end,
                                               int32_t (&tk)[CHUNK_J], int lane)
{
#pragma unroll
    for (int j = 0; j < CHUNK_J; ++j) tk[j] = row_token(a, g, lo + lane + WAVE * j, end);
}

/* One row's outline, by one wave.  WRITE = false: status and counts (the
 * first walk); WRITE = true: the worker records of a row whose outline is well
 * formed, its first worker w0 and first context token t0 given.  ev: the
 * wave's CHUNK entries of LDS. */
template <bool WRITE>
__device__ __forceinline__ void outline_row(const ForkArgs &a, int64_t i, int64_t w0, int64_t t0, uint32_t *ev,
                                            int lane)
{
    const bool contig = a.tm.contiguous != 0;
    const int64_t g = a.starts[i];
    const int32_t L = a.lengths[i];
    int64_t o;
    if (WRITE) {
        const int64_t n_e = a.counts[3 * i];
        if (a.status[i] != 0 || n_e == 0) return;
        if (n_e <= SUMM_ENTRIES) {
            /* the first walk kept every entry of this outline: the records
             * without a second walk (lane k: entry k) */
            const uint64_t x = lane < n_e ? a.summ[i * SUMM_ENTRIES + lane] : 0ull;
            const int32_t sl = a.seed ? (int32_t)((x >> 32) & 0x7fffffffu) : 0;
            const int64_t before = dpp_incl_scan<OpAdd>(sl, lane) - sl; /* seeds of entries 0 .. k-1 */
            if (lane < n_e) {
                const int64_t w = w0 + lane;
                a.ctx_starts[w] = t0 + lane * ((int64_t)L + 1) + before;
                a.ctx_lengths[w] = (int32_t)((int64_t)L + 1 + sl);
                a.ctx_row[w] = (int32_t)i;
                a.ctx_entry[w] = lane;
                a.ctx_kind[w] = (x >> 63) ? (int32_t)T_TRI : (int32_t)T_SUB;
            }
            return;
        }
        o = a.outl[i];
    } else {
        uint32_t st = 0;
        o = -1;
        if (L < 0 || g < 0) st = PARASON_PACK_BAD_ROW;
        else if (L == 0) st = PARASON_PACK_NO_OUTLINE_END;
        /* backwards from the row's end in chunks: the first chunk holds the
         * last token, which must be </Outlines>; then the last <Outlines>
         * before it, and the class of the token right before that when it
         * is in the same chunk (1: <Parallel>, 0: not, -1: not seen) */
        int32_t par_before = -1;
        for (int64_t e = (int64_t)L; st == 0 && e > 0 && o < 0; e -= BACK) {
            const int64_t lo = e > BACK ? e - BACK : 0;
            uint32_t c[BACK_J];
            int32_t best = -1;
            bool end_mine = false;
            int32_t tk[BACK_J];
#pragma unroll
            for (int j = 0; j < BACK_J; ++j) tk[j] = row_token(a, g, lo + lane + WAVE * j, e);
#pragma unroll
            for (int j = 0; j < BACK_J; ++j) {
                const int64_t p = lo + lane + WAVE * j;
                c[j] = p < e ? classify(a.tm, tk[j], contig) : C_TEXT;
                if (p < (int64_t)L - 1 && c[j] == C_OUT) best = (int32_t)p > best ? (int32_t)p : best;
                end_mine = end_mine || (p == (int64_t)L - 1 && c[j] == C_END_OUT);
            }
            if (e == (int64_t)L && __ballot(end_mine) == 0) {
                st = PARASON_PACK_NO_OUTLINE_END;
                break;
            }
            o = wave_max_pos(best, lane);
            if (o >= 1 && o - 1 >= lo) {
                bool par_mine = false;
#pragma unroll
                for (int j = 0; j < BACK_J; ++j) par_mine = par_mine || (lo + lane + WAVE * j == o - 1 && c[j] == C_PAR);
                par_before = __ballot(par_mine) != 0 ? 1 : 0;
            }
        }
        if (st == 0) {
            /* the tag before <Outlines> must be <Parallel>: right before it,
             * or with only Text between when lenient */
            bool par_ok;
            if (a.lenient) {
                const int64_t q = o >= 1 ? last_tag_before(a, g, o, lane, contig) : -1;
                par_ok = q >= 0 && classify(a.tm, a.tokens[g + q], contig) == C_PAR;
            } else {
                par_ok = o >= 1 && (par_before >= 0 ? par_before == 1
                                                    : classify(a.tm, a.tokens[g + o - 1], contig) == C_PAR);
            }
            if (o < 0 || !par_ok) st = PARASON_PACK_NO_OUTLINE;
        }
        if (st != 0) {
            if (lane == 0) {
                a.status[i] = st;
                a.counts[3 * i] = 0;
                a.counts[3 * i + 1] = 0;
                a.counts[3 * i + 2] = 0;
                a.outl[i] = -1;
            }
            return;
        }
    }
    /* walk the outline [o + 1, L - 1) in chunks; events are its tags */
    const int64_t end = (int64_t)L - 1;
    int64_t m = 0;                       /* tags before this chunk */
    int64_t prev_pos = o;                /* the tag before the current one */
    uint32_t prev_cls = C_OUT;
    int64_t text = 0;                    /* entry text tokens so far (the same in every lane) */
    bool ok = true;
    /* the next chunk's tokens are loaded while this one is walked */
    int32_t tk[CHUNK_J];
    outline_tokens(a, g, o + 1, end, tk, lane);
    for (int64_t lo = o + 1; lo < end; lo += CHUNK) {
        int32_t tn[CHUNK_J];
        outline_tokens(a, g, lo + CHUNK, end, tn, lane);
        uint64_t b[CHUNK_J];
        uint32_t c[CHUNK_J];
#pragma unroll
        for (int j = 0; j < CHUNK_J; ++j) {
            const int64_t p = lo + lane + WAVE * j;
            c[j] = p < end ? classify(a.tm, tk[j], contig) : C_TEXT;
            b[j] = __ballot(c[j] != C_TEXT);
            tk[j] = tn[j];
        }
        uint32_t base = 0;
#pragma unroll
        for (int j = 0; j < CHUNK_J; ++j) {
            if (c[j] != C_TEXT) {
                const uint32_t idx = base + __builtin_amdgcn_mbcnt_hi((uint32_t)(b[j] >> 32),
                                                                      __builtin_amdgcn_mbcnt_lo((uint32_t)b[j], 0u));
                ev[idx] = ((uint32_t)(lane + WAVE * j) << 4) | c[j];
            }
            base += (uint32_t)__popcll(b[j]);
        }
        wave_lds_sync();
        for (uint32_t e0 = 0; e0 < base; e0 += WAVE) { /* the same trip count in every lane */
            const uint32_t e = e0 + (uint32_t)lane;
            const bool act = e < base;
            int64_t len = 0; /* text tokens of the entry this lane closes */
            int64_t J = 0, tstart = 0;
            uint32_t pc = 0;
            if (act) {
                const uint32_t x = ev[e];
                const int64_t P = lo + (x >> 4);
                const uint32_t cl = x & 15u;
                int64_t pp = prev_pos;
                pc = prev_cls;
                if (e > 0) {
                    const uint32_t y = ev[e - 1];
                    pp = lo + (y >> 4);
                    pc = y & 15u;
                }
                J = m + e;
                if ((J & 1) == 0) {
                    /* an entry opens after <Outlines> or the previous entry:
                     * right after it, or after a gap when lenient */
                    ok = ok && (cl == C_SUB || cl == C_TRI) && (a.lenient || P == pp + 1);
                } else {
                    /* and closes with its own tag after at least one text token */
                    ok = ok && (pc == C_SUB || pc == C_TRI) && cl == pc + 1 && P >= pp + 2;
                    len = P - pp - 1;
                    tstart = pp + 1;
                }
            }
            if (!WRITE && act && (J & 1) && (J >> 1) < SUMM_ENTRIES)
                a.summ[i * SUMM_ENTRIES + (J >> 1)] = (uint64_t)(uint32_t)tstart |
                                                     ((uint64_t)(uint32_t)len << 32) |
                                                     ((uint64_t)(pc == C_TRI) << 63);
            /* entry text lengths and their sums within a chunk are below L */
            const int64_t incl = dpp_incl_scan<OpAdd>((int32_t)len, lane);
            if (WRITE && act && (J & 1)) {
                const int64_t k = J >> 1;
                const int64_t w = w0 + k;
                const int64_t seed_before = text + incl - len; /* texts of entries 0 .. k-1 */
                a.ctx_starts[w] = t0 + k * ((int64_t)L + 1) + (a.seed ? seed_before : 0);
                a.ctx_lengths[w] = (int32_t)((int64_t)L + 1 + (a.seed ? len : 0));
                a.ctx_row[w] = (int32_t)i;
                a.ctx_entry[w] = (int32_t)k;
                a.ctx_kind[w] = pc == C_SUB ? (int32_t)T_SUB : (int32_t)T_TRI;
            }
            text += lane63((int32_t)incl);
        }
        if (base > 0) {
            const uint32_t y = ev[base - 1];
            prev_pos = lo + (y >> 4);
            prev_cls = y & 15u;
        }
        m += base;
        __builtin_amdgcn_wave_barrier(); /* ev is rewritten by the next chunk */
    }
    if (!WRITE) {
        ok = __ballot(!ok) == 0;
        /* an even, non-zero number of tags, the last one right before
         * </Outlines> (or followed by a gap when lenient) */
        ok = ok && m >= 2 && (m & 1) == 0 && (a.lenient || prev_pos == end - 1);
        const int64_t n_e = ok ? m / 2 : 0;
        int64_t toks = n_e * ((int64_t)L + 1) + (a.seed ? text : 0);
        uint32_t st = ok ? 0u : (uint32_t)PARASON_PACK_BAD_ENTRY;
        if (ok && (int64_t)L + 1 + (a.seed ? text : 0) > (int64_t)INT32_MAX) {
            st = PARASON_PACK_TOO_LONG;
            toks = 0;
        }
        if (lane == 0) {
            a.status[i] = st;
            a.counts[3 * i] = st == 0 ? n_e : 0;
            a.counts[3 * i + 1] = st == 0 ? toks : 0;
            /* fork_copy reads the row once per group of COPY_GROUP workers */
            a.counts[3 * i + 2] = st == 0 ? (n_e + COPY_GROUP - 1) / COPY_GROUP * (int64_t)L : 0;
            a.outl[i] = (int32_t)o;
        }
    }
}

/* One wave per row (grid-stride).  WRITE = false: status and counts;
 * WRITE = true: the worker records of rows whose outline is well formed. */
template <bool WRITE>
__global__ void __launch_bounds__(OUTLINE_WAVES * WAVE) fork_outline(ForkArgs a)
{
    __shared__ uint32_t ev_all[OUTLINE_WAVES][CHUNK]; /* per wave: (offset in chunk << 4) | class, in position order */
    const int lane = threadIdx.x & (WAVE - 1);
    const int wv = threadIdx.x / WAVE;
    if (WRITE && a.over[0]) return;
    const int64_t n_waves = (int64_t)gridDim.x * OUTLINE_WAVES;
    for (int64_t i = uniform64((int64_t)blockIdx.x * OUTLINE_WAVES + wv); i < a.n; i += n_waves)
        outline_row<WRITE>(a, i, WRITE ? a.worker_off[i] : 0, WRITE ? a.tok_off[i] : 0, ev_all[wv], lane);
}

/* Up to FORK_SINGLE rows: the scans of the three counts and the worker
 * records in one launch instead of pack_single and fork_outline<true>.  Every
 * block scans the counts of all rows (24 bytes per row, read from L2; each
 * thread FORK_REC_RPT consecutive rows), then its FORK_REC_WAVES waves write
 * the records of the block's rows, one row per wave.  The thread holding a
 * row in the scan writes its offsets (in the row's own block); the block
 * holding the last row writes the totals and the capacity flag, which every
 * block computes alike. */
constexpr int FORK_SINGLE = 1024;
constexpr int FORK_REC_WAVES = 8; /* 16: 1.3 us slower at 1,024 rows; 4: as fast */
constexpr int FORK_REC_THREADS = FORK_REC_WAVES * WAVE;
constexpr int FORK_REC_RPT = FORK_SINGLE / FORK_REC_THREADS;

__global__ void __launch_bounds__(FORK_REC_THREADS) fork_records(ForkArgs a, PackScan<3> ps)
{
    __shared__ int64_t part[3][FORK_REC_WAVES];
    __shared__ int64_t offs[2][FORK_REC_WAVES]; /* first worker and first context token of the block's rows */
    __shared__ uint32_t ev_all[FORK_REC_WAVES][CHUNK];
    const int t = (int)threadIdx.x, lane = t & (WAVE - 1), wv = t / WAVE;
    const int64_t q0 = (int64_t)t * FORK_REC_RPT; /* this thread's rows in the scan */
    int64_t v[FORK_REC_RPT][3], off[3], total[3];
#pragma unroll
    for (int j = 0; j < FORK_REC_RPT; ++j) {
#pragma unroll
        for (int k = 0; k < 3; ++k) v[j][k] = q0 + j < a.n ? a.counts[3 * (q0 + j) + k] : 0;
    }
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        int64_t sum = 0;
#pragma unroll
        for (int j = 0; j < FORK_REC_RPT; ++j) sum += v[j][k];
        const int64_t inc = wave_inclusive_scan(sum);
        if (lane == WAVE - 1) part[k][wv] = inc;
        off[k] = inc - sum;
    }
    __syncthreads();
    int32_t over = 0;
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        total[k] = 0;
        for (int w = 0; w < FORK_REC_WAVES; ++w) {
            off[k] += w < wv ? part[k][w] : 0;
            total[k] += part[k][w];
        }
        over |= total[k] > ps.cap[k] ? 1 : 0;
    }
    const int64_t r0 = (int64_t)blockIdx.x * FORK_REC_WAVES; /* the block's rows */
#pragma unroll
    for (int j = 0; j < FORK_REC_RPT; ++j) {
        const int64_t r = q0 + j;
        if (r >= r0 && r < r0 + FORK_REC_WAVES && r < a.n) {
#pragma unroll
            for (int k = 0; k < 3; ++k) ps.out[k][r] = off[k];
            offs[0][r - r0] = off[0];
            offs[1][r - r0] = off[1];
        }
#pragma unroll
        for (int k = 0; k < 3; ++k) off[k] += v[j][k];
    }
    if (blockIdx.x == gridDim.x - 1 && t == 0) {
#pragma unroll
        for (int k = 0; k < 3; ++k) ps.out[k][a.n] = total[k];
        ps.totals[0] = total[0];
        ps.totals[1] = total[1];
        ps.totals[2] = over;
        ps.over[0] = over;
    }
    __syncthreads();
    const int64_t i = r0 + wv;
    if (over || i >= a.n) return;
    outline_row<true>(a, i, offs[0][wv], offs[1][wv], ev_all[wv], lane);
}

/* ---- tiled copies -------------------------------------------------------- */

/* The copies are tiled over their output by waves: each wave step covers
 * WTILE consecutive output positions (WV 16-byte vectors per lane, all loads
 * issued before the first store), finds the row holding the first of them by
 * a 64-way search, and walks the pieces of that range.  Waves work
 * independently, so the chains of dependent loads of many tiles (search, row
 * and worker records, data) overlap on every CU. */
#ifndef PARASON_COPY_WV
#define PARASON_COPY_WV 4
#endif
constexpr int WV = PARASON_COPY_WV;      /* 16-byte vectors per lane per wave step */
constexpr int64_t WTILE = 4 * WV * WAVE; /* output positions per wave step */
constexpr int TAIL_U = 16;               /* elements per lane per step of a context's tail */
constexpr int COPY_WAVES = PACK_THREADS / WAVE;

typedef int v4i_t __attribute__((ext_vector_type(4)));

/* 16 bytes from a 4-byte aligned address (global memory takes unaligned
 * 16-byte loads at dword granularity). */
__device__ __forceinline__ v4i_t load16(const int32_t *p)
{
    v4i_t v;
    __builtin_memcpy(&v, p, 16);
    return v;
}

/* Largest index s in [0, count) with offs[s] <= x (offs ascending, offs[0] <= x),
 * by one wave in 64-way rounds; the result is returned to every lane. */
__device__ __forceinline__ int64_t wave_find(const int64_t *offs, int64_t count, int64_t x, int lane)
{
    int64_t lo = 0, hi = count;
    while (hi - lo > 1) {
        const int64_t step = (hi - lo + WAVE - 1) / WAVE;
        const int64_t idx = lo + lane * step;
        const uint64_t m = __ballot(idx < hi && offs[idx] <= x);
        const int64_t last = 63 - __builtin_clzll(m | 1ull);
        lo = lo + last * step;
        hi = min(hi, lo + step);
    }
    return lo;
}

/* Elements lane + j * WAVE of a range of n: how many of them this lane holds. */
__device__ __forceinline__ int lane_count(int64_t n, int lane)
{
    return n > lane ? (int)((n - lane + WAVE - 1) / WAVE) : 0;
}

/* dst[o_k + p] = src[p] for p in [p0, p1) and every k < nd, by one wave
 * (p1 - p0 <= WTILE): each source token is loaded once (dword loads, 4 * WV
 * per lane) and stored nd times; o_k is lane k's value of o.  Sharing the
 * loads beats per-destination 16-byte copies here: the contexts of a group
 * start at unrelated alignments. */
__device__ __forceinline__ void wave_copy_multi(int32_t *__restrict__ dst, int64_t o, int nd, int64_t p0, int64_t p1,
                                                const int32_t *__restrict__ src, int lane)
{
    constexpr int U = 4 * WV;
    const int jm = lane_count(p1 - p0, lane);
    const int32_t *sp = src + p0 + lane;
    int32_t v[U];
#pragma unroll
    for (int j = 0; j < U; ++j) v[j] = j < jm ? sp[j * WAVE] : 0;
    for (int k = 0; k < nd; ++k) {
        int32_t *dp = dst + __shfl(o, k, WAVE) + p0 + lane;
#pragma unroll
        for (int j = 0; j < U; ++j)
            if (j < jm) dp[j * WAVE] = v[j];
    }
}

/* dst[d] = src[d - shift] for d in [d0, d1), by one wave (d1 - d0 <= WTILE):
 * 16-byte stores aligned on dst and 16-byte loads from src at whatever dword
 * alignment that gives; the at most three elements before dst's first 16-byte
 * boundary and the at most three after the last one are copied singly. */
__device__ __forceinline__ void wave_copy(int32_t *__restrict__ dst, int64_t d0, int64_t d1,
                                          const int32_t *__restrict__ src, int64_t shift, int lane)
{
    if (d0 >= d1) return;
    const int64_t b0 = min(d0 + (int64_t)(((16u - ((uint32_t)(uintptr_t)(dst + d0) & 15u)) & 15u) >> 2), d1);
    const int64_t nvec = (d1 - b0) >> 2;
    const int64_t b1 = b0 + 4 * nvec;
    if (lane < 6) { /* lanes 0-2: the head, lanes 3-5: the tail */
        const int64_t d = lane < 3 ? d0 + lane : b1 + (lane - 3);
        if (lane < 3 ? d < b0 : d < d1) dst[d] = src[d - shift];
    }
    if (nvec == 0) return;
    /* every lane loads WV vectors (beyond the range: the last one again), so
     * that the loads are unconditional and issue back to back */
    const int32_t *sp = src + (b0 - shift);
    v4i_t *dp = reinterpret_cast<v4i_t *>(dst + b0);
    v4i_t v[WV];
#pragma unroll
    for (int j = 0; j < WV; ++j) v[j] = load16(sp + 4 * min((int64_t)(lane + WAVE * j), nvec - 1));
    /* streaming stores: the joined rows are not read again by this call
     * (dword stores of fork_copy's contexts measured slower this way) */
#pragma unroll
    for (int j = 0; j < WV; ++j)
        if (lane + WAVE * j < nvec) __builtin_nontemporal_store(v[j], dp + lane + WAVE * j);
}

/* A worker context's tail at dst[d0 .. d1): sub (the <Thread> id) at d0, then
 * src[f ..] (the entry's text), by one wave in steps of TAIL_U per lane.
 * f >= 1: the element before the text (its opening tag) is loaded for d0 and
 * replaced. */
__device__ __forceinline__ void wave_tail(int32_t *__restrict__ dst, int64_t d0, int64_t d1,
                                          const int32_t *__restrict__ src, int64_t f, int32_t sub, int lane)
{
    for (int64_t base = 0; base < d1 - d0; base += TAIL_U * WAVE) {
        const int jm = lane_count(min(d1 - d0 - base, (int64_t)TAIL_U * WAVE), lane);
        const int32_t *sp = src + (f - 1) + base + lane;
        int32_t *dp = dst + d0 + base + lane;
        int32_t v[TAIL_U];
#pragma unroll
        for (int j = 0; j < TAIL_U; ++j) v[j] = j < jm ? sp[j * WAVE] : 0;
        if (base == 0 && lane == 0) v[0] = sub;
#pragma unroll
        for (int j = 0; j < TAIL_U; ++j)
            if (j < jm) dp[j * WAVE] = v[j];
    }
}

/* Positions of the first text tokens of entries ea .. ea + nd - 1 of the
 * outline that starts at o in the row src of length L (each entry's
 * <Subtask>/<Trial> tag plus one), found by one wave in 64-token ballot
 * rounds; lane k < nd receives entry ea + k's.  Used with lenient gaps, where
 * gaps break the closed form of the position.  slot: COPY_GROUP int64 of LDS
 * owned by the wave.  The row's outline passed the walk, so the entries exist. */
__device__ __forceinline__ int64_t group_text_pos(const ForkArgs &a, const int32_t *src, int64_t o, int64_t L,
                                                  int64_t ea, int nd, int64_t *slot, int lane)
{
    const bool contig = a.tm.contiguous != 0;
    int64_t seen = 0;
    for (int64_t lo = o + 1; lo < L - 1 && seen < ea + nd; lo += WAVE) {
        const int64_t p = lo + lane;
        const uint32_t c = p < L - 1 ? classify(a.tm, src[p], contig) : C_TEXT;
        const bool open = c == C_SUB || c == C_TRI;
        const uint64_t b = __ballot(open);
        const int64_t rk =
            seen + __builtin_amdgcn_mbcnt_hi((uint32_t)(b >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)b, 0u));
        if (open && rk >= ea && rk < ea + nd) slot[rk - ea] = p + 1;
        seen += __popcll(b);
    }
    wave_lds_sync();
    const int64_t f = lane < nd ? slot[lane] : 0;
    __builtin_amdgcn_wave_barrier(); /* slot is rewritten by the next group */
    return f;
}

/* Contexts, tiled over copy units: a forked row of length L with k workers
 * has ceil(k / COPY_GROUP) * L units, one per row token and group of up to
 * COPY_GROUP workers (unit_off is their scan).  A wave step takes WTILE
 * consecutive units: it loads those row tokens once and stores them into the
 * contexts of the group's workers; the step that reaches the end of the row
 * also writes the group's <Thread> tokens and seeds.  The row is read from
 * memory once per group, not once per worker. */
__global__ void __launch_bounds__(PACK_THREADS) fork_copy(ForkArgs a)
{
    __shared__ int64_t slots[COPY_WAVES][COPY_GROUP];
    const int lane = threadIdx.x & (WAVE - 1);
    const int wv = threadIdx.x / WAVE;
    if (a.over[0]) return;
    const int64_t UT = a.unit_off[a.n];
    const int64_t NW = (int64_t)gridDim.x * COPY_WAVES;
    for (int64_t t = (int64_t)blockIdx.x * COPY_WAVES + wv; t * WTILE < UT; t += NW) {
        const int64_t lo = t * WTILE, hi = min(lo + WTILE, UT);
        for (int64_t r = wave_find(a.unit_off, a.n, lo, lane); r < a.n; ++r) {
            /* the row's records in one round of loads, before any branch */
            const int64_t uo = a.unit_off[r], ue = a.unit_off[r + 1];
            const int64_t L = a.lengths[r], g0 = a.starts[r];
            const int64_t w0 = a.worker_off[r], w1 = a.worker_off[r + 1];
            const int64_t o = a.outl[r], to = a.tok_off[r];
            if (uo >= hi) break;
            if (ue <= max(lo, uo)) continue; /* no units (not forked), or all before the tile */
            const int32_t *src = a.tokens + g0;
            for (int64_t g = (max(lo, uo) - uo) / L; uo + g * L < min(hi, ue); ++g) {
                const int64_t gs = uo + g * L;
                const int64_t p0 = max(lo, gs) - gs, p1 = min(hi, gs + L) - gs;
                const int64_t wa = w0 + g * COPY_GROUP;
                const int nd = (int)min((int64_t)COPY_GROUP, w1 - wa);
                /* lane k: worker wa + k */
                const int64_t cs = lane < nd ? a.ctx_starts[wa + lane] : 0;
                const int64_t len = lane < nd ? (int64_t)a.ctx_lengths[wa + lane] : 0;
                wave_copy_multi(a.ctx_tokens, cs, nd, p0, p1, src, lane);
                if (p1 < L) continue;
                /* the group's tails: <Thread>, then entry e's text when seeding;
                 * workers are numbered entry by entry, so worker wa + k runs
                 * entry g * COPY_GROUP + k */
                const int64_t e = g * COPY_GROUP + lane;
                /* first text token of entry e: without gaps, o + 2 + 2e + the texts
                 * before it (see fork_outline); with gaps, searched */
                int64_t ft;
                if (!(a.lenient && a.seed)) ft = o + 2 + 2 * e + (cs - to - e * (L + 1));
                else if (w1 - w0 <= SUMM_ENTRIES) ft = lane < nd ? (int64_t)(uint32_t)a.summ[r * SUMM_ENTRIES + lane] : 0;
                else ft = group_text_pos(a, src, o, L, g * COPY_GROUP, nd, slots[wv], lane);
                for (int k = 0; k < nd; ++k) {
                    const int64_t c = __shfl(cs, k, WAVE);
                    wave_tail(a.ctx_tokens, c + L, c + __shfl(len, k, WAVE), src, __shfl(ft, k, WAVE), a.thread_id,
                              lane);
                }
            }
        }
    }
}

/* ---- join --------------------------------------------------------------- */

struct JoinArgs {
    const int32_t *tokens;
    const int64_t *starts;
    const int32_t *lengths;
    int64_t n;
    const int64_t *worker_off;
    int64_t n_workers;
    const int32_t *wtokens;
    const int64_t *wstarts;
    const int32_t *wlengths;
    int32_t thread_id, end_thread_id, end_par_id;
    bool close, append_only;
    uint32_t *status;
    int64_t *out_len64;     /* [n] joined lengths for the scan (0 for rows not written) */
    int32_t *out_lengths;
    const int64_t *out_starts;
    const int32_t *over;
    int32_t *out_tokens;
};

/* Joined length and status of row i (the checks of its worker sequences);
 * writes status, out_len64 and out_lengths and returns the length. */
__device__ __forceinline__ int64_t join_row(const JoinArgs &a, int64_t i)
{
    const int64_t L = a.lengths[i], g = a.starts[i];
    const int64_t w0 = a.worker_off[i], w1 = a.worker_off[i + 1];
    uint32_t st = 0;
    int64_t tot = 0;
    if (L < 0 || g < 0 || w0 < 0 || w1 < w0 || w1 > a.n_workers) {
        st = PARASON_PACK_BAD_ROW;
    } else {
        tot = (a.append_only ? 0 : L) + (a.close ? 1 : 0);
        /* JOIN_UNROLL workers at a time: their records in one round of loads,
         * then the tokens after the row and at the end in one more */
        for (int64_t wb = w0; wb < w1; wb += JOIN_UNROLL) {
            /* every load unconditional, from a valid address (the last
             * worker of the row, or this row's own status word, in place of
             * one not needed), and the value selected after it: a load under
             * a condition waits for the one before it */
            int64_t wl[JOIN_UNROLL], ws[JOIN_UNROLL];
#pragma unroll
            for (int u = 0; u < JOIN_UNROLL; ++u) {
                const bool in = wb + u < w1;
                const int64_t w = in ? wb + u : w1 - 1;
                const int64_t l = a.wlengths[w], s = a.wstarts[w];
                wl[u] = in ? l : 0;
                ws[u] = in ? s : 0;
            }
            int32_t first[JOIN_UNROLL], last[JOIN_UNROLL];
            bool chk[JOIN_UNROLL];
            const int32_t *safe = reinterpret_cast<const int32_t *>(a.status + i);
#pragma unroll
            for (int u = 0; u < JOIN_UNROLL; ++u) {
                const int64_t tail = wl[u] > L ? wl[u] - L : 0;
                chk[u] = wb + u < w1 && wl[u] >= 0 && ws[u] >= 0 && tail >= 2;
                const int32_t f = *(chk[u] ? a.wtokens + ws[u] + L : safe);
                const int32_t e = *(chk[u] ? a.wtokens + ws[u] + wl[u] - 1 : safe);
                first[u] = chk[u] ? f : 0;
                last[u] = chk[u] ? e : 0;
            }
#pragma unroll
            for (int u = 0; u < JOIN_UNROLL; ++u) {
                if (wb + u >= w1) break;
                if (wl[u] < 0 || ws[u] < 0) {
                    st |= PARASON_PACK_BAD_ROW;
                    continue;
                }
                if (!chk[u] || first[u] != a.thread_id || last[u] != a.end_thread_id) st |= PARASON_PACK_BAD_THREAD;
                tot += wl[u] > L ? wl[u] - L : 0;
            }
        }
        if (st & PARASON_PACK_BAD_ROW) tot = 0;
        else if (tot > (int64_t)INT32_MAX) {
            st |= PARASON_PACK_TOO_LONG;
            tot = 0;
        }
    }
    a.status[i] = st;
    a.out_len64[i] = tot;
    a.out_lengths[i] = (int32_t)tot;
    return tot;
}

__global__ void __launch_bounds__(JOIN_SIZE_THREADS) join_size(JoinArgs a)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < a.n) join_row(a, i);
}

/* Joined rows, tiled over their tokens by waves like fork_copy.  Inside a
 * row the pieces are the row, each worker's span (its sequence from the
 * <Thread> after the row on) and </Parallel>; the span positions of 64
 * workers at a time come from one wave prefix scan of their lengths.
 * SCAN (up to JOIN_SINGLE rows): every block first scans the joined lengths
 * itself into LDS, where its waves then search the rows (block 0 also writes
 * the offsets, the total and the capacity flag), in place of the separate
 * scan launch and the searches in global memory. */
template <bool SCAN>
__global__ void __launch_bounds__(PACK_THREADS) join_copy(JoinArgs a, PackScan<1> ps)
{
    constexpr int RPT = JOIN_SINGLE / PACK_THREADS; /* rows per thread of the scan */
    __shared__ int64_t soff[SCAN ? JOIN_SINGLE + 1 : 1];
    __shared__ int64_t part[PACK_THREADS / WAVE];
    const int lane = threadIdx.x & (WAVE - 1);
    const int wv = threadIdx.x / WAVE;
    const int64_t *out_starts = a.out_starts;
    if (SCAN) {
        const int64_t r0 = (int64_t)threadIdx.x * RPT;
        int64_t v[RPT], sum = 0;
#pragma unroll
        for (int j = 0; j < RPT; ++j) {
            v[j] = r0 + j < a.n ? a.out_len64[r0 + j] : 0;
            sum += v[j];
        }
        const int64_t inc = wave_inclusive_scan(sum);
        if (lane == WAVE - 1) part[wv] = inc;
        __syncthreads();
        int64_t off = inc - sum, total = 0;
        for (int w = 0; w < PACK_THREADS / WAVE; ++w) {
            off += w < wv ? part[w] : 0;
            total += part[w];
        }
        const int32_t over = total > ps.cap[0] ? 1 : 0;
#pragma unroll
        for (int j = 0; j < RPT; ++j) {
            if (r0 + j < a.n) {
                soff[r0 + j] = off;
                if (blockIdx.x == 0) ps.out[0][r0 + j] = off;
            }
            off += v[j];
        }
        if (threadIdx.x == 0) {
            soff[a.n] = total;
            if (blockIdx.x == 0) {
                ps.out[0][a.n] = total;
                ps.totals[0] = total;
                ps.totals[1] = over;
                ps.over[0] = over;
            }
        }
        __syncthreads();
        if (over) return;
        out_starts = soff;
    } else if (a.over[0]) {
        return;
    }
    const int64_t T = out_starts[a.n];
    const int64_t NW = (int64_t)gridDim.x * COPY_WAVES;
    for (int64_t t = (int64_t)blockIdx.x * COPY_WAVES + wv; t * WTILE < T; t += NW) {
        const int64_t lo = t * WTILE, hi = min(lo + WTILE, T);
        for (int64_t i = wave_find(out_starts, a.n, lo, lane); i < a.n; ++i) {
            /* the row's records in one round of loads, before any branch */
            const int64_t os = out_starts[i], len = a.out_len64[i];
            const int64_t L = a.lengths[i], g0 = a.starts[i];
            const int64_t wb = a.worker_off[i], we = a.worker_off[i + 1];
            if (os >= hi) break;
            if (len == 0) continue;
            int64_t pos = os;
            if (!a.append_only) {
                if (pos + L > lo) wave_copy(a.out_tokens, max(lo, pos), min(hi, pos + L), a.tokens + g0, pos, lane);
                pos += L;
            }
            for (int64_t w = wb; w < we && pos < hi; w += WAVE) {
                const bool in = w + lane < we;
                const int64_t wl = in ? (int64_t)a.wlengths[w + lane] : 0;
                const int64_t ws = in ? a.wstarts[w + lane] : 0;
                const int64_t tail = wl > L ? wl - L : 0;
                const int64_t incl = wave_incl_scan(tail, lane);
                const int64_t at = pos + incl - tail; /* this lane's span in the joined row */
                uint64_t m = __ballot(in && tail > 0 && at < hi && at + tail > lo);
                while (m) {
                    const int k = __builtin_ctzll(m);
                    m &= m - 1;
                    const int64_t s0 = __shfl(at, k, WAVE);
                    const int64_t tl = __shfl(tail, k, WAVE);
                    wave_copy(a.out_tokens, max(lo, s0), min(hi, s0 + tl), a.wtokens + __shfl(ws, k, WAVE) + L, s0,
                              lane);
                }
                pos += __shfl(incl, WAVE - 1, WAVE);
            }
            if (a.close && pos >= lo && pos < hi && lane == 0) a.out_tokens[pos] = a.end_par_id;
        }
    }
}

} /* namespace pk */
