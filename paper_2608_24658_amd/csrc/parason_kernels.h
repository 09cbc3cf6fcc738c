/*
 * parason_kernels.h -- gfx950 kernels of the Parason accounting/reward path.
 *
 * Data flow of one parason_run (all on the caller's stream):
 *
 *   plan_tiles / plan_top / plan_rows  (one plan_rows block for one tile)
 *        Each row is cut into segments of SEG_VEC 16-byte vectors, starting at
 *        the 128-byte line that holds its first token.  A three-pass exclusive
 *        scan gives seg_off[i] (first segment of row i) and the segment count
 *        seg_off[n]; mode[i] is cleared.  A batch that takes rows_par and has
 *        at most SCAN_PLAN_ROWS rows skips these launches: every scan block
 *        makes the plan in LDS itself (scan_plan).
 *   scan_rows  (HBM-bound; one wave per segment, persistent grid)
 *        Streams every token once with 16-byte loads, tests it against the
 *        twelve tag ids with a wave ballot and compacts the rare tags (about
 *        0.1-1% of tokens) in position order.  A row whose segments all fall in
 *        one wave's range collects its events in that wave's LDS buffer and is
 *        written out, coalesced, as one compact list (mode[i] = 1).  Other rows
 *        leave their events in per-segment lists (mode[i] = 0) and are listed
 *        as split.  Every list the scan writes is in the wave's region of the
 *        slot pool; seg[s] holds its length and first slot.
 *   gather_rows  (one wave per split row)
 *        Gathers a split row's per-segment events through LDS into one compact
 *        list with row positions in the row's gather slots (mode[i] = 1).
 *   rows_par  (small batches: one wave per row, four events per lane)
 *        Validity from local checks and a depth prefix sum; latency and branch
 *        tokens level by level with segmented scans (DPP).  A row it cannot
 *        hold runs through the automaton on one lane, with MID_DEPTH frames in
 *        LDS, as in rows_mid.
 *   rows_fast  (larger batches: one thread per row)
 *        The grammar's pushdown automaton over the row's events; Text runs are
 *        the gaps between event positions.  A segment whose events the scan
 *        could not store (marked DENSE) is classified again token by token.
 *        Frames of open blocks in LDS (FAST_DEPTH per row, 64 outline entries
 *        per block); a row that needs more is handed to rows_mid.
 *   rows_mid  (after rows_fast: one thread per handed-over row, MID_DEPTH
 *        frames in LDS)
 *        The same automaton for deeper rows; a row that needs more still is
 *        handed to rows_deep.
 *   rows_deep  (one thread, only rows rows_mid or rows_par handed over)
 *        The same automaton with frames and entry types in global workspace.
 *        Only with batch-wide statistics is this a launch of its own; with
 *        per-group statistics the first block of group_reward runs these rows
 *        and then the rewards of their groups (mode[i] bit MODE_DEEP marks
 *        them, so every other block skips those groups).
 *   group_reward  (one thread per row)
 *        Statistics and Definition 3.1 in IEEE double, fixed order.
 *
 * Paper references: grammar -- figure "Context-Free Grammar for Parason"
 * (Sec. 3.2); latency -- Sec. 4 "Evaluation"; ratios, eta and the reward --
 * Sec. 3.3, Definition 3.1.
 */
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device_common.h"

namespace pk {

/* mode[i], one byte per row: where its events are, and whether the deep tier
 * evaluates it. */
constexpr uint8_t MODE_COMPACT = 1; /* one compact list with row positions (else per-segment lists) */
constexpr uint8_t MODE_DEEP = 2;    /* listed for the single-thread tier with global frames */

/* ------------------------------------------------------------------ plan */

/* tile_sum[b] = number of segments of rows [b*PLAN_TILE, (b+1)*PLAN_TILE). */
__global__ void __launch_bounds__(PLAN_THREADS) plan_tiles(const int64_t *__restrict__ starts,
                                                           const int32_t *__restrict__ lengths, int64_t n,
                                                           int64_t mis, int64_t *__restrict__ tile_sum)
{
    __shared__ int64_t part[PLAN_THREADS / WAVE];
    int64_t r0 = (int64_t)blockIdx.x * PLAN_TILE;
    int64_t s = 0;
    for (int j = 0; j < ROWS_PER_THREAD; ++j) {
        int64_t r = r0 + (int64_t)j * PLAN_THREADS + threadIdx.x; /* coalesced */
        if (r < n) s += row_segments(starts[r], lengths[r], mis);
    }
    s = wave_inclusive_scan(s);
    if ((threadIdx.x & (WAVE - 1)) == WAVE - 1) part[threadIdx.x / WAVE] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        int64_t t = 0;
        for (int w = 0; w < PLAN_THREADS / WAVE; ++w) t += part[w];
        tile_sum[blockIdx.x] = t;
    }
}

/* tile_off = exclusive scan of tile_sum; seg_off[n] = total; clears counters. */
__global__ void __launch_bounds__(1024) plan_top(const int64_t *__restrict__ tile_sum, int64_t n_tiles,
                                                 int64_t *__restrict__ tile_off, int64_t *__restrict__ seg_off,
                                                 int64_t n, int32_t *__restrict__ counters)
{
    __shared__ int64_t part[1024 / WAVE];
    __shared__ int64_t carry_s;
    if (threadIdx.x == 0) carry_s = 0;
    if (threadIdx.x < 4) counters[threadIdx.x] = 0;
    __syncthreads();
    for (int64_t base = 0; base < n_tiles; base += 1024) {
        int64_t i = base + threadIdx.x;
        int64_t v = i < n_tiles ? tile_sum[i] : 0;
        int64_t inc = wave_inclusive_scan(v);
        if ((threadIdx.x & (WAVE - 1)) == WAVE - 1) part[threadIdx.x / WAVE] = inc;
        __syncthreads();
        int64_t before = carry_s;
        for (int w = 0; w < (int)(threadIdx.x / WAVE); ++w) before += part[w];
        if (i < n_tiles) tile_off[i] = before + inc - v;
        __syncthreads();
        if (threadIdx.x == 0) {
            int64_t t = 0;
            for (int w = 0; w < 1024 / WAVE; ++w) t += part[w];
            carry_s += t;
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) seg_off[n] = carry_s;
}

/* seg_off[i] = first segment of row i; mode[i] = 0 (events in per-segment lists). */
/* SINGLE: the batch is one tile, and this one block also does plan_top's
 * work (seg_off[n], clearing the counters), so a small batch is planned with
 * one launch instead of three. */
template <bool SINGLE>
__global__ void __launch_bounds__(PLAN_THREADS) plan_rows(const int64_t *__restrict__ starts,
                                                          const int32_t *__restrict__ lengths, int64_t n,
                                                          int64_t mis, const int64_t *__restrict__ tile_off,
                                                          int64_t *__restrict__ seg_off, uint8_t *__restrict__ mode,
                                                          int32_t *__restrict__ counters)
{
    if (SINGLE && threadIdx.x < 4) counters[threadIdx.x] = 0;
    __shared__ int64_t part[PLAN_THREADS / WAVE];
    /* thread t owns the ROWS_PER_THREAD consecutive rows starting at r0 + t*ROWS_PER_THREAD */
    int64_t r0 = (int64_t)blockIdx.x * PLAN_TILE + (int64_t)threadIdx.x * ROWS_PER_THREAD;
    int64_t cnt[ROWS_PER_THREAD];
    int64_t s = 0;
#pragma unroll
    for (int j = 0; j < ROWS_PER_THREAD; ++j) {
        int64_t r = r0 + j;
        cnt[j] = r < n ? row_segments(starts[r], lengths[r], mis) : 0;
        s += cnt[j];
    }
    int64_t inc = wave_inclusive_scan(s);
    if ((threadIdx.x & (WAVE - 1)) == WAVE - 1) part[threadIdx.x / WAVE] = inc;
    __syncthreads();
    int64_t off = (SINGLE ? 0 : tile_off[blockIdx.x]) + inc - s;
    for (int w = 0; w < (int)(threadIdx.x / WAVE); ++w) off += part[w];
#pragma unroll
    for (int j = 0; j < ROWS_PER_THREAD; ++j) {
        int64_t r = r0 + j;
        if (r < n) {
            seg_off[r] = off;
            mode[r] = 0;
        }
        off += cnt[j];
    }
    if (SINGLE && threadIdx.x == PLAN_THREADS - 1) seg_off[n] = off; /* the last thread ends at the total */
}

/* ------------------------------------------------------------------ automaton */

/* The open block on top of the stack (kept in registers). */
struct Top {
    int32_t saved_acc;  /* latency of the enclosing body when <Parallel> came */
    int32_t block_main; /* <Parallel> + outline tokens so far */
    int32_t max_w;      /* longest finished thread */
    int32_t n_e;        /* outline entries */
    int32_t k;          /* threads so far */
    uint32_t saved_ctx; /* branch type of the enclosing context */
    uint64_t ent;       /* fast store: entry-type bits; deep store: first bit index */
};

/* LDS store: DEPTH frames per thread in LDS, entry types as a 64-bit mask. */
template <int DEPTH>
struct LdsStore {
    int32_t *lds; /* [DEPTH][FRAME_WORDS][blockDim] */
    int tid, nt;
    __device__ int32_t &at(int d, int f) { return lds[(d * FRAME_WORDS + f) * nt + tid]; }
    __device__ bool push(const Top &t, int d)
    {
        if (d > DEPTH) return false;
        at(d - 1, 0) = t.saved_acc;
        at(d - 1, 1) = t.block_main;
        at(d - 1, 2) = t.max_w;
        at(d - 1, 3) = t.n_e;
        at(d - 1, 4) = t.k;
        at(d - 1, 5) = (int32_t)t.saved_ctx;
        at(d - 1, 6) = (int32_t)(uint32_t)t.ent;
        at(d - 1, 7) = (int32_t)(uint32_t)(t.ent >> 32);
        return true;
    }
    __device__ void pop(Top &t, int d)
    {
        t.saved_acc = at(d - 1, 0);
        t.block_main = at(d - 1, 1);
        t.max_w = at(d - 1, 2);
        t.n_e = at(d - 1, 3);
        t.k = at(d - 1, 4);
        t.saved_ctx = (uint32_t)at(d - 1, 5);
        t.ent = (uint64_t)(uint32_t)at(d - 1, 6) | ((uint64_t)(uint32_t)at(d - 1, 7) << 32);
    }
    __device__ void begin_block(Top &t) { t.ent = 0; }
    __device__ void end_block(const Top &) {}
    __device__ bool add_entry(Top &t, bool trial)
    {
        if (t.n_e >= FAST_ENTRIES) return false;
        if (trial) t.ent |= (uint64_t)1 << t.n_e;
        return true;
    }
    __device__ uint32_t entry_type(const Top &t, int32_t k) { return ((t.ent >> k) & 1u) ? T_TRI : T_SUB; }
};

/* Deep store: frames and entry bits in global workspace (single thread). */
struct GlobalStore {
    int32_t *frames;    /* [max_frames][FRAME_WORDS] */
    uint32_t *bits;     /* max_bits bits */
    int64_t max_frames; /* at most DEEP_FRAMES */
    int64_t max_bits;   /* at most DEEP_ENTRY_BITS */
    int64_t esp;      /* next free entry bit */
    __device__ bool push(const Top &t, int d)
    {
        if ((int64_t)d > max_frames) return false;
        int32_t *f = frames + (int64_t)(d - 1) * FRAME_WORDS;
        f[0] = t.saved_acc;
        f[1] = t.block_main;
        f[2] = t.max_w;
        f[3] = t.n_e;
        f[4] = t.k;
        f[5] = (int32_t)t.saved_ctx;
        f[6] = (int32_t)(uint32_t)t.ent;
        f[7] = (int32_t)(uint32_t)(t.ent >> 32);
        return true;
    }
    __device__ void pop(Top &t, int d)
    {
        const int32_t *f = frames + (int64_t)(d - 1) * FRAME_WORDS;
        t.saved_acc = f[0];
        t.block_main = f[1];
        t.max_w = f[2];
        t.n_e = f[3];
        t.k = f[4];
        t.saved_ctx = (uint32_t)f[5];
        t.ent = (uint64_t)(uint32_t)f[6] | ((uint64_t)(uint32_t)f[7] << 32);
    }
    __device__ void begin_block(Top &t) { t.ent = (uint64_t)esp; }
    __device__ void end_block(const Top &t) { esp = (int64_t)t.ent; }
    __device__ bool add_entry(Top &t, bool trial)
    {
        int64_t b = (int64_t)t.ent + t.n_e;
        if (b >= max_bits) return false;
        uint32_t w = bits[b >> 5], m = 1u << (b & 31);
        bits[b >> 5] = trial ? (w | m) : (w & ~m);
        esp = b + 1;
        return true;
    }
    __device__ uint32_t entry_type(const Top &t, int32_t k)
    {
        int64_t b = (int64_t)t.ent + k;
        return ((bits[b >> 5] >> (b & 31)) & 1u) ? T_TRI : T_SUB;
    }
};

enum : uint32_t { S_START, S_BODY, S_P_OPEN, S_O_OPEN, S_ENTRY, S_E_DONE, S_O_DONE, S_W_DONE, S_TRAIL };

/* Pushdown automaton of the grammar, fed with tag events in position order.
 * Text runs are the gaps between consecutive event positions.  LENIENT:
 * PARASON_CFG_LENIENT_GAPS (a compile-time choice, so that the strict
 * automaton carries no code for it). */
template <class Store, bool LENIENT>
struct Automaton {
    Store st;
    int32_t prev;      /* position of the last token consumed */
    uint32_t state;
    int32_t acc;       /* latency of the current body (main or thread) */
    int32_t depth, n_blocks, max_depth;
    int32_t n_sub, n_tri;
    uint32_t ctx;      /* innermost enclosing thread's branch type */
    uint32_t open_tag; /* class of the open entry tag */
    int32_t entry_len; /* Text tokens of the open entry */
    int32_t err;       /* first error position, -1 while none */
    bool mismatch;
    bool overflow;     /* the store ran out: hand the row to the slow path */
    Top top;

    __device__ void init()
    {
        prev = -1;
        state = S_START;
        acc = 0;
        depth = n_blocks = max_depth = 0;
        n_sub = n_tri = 0;
        ctx = T_MAIN;
        open_tag = 0;
        entry_len = 0;
        err = -1;
        mismatch = false;
        overflow = false;
    }

    __device__ void attribute(int32_t n)
    {
        n_sub += ctx == T_SUB ? n : 0;
        n_tri += ctx == T_TRI ? n : 0;
    }

    /* n > 0 Text tokens at prev+1 .. prev+n.  Returns false on error. */
    __device__ bool text(int32_t n)
    {
        switch (state) {
        case S_BODY:
            acc += n;
            attribute(n);
            break;
        case S_ENTRY:
            top.block_main += n;
            entry_len += n;
            attribute(n);
            break;
        case S_TRAIL:
            acc += n;
            break;
        default:
            /* between structural tags of an open region (after <Parallel>,
             * <Outlines>, an entry, </Outlines> or a thread): when lenient a
             * gap, decoded by the enclosing path like the outline */
            if (!LENIENT || state == S_START) {
                err = prev + 1;
                return false;
            }
            top.block_main += n;
            attribute(n);
            break;
        }
        prev += n;
        return true;
    }

    __device__ bool fail(int32_t p)
    {
        err = p;
        return false;
    }

    __device__ void open_thread()
    {
        uint32_t t = top.k < top.n_e ? st.entry_type(top, top.k) : T_MAIN;
        ctx = t;
        acc = 1;
        attribute(1);
        state = S_BODY;
    }

    /* The tag of class c at position p (prev == p - 1).  False on error or
     * store overflow. */
    __device__ bool tag(int32_t p, uint32_t c)
    {
        switch (state) {
        case S_START:
            if (c != C_THINK) return fail(p);
            acc = 1;
            state = S_BODY;
            break;
        case S_BODY:
            if (c == C_PAR) {
                if (depth >= 1 && !st.push(top, depth)) {
                    overflow = true;
                    return false;
                }
                top.saved_acc = acc;
                top.block_main = 1;
                top.max_w = 0;
                top.n_e = 0;
                top.k = 0;
                top.saved_ctx = ctx;
                st.begin_block(top);
                depth += 1;
                n_blocks += 1;
                max_depth = max(max_depth, depth);
                attribute(1);
                state = S_P_OPEN;
            } else if (c == C_END_THINK && depth == 0) {
                acc += 1;
                state = S_TRAIL;
            } else if (c == C_END_THR && depth > 0) {
                acc += 1;
                attribute(1);
                top.max_w = max(top.max_w, acc);
                top.k += 1;
                ctx = top.saved_ctx;
                state = S_W_DONE;
            } else {
                return fail(p);
            }
            break;
        case S_P_OPEN:
            if (c != C_OUT) return fail(p);
            top.block_main += 1;
            attribute(1);
            state = S_O_OPEN;
            break;
        case S_O_OPEN:
        case S_E_DONE:
            if (c == C_SUB || c == C_TRI) {
                top.block_main += 1;
                attribute(1);
                open_tag = c;
                entry_len = 0;
                state = S_ENTRY;
            } else if (c == C_END_OUT && state == S_E_DONE) {
                top.block_main += 1;
                attribute(1);
                state = S_O_DONE;
            } else {
                return fail(p);
            }
            break;
        case S_ENTRY:
            if (entry_len == 0 || c != open_tag + 1) return fail(p);
            if (!st.add_entry(top, open_tag == C_TRI)) {
                overflow = true;
                return false;
            }
            top.n_e += 1;
            top.block_main += 1;
            attribute(1);
            state = S_E_DONE;
            break;
        case S_O_DONE:
        case S_W_DONE:
            if (c == C_THR) {
                open_thread();
            } else if (c == C_END_PAR && state == S_W_DONE) {
                if (top.k != top.n_e) mismatch = true;
                attribute(1);
                int32_t lat = top.block_main + top.max_w + 1;
                acc = top.saved_acc + lat;
                st.end_block(top);
                depth -= 1;
                if (depth >= 1) st.pop(top, depth);
                state = S_BODY;
            } else {
                return fail(p);
            }
            break;
        default: /* S_TRAIL: only Text may follow </think> */
            return fail(p);
        }
        prev = p;
        return true;
    }

    __device__ bool event(int32_t p, uint32_t c)
    {
        int32_t gap = p - prev - 1;
        if (gap > 0 && !text(gap)) return false;
        return tag(p, c);
    }

    /* End of the row (no error or overflow so far). */
    __device__ void finish(int32_t len)
    {
        int32_t gap = len - prev - 1;
        if (gap > 0 && !text(gap)) return;
        if (state != S_TRAIL) err = len;
    }
};

struct RowOut {
    int32_t *total, *latency, *n_subtask, *n_trial, *n_blocks, *max_depth, *first_error_pos;
    uint32_t *flags;
};

__device__ __forceinline__ void write_row(const RowOut &o, int64_t r, int32_t total, int32_t lat, int32_t ns,
                                          int32_t nt, int32_t nb, int32_t md, int32_t fe, uint32_t fl)
{
    o.total[r] = total;
    o.latency[r] = lat;
    o.n_subtask[r] = ns;
    o.n_trial[r] = nt;
    o.n_blocks[r] = nb;
    o.max_depth[r] = md;
    o.first_error_pos[r] = fe;
    o.flags[r] = fl;
}

template <class Store, bool LENIENT>
__device__ __forceinline__ void write_result(const RowOut &o, int64_t r, int32_t len, const Automaton<Store, LENIENT> &A)
{
    if (A.err < 0) {
        uint32_t fl = PARASON_FLAG_VALID;
        if (A.mismatch) fl |= PARASON_FLAG_COUNT_MISMATCH;
        if (A.n_blocks > 0) fl |= PARASON_FLAG_TRIGGERED;
        write_row(o, r, len, A.acc, A.n_sub, A.n_tri, A.n_blocks, A.max_depth, -1, fl);
    } else {
        write_row(o, r, len, len, 0, 0, 0, 0, A.err, A.err == len ? PARASON_FLAG_TRUNCATED : 0u);
    }
}

struct RowArgs {
    const int32_t *tok_base;
    int64_t mis;
    const int64_t *starts;
    const int32_t *lengths;
    int64_t n;
    const int64_t *seg_off;
    int64_t seg_cap;
    const SegRec *seg;
    const uint32_t *slots;
    int64_t deep_frames;    /* frames of the deep tier's store in workspace ... */
    int64_t deep_bits;      /* ... and its entry bits */
    TagMatch tm;
    RowOut out;
};

/* Feed row r's events to A.  Returns false when A stopped early.
 *
 * Three sources, all feeding the one call of A.event below: a compact list
 * (the whole row: seg[first], row positions), or per segment
 * its stored list (segment positions) or, for a segment marked DENSE, its
 * tokens classified again one by one.  Lists start at slots + seg[s].list.
 * With two inlined copies of the automaton (one per source) the
 * gfx950 build returned wrong results for dense segments although the same
 * source is correct when compiled for the CPU, so the sources are merged into
 * one fetch loop. */
template <class Store, bool LENIENT>
__device__ bool drive_row(const RowArgs &a, int64_t r, int64_t g, int32_t len, bool compact,
                          Automaton<Store, LENIENT> &A)
{
    const int64_t s0 = a.seg_off[r], s1 = a.seg_off[r + 1];
    const int64_t vrow0 = row_first_vec(g), vend = row_end_vec(g, len);
    int64_t s = s0;              /* next segment to open */
    const uint32_t *ev = nullptr;
    int32_t e = 0, cnt = 0;      /* stored-event cursor and list length */
    int64_t base = 0;            /* row position of stored position 0 */
    bool dense = false;
    int64_t q = 0, q_end = 0;    /* dense cursor (element index on the token grid) */
    uint4 quad = make_uint4(0u, 0u, 0u, 0u);
    if (compact) {
        const SegRec rec = a.seg[s0];
        ev = a.slots + rec.list;
        cnt = rec.count;
        s = s1;
    }
    for (;;) {
        int32_t p = 0;
        uint32_t c = 0;
        for (;;) {
            if (!dense && e < cnt) {
                /* lists start 16-byte aligned and take multiples of 4 slots:
                 * read them 16 bytes at a time */
                if ((e & 3) == 0) quad = *reinterpret_cast<const uint4 *>(ev + e);
                const uint32_t k = (uint32_t)e & 3u;
                const uint32_t w = k == 0 ? quad.x : k == 1 ? quad.y : k == 2 ? quad.z : quad.w;
                ++e;
                p = (int32_t)(base + (w >> 4));
                c = w & 15u;
                break;
            }
            if (dense) {
                while (q < q_end) {
                    const int32_t t = a.tok_base[q];
                    const int64_t pp = q - g;
                    ++q;
                    if (pp < 0 || pp >= len) continue;
                    c = classify(a.tm, t, a.tm.contiguous != 0);
                    if (c) {
                        p = (int32_t)pp;
                        break;
                    }
                }
                if (c) break;
                dense = false;
            }
            if (s >= s1) break;
            /* open segment s */
            const int64_t v0 = vrow0 + (s - s0) * SEG_VEC;
            const SegRec rec = a.seg[s];
            const int32_t n_s = rec.count;
            base = 4 * v0 - g;
            e = 0;
            if (n_s != DENSE) {
                cnt = n_s;
                ev = a.slots + rec.list; /* not read when n_s is 0 */
            } else {
                cnt = 0;
                dense = true;
                q = 4 * v0;
                q_end = 4 * min(v0 + (int64_t)SEG_VEC, vend);
            }
            ++s;
        }
        if (c == 0) break; /* no more events */
        if (!A.event(p, c)) return false;
    }
    return true;
}

/* One thread per row.  mode[r] == MODE_COMPACT: the scan left the row's events as one
 * compact list; 0: per-segment lists.  A row that needs more than FAST_DEPTH
 * frames (or more than 64 entries in an open block) is listed for rows_mid.
 * Few frames keep the LDS per block small, so that many waves hide the
 * latency of the branchy automaton. */
template <bool LENIENT>
__global__ void __launch_bounds__(64) rows_fast(RowArgs a, const uint8_t *__restrict__ mode,
                                                int32_t *__restrict__ counters, int32_t *__restrict__ mid_rows,
                                                int32_t lane_shift)
{
    __shared__ int32_t lds[FAST_DEPTH * FRAME_WORDS * 64];
    /* every (1 << lane_shift)-th lane takes a row (64 >> lane_shift rows per wave) */
    if ((threadIdx.x & ((1u << lane_shift) - 1u)) != 0) return;
    const int64_t r = (int64_t)blockIdx.x * (blockDim.x >> lane_shift) + (threadIdx.x >> lane_shift);
    if (r >= a.n) return;
    const int64_t start = a.starts[r];
    const int32_t len = a.lengths[r];
    if (start < 0 || len < 0) {
        write_row(a.out, r, 0, 0, 0, 0, 0, 0, 0, PARASON_FLAG_BAD_ROW);
        return;
    }
    if (a.seg_off[a.n] > a.seg_cap) {
        write_row(a.out, r, len, 0, 0, 0, 0, 0, 0, PARASON_FLAG_WS_OVERFLOW);
        return;
    }
    Automaton<LdsStore<FAST_DEPTH>, LENIENT> A;
    A.st.lds = lds;
    A.st.tid = threadIdx.x;
    A.st.nt = blockDim.x;
    A.init();
    if (drive_row(a, r, start + a.mis, len, (mode[r] & MODE_COMPACT) != 0, A)) A.finish(len);
    if (A.overflow) {
        mid_rows[atomicAdd(&counters[0], 1)] = (int32_t)r;
        return; /* rows_mid writes this row */
    }
    write_result(a.out, r, len, A);
}

/* The rows rows_fast listed, one thread each (grid-stride over the list), with
 * MID_DEPTH frames per row in LDS; rows that need still more are listed for
 * rows_deep. */
template <bool LENIENT>
__global__ void __launch_bounds__(64) rows_mid(RowArgs a, uint8_t *__restrict__ mode,
                                               int32_t *__restrict__ counters, const int32_t *__restrict__ mid_rows,
                                               int32_t *__restrict__ deep_rows)
{
    __shared__ int32_t lds[MID_DEPTH * FRAME_WORDS * 64];
    const int32_t n_mid = counters[0];
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_mid;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t r = mid_rows[i];
        const int32_t len = a.lengths[r];
        Automaton<LdsStore<MID_DEPTH>, LENIENT> A;
        A.st.lds = lds;
        A.st.tid = threadIdx.x;
        A.st.nt = blockDim.x;
        A.init();
        if (drive_row(a, r, a.starts[r] + a.mis, len, (mode[r] & MODE_COMPACT) != 0, A)) A.finish(len);
        if (A.overflow) {
            mode[r] |= MODE_DEEP;
            int32_t slot = atomicAdd(&counters[1], 1);
            deep_rows[slot] = (int32_t)r;
        } else {
            write_result(a.out, r, len, A);
        }
    }
}

/* Rows whose nesting or entry count exceeded the LDS stores, one after the
 * other, on the calling thread with frames in global workspace. */
template <bool LENIENT>
__device__ void run_deep_rows(const RowArgs &a, const uint8_t *__restrict__ mode, int32_t n_deep,
                              const int32_t *__restrict__ deep_rows, int32_t *__restrict__ frames,
                              uint32_t *__restrict__ bits)
{
    for (int32_t i = 0; i < n_deep; ++i) {
        const int64_t r = deep_rows[i];
        const int32_t len = a.lengths[r];
        Automaton<GlobalStore, LENIENT> A;
        A.st.frames = frames;
        A.st.bits = bits;
        A.st.max_frames = a.deep_frames;
        A.st.max_bits = a.deep_bits;
        A.st.esp = 0;
        A.init();
        if (drive_row(a, r, a.starts[r] + a.mis, len, (mode[r] & MODE_COMPACT) != 0, A)) A.finish(len);
        if (A.overflow)
            write_row(a.out, r, len, 0, 0, 0, 0, 0, 0, PARASON_FLAG_DEPTH_LIMIT);
        else
            write_result(a.out, r, len, A);
    }
}

/* The deep rows on a single thread, as a launch of its own: used when the
 * batch-wide statistics need every row before the reward. */
template <bool LENIENT>
__global__ void __launch_bounds__(64) rows_deep(RowArgs a, const uint8_t *__restrict__ mode,
                                                const int32_t *__restrict__ counters,
                                                const int32_t *__restrict__ deep_rows, int32_t *__restrict__ frames,
                                                uint32_t *__restrict__ bits)
{
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    run_deep_rows<LENIENT>(a, mode, counters[1], deep_rows, frames, bits);
}

/* ------------------------------------------------------------------ rows_par */

constexpr int PAR_EVENTS = 512; /* events of a row rows_par holds in LDS */
constexpr int PAR_LEVELS = 16;  /* nesting rows_par evaluates */

/* The classes that may follow state st (one bit per class). */
constexpr uint32_t allowed_classes(uint32_t st)
{
    switch (st) {
    case S_START: return 1u << C_THINK;
    case S_BODY: return (1u << C_PAR) | (1u << C_END_THINK) | (1u << C_END_THR);
    case S_P_OPEN: return 1u << C_OUT;
    case S_O_OPEN: return (1u << C_SUB) | (1u << C_TRI);
    case S_ENTRY: return (1u << C_END_SUB) | (1u << C_END_TRI);
    case S_E_DONE: return (1u << C_SUB) | (1u << C_TRI) | (1u << C_END_OUT);
    case S_O_DONE: return 1u << C_THR;
    case S_W_DONE: return (1u << C_THR) | (1u << C_END_PAR);
    default: return 0u; /* S_TRAIL */
    }
}

/* The state after a tag of class c: the class alone decides it. */
constexpr uint32_t state_after(int32_t c)
{
    switch (c) {
    case C_THINK: return S_BODY;
    case C_END_THINK: return S_TRAIL;
    case C_PAR: return S_P_OPEN;
    case C_END_PAR: return S_BODY;
    case C_OUT: return S_O_OPEN;
    case C_END_OUT: return S_O_DONE;
    case C_SUB:
    case C_TRI: return S_ENTRY;
    case C_END_SUB:
    case C_END_TRI: return S_E_DONE;
    case C_THR: return S_BODY;
    default: return S_W_DONE; /* C_END_THR */
    }
}

/* The two functions above as bit tables, for lanes whose classes differ (a
 * switch there runs every case under an execution mask):
 *   state_at(pc)      the state after a tag of class pc, S_START for pc = -1
 *                     (the row's start): one nibble per pc + 1;
 *   class_allowed     bit 13 * st + c of a 128-bit table;
 *   text_allowed      Text may stand in state st (strict grammar). */
constexpr uint64_t state_table()
{
    uint64_t t = S_START;
    for (int32_t c = 0; c <= (int32_t)C_END_THR; ++c) t |= (uint64_t)state_after(c) << (4 * (c + 1));
    return t;
}
constexpr uint64_t allowed_table(int word)
{
    uint64_t t = 0;
    for (uint32_t st = S_START; st <= S_TRAIL; ++st)
        for (uint32_t c = 0; c <= C_END_THR; ++c) {
            const uint32_t bit = 13u * st + c;
            if ((allowed_classes(st) >> c) & 1u && bit / 64u == (uint32_t)word) t |= 1ull << (bit % 64u);
        }
    return t;
}
constexpr uint64_t STATE_TAB = state_table();
constexpr uint64_t ALLOWED_TAB0 = allowed_table(0), ALLOWED_TAB1 = allowed_table(1);
constexpr uint32_t TEXT_STATES = (1u << S_BODY) | (1u << S_TRAIL) | (1u << S_ENTRY);
static_assert(13u * S_TRAIL + C_END_THR < 128u, "the table holds every state and class");
static_assert(C_END_THR + 2 <= 16, "a nibble per class and the start");

__device__ __forceinline__ uint32_t state_at(int32_t pc) { return (uint32_t)(STATE_TAB >> (4 * (pc + 1))) & 15u; }
__device__ __forceinline__ bool class_allowed(uint32_t st, int32_t c)
{
    const uint32_t bit = 13u * st + (uint32_t)c;
    return ((bit < 64u ? ALLOWED_TAB0 : ALLOWED_TAB1) >> (bit & 63u)) & 1u;
}
__device__ __forceinline__ bool text_allowed(uint32_t st) { return (TEXT_STATES >> st) & 1u; }

/* Inclusive prefix sum and running maximum over the wave's lanes. */
__device__ __forceinline__ int32_t wave_incl_scan32(int32_t v, int lane) { return dpp_incl_scan<OpAdd>(v, lane); }
__device__ __forceinline__ int32_t wave_incl_max32(int32_t v, int lane) { return dpp_incl_scan<OpMax>(v, lane); }

template <bool MAX>
__device__ __forceinline__ int32_t wave_seg_scan(int32_t v, bool head, int32_t carry, int lane)
{
    return MAX ? dpp_seg_scan<OpMax>(v, head, carry, lane) : dpp_seg_scan<OpAdd>(v, head, carry, lane);
}

/* Reductions over the wave, the result in every lane. */
__device__ __forceinline__ int32_t wave_sum32(int32_t v)
{
    return lane63(dpp_incl_scan<OpAdd>(v, (int)(threadIdx.x & (WAVE - 1))));
}
__device__ __forceinline__ int32_t wave_min32(int32_t v)
{
    return lane63(dpp_incl_scan<OpMin>(v, (int)(threadIdx.x & (WAVE - 1))));
}
__device__ __forceinline__ int32_t wave_max32(int32_t v)
{
    return lane63(dpp_incl_scan<OpMax>(v, (int)(threadIdx.x & (WAVE - 1))));
}

/* The largest lane j with x (held by lane j) <= f, for x non-decreasing over
 * the lanes and x of lane 0 <= f (every lane must call it). */
__device__ __forceinline__ int32_t last_lane_at_most(int32_t x, int32_t f)
{
    int32_t lo = 0;
#pragma unroll
    for (int step = WAVE / 2; step > 0; step >>= 1) {
        const int32_t cand = lo + step;
        lo = __shfl(x, cand, WAVE) <= f ? cand : lo;
    }
    return lo;
}

/* Events in passes of PAR_PASS: event i0 + PAR_K * lane + k is element k of
 * the lane, so a row of up to PAR_PASS events takes one wave scan per
 * quantity instead of one per 64 events (the scans are latency: a chain of
 * DPP steps and cross-row reads each). */
constexpr int PAR_K = 4;
constexpr int PAR_PASS = PAR_K * WAVE;
static_assert(PAR_EVENTS % PAR_PASS == 0, "passes end inside the LDS arrays");

__device__ __forceinline__ void par_load(const int32_t *s, int32_t ib, int32_t (&v)[PAR_K])
{
    const int4 x = *reinterpret_cast<const int4 *>(s + ib);
    v[0] = x.x;
    v[1] = x.y;
    v[2] = x.z;
    v[3] = x.w;
}

__device__ __forceinline__ void par_store(int32_t *s, int32_t ib, const int32_t (&v)[PAR_K])
{
    *reinterpret_cast<int4 *>(s + ib) = make_int4(v[0], v[1], v[2], v[3]);
}

__device__ __forceinline__ int32_t par_pick(const int32_t (&v)[PAR_K], int32_t k)
{
    return k == 0 ? v[0] : k == 1 ? v[1] : k == 2 ? v[2] : v[3];
}

/* Inclusive scan over the wave's events in order, continuing from carry. */
template <class Op>
__device__ __forceinline__ void par_incl_scan(int32_t (&v)[PAR_K], int32_t carry, int lane)
{
#pragma unroll
    for (int k = 1; k < PAR_K; ++k) v[k] = Op::f(v[k - 1], v[k]);
    const int32_t before = Op::f(carry, lane_before(dpp_incl_scan<Op>(v[PAR_K - 1], lane), Op::ident));
#pragma unroll
    for (int k = 0; k < PAR_K; ++k) v[k] = Op::f(before, v[k]);
}

/* Segmented form: restarts at events with head set; events before the first
 * head continue from carry. */
template <class Op>
__device__ __forceinline__ void par_seg_scan(int32_t (&v)[PAR_K], const bool (&head)[PAR_K], int32_t carry, int lane)
{
    bool any = head[0];
#pragma unroll
    for (int k = 1; k < PAR_K; ++k) {
        if (!head[k]) v[k] = Op::f(v[k - 1], v[k]);
        any = any || head[k];
    }
    const int32_t in = lane_before(dpp_seg_scan<Op>(v[PAR_K - 1], any, carry, lane), carry);
    bool seen = false;
#pragma unroll
    for (int k = 0; k < PAR_K; ++k) {
        seen = seen || head[k];
        if (!seen) v[k] = Op::f(in, v[k]);
    }
}

/* One wave per row, its lanes over the row's events, four consecutive events
 * per lane (a small batch).  The same results as the automaton, from the
 * structure of the grammar:
 *   - the state before a tag is fixed by the class of the tag before it, and
 *     the nesting depth before it is a prefix sum, so every check of the
 *     automaton is local to an event and its predecessor; the row's first
 *     error is the smallest error position over the events (phase A);
 *   - for a valid row, with saved(P) = sum_k tokens(W_k) - max_k lat(W_k)
 *     over the threads W_k of block P, and lat(W) = tokens(W) - the saved
 *     tokens of the blocks directly inside W, the latency is the row's
 *     length less the saved tokens of its top-level blocks; a thread's own
 *     tokens (its tokens less those of the threads nested in it) take the
 *     type of the outline entry it pairs with.  Evaluated level by level,
 *     deepest first, with segmented scans, one pass over the events per
 *     level (phase B).
 * Rows holding more than PAR_EVENTS events, nested deeper than PAR_LEVELS,
 * or with a dense segment, run through the automaton on lane 0 (the single
 * automaton call site of this kernel).  Split rows are read from their
 * segments' lists directly (no gather_rows launch for a small batch). */
template <bool LENIENT>
__global__ void __launch_bounds__(64) rows_par(RowArgs a, uint8_t *__restrict__ mode,
                                               int32_t *__restrict__ counters, int32_t *__restrict__ deep_rows)
{
    __shared__ __align__(16) int32_t sP[PAR_EVENTS], sC[PAR_EVENTS], sD[PAR_EVENTS], sT[PAR_EVENTS];
    __shared__ __align__(16) int32_t sTOK[PAR_EVENTS], sLAT[PAR_EVENTS], sOWN[PAR_EVENTS], sSAV[PAR_EVENTS];
    const int lane = threadIdx.x;
    const int64_t r = blockIdx.x;
    if (r >= a.n) return;
    /* the row's records in one round of loads, before any branch */
    const int64_t start = a.starts[r];
    const int32_t len = a.lengths[r];
    const int64_t S = a.seg_off[a.n], s0 = a.seg_off[r], s1 = a.seg_off[r + 1];
    const uint8_t md = mode[r];
    if (start < 0 || len < 0) {
        if (lane == 0) write_row(a.out, r, 0, 0, 0, 0, 0, 0, 0, PARASON_FLAG_BAD_ROW);
        return;
    }
    if (S > a.seg_cap) {
        if (lane == 0) write_row(a.out, r, len, 0, 0, 0, 0, 0, 0, PARASON_FLAG_WS_OVERFLOW);
        return;
    }
    /* the row's events into LDS, in position order: from its compact list (row
     * positions), or from its segments' lists (segment positions), gathered
     * here as gather_rows does for the per-lane kernel */
    const int64_t g = start + a.mis;
    int32_t m = 0;
    bool held = true;
    if (md & MODE_COMPACT) {
        const SegRec rec = a.seg[s0];
        m = rec.count;
        held = m <= PAR_EVENTS;
        const uint32_t *list = a.slots + rec.list;
        for (int32_t i0 = 0; held && i0 < m; i0 += 4 * WAVE) { /* four loads per lane in flight */
            uint32_t w[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int32_t i = i0 + u * WAVE + lane;
                w[u] = i < m ? list[i] : 0u;
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int32_t i = i0 + u * WAVE + lane;
                if (i < m) {
                    sP[i] = (int32_t)(w[u] >> 4);
                    sC[i] = (int32_t)(w[u] & 15u);
                }
            }
        }
    } else {
        /* PAR_PASS segments at a time, four per lane: their records in one
         * round of loads and an exclusive scan of their counts; then an LDS
         * map from event to segment (each segment that holds events marks its
         * first event, a running maximum spreads the marks) and the events'
         * loads in one round per PAR_PASS events.  Until phase A, sD holds the
         * map and sLAT, sOWN each segment's first slot and first event. */
        const int64_t vrow0 = row_first_vec(g);
        for (int64_t c0 = s0; held && c0 < s1; c0 += PAR_PASS) {
            const int32_t jb = PAR_K * lane; /* the chunk's segment of element 0 */
            int32_t cnt[PAR_K], lst[PAR_K], incl[PAR_K];
            bool dense = false;
#pragma unroll
            for (int k = 0; k < PAR_K; ++k) {
                const int64_t s = c0 + jb + k;
                const SegRec rec = s < s1 ? a.seg[s] : SegRec{0, 0u};
                cnt[k] = rec.count;
                lst[k] = (int32_t)rec.list; /* meaningless for a segment without events */
                incl[k] = cnt[k];
                dense = dense || cnt[k] == DENSE;
            }
            par_incl_scan<OpAdd>(incl, 0, lane); /* DENSE counts cannot overflow it */
            const int32_t total = lane63(incl[PAR_K - 1]);
            /* a dense segment or too many events: the automaton below */
            held = __ballot(dense) == 0 && m + total <= PAR_EVENTS;
            if (!held || total == 0) continue;
            for (int32_t f0 = 0; f0 < total; f0 += PAR_PASS) par_store(sD, f0 + jb, {-1, -1, -1, -1});
            __syncthreads();
#pragma unroll
            for (int k = 0; k < PAR_K; ++k) {
                if (cnt[k] > 0) {
                    const int32_t e0 = incl[k] - cnt[k];
                    sD[e0] = jb + k;
                    sLAT[jb + k] = lst[k];
                    sOWN[jb + k] = e0;
                }
            }
            __syncthreads();
            int32_t carry = -1;
            for (int32_t f0 = 0; f0 < total; f0 += PAR_PASS) {
                int32_t j[PAR_K];
                uint32_t w[PAR_K];
                par_load(sD, f0 + jb, j);
                par_incl_scan<OpMax>(j, carry, lane); /* every event's segment (position 0 is marked) */
#pragma unroll
                for (int k = 0; k < PAR_K; ++k) {
                    const int32_t f = f0 + jb + k, jj = max(j[k], 0);
                    w[k] = f < total ? a.slots[(int64_t)(uint32_t)sLAT[jj] + (f - sOWN[jj])] : 0u;
                }
#pragma unroll
                for (int k = 0; k < PAR_K; ++k) {
                    const int32_t f = f0 + jb + k;
                    if (f < total) {
                        const int64_t seg = c0 + j[k];
                        sP[m + f] = (int32_t)(4 * (vrow0 + (seg - s0) * SEG_VEC) - g + (int64_t)(w[k] >> 4));
                        sC[m + f] = (int32_t)(w[k] & 15u);
                    }
                }
                carry = lane63(j[PAR_K - 1]);
            }
            __syncthreads(); /* the next chunk rewrites the map */
            m += total;
        }
    }
    /* phase A: validity, first error, depth and open threads before each event */
    int32_t prev_c = -1, prev_p = -1, depth = 0, threads = 0, err = INT32_MAX, max_depth = 0, n_blocks = 0;
    bool fallback = !held; /* the row goes to the automaton below */
    do {
        if (fallback) break;
        __syncthreads();
        for (int32_t i0 = 0; i0 < m && err == INT32_MAX; i0 += PAR_PASS) {
            const int32_t ib = i0 + PAR_K * lane;
            int32_t c[PAR_K], p[PAR_K], dd[PAR_K], dt[PAR_K];
            par_load(sC, ib, c);
            par_load(sP, ib, p);
#pragma unroll
            for (int k = 0; k < PAR_K; ++k) {
                if (ib + k >= m) c[k] = p[k] = 0;
                dd[k] = ib + k < m ? (c[k] == C_PAR) - (c[k] == C_END_PAR) : 0;
                dt[k] = ib + k < m ? (c[k] == C_THR) - (c[k] == C_END_THR) : 0;
            }
            int32_t d_in[PAR_K], t_in[PAR_K]; /* depth and open threads after each event */
#pragma unroll
            for (int k = 0; k < PAR_K; ++k) {
                d_in[k] = dd[k];
                t_in[k] = dt[k];
            }
            par_incl_scan<OpAdd>(d_in, depth, lane);
            par_incl_scan<OpAdd>(t_in, threads, lane);
            int32_t pc = lane_before(c[PAR_K - 1], prev_c), pp = lane_before(p[PAR_K - 1], prev_p);
            int32_t e = INT32_MAX, open_depth = 0, pars = 0;
            int32_t dbv[PAR_K], tbv[PAR_K];
#pragma unroll
            for (int k = 0; k < PAR_K; ++k) {
                /* the checks of one event, without branches (bitwise, not
                 * short-circuit: lanes hold different classes) */
                const int32_t db = d_in[k] - dd[k], tb = t_in[k] - dt[k];
                const int32_t ck = c[k];
                const bool act = ib + k < m;
                const uint32_t st = state_at(pc);
                const int32_t gap = p[k] - pp - 1;
                const bool text_ok = (gap == 0) | text_allowed(st) | (LENIENT & (st != S_START));
                const bool closes_entry = (ck == C_END_SUB) | (ck == C_END_TRI);
                const bool tag_ok = class_allowed(st, ck) & !((ck == C_END_THINK) & (db != 0)) &
                                    !((ck == C_END_THR) & (db == 0)) & !(closes_entry & ((ck != pc + 1) | (gap == 0)));
                const int32_t ek = text_ok ? (tag_ok ? INT32_MAX : p[k]) : pp + 1;
                const bool opens = act & (ck == C_PAR);
                e = min(e, act ? ek : INT32_MAX);
                open_depth = max(open_depth, opens ? db + 1 : 0);
                pars += opens ? 1 : 0;
                dbv[k] = db;
                tbv[k] = tb;
                pc = c[k];
                pp = p[k];
            }
            par_store(sD, ib, dbv);
            par_store(sT, ib, tbv);
            err = wave_min32(e);
            max_depth = max(max_depth, wave_max32(open_depth));
            n_blocks += wave_sum32(pars);
            /* the pass's last event: the one before the next pass's first */
            const int32_t last = min(m - i0, PAR_PASS) - 1;
            prev_c = __builtin_amdgcn_readlane(par_pick(c, last % PAR_K), last / PAR_K);
            prev_p = __builtin_amdgcn_readlane(par_pick(p, last % PAR_K), last / PAR_K);
            depth = lane63(d_in[PAR_K - 1]);
            threads = lane63(t_in[PAR_K - 1]);
        }
        if (err == INT32_MAX) {
            /* the end of the row: the text after the last tag, then </think> must have come */
            const uint32_t st = state_at(prev_c);
            const int32_t gap = len - prev_p - 1;
            const bool text_ok = gap == 0 || text_allowed(st) || (LENIENT && st != S_START);
            if (!text_ok) err = prev_p + 1;
            else if (st != S_TRAIL) err = len;
        }
        if (err != INT32_MAX) {
            if (lane == 0) write_row(a.out, r, len, len, 0, 0, 0, 0, err, err == len ? PARASON_FLAG_TRUNCATED : 0u);
            return;
        }
        fallback = max_depth > PAR_LEVELS;
    } while (0);
    if (fallback) {
        /* a row this kernel does not hold (more than PAR_EVENTS events, a dense
         * segment, nesting deeper than PAR_LEVELS): the automaton on one lane
         * with MID_DEPTH frames in LDS (sTOK, unused on this path), as rows_mid
         * would; a row that needs still more is listed for rows_deep */
        if (lane == 0) {
            Automaton<LdsStore<MID_DEPTH>, LENIENT> A;
            A.st.lds = sTOK;
            A.st.tid = 0;
            A.st.nt = 1;
            A.init();
            if (drive_row(a, r, g, len, (md & MODE_COMPACT) != 0, A)) A.finish(len);
            if (A.overflow) {
                mode[r] = md | MODE_DEEP;
                deep_rows[atomicAdd(&counters[1], 1)] = (int32_t)r;
            }
            else write_result(a.out, r, len, A);
        }
        return;
    }
    __syncthreads();

    /* phase B: level by level, deepest first */
    int32_t my_sub = 0, my_tri = 0, my_saved = 0;
    bool my_mismatch = false;
    for (int32_t lev = max_depth; lev >= 1; --lev) {
        /* one pass per level: the threads of level lev (tokens, latency, own
         * tokens), then, from those values still in registers, the blocks of
         * level lev (saved tokens, thread types, count mismatch) */
        int32_t c_thr = -1, c_S = 0, c_CH = 0;
        int32_t c_sum = 0, c_max = 0, c_n = 0, c_par = -1, c_eout = -1;
        for (int32_t i0 = 0; i0 < m; i0 += PAR_PASS) {
            const int32_t ib = i0 + PAR_K * lane;
            int32_t c[PAR_K], db[PAR_K], tb[PAR_K], sav[PAR_K], tk[PAR_K];
            par_load(sC, ib, c);
            par_load(sD, ib, db);
            par_load(sT, ib, tb);
            par_load(sSAV, ib, sav);
            par_load(sTOK, ib, tk);
            bool thr[PAR_K], ethr[PAR_K], par[PAR_K], epar[PAR_K];
            int32_t ti[PAR_K], S[PAR_K], CH[PAR_K], pi[PAR_K], oi[PAR_K];
#pragma unroll
            for (int k = 0; k < PAR_K; ++k) {
                const bool act = ib + k < m;
                thr[k] = act & (c[k] == C_THR) & (tb[k] == lev - 1);
                ethr[k] = act & (c[k] == C_END_THR) & (tb[k] == lev);
                const bool epar_in = act & (c[k] == C_END_PAR) & (db[k] == lev + 1);
                const bool ethr_in = act & (c[k] == C_END_THR) & (tb[k] == lev + 1);
                par[k] = act & (c[k] == C_PAR) & (db[k] == lev - 1);
                epar[k] = act & (c[k] == C_END_PAR) & (db[k] == lev);
                const bool eout = act & (c[k] == C_END_OUT) & (db[k] == lev) & (tb[k] == lev - 1);
                ti[k] = thr[k] ? ib + k : -1;
                S[k] = epar_in ? sav[k] : 0;
                CH[k] = ethr_in ? tk[k] : 0;
                pi[k] = par[k] ? ib + k : -1;
                oi[k] = eout ? ib + k : -1;
            }
            par_incl_scan<OpMax>(ti, c_thr, lane);  /* the thread each event is in */
            par_seg_scan<OpAdd>(S, thr, c_S, lane);
            par_seg_scan<OpAdd>(CH, thr, c_CH, lane);
            par_incl_scan<OpMax>(pi, c_par, lane);  /* the block each event is in ... */
            par_incl_scan<OpMax>(oi, c_eout, lane); /* ... and its outline's end */
            int32_t sum[PAR_K], mx[PAR_K], nt[PAR_K], own[PAR_K];
#pragma unroll
            for (int k = 0; k < PAR_K; ++k) {
                const int32_t tok = ethr[k] ? sP[ib + k] - sP[max(ti[k], 0)] + 1 : 0;
                if (ethr[k]) sTOK[ib + k] = tok; /* read by the next level's threads */
                sum[k] = tok;
                mx[k] = ethr[k] ? tok - S[k] : 0; /* the thread's latency */
                own[k] = tok - CH[k];
                nt[k] = ethr[k] ? 1 : 0;
            }
            par_seg_scan<OpAdd>(sum, par, c_sum, lane);
            par_seg_scan<OpMax>(mx, par, c_max, lane);
            par_seg_scan<OpAdd>(nt, par, c_n, lane);
#pragma unroll
            for (int k = 0; k < PAR_K; ++k) {
                const int32_t n_e = (oi[k] - pi[k] - 2) / 2;
                if (ethr[k]) {
                    const int32_t kk = nt[k] - 1; /* thread kk pairs with entry kk */
                    if (kk < n_e) {
                        const int32_t t = sC[pi[k] + 2 + 2 * kk];
                        my_sub += t == C_SUB ? own[k] : 0;
                        my_tri += t == C_TRI ? own[k] : 0;
                    }
                }
                if (epar[k]) {
                    const int32_t saved = sum[k] - mx[k];
                    sSAV[ib + k] = saved;
                    my_mismatch = my_mismatch || nt[k] != n_e;
                    my_saved += lev == 1 ? saved : 0;
                }
            }
            c_thr = lane63(ti[PAR_K - 1]);
            c_S = lane63(S[PAR_K - 1]);
            c_CH = lane63(CH[PAR_K - 1]);
            c_sum = lane63(sum[PAR_K - 1]);
            c_max = lane63(mx[PAR_K - 1]);
            c_n = lane63(nt[PAR_K - 1]);
            c_par = lane63(pi[PAR_K - 1]);
            c_eout = lane63(oi[PAR_K - 1]);
        }
        __syncthreads();
    }
    const int32_t n_sub = wave_sum32(my_sub), n_tri = wave_sum32(my_tri), saved = wave_sum32(my_saved);
    const bool mismatch = __ballot(my_mismatch) != 0;
    if (lane == 0) {
        uint32_t fl = PARASON_FLAG_VALID;
        if (mismatch) fl |= PARASON_FLAG_COUNT_MISMATCH;
        if (n_blocks > 0) fl |= PARASON_FLAG_TRIGGERED;
        write_row(a.out, r, len, len - saved, n_sub, n_tri, n_blocks, max_depth, -1, fl);
    }
}

/* ------------------------------------------------------------------ scan */

typedef int v4i __attribute__((ext_vector_type(4)));

/* 16-byte streaming load (each token is read exactly once). */
__device__ __forceinline__ int4 load_vec(const int4 *p)
{
    v4i v = __builtin_nontemporal_load(reinterpret_cast<const v4i *>(p));
    return make_int4(v.x, v.y, v.z, v.w);
}

/* Tag tests of the token scan: contiguous ids (a range check), hashed ids (one
 * lookup in the slot table held across the wave's lanes, tab = slot_id[lane])
 * or, for tag sets no shift pair separates, twelve compares. */
enum : int { TM_CONTIG = 0, TM_HASH = 1, TM_LINEAR = 2 };

template <int MODE>
__device__ __forceinline__ bool is_tag(const TagMatch &tm, int32_t t, int32_t tab)
{
    if (MODE == TM_CONTIG) return (uint32_t)t - (uint32_t)tm.base < 12u;
    if (MODE == TM_HASH) return __builtin_amdgcn_ds_bpermute((int)(tag_slot(tm, t) << 2), tab) == t;
    bool h = false;
#pragma unroll
    for (int k = 0; k < 12; ++k) h = h || (t == tm.ids[k]);
    return h;
}

/* The class of a token known to be a tag: for contiguous ids one shift of
 * the 64-bit nibble table (the id is base + o with o < 12). */
template <int MODE>
__device__ __forceinline__ uint32_t tag_class(const TagMatch &tm, int32_t t)
{
    if (MODE == TM_CONTIG) {
        const uint64_t lut = (uint64_t)tm.lut_hi << 32 | tm.lut_lo;
        return (uint32_t)(lut >> (4u * ((uint32_t)t - (uint32_t)tm.base))) & 15u;
    }
    return classify(tm, t, false);
}

/* Tags of the LOADS vectors x[i] (vector v0 + i*WAVE + lane of this lane) are
 * appended to dst[0 .. cap) in position order as (q + bias) << 4 | class, where
 * q = 4*(i*WAVE + lane) + j is the position in the segment; cnt counts all of
 * them, stored or not.  EDGE: the segment holds the first or last vector of its
 * row, so only positions q_lo <= q < q_hi belong to the row. */
template <int MODE, bool EDGE>
__device__ __forceinline__ void scan_vectors(const int4 (&x)[LOADS], int32_t q_lo, int32_t q_hi,
                                             uint32_t *__restrict__ dst, uint32_t cap, int32_t bias, uint32_t &cnt,
                                             const TagMatch &tm, int32_t tab, int lane)
{
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
        const int32_t t[4] = {x[i].x, x[i].y, x[i].z, x[i].w};
        if (MODE == TM_CONTIG) {
            /* Contiguous ids are base .. base + 11 with base >= 0: a vector
             * holds a tag only if its largest (signed) token reaches base.
             * Three VALU operations per lane instead of eight settle the
             * vectors without a tag (about four in five at 0.1 % tags). */
            const int32_t hi = max(max(t[0], t[1]), max(t[2], t[3]));
            if (__ballot(hi >= tm.base) == 0) continue; /* wave-uniform */
        }
        const int32_t q0 = 4 * (i * WAVE + lane);
        uint64_t b[4];
        uint32_t mine = 0; /* this lane's tags, bit j for token j */
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            bool hit = is_tag<MODE>(tm, t[j], tab);
            if (EDGE) hit = hit && q0 + j >= q_lo && q0 + j < q_hi;
            b[j] = __ballot(hit);
            mine |= hit ? 1u << j : 0u;
        }
        if ((b[0] | b[1] | b[2] | b[3]) == 0) continue; /* wave-uniform: most vectors hold no tag */
        uint32_t pre = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j)
            pre = __builtin_amdgcn_mbcnt_hi((uint32_t)(b[j] >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)b[j], pre));
        /* the lane's tags in position order, one store each (a lane almost
         * never holds more than one tag of a vector) */
        for (uint32_t idx = cnt + pre; mine != 0; ++idx) {
            const uint32_t j = (uint32_t)__builtin_ctz(mine);
            mine &= mine - 1u;
            const int32_t tj = j == 0 ? t[0] : j == 1 ? t[1] : j == 2 ? t[2] : t[3];
            if (idx < cap) dst[idx] = ((uint32_t)(q0 + (int32_t)j + bias) << 4) | tag_class<MODE>(tm, tj);
        }
        cnt += (uint32_t)(__popcll(b[0]) + __popcll(b[1]) + __popcll(b[2]) + __popcll(b[3]));
    }
}

__device__ __forceinline__ void issue_loads(int4 (&x)[LOADS], const int4 *src, int64_t v0, int64_t v1, bool edge,
                                            int lane)
{
    const int4 *p = src + v0 + lane;
    if (!edge) {
#pragma unroll
        for (int i = 0; i < LOADS; ++i) x[i] = load_vec(p + i * WAVE);
    } else {
#pragma unroll
        for (int i = 0; i < LOADS; ++i)
            x[i] = (v0 + i * WAVE + lane < v1) ? load_vec(p + i * WAVE) : make_int4(-1, -1, -1, -1);
    }
}

/* seg[s].count = DENSE for s in [a, b): the row kernels classify those
 * segments' tokens again. */

__device__ __forceinline__ void mark_dense(SegRec *seg, int64_t a, int64_t b, int lane)
{
    for (int64_t s = a + lane; s < b; s += WAVE) seg[s].count = DENSE;
}

struct ScanArgs {
    const int32_t *tok_base;
    int64_t mis;
    const int64_t *starts;
    const int32_t *lengths;
    int64_t n;
    const int64_t *seg_off;
    int64_t seg_cap;
    SegRec *seg;
    uint32_t *slots;
    uint32_t pool_base;  /* the pool: slots [pool_base, pool_base + pool_slots); wave w's */
    uint32_t pool_slots; /* region starts at pool_base + POOL_PER_SEG * s_begin + x * w and ends at
                            pool_base + POOL_PER_SEG * s_end + x * (w + 1), with
                            x = (pool_slots - POOL_PER_SEG * S) / W rounded down to 4 */
    uint8_t *mode;
    TagMatch tm;
    int32_t *split_count; /* rows of more than one segment that no scan wave owns ... */
    int32_t *split_rows;  /* ... listed here for gather_rows */
    int32_t *counters;    /* cleared by a scan that plans the batch itself */
};

/* Row being collected by a scan wave, in processing order. */
struct RowCollect {
    uint32_t lcnt; /* events in the wave's LDS buffer */
    bool global;   /* events go to per-segment lists; the row kernel evaluates the row */
    uint32_t pc;    /* next free slot of the wave's pool region (a multiple of 4) ... */
    uint32_t p_end; /* ... and its end */
};

constexpr int EVL = 1024;                 /* LDS events per wave */
constexpr int SCAN_WAVES = 4;             /* waves per scan block */
constexpr int SCAN_THREADS = WAVE * SCAN_WAVES;
constexpr int SCAN_PLAN_ROWS = 2048;      /* rows up to which a scan block plans the batch itself */
/* Waves per block of a scan that plans in LDS.  Every block plans the whole
 * batch before its first load, so half as many blocks of twice the size plan
 * it half as often and are all dispatched sooner (a 2,048-row step: 2.7 us
 * less); the same per-CU occupancy. */
constexpr int SCAN_PLAN_WAVES = 8;
template <bool PLAN>
constexpr int scan_waves() { return PLAN ? SCAN_PLAN_WAVES : SCAN_WAVES; }

/* The whole of row `row` is in the wave's LDS buffer lev[0 .. lcnt): copy it,
 * coalesced, to the wave's pool region as one compact list for the row kernel
 * (mode 1).  A list that does not fit makes the row kernel classify the row's
 * segments again. */
__device__ __forceinline__ void flush_row(const ScanArgs &a, int64_t row, int64_t first, int64_t last, uint32_t lcnt,
                                          const uint32_t *lev, RowCollect &rc, int lane)
{
    const uint32_t need = (lcnt + 3u) & ~3u;
    if (need > rc.p_end - rc.pc) {
        mark_dense(a.seg, first, last + 1, lane);
        return;
    }
    uint32_t *dst = a.slots + rc.pc;
    /* lane i copies events other lanes wrote: the wave's LDS stores above
     * come first (a wave's LDS accesses are performed in program order; this
     * keeps the compiler from moving them across) */
    __builtin_amdgcn_wave_barrier();
    for (uint32_t i = lane; i < lcnt; i += WAVE) dst[i] = lev[i];
    if (lane == 0) {
        a.seg[first] = SegRec{(int32_t)lcnt, rc.pc};
        a.mode[row] = MODE_COMPACT;
    }
    rc.pc += need;
}

/* Scan one segment whose loads are in x.  A row owned by the wave collects
 * its events in the wave's LDS buffer; any other row leaves its events in the
 * per-segment lists for the row kernels.  Returns true when this segment
 * completes a row whose events are all in the LDS buffer (rc.lcnt of them). */
template <int MODE, bool PLAN>
__device__ __forceinline__ bool collect_segment(const ScanArgs &a, const int4 (&x)[LOADS], const SegView &w,
                                                RowCollect &rc, uint32_t *lev, int32_t tab, int lane)
{
    if (w.s == w.first) {
        rc.lcnt = 0;
        rc.global = !w.owned;
        if (PLAN) {
            /* the scan planned the batch itself: the wave holding a row's first
             * segment clears its mode (flush_row may set it again below) */
            if (lane == 0) a.mode[w.row] = 0;
        } else if (!w.owned && w.last > w.first && w.len < (1 << 27) && lane == 0) {
            /* the wave holding the first segment of a split row lists it for
             * gather_rows (rows of 2^27 tokens or more stay per segment) */
            a.split_rows[atomicAdd(a.split_count, 1)] = (int32_t)w.row;
        }
    }
    uint32_t cnt = 0; /* wave-uniform */
    if (!rc.global) {
        const int32_t bias = (int32_t)(4 * w.v0 - w.g); /* row position of segment position 0 */
        const uint32_t cap = (uint32_t)EVL - rc.lcnt;
        if (!w.edge) scan_vectors<MODE, false>(x, 0, SEG_TOK, lev + rc.lcnt, cap, bias, cnt, a.tm, tab, lane);
        else scan_vectors<MODE, true>(x, w.q_lo, w.q_hi, lev + rc.lcnt, cap, bias, cnt, a.tm, tab, lane);
        if (cnt > cap) {
            /* the row's events overflow the LDS buffer: its segments so far are
             * classified again by the row kernel, the rest use per-segment lists */
            mark_dense(a.seg, w.first, w.s + 1, lane);
            rc.global = true;
        } else {
            rc.lcnt += cnt;
        }
    } else {
        /* the segment's own list, in the wave's pool region */
        const uint32_t room = min(rc.p_end - rc.pc, (uint32_t)SEG_TOK); /* a multiple of 4 */
        uint32_t *dst = a.slots + rc.pc;
        if (!w.edge) scan_vectors<MODE, false>(x, 0, SEG_TOK, dst, room, 0, cnt, a.tm, tab, lane);
        else scan_vectors<MODE, true>(x, w.q_lo, w.q_hi, dst, room, 0, cnt, a.tm, tab, lane);
        const bool stored = cnt <= room;
        if (lane == 0) a.seg[w.s] = SegRec{stored ? (int32_t)cnt : DENSE, rc.pc};
        if (stored) rc.pc += (cnt + 3u) & ~3u;
    }
    return w.s == w.last && !rc.global;
}

/* The segment plan of a batch of at most SCAN_PLAN_ROWS rows, made by one
 * scan block in LDS (off[r] = first segment of row r, off[n] = the total):
 * the segment counts with coalesced loads (row t + SCAN_THREADS * j for thread
 * t), then an exclusive scan with each thread over SCAN_PLAN_ROWS /
 * SCAN_THREADS consecutive rows.  Block 0 also writes the plan to seg_off for
 * the row kernels, clears the mode of rows without segments (no scan wave
 * sees them; all rows when the batch overflows the workspace) and the
 * counters; every other row's mode is cleared by the wave holding its first
 * segment.  The rows' starts and lengths stay in LDS (st, ln) for the block's
 * segment cursors. */
template <int NW>
__device__ __forceinline__ void scan_plan(const ScanArgs &a, int64_t *off, int64_t *part, int64_t *st, int32_t *ln)
{
    constexpr int THREADS = WAVE * NW;
    constexpr int RPT = SCAN_PLAN_ROWS / THREADS;
    static_assert(SCAN_PLAN_ROWS % THREADS == 0, "whole rows per thread");
    const int t = (int)threadIdx.x, lane = t & (WAVE - 1), wv = t / WAVE;
#pragma unroll
    for (int j = 0; j < RPT; ++j) {
        const int64_t r = t + (int64_t)THREADS * j;
        if (r < a.n) {
            const int64_t start = a.starts[r];
            const int32_t len = a.lengths[r];
            st[r] = start;
            ln[r] = len;
            off[r] = row_segments(start, len, a.mis);
        } else {
            off[r] = 0;
        }
    }
    __syncthreads();
    int64_t c[RPT], sum = 0;
#pragma unroll
    for (int k = 0; k < RPT; ++k) {
        c[k] = off[t * RPT + k];
        sum += c[k];
    }
    const int64_t inc = wave_inclusive_scan(sum);
    if (lane == WAVE - 1) part[wv] = inc;
    __syncthreads();
    int64_t run = inc - sum, total = 0;
    for (int w = 0; w < NW; ++w) {
        run += w < wv ? part[w] : 0;
        total += part[w];
    }
#pragma unroll
    for (int k = 0; k < RPT; ++k) {
        if (t * RPT + k < a.n) off[t * RPT + k] = run;
        run += c[k];
    }
    if (t == 0) off[a.n] = total; /* rows beyond n are not rewritten, so no other thread writes off[n] */
    __syncthreads();
    if (blockIdx.x == 0) {
        /* when the batch overflows the workspace no scan wave runs, so every
         * mode byte is cleared here */
        const bool overflow = off[a.n] > a.seg_cap;
        int64_t *seg_off = const_cast<int64_t *>(a.seg_off);
        for (int64_t r = t; r <= a.n; r += THREADS) {
            seg_off[r] = off[r];
            if (r < a.n && (overflow || off[r + 1] == off[r])) a.mode[r] = 0;
        }
        if (t < 4) a.counters[t] = 0;
    }
}

/* Work distribution of a large scan.  Compute units do not all stream at the
 * same rate (on MI355X, with equal shares, the waves of four of the eight dies
 * finished about 9 % later than the others), so equal static shares leave
 * part of the chip idle at the end.  A scan with at least DYN_MIN_PER_WAVE segments per
 * wave therefore gives each wave an equal contiguous share of the first
 * S1 = S - S * DYN_NUM / DYN_DEN segments, and hands out the rest in chunks,
 * in segment order, through one counter: rounds of one chunk per wave whose
 * size halves from c0 = (S - S1) / (2 W) down to DYN_KMIN, then chunks of
 * DYN_KMIN to the end.  A wave that finishes early takes more chunks.  Rows cut
 * by a chunk boundary are split rows, handled as those cut by a share's
 * boundary.  Every range (share or chunk) has its own region of the slot pool:
 * range q (shares 0 .. W-1, then chunk i as W + i) covering segments [b, e)
 * owns slots [POOL_PER_SEG * b + x * q, POOL_PER_SEG * e + x * (q + 1)) past
 * pool_base, x = (pool_slots - POOL_PER_SEG * S) / (W + chunks) rounded down
 * to 4, so regions are disjoint and in segment order. */
constexpr int64_t DYN_MIN_PER_WAVE = 256;
constexpr int64_t DYN_NUM = 3, DYN_DEN = 16;
constexpr int64_t DYN_KMIN = 32;
constexpr int64_t BLK_CHUNK = 2; /* segments per chunk of a block's own pool ... */
constexpr int64_t BLK_MIN = 64;  /* ... which a block has from this many segments on */

struct ScanSched {
    int64_t S, S1, c0, base_final, n_chunks, W;
    int32_t rounds;
    bool dyn;
    int64_t kmin; /* every field is wave-uniform */

    /* S units (segments) over W waves; kmin: the smallest chunk; num / den of
     * the units handed out in chunks (all wave-uniform) */
    __device__ void init(int64_t S_, int64_t W_, bool allow, int64_t kmin_ = DYN_KMIN, int64_t num = DYN_NUM,
                         int64_t den = DYN_DEN)
    {
        S = S_;
        W = W_;
        kmin = kmin_;
        dyn = allow && S >= DYN_MIN_PER_WAVE * kmin / DYN_KMIN * W;
        S1 = dyn ? S - S / den * num - S % den * num / den : S;
        c0 = (S - S1) / (2 * W);
        rounds = 0;
        int64_t b = S1;
        while ((c0 >> rounds) >= kmin) {
            b += W * (c0 >> rounds);
            ++rounds;
        }
        base_final = b;
        n_chunks = dyn ? W * rounds + (S - b + kmin - 1) / kmin : 0;
    }
    /* units [b, e) of chunk i < n_chunks */
    __device__ void chunk(int64_t i, int64_t &b, int64_t &e) const
    {
        if (i >= W * rounds) {
            b = base_final + (i - W * rounds) * kmin;
            e = min(b + kmin, S);
            return;
        }
        int64_t base = S1;
        int32_t r = 0;
        while (i >= W) {
            base += W * (c0 >> r);
            i -= W;
            ++r;
        }
        b = base + i * (c0 >> r);
        e = b + (c0 >> r);
    }
};

/* Scan segments [s_begin, s_end) (a share or a chunk), filling the pool region
 * [pc, p_end).  Two register buffers: segment s + 1 is in flight while s is
 * compacted (and a finished row's events flushed), so the wave always has a
 * segment in flight. */
template <int MODE, bool PLAN>
__device__ __forceinline__ void scan_range(const ScanArgs &a, const int64_t *seg_off, const int64_t *starts,
                                           const int32_t *lengths, int64_t s_begin, int64_t s_end,
                                           uint32_t pc, uint32_t p_end, uint32_t *lev, int32_t tab, int lane)
{
    const int4 *src = reinterpret_cast<const int4 *>(a.tok_base);
    SegCursor cur;
    cur.seg_off = seg_off;
    cur.starts = starts;
    cur.lengths = lengths;
    cur.mis = a.mis;
    cur.s_begin = s_begin;
    cur.s_end = s_end;
    cur.seek(s_begin, a.n);

    RowCollect rc;
    rc.lcnt = 0;
    rc.global = true; /* a row already begun in the previous range */
    rc.pc = pc;
    rc.p_end = p_end;
    SegView w = cur.view(s_begin);
    int4 xa[LOADS], xb[LOADS];
    issue_loads(xa, src, w.v0, w.v1, w.edge, lane);
    int64_t s = s_begin;
    while (true) {
        SegView wn;
        bool more = s + 1 < s_end;
        if (more) {
            wn = cur.view(s + 1);
            issue_loads(xb, src, wn.v0, wn.v1, wn.edge, lane);
        }
        if (collect_segment<MODE, PLAN>(a, xa, w, rc, lev, tab, lane))
            flush_row(a, w.row, w.first, w.last, rc.lcnt, lev, rc, lane);
        if (!more) break;
        ++s;
        w = wn;
        more = s + 1 < s_end;
        if (more) {
            wn = cur.view(s + 1);
            issue_loads(xa, src, wn.v0, wn.v1, wn.edge, lane);
        }
        if (collect_segment<MODE, PLAN>(a, xb, w, rc, lev, tab, lane))
            flush_row(a, w.row, w.first, w.last, rc.lcnt, lev, rc, lane);
        if (!more) break;
        ++s;
        w = wn;
    }
}

/* One wave per segment: each wave scans its share of the segments, then (a
 * large scan) takes chunks of the rest until none is left. */
template <int MODE, bool PLAN>
__global__ void __launch_bounds__(WAVE * scan_waves<PLAN>(), PARASON_SCAN_WAVES_PER_SIMD) scan_rows(ScanArgs a)
{
    constexpr int NW = scan_waves<PLAN>();
    __shared__ uint32_t lds_ev[NW][EVL];
    __shared__ int64_t plan_off[PLAN ? SCAN_PLAN_ROWS + 1 : 1];
    __shared__ int64_t plan_st[PLAN ? SCAN_PLAN_ROWS : 1];
    __shared__ int32_t plan_ln[PLAN ? SCAN_PLAN_ROWS : 1];
    __shared__ int64_t plan_part[NW];
    const int lane = threadIdx.x & (WAVE - 1);
    const int wib = __builtin_amdgcn_readfirstlane(threadIdx.x / WAVE);
    const int64_t wave = uniform64((int64_t)blockIdx.x * NW + wib);
    const int64_t n_waves = (int64_t)gridDim.x * NW;
    const int64_t *seg_off = a.seg_off;
    /* a batch the scan plans (a small one): block k scans segments
     * [S k / nb, S (k + 1) / nb), its waves an equal share each of the first
     * L1 = L - 3 L / 16 of them, then the rest in chunks of BLK_CHUNK handed
     * out by an LDS counter, so that the block's waves end together (a block
     * of fewer than BLK_MIN segments keeps equal shares of all of them: its
     * waves are done before a counter would pay); ranges are numbered
     * k Q + wave (shares), k Q + NW + j (chunks), Q above any block's share
     * and chunk count. */
    __shared__ uint32_t blk_next;
    if (PLAN) {
        if (threadIdx.x == 0) blk_next = 0; /* before scan_plan's barriers */
        scan_plan<NW>(a, plan_off, plan_part, plan_st, plan_ln);
        seg_off = plan_off;
    }
    const int64_t S = uniform64(seg_off[a.n]);
    if (S > a.seg_cap) return; /* the row kernel reports PARASON_FLAG_WS_OVERFLOW */
    uint32_t *lev = lds_ev[wib];
    const int32_t tab = MODE == TM_HASH ? a.tm.slot_id[lane] : 0;
    int64_t b, e, q, Bk = 0, Ek = 0, L1 = 0, Q = 0;
    bool blk_dyn = false;
    uint32_t extra;
    ScanSched sch;
    if (PLAN) {
        /* 64-bit divisions are long on the scalar unit: by shifts when the
         * block count is a power of two (two blocks per compute unit) */
        const uint32_t nb = gridDim.x;
        const bool pow2 = (nb & (nb - 1)) == 0;
        const int sh = __builtin_ctz(nb);
        const int64_t k = blockIdx.x;
        Bk = uniform64(pow2 ? (S * k) >> sh : S * k / nb);
        Ek = uniform64(pow2 ? (S * (k + 1)) >> sh : S * (k + 1) / nb);
        Q = uniform64(NW + ((pow2 ? S >> sh : S / nb) + 1) * DYN_NUM / DYN_DEN / BLK_CHUNK + 2);
        /* slot indices fit 32 bits, which the host checks */
        extra = ((a.pool_slots - POOL_PER_SEG * (uint32_t)S) / (uint32_t)(nb * Q)) & ~3u;
        blk_dyn = Ek - Bk >= BLK_MIN;
        L1 = blk_dyn ? (Ek - Bk) - (Ek - Bk) * DYN_NUM / DYN_DEN : Ek - Bk;
        b = uniform64(Bk + L1 * wib / NW);
        e = uniform64(Bk + L1 * (wib + 1) / NW);
        q = k * Q + wib;
    } else {
        sch.init(S, n_waves, true);
        /* S1 < 2^40 and n_waves < 2^20 (checked on the host), so S1 * wave fits */
        b = uniform64(sch.S1 * wave / n_waves);
        e = uniform64(sch.S1 * (wave + 1) / n_waves);
        q = wave;
        extra = ((a.pool_slots - POOL_PER_SEG * (uint32_t)S) / (uint32_t)(n_waves + sch.n_chunks)) & ~3u;
    }
    while (true) {
        if (b < e) {
            const uint32_t pc = __builtin_amdgcn_readfirstlane(a.pool_base + POOL_PER_SEG * (uint32_t)b + extra * (uint32_t)q);
            const uint32_t p_end =
                __builtin_amdgcn_readfirstlane(a.pool_base + POOL_PER_SEG * (uint32_t)e + extra * (uint32_t)(q + 1));
            scan_range<MODE, PLAN>(a, seg_off, PLAN ? plan_st : a.starts, PLAN ? plan_ln : a.lengths, b, e, pc, p_end,
                                   lev, tab, lane);
        }
        if (PLAN) {
            if (!blk_dyn) break;
            uint32_t j = 0;
            if (lane == 0) j = atomicAdd(&blk_next, 1u);
            j = __builtin_amdgcn_readfirstlane(j);
            b = uniform64(Bk + L1 + (int64_t)j * BLK_CHUNK);
            if (b >= Ek) break;
            e = uniform64(min(b + BLK_CHUNK, Ek));
            q = blockIdx.x * Q + NW + j;
            continue;
        }
        if (!sch.dyn) break;
        int32_t i = 0;
        if (lane == 0) i = atomicAdd(&a.counters[3], 1);
        i = __builtin_amdgcn_readfirstlane(i);
        if ((int64_t)i >= sch.n_chunks) break;
        sch.chunk(i, b, e);
        b = uniform64(b);
        e = uniform64(e);
        q = n_waves + i;
    }
}

/* The ceiling the token scan is measured against: a plain streaming read of
 * the same buffer with the scan's 16-byte nontemporal loads and persistent
 * grid, every unit handed out in chunks through a counter as ScanSched does
 * (a chunk unit is one 8 KB step of eight loads per lane, all issued before
 * any is used), and no other work.  Each wave stores the XOR of what it read to
 * sink[wave % sink_len] (so the loads are kept).  *next must be zero at the
 * launch (probe_reset clears it). */
constexpr int PROBE_LOADS = 8;
constexpr int PROBE_CHUNK = PROBE_LOADS * WAVE; /* 16-byte vectors per chunk */
constexpr int64_t PROBE_KMIN = 16;              /* the smallest chunk: 16 steps of 8 KB */

__global__ void probe_reset(int32_t *next) { *next = 0; }

__global__ void __launch_bounds__(WAVE * SCAN_WAVES) read_probe(const int4 *__restrict__ src, int64_t n_vec,
                                                                const int32_t *__restrict__ tail, int32_t n_tail,
                                                                uint32_t *__restrict__ sink, int64_t sink_len,
                                                                int32_t *__restrict__ next)
{
    const int lane = threadIdx.x & (WAVE - 1);
    const int64_t wave = uniform64((int64_t)blockIdx.x * SCAN_WAVES + threadIdx.x / WAVE);
    const int64_t n_waves = (int64_t)gridDim.x * SCAN_WAVES;
    const int64_t n_chunks = n_vec / PROBE_CHUNK;
    ScanSched sch;
    /* units of 8 KB, all of them in chunks: the waves of a pure read
     * stream at rates several times apart, more than the scan's equal
     * shares leave room for */
    sch.init(n_chunks, n_waves, true, PROBE_KMIN, 1, 1);
    int64_t c0 = uniform64(sch.S1 * wave / n_waves), c1 = uniform64(sch.S1 * (wave + 1) / n_waves);
    uint32_t acc = 0;
    while (true) {
        for (int64_t c = c0; c < c1; ++c) {
            int4 x[PROBE_LOADS];
            const int4 *p = src + c * PROBE_CHUNK + lane;
#pragma unroll
            for (int i = 0; i < PROBE_LOADS; ++i) x[i] = load_vec(p + i * WAVE);
#pragma unroll
            for (int i = 0; i < PROBE_LOADS; ++i) acc ^= (uint32_t)(x[i].x ^ x[i].y ^ x[i].z ^ x[i].w);
        }
        if (!sch.dyn) break;
        int32_t i = 0;
        if (lane == 0) i = atomicAdd(next, 1);
        i = __builtin_amdgcn_readfirstlane(i);
        if ((int64_t)i >= sch.n_chunks) break;
        sch.chunk(i, c0, c1);
        c0 = uniform64(c0);
        c1 = uniform64(c1);
    }
    if (wave == n_waves - 1) {
        /* the vectors after the last whole chunk, then the last 0-3 elements */
        for (int64_t v = n_chunks * PROBE_CHUNK + lane; v < n_vec; v += WAVE) {
            const int4 x = load_vec(src + v);
            acc ^= (uint32_t)(x.x ^ x.y ^ x.z ^ x.w);
        }
        if (lane < n_tail) acc ^= (uint32_t)tail[lane];
    }
    /* XOR over the wave by DPP (row_shr) and readlane, as the scans do */
    uint32_t v = acc;
    v ^= (uint32_t)row_shr<1>((int32_t)v, 0);
    v ^= (uint32_t)row_shr<2>((int32_t)v, 0);
    v ^= (uint32_t)row_shr<4>((int32_t)v, 0);
    v ^= (uint32_t)row_shr<8>((int32_t)v, 0);
    const uint32_t w = (uint32_t)__builtin_amdgcn_readlane((int32_t)v, 15) ^
                       (uint32_t)__builtin_amdgcn_readlane((int32_t)v, 31) ^
                       (uint32_t)__builtin_amdgcn_readlane((int32_t)v, 47) ^ (uint32_t)lane63((int32_t)v);
    if (lane == 0) sink[wave % sink_len] = w;
}

/* ------------------------------------------------------------------ gather */

struct GatherArgs {
    const int64_t *starts;
    int64_t n, mis;
    const int64_t *seg_off;
    int64_t seg_cap;
    SegRec *seg;
    uint32_t *slots;
    uint8_t *mode;
    const int32_t *split_count;
    const int32_t *split_rows;
};

constexpr int GATHER_EVENTS = 1024; /* LDS events per gather wave */

/* Gather the events of row `row` (split between scan waves: one list per
 * segment, segment positions) into one list in the row's gather slots
 * (GATHER_SLOTS per segment of the row, from slot GATHER_SLOTS * seg_off[row]),
 * in position order, with row positions (the compact form, mode 1), through
 * the wave's LDS buffer lds[0 .. GATHER_EVENTS).  A row with a DENSE segment,
 * or with more events than its gather slots or the buffer hold, is left as it
 * is; the whole wave calls this. */
__device__ __forceinline__ void gather_row(const GatherArgs &a, int64_t row, uint32_t *lds, int lane)
{
    const int64_t s0 = uniform64(a.seg_off[row]), s1 = uniform64(a.seg_off[row + 1]);
    const int64_t g = uniform64(a.starts[row] + a.mis);
    const int64_t vrow0 = row_first_vec(g);
    bool dense = false;
    int64_t total = 0;
    for (int64_t c0 = s0; c0 < s1; c0 += WAVE) {
        const int64_t s = c0 + lane;
        const int32_t cnt = s < s1 ? a.seg[s].count : 0;
        dense = dense || cnt == DENSE;
        total += lane63(wave_incl_scan32(cnt, lane)); /* DENSE counts cannot overflow it */
    }
    if (__ballot(dense) != 0 || total > GATHER_EVENTS || total > (s1 - s0) * GATHER_SLOTS) return;
    int64_t carry = 0; /* events of the segments before this chunk */
    for (int64_t c0 = s0; c0 < s1; c0 += WAVE) {
        const int64_t s = c0 + lane;
        const SegRec rec = s < s1 ? a.seg[s] : SegRec{0, 0u};
        const int32_t cnt = rec.count;
        const uint32_t list = rec.list; /* meaningless for a segment without events */
        const int32_t incl = wave_incl_scan32(cnt, lane);
        const int32_t excl = incl - cnt;
        const int32_t n_c = lane63(incl);
        for (int32_t f0 = 0; f0 < n_c; f0 += WAVE) {
            const int32_t f = f0 + lane; /* the chunk's f-th event, of segment c0 + j */
            const int32_t j = last_lane_at_most(excl, f);
            const int32_t first = __shfl(excl, j, WAVE);
            const uint32_t lj = __shfl(list, j, WAVE);
            if (f < n_c) {
                const int64_t seg = c0 + j;
                const uint32_t w = a.slots[(int64_t)lj + (f - first)];
                /* row position of segment position 0 */
                const int64_t base = 4 * (vrow0 + (seg - s0) * SEG_VEC) - g;
                lds[carry + f] = ((uint32_t)(base + (int64_t)(w >> 4)) << 4) | (w & 15u);
            }
        }
        carry += n_c;
    }
    /* lanes store what other lanes loaded: every load above first */
    __builtin_amdgcn_wave_barrier();
    uint32_t *dst = a.slots + s0 * GATHER_SLOTS;
    for (int64_t i = lane; i < carry; i += WAVE) dst[i] = lds[i];
    if (lane == 0) {
        a.seg[s0] = SegRec{(int32_t)carry, (uint32_t)(s0 * GATHER_SLOTS)};
        a.mode[row] = MODE_COMPACT;
    }
}

/* The rows the scan listed as split between its waves, for the per-lane row
 * kernel: one wave per listed row (grid-stride over the list). */
__global__ void __launch_bounds__(256) gather_rows(GatherArgs a)
{
    __shared__ uint32_t lds[256 / WAVE][GATHER_EVENTS];
    const int lane = threadIdx.x & (WAVE - 1);
    const int wib = __builtin_amdgcn_readfirstlane(threadIdx.x / WAVE);
    const int64_t wave = uniform64(((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / WAVE);
    const int64_t n_waves = (int64_t)gridDim.x * (blockDim.x / WAVE);
    if (a.seg_off[a.n] > a.seg_cap) return; /* the scan wrote nothing: the row kernel reports it */
    const int32_t n_split = __builtin_amdgcn_readfirstlane(*a.split_count);
    for (int64_t i = wave; i < n_split; i += n_waves) gather_row(a, uniform64(a.split_rows[i]), lds[wib], lane);
}

/* ------------------------------------------------------------------ reward */

/* Batch-wide statistics (PARASON_CFG_BATCH_STATS), in workspace. */
struct BatchStats {
    double mu[3];    /* latency, Subtask ratio, Trial ratio */
    double sigma[3];
    int32_t all_equal[3];
    int32_t not_evaluated; /* rows flagged not evaluated */
};

struct RewardArgs {
    const int32_t *total, *latency, *n_subtask, *n_trial;
    const uint32_t *flags;
    const uint8_t *correct;
    int64_t n_groups;
    int32_t G;
    const BatchStats *batch; /* non-null: one normalisation group = the whole batch */
    int64_t n;
    double alpha, beta_s, beta_r, rho, rho_clip;
    uint32_t cfg_flags;
    float *reward, *r_subtask, *r_trial, *eta;
    float *accel;   /* optional: total / latency */
    int32_t *saved; /* optional: total - latency */
};

constexpr uint32_t NOT_EVALUATED = PARASON_FLAG_DEPTH_LIMIT | PARASON_FLAG_WS_OVERFLOW | PARASON_FLAG_BAD_ROW;

__device__ __forceinline__ double ratio(int32_t n, int32_t total)
{
    return total > 0 ? __ddiv_rn((double)n, (double)total) : 0.0;
}

/* Do all rows of the group have the same ratio n/total?  Exact (cross-multiplied). */
__device__ __forceinline__ bool same_ratio(const int32_t *nn, const int32_t *tt, int64_t r0, int32_t G)
{
    int64_t n0 = tt[r0] > 0 ? nn[r0] : 0, d0 = tt[r0] > 0 ? tt[r0] : 1;
    for (int32_t i = 1; i < G; ++i) {
        int64_t ni = tt[r0 + i] > 0 ? nn[r0 + i] : 0, di = tt[r0 + i] > 0 ? tt[r0 + i] : 1;
        if (ni * d0 != n0 * di) return false;
    }
    return true;
}

/* mean and population standard deviation of x over the group, by index order */
struct Moments {
    double mu, sigma;
};

template <class F>
__device__ __forceinline__ Moments moments(F x, int32_t G)
{
    double s = 0.0;
    for (int32_t i = 0; i < G; ++i) s = __dadd_rn(s, x(i));
    double mu = __ddiv_rn(s, (double)G);
    double ss = 0.0;
    for (int32_t i = 0; i < G; ++i) {
        double d = __dsub_rn(x(i), mu);
        ss = __dadd_rn(ss, __dmul_rn(d, d));
    }
    return Moments{mu, __dsqrt_rn(__ddiv_rn(ss, (double)G))};
}

__device__ __forceinline__ double zscore(double x, Moments m, bool all_equal)
{
    return (all_equal || m.sigma == 0.0) ? 0.0 : __ddiv_rn(__dsub_rn(x, m.mu), m.sigma);
}

/* A row's accounting outputs and correctness, loaded once. */
struct RowVals {
    uint32_t fl;
    int32_t lat, tot, ns, nt;
    uint8_t correct;
};

__device__ __forceinline__ RowVals row_vals(const RewardArgs &a, int64_t r)
{
    return RowVals{a.flags[r], a.latency[r], a.total[r], a.n_subtask[r], a.n_trial[r], a.correct[r]};
}

__device__ __forceinline__ void write_reward(const RewardArgs &a, int64_t r, const RowVals &v, double zT, double zs,
                                             double zr, double xs, double xr)
{
    const int32_t tot = v.tot;
    const double e = tot > 0 ? __dsub_rn(1.0, __ddiv_rn((double)v.lat, (double)tot)) : 0.0;
    const bool valid = (v.fl & PARASON_FLAG_VALID) != 0;
    const bool c = v.correct != 0 && (valid || (a.cfg_flags & PARASON_CFG_INVALID_KEEPS_CORRECTNESS));
    const double accel = __dmul_rn(a.rho, e);
    const double clipped = accel < a.rho_clip ? accel : a.rho_clip;
    double inner = __dsub_rn(1.0, __dmul_rn(a.alpha, zT));
    inner = __dadd_rn(inner, __dmul_rn(a.beta_s, zs));
    inner = __dadd_rn(inner, __dmul_rn(a.beta_r, zr));
    inner = __dadd_rn(inner, clipped);
    const double R = __dadd_rn(-1.0, __dmul_rn(__dmul_rn(2.0, c ? 1.0 : 0.0), inner));
    a.reward[r] = (float)R;
    if (a.r_subtask) a.r_subtask[r] = (float)xs;
    if (a.r_trial) a.r_trial[r] = (float)xr;
    if (a.eta) a.eta[r] = (float)e;
    /* a row with tokens has latency >= 1 (an invalid row's latency is its length) */
    if (a.accel) a.accel[r] = tot > 0 ? (float)__ddiv_rn((double)tot, (double)v.lat) : 1.0f;
    if (a.saved) a.saved[r] = tot - v.lat;
}

__device__ __forceinline__ void write_nan(const RewardArgs &a, int64_t r, const RowVals &v)
{
    const float nan = __int_as_float(0x7fc00000);
    a.reward[r] = nan;
    if (a.r_subtask) a.r_subtask[r] = nan;
    if (a.r_trial) a.r_trial[r] = nan;
    if (a.eta) a.eta[r] = nan;
    if (a.accel) a.accel[r] = nan;
    if (a.saved) a.saved[r] = (v.fl & NOT_EVALUATED) ? 0 : v.tot - v.lat;
}

/* A group of G rows (G a power of two up to 64) in G consecutive lanes of one
 * wave: each lane loads its own row once and reads the others' values with
 * shuffles, in the group's order.  GC > 0 fixes G at compile time (the
 * paper's G = 8), so that the group's shuffles are unrolled and issue
 * together instead of one sum step after another. */
template <int GC>
__device__ __forceinline__ void group_reward_lanes(const RewardArgs &a, int64_t r, int32_t G_run, const RowVals &v)
{
    const int32_t G = GC > 0 ? GC : G_run;
    const int lane = threadIdx.x & (WAVE - 1);
    const int gl = lane & ~(G - 1); /* the group's first lane */
    const uint64_t gmask = (G == WAVE ? ~0ull : ((1ull << G) - 1ull)) << gl;
    const uint32_t fl = v.fl;
    const int32_t lat = v.lat, tot = v.tot, ns = v.ns, nt = v.nt;
    if ((__ballot(!(fl & NOT_EVALUATED)) & gmask) != gmask) {
        write_nan(a, r, v);
        return; /* the whole group returns here */
    }
    const bool lat_equal = (__ballot(lat == __shfl(lat, gl, WAVE)) & gmask) == gmask;
    /* exact equality of the ratios, cross-multiplied against the group's first row */
    const int64_t d = tot > 0 ? tot : 1;
    const int64_t d0 = __shfl(d, gl, WAVE);
    const int64_t s_n = tot > 0 ? ns : 0, t_n = tot > 0 ? nt : 0;
    const bool sub_equal = (__ballot(s_n * d0 == __shfl(s_n, gl, WAVE) * d) & gmask) == gmask;
    const bool tri_equal = (__ballot(t_n * d0 == __shfl(t_n, gl, WAVE) * d) & gmask) == gmask;
    const double xT = (double)lat, xs = ratio(ns, tot), xr = ratio(nt, tot);
    const Moments mT = moments([&](int32_t j) { return __shfl(xT, gl + j, WAVE); }, G);
    const Moments ms = moments([&](int32_t j) { return __shfl(xs, gl + j, WAVE); }, G);
    const Moments mr = moments([&](int32_t j) { return __shfl(xr, gl + j, WAVE); }, G);
    write_reward(a, r, v, zscore(xT, mT, lat_equal), zscore(xs, ms, sub_equal), zscore(xr, mr, tri_equal), xs, xr);
}

/* Row r's reward from its group's values in memory, in the group's row order
 * (any group size, any thread layout). */
__device__ __forceinline__ void group_reward_memory(const RewardArgs &a, int64_t r)
{
    const int32_t G = a.G;
    const int64_t r0 = r - r % G;
    bool evaluated = true;
    bool lat_equal = true;
    for (int32_t i = 0; i < G; ++i) {
        evaluated = evaluated && !(a.flags[r0 + i] & NOT_EVALUATED);
        lat_equal = lat_equal && a.latency[r0 + i] == a.latency[r0];
    }
    const RowVals v = row_vals(a, r);
    if (!evaluated) {
        write_nan(a, r, v);
        return;
    }
    const bool sub_equal = same_ratio(a.n_subtask, a.total, r0, G);
    const bool tri_equal = same_ratio(a.n_trial, a.total, r0, G);
    auto xT = [&](int32_t i) { return (double)a.latency[r0 + i]; };
    auto xs = [&](int32_t i) { return ratio(a.n_subtask[r0 + i], a.total[r0 + i]); };
    auto xr = [&](int32_t i) { return ratio(a.n_trial[r0 + i], a.total[r0 + i]); };
    const Moments mT = moments(xT, G), ms = moments(xs, G), mr = moments(xr, G);
    const int32_t i = (int32_t)(r - r0);
    write_reward(a, r, v, zscore(xT(i), mT, lat_equal), zscore(xs(i), ms, sub_equal), zscore(xr(i), mr, tri_equal),
                 xs(i), xr(i));
}

/* The deep tier's rows (listed by rows_par or rows_mid), run by the first
 * block of group_reward instead of a launch of their own. */
struct DeepArgs {
    RowArgs rows;
    const uint8_t *mode;
    const int32_t *counters; /* counters[1]: rows in deep_rows */
    const int32_t *deep_rows;
    int32_t *frames;
    uint32_t *bits;
};

/* One thread per row.  A group within one wave shares its values by shuffles
 * (group_reward_lanes); otherwise every thread of a group computes the group's
 * moments itself from memory.  Either way the sums run in the group's row
 * order, so every thread of a group holds the same values; a group takes G
 * threads instead of one, which keeps the GPU busy when a batch has few
 * groups (an RL step has 128).
 *
 * Rows listed for the deep tier (normally none) are evaluated here first, by
 * thread 0 of block 0; after a barrier that block computes the rewards of the
 * groups holding them (a group listed twice is written twice, with the same
 * values).  Every block skips those groups: it tells them by the MODE_DEEP
 * mark, which nothing writes during this launch, so no block reads a row
 * another block is writing. */
template <bool LENIENT>
__global__ void __launch_bounds__(256) group_reward(RewardArgs a, DeepArgs d)
{
    const int32_t G = a.G;
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    /* the row's values in the same round of loads as the deep count (rows of
     * groups the deep tier writes during this launch are not read from v) */
    const RowVals v = row_vals(a, min(r, a.n - 1));
    const int32_t n_deep = d.counters[1]; /* the same for every thread */
    if (n_deep > 0 && blockIdx.x == 0) {
        if (threadIdx.x == 0) run_deep_rows<LENIENT>(d.rows, d.mode, n_deep, d.deep_rows, d.frames, d.bits);
        __syncthreads();
        for (int64_t k = threadIdx.x; k < (int64_t)n_deep * G; k += blockDim.x) {
            const int64_t rd = d.deep_rows[k / G];
            group_reward_memory(a, rd - rd % G + k % G);
        }
    }
    if (r >= a.n) return; /* n is a multiple of G: whole groups only */
    if (n_deep > 0) {
        const int64_t r0 = r - r % G;
        bool deep = false;
        for (int32_t i = 0; i < G; ++i) deep = deep || (d.mode[r0 + i] & MODE_DEEP) != 0;
        if (deep) return; /* the whole group returns here */
    }
    if (G == 8) group_reward_lanes<8>(a, r, G, v);
    else if (G <= WAVE && (G & (G - 1)) == 0) group_reward_lanes<0>(a, r, G, v);
    else group_reward_memory(a, r);
}

/* One thread per row; mu, sigma of the whole batch from batch_stats. */
__global__ void __launch_bounds__(256) batch_reward(RewardArgs a)
{
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= a.n) return;
    const BatchStats &b = *a.batch;
    const RowVals v = row_vals(a, r);
    if (b.not_evaluated) {
        write_nan(a, r, v);
        return;
    }
    const double xT = (double)v.lat, xs = ratio(v.ns, v.tot), xr = ratio(v.nt, v.tot);
    write_reward(a, r, v, zscore(xT, Moments{b.mu[0], b.sigma[0]}, b.all_equal[0] != 0),
                 zscore(xs, Moments{b.mu[1], b.sigma[1]}, b.all_equal[1] != 0),
                 zscore(xr, Moments{b.mu[2], b.sigma[2]}, b.all_equal[2] != 0), xs, xr);
}

/* ------------------------------------------------------------------ batch reductions */

struct StatsArgs {
    const int32_t *total, *latency, *n_subtask, *n_trial;
    const uint32_t *flags;
    int64_t n;
    double *dpart;    /* [tiles][3] */
    int64_t *ipart;   /* [tiles][4]: not evaluated, latency differs, Subtask ratio differs, Trial ratio differs */
    BatchStats *stats;
};

/* PASS 1: sums of the three statistics and the equality checks; PASS 2: sums
 * of squared deviations from the batch means. */
template <int PASS>
__global__ void __launch_bounds__(RED_THREADS) batch_stats_tiles(StatsArgs a)
{
    __shared__ double dl[3 * RED_THREADS];
    __shared__ int64_t il[4 * RED_THREADS];
    const int64_t r0 = (int64_t)blockIdx.x * RED_TILE + (int64_t)threadIdx.x * ROWS_PER_THREAD;
    double d[3] = {0.0, 0.0, 0.0};
    int64_t c[4] = {0, 0, 0, 0};
    const int64_t s0 = a.n_subtask[0], t0 = a.total[0] > 0 ? a.total[0] : 1, u0 = a.n_trial[0];
    const int64_t n0s = a.total[0] > 0 ? s0 : 0, n0r = a.total[0] > 0 ? u0 : 0;
    for (int j = 0; j < ROWS_PER_THREAD; ++j) {
        const int64_t r = r0 + j;
        if (r >= a.n) break;
        const double x[3] = {(double)a.latency[r], ratio(a.n_subtask[r], a.total[r]), ratio(a.n_trial[r], a.total[r])};
        if (PASS == 1) {
#pragma unroll
            for (int k = 0; k < 3; ++k) d[k] = __dadd_rn(d[k], x[k]);
            const int64_t tr = a.total[r] > 0 ? a.total[r] : 1;
            const int64_t ns = a.total[r] > 0 ? a.n_subtask[r] : 0, nr = a.total[r] > 0 ? a.n_trial[r] : 0;
            c[0] += (a.flags[r] & NOT_EVALUATED) != 0;
            c[1] += a.latency[r] != a.latency[0];
            c[2] += ns * t0 != n0s * tr;
            c[3] += nr * t0 != n0r * tr;
        } else {
#pragma unroll
            for (int k = 0; k < 3; ++k) {
                const double dv = __dsub_rn(x[k], a.stats->mu[k]);
                d[k] = __dadd_rn(d[k], __dmul_rn(dv, dv));
            }
        }
    }
    block_tree_sum<double, 3>(d, dl);
    if (PASS == 1) block_tree_sum<int64_t, 4>(c, il);
    if (threadIdx.x == 0) {
        for (int k = 0; k < 3; ++k) a.dpart[blockIdx.x * 3 + k] = d[k];
        if (PASS == 1)
            for (int k = 0; k < 4; ++k) a.ipart[blockIdx.x * 4 + k] = c[k];
    }
}

template <int PASS>
__global__ void __launch_bounds__(RED_THREADS) batch_stats_final(StatsArgs a, int64_t tiles)
{
    __shared__ double dl[3 * RED_THREADS];
    __shared__ int64_t il[4 * RED_THREADS];
    double d[3];
    sum_partials<double, 3>(a.dpart, tiles, d, dl);
    if (PASS == 1) {
        int64_t c[4];
        sum_partials<int64_t, 4>(a.ipart, tiles, c, il);
        if (threadIdx.x == 0) {
            for (int k = 0; k < 3; ++k) a.stats->mu[k] = __ddiv_rn(d[k], (double)a.n);
            a.stats->not_evaluated = c[0] != 0;
            for (int k = 0; k < 3; ++k) a.stats->all_equal[k] = c[k + 1] == 0;
        }
    } else if (threadIdx.x == 0) {
        for (int k = 0; k < 3; ++k) a.stats->sigma[k] = __dsqrt_rn(__ddiv_rn(d[k], (double)a.n));
    }
}

struct MetricsArgs {
    const int32_t *total, *latency, *n_subtask, *n_trial;
    const uint32_t *flags;
    const uint8_t *correct;
    const float *reward;
    int64_t n;
    int64_t *ipart; /* [tiles][9] */
    double *dpart;  /* [tiles][1] */
    double *metrics;
};

constexpr int NMI = 9; /* valid, triggered, correct, truncated, mismatch, sum total, latency, Subtask, Trial */

__global__ void __launch_bounds__(RED_THREADS) metrics_tiles(MetricsArgs a)
{
    __shared__ int64_t il[NMI * RED_THREADS];
    __shared__ double dl[RED_THREADS];
    const int64_t r0 = (int64_t)blockIdx.x * RED_TILE + (int64_t)threadIdx.x * ROWS_PER_THREAD;
    int64_t c[NMI];
#pragma unroll
    for (int k = 0; k < NMI; ++k) c[k] = 0;
    double d[1] = {0.0};
    for (int j = 0; j < ROWS_PER_THREAD; ++j) {
        const int64_t r = r0 + j;
        if (r >= a.n) break;
        const uint32_t f = a.flags[r];
        c[0] += (f & PARASON_FLAG_VALID) != 0;
        c[1] += (f & PARASON_FLAG_TRIGGERED) != 0;
        c[2] += a.correct[r] != 0;
        c[3] += (f & PARASON_FLAG_TRUNCATED) != 0;
        c[4] += (f & PARASON_FLAG_COUNT_MISMATCH) != 0;
        c[5] += a.total[r];
        c[6] += a.latency[r];
        c[7] += a.n_subtask[r];
        c[8] += a.n_trial[r];
        d[0] = __dadd_rn(d[0], (double)a.reward[r]);
    }
    block_tree_sum<int64_t, NMI>(c, il);
    block_tree_sum<double, 1>(d, dl);
    if (threadIdx.x == 0) {
        for (int k = 0; k < NMI; ++k) a.ipart[blockIdx.x * NMI + k] = c[k];
        a.dpart[blockIdx.x] = d[0];
    }
}

__global__ void __launch_bounds__(RED_THREADS) metrics_final(MetricsArgs a, int64_t tiles)
{
    __shared__ int64_t il[NMI * RED_THREADS];
    __shared__ double dl[RED_THREADS];
    int64_t c[NMI];
    double d[1];
    sum_partials<int64_t, NMI>(a.ipart, tiles, c, il);
    sum_partials<double, 1>(a.dpart, tiles, d, dl);
    if (threadIdx.x != 0) return;
    double *m = a.metrics;
    const double n = (double)a.n;
    const int64_t st = c[5], sl = c[6];
    for (int k = 0; k < PARASON_METRIC_COUNT; ++k) m[k] = 0.0;
    m[PARASON_METRIC_ROWS] = n;
    m[PARASON_METRIC_VALID] = (double)c[0];
    m[PARASON_METRIC_TRIGGERED] = (double)c[1];
    m[PARASON_METRIC_CORRECT] = (double)c[2];
    m[PARASON_METRIC_TRUNCATED] = (double)c[3];
    m[PARASON_METRIC_COUNT_MISMATCH] = (double)c[4];
    m[PARASON_METRIC_SUM_TOTAL] = (double)st;
    m[PARASON_METRIC_SUM_LATENCY] = (double)sl;
    m[PARASON_METRIC_SUM_SUBTASK] = (double)c[7];
    m[PARASON_METRIC_SUM_TRIAL] = (double)c[8];
    if (a.n > 0) {
        m[PARASON_METRIC_TRIGGER_RATIO] = __ddiv_rn((double)c[1], n);
        m[PARASON_METRIC_MEAN_LATENCY] = __ddiv_rn((double)sl, n);
        m[PARASON_METRIC_MEAN_TOTAL] = __ddiv_rn((double)st, n);
        m[PARASON_METRIC_MEAN_SAVED] = __ddiv_rn((double)(st - sl), n);
        m[PARASON_METRIC_ACCURACY] = __ddiv_rn((double)c[2], n);
        m[PARASON_METRIC_MEAN_REWARD] = __ddiv_rn(d[0], n);
    }
    if (sl > 0) m[PARASON_METRIC_ACCELERATION] = __ddiv_rn((double)st, (double)sl);
    if (st > 0) {
        m[PARASON_METRIC_SUBTASK_SHARE] = __ddiv_rn((double)c[7], (double)st);
        m[PARASON_METRIC_TRIAL_SHARE] = __ddiv_rn((double)c[8], (double)st);
    }
}

} /* namespace pk */
