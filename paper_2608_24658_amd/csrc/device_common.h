/*
 * device_common.h -- constants and device helpers shared by the kernels of
 * libparason.so: token classes and the tag test, the segment plan's geometry
 * and cursor, wave helpers and the deterministic block reductions.  Only
 * inline device code lives here; every kernel is defined in exactly one
 * translation unit.
 */
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "parason.h"

namespace pk {

constexpr int WAVE = 64;
#ifndef PARASON_SEG_VEC
#define PARASON_SEG_VEC 256
#endif
#ifndef PARASON_SCAN_WAVES_PER_SIMD
#define PARASON_SCAN_WAVES_PER_SIMD 4
#endif
constexpr int SEG_VEC = PARASON_SEG_VEC; /* 16-byte vectors per segment (1024 tokens) */
constexpr int SEG_TOK = 4 * SEG_VEC;     /* tokens per segment */
constexpr int LOADS = SEG_VEC / WAVE;    /* vector loads per lane per segment */
/* Where the tag events of a segment (or of a whole row) are kept: one array
 * of 4-byte slots, a list being a run of slots starting at a multiple of 4.
 * The first GATHER_SLOTS per segment are a per-row area (the segments of a
 * row are consecutive) that gather_rows writes compact lists into; the rest is
 * the pool the scan writes into, cut into one region per scan wave:
 * POOL_PER_SEG slots for each segment of the wave's range, plus an equal
 * share of what the batch's segments leave of the pool (at least POOL_MIN
 * slots), so that a wave with one or two segments of a small batch can still
 * hold an outline-heavy segment.  A wave fills its region in order, so no
 * atomics are needed, and tags, which are rare, use about 1.5 % of the token
 * bytes in all. */
constexpr int GATHER_SLOTS = 4;
constexpr int POOL_PER_SEG = 8;
constexpr int64_t POOL_MIN = (int64_t)1 << 20;
/* A segment's event list (or, in its first segment, a compact row's): its
 * length and its first slot.  Slot indices fit 32 bits for any batch one GPU
 * holds (the host refuses larger ones). */
struct SegRec {
    int32_t count;
    uint32_t list;
};

/* seg count of a segment whose events were not stored: the row kernels
 * classify its tokens again (counts of stored lists are at most 2048) */
constexpr int32_t DENSE = 1 << 20;
static_assert(SEG_VEC % WAVE == 0, "a segment is a whole number of wave-wide loads");
static_assert(GATHER_SLOTS % 4 == 0 && POOL_PER_SEG % 4 == 0, "stored events are read 16 bytes at a time");
constexpr int PLAN_TILE = 4096;          /* rows per plan tile */
constexpr int PLAN_THREADS = 256;
constexpr int ROWS_PER_THREAD = PLAN_TILE / PLAN_THREADS;
#ifndef PARASON_FAST_DEPTH
#define PARASON_FAST_DEPTH 4
#endif
constexpr int FAST_DEPTH = PARASON_FAST_DEPTH; /* LDS frames per row (depth <= FAST_DEPTH + 1) */
constexpr int MID_DEPTH = 32;            /* LDS frames per row handed to the second tier */
constexpr int FAST_ENTRIES = 64;         /* entries per open block on the fast path */
constexpr int FRAME_WORDS = 8;
/* frames hold the enclosing blocks (the innermost open block stays in
 * registers), so PARASON_MAX_DEPTH - 1 of them evaluate a row nested
 * PARASON_MAX_DEPTH deep and flag one nested deeper */
constexpr int64_t DEEP_FRAMES = PARASON_MAX_DEPTH - 1;
constexpr int64_t DEEP_ENTRY_BITS = PARASON_MAX_OPEN_ENTRIES;
/* A row nests at most one level per 6 tokens and opens at most one outline
 * entry per 3, so a store of these per 1024-token segment of the batch holds
 * any row (up to DEEP_FRAMES and DEEP_ENTRY_BITS). */
constexpr int64_t DEEP_FRAMES_PER_SEG = SEG_TOK / 6 + 1;
constexpr int64_t DEEP_BITS_PER_SEG = SEG_TOK / 3 + 1;

/* Token classes: 0 = Text, 1..12 = tags in tag_ids order. */
enum : uint32_t {
    C_TEXT = 0, C_THINK, C_END_THINK, C_PAR, C_END_PAR, C_OUT, C_END_OUT,
    C_SUB, C_END_SUB, C_TRI, C_END_TRI, C_THR, C_END_THR
};

/* Branch type of the innermost enclosing thread. */
enum : uint32_t { T_MAIN = 0, T_SUB = 1, T_TRI = 2 };

constexpr int TAG_SLOTS = 64; /* slots of the tag hash: one per lane */

struct TagMatch {
    int32_t ids[12];
    int32_t base;     /* contiguous case: smallest id */
    uint32_t lut_lo;  /* contiguous case: class of id base+o in nibble o (o < 8) */
    uint32_t lut_hi;  /* nibbles for o = 8..11 */
    int32_t contiguous;
    /* other tag sets, when a pair of shifts separates them: slot(t) =
     * ((t >> hash_a) ^ (t >> hash_b)) mod 64 is distinct for the twelve ids,
     * slot_id[s] is the id in slot s (or an id of another slot, which no token
     * hashing to s can equal) */
    int32_t hashed;
    int32_t hash_a, hash_b;
    int32_t slot_id[TAG_SLOTS];
};

__device__ __forceinline__ uint32_t tag_slot(const TagMatch &tm, int32_t t)
{
    const uint32_t u = (uint32_t)t;
    return ((u >> tm.hash_a) ^ (u >> tm.hash_b)) & (uint32_t)(TAG_SLOTS - 1);
}

__device__ __forceinline__ uint32_t classify(const TagMatch &tm, int32_t t, bool contig)
{
    if (contig) {
        uint32_t o = (uint32_t)t - (uint32_t)tm.base;
        if (o >= 12u) return C_TEXT;
        return o < 8u ? (tm.lut_lo >> (4u * o)) & 15u : (tm.lut_hi >> (4u * (o - 8u))) & 15u;
    }
    uint32_t c = C_TEXT;
#pragma unroll
    for (int k = 0; k < 12; ++k) c = (t == tm.ids[k]) ? (uint32_t)(k + 1) : c;
    return c;
}

/* First 16-byte vector of a row's segments: the 128-byte line (8 vectors) that
 * holds its first token, so every wave-wide load covers whole L2 lines. */
__device__ __forceinline__ int64_t row_first_vec(int64_t g) { return (g >> 5) << 3; }

/* One past the last vector holding a token of the row. */
__device__ __forceinline__ int64_t row_end_vec(int64_t g, int32_t len) { return (g + (int64_t)len + 3) >> 2; }

__device__ __forceinline__ int64_t row_segments(int64_t start, int32_t len, int64_t mis)
{
    if (start < 0 || len <= 0) return 0;
    int64_t g = start + mis;
    int64_t nvec = row_end_vec(g, len) - row_first_vec(g);
    return (nvec + SEG_VEC - 1) / SEG_VEC;
}

__device__ __forceinline__ int64_t uniform64(int64_t x)
{
    uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
    uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)x >> 32));
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

/* Inclusive prefix sum over the 64 lanes of a wave. */
__device__ __forceinline__ int64_t wave_inclusive_scan(int64_t v)
{
    const int lane = threadIdx.x & (WAVE - 1);
#pragma unroll
    for (int d = 1; d < WAVE; d <<= 1) {
        int64_t o = __shfl_up(v, d, WAVE);
        if (lane >= d) v += o;
    }
    return v;
}

/* Wave scans and reductions by DPP: shifts within rows of 16 lanes
 * (row_shr), carries between the four rows from the rows' last lanes
 * (readlane).  A chain of shuffles would go through the LDS crossbar, one
 * round trip per step; these stay in the VALU.  Every lane must call them. */
constexpr int DPP_ROW_SHR = 0x110; /* row_shr:n is DPP_ROW_SHR + n */
constexpr int DPP_WAVE_SHR1 = 0x138;

template <int N>
__device__ __forceinline__ int32_t row_shr(int32_t v, int32_t ident)
{
    return __builtin_amdgcn_update_dpp(ident, v, DPP_ROW_SHR + N, 0xf, 0xf, false);
}

/* v of lane - 1 (ident in lane 0). */
__device__ __forceinline__ int32_t lane_before(int32_t v, int32_t ident)
{
    return __builtin_amdgcn_update_dpp(ident, v, DPP_WAVE_SHR1, 0xf, 0xf, false);
}

__device__ __forceinline__ int32_t lane63(int32_t v) { return __builtin_amdgcn_readlane(v, WAVE - 1); }

struct OpAdd {
    static constexpr int32_t ident = 0;
    __device__ static int32_t f(int32_t x, int32_t y) { return x + y; }
};
struct OpMax {
    static constexpr int32_t ident = INT32_MIN;
    __device__ static int32_t f(int32_t x, int32_t y) { return x > y ? x : y; }
};
struct OpMin {
    static constexpr int32_t ident = INT32_MAX;
    __device__ static int32_t f(int32_t x, int32_t y) { return x < y ? x : y; }
};

template <class Op>
__device__ __forceinline__ int32_t dpp_incl_scan(int32_t v, int lane)
{
    v = Op::f(v, row_shr<1>(v, Op::ident));
    v = Op::f(v, row_shr<2>(v, Op::ident));
    v = Op::f(v, row_shr<4>(v, Op::ident));
    v = Op::f(v, row_shr<8>(v, Op::ident));
    const int32_t t0 = __builtin_amdgcn_readlane(v, 15), t1 = __builtin_amdgcn_readlane(v, 31),
                  t2 = __builtin_amdgcn_readlane(v, 47);
    const int32_t p2 = Op::f(t0, t1), p3 = Op::f(p2, t2);
    const int row = lane >> 4;
    return row == 0 ? v : Op::f(row == 1 ? t0 : (row == 2 ? p2 : p3), v);
}

/* Segmented form: restarts at lanes with head set; lanes before the first
 * head continue from carry.  Row r starts from C_r: C_0 = carry, and
 * C_{r+1} is row r's last lane if the row holds a head, else op(C_r, it). */
template <class Op>
__device__ __forceinline__ int32_t dpp_seg_scan(int32_t v, bool head, int32_t carry, int lane)
{
    int32_t f = head ? 1 : 0;
#define PARASON_SEG_STEP(N)                          \
    {                                                \
        const int32_t vo = row_shr<N>(v, Op::ident); \
        const int32_t fo = row_shr<N>(f, 0);         \
        if (!f) {                                    \
            v = Op::f(vo, v);                        \
            f = fo;                                  \
        }                                            \
    }
    PARASON_SEG_STEP(1)
    PARASON_SEG_STEP(2)
    PARASON_SEG_STEP(4)
    PARASON_SEG_STEP(8)
#undef PARASON_SEG_STEP
    const int32_t v0 = __builtin_amdgcn_readlane(v, 15), v1 = __builtin_amdgcn_readlane(v, 31),
                  v2 = __builtin_amdgcn_readlane(v, 47);
    const int32_t f0 = __builtin_amdgcn_readlane(f, 15), f1 = __builtin_amdgcn_readlane(f, 31),
                  f2 = __builtin_amdgcn_readlane(f, 47);
    const int32_t c1 = f0 ? v0 : Op::f(carry, v0);
    const int32_t c2 = f1 ? v1 : Op::f(c1, v1);
    const int32_t c3 = f2 ? v2 : Op::f(c2, v2);
    const int row = lane >> 4;
    const int32_t c = row == 0 ? carry : (row == 1 ? c1 : (row == 2 ? c2 : c3));
    return f ? v : Op::f(c, v);
}

/* A segment as the scan wave sees it (all fields wave-uniform). */
struct SegView {
    int64_t s;                  /* segment id */
    int64_t row, first, last;   /* its row and the row's first and last segment */
    int64_t v0, v1;             /* its vectors [v0, v1) */
    int64_t g;                  /* row start on the element grid of tok_base */
    int32_t len;
    int32_t q_lo, q_hi;         /* segment positions that belong to the row */
    bool edge;                  /* holds the first or the last vector of the row */
    bool owned;                 /* every segment of the row is in this wave's range */
};

/* Walks a wave's contiguous range of segment ids, row by row. */
struct SegCursor {
    const int64_t *seg_off;
    const int64_t *starts;
    const int32_t *lengths;
    int64_t mis, s_begin, s_end;
    int64_t row, row_first, row_next;
    int64_t g, vrow0, vend;
    int32_t len;
    int32_t nvec;  /* vectors of the row: vend - vrow0 (rows are shorter than 2^31 tokens) */
    int32_t head;  /* row position 0 relative to the row's first vector element: 0 .. 31 */
    bool owned_row;
    bool loaded;

    /* Called by the whole wave. */
    __device__ void seek(int64_t s, int64_t n)
    {
        /* the row holding s: the last row with seg_off[row] <= s, by a 64-way
         * search (each round one load per lane), so that a wave's first load
         * waits for log64(n) dependent loads, not log2(n) */
        const int lane = threadIdx.x & (WAVE - 1);
        int64_t lo = 0, hi = n;
        while (hi - lo > 1) {
            const int64_t step = (hi - lo + WAVE - 1) / WAVE;
            const int64_t idx = lo + lane * step;
            const uint64_t m = __ballot(idx < hi && seg_off[idx] <= s);
            lo += (63 - __builtin_clzll(m | 1ull)) * step;
            hi = min(hi, lo + step);
        }
        row = uniform64(lo);
        row_first = uniform64(seg_off[row]);
        row_next = uniform64(seg_off[row + 1]);
        loaded = false;
    }

    __device__ SegView view(int64_t s)
    {
        while (row_next <= s) {
            ++row;
            row_first = row_next;
            row_next = uniform64(seg_off[row + 1]);
            loaded = false;
        }
        if (!loaded) {
            g = uniform64(starts[row] + mis);
            len = __builtin_amdgcn_readfirstlane(lengths[row]);
            vrow0 = row_first_vec(g);
            vend = row_end_vec(g, len);
            nvec = (int32_t)(vend - vrow0);
            head = (int32_t)(g - 4 * vrow0);
            /* LDS events hold (position << 4 | class) in 32 bits */
            owned_row = row_first >= s_begin && row_next <= s_end && len < (1 << 27);
            loaded = true;
        }
        /* the segment relative to the row, in 32 bits (a row has fewer than
         * 2^21 segments); only the absolute vector indices are 64-bit */
        const int32_t k = (int32_t)(s - row_first);
        const int32_t v0r = k * SEG_VEC;
        const int32_t v1r = min(v0r + SEG_VEC, nvec);
        SegView w;
        w.s = s;
        w.row = row;
        w.first = row_first;
        w.last = row_next - 1;
        w.g = g;
        w.len = len;
        w.v0 = vrow0 + v0r;
        w.v1 = vrow0 + v1r;
        w.edge = k == 0 || v1r == nvec;
        /* row positions 0 .. len-1 relative to the segment's first element:
         * they start inside the first segment only (head < 32) and end inside
         * the last one only, so every other segment is whole */
        w.q_lo = k == 0 ? head : 0;
        w.q_hi = v1r == nvec ? (int32_t)((int64_t)head + len - 4 * (int64_t)v0r) : 4 * (v1r - v0r);
        w.owned = owned_row;
        return w;
    }
};

/* ------------------------------------------------------------------ batch reductions */

/* Deterministic sums: every thread adds its ROWS_PER_THREAD consecutive rows in
 * index order, the block combines the threads in a fixed pairwise tree, and one
 * block adds the block partials in block order. */
constexpr int RED_THREADS = 256;
constexpr int RED_TILE = RED_THREADS * ROWS_PER_THREAD;
static_assert(RED_TILE == PLAN_TILE, "the reductions reuse the plan's tile count");

template <class T, int K>
__device__ __forceinline__ void block_tree_sum(T (&v)[K], T *lds /* [K][RED_THREADS] */)
{
    const int t = threadIdx.x;
#pragma unroll
    for (int k = 0; k < K; ++k) lds[k * RED_THREADS + t] = v[k];
    __syncthreads();
    for (int stride = RED_THREADS / 2; stride > 0; stride >>= 1) {
        if (t < stride) {
#pragma unroll
            for (int k = 0; k < K; ++k) lds[k * RED_THREADS + t] += lds[k * RED_THREADS + t + stride];
        }
        __syncthreads();
    }
#pragma unroll
    for (int k = 0; k < K; ++k) v[k] = lds[k * RED_THREADS];
    __syncthreads();
}

/* Sum of part[0 .. m) (each of K values) in index order by one block. */
template <class T, int K>
__device__ __forceinline__ void sum_partials(const T *part, int64_t m, T (&out)[K], T *lds)
{
    T v[K];
#pragma unroll
    for (int k = 0; k < K; ++k) v[k] = 0;
    const int64_t per = (m + RED_THREADS - 1) / RED_THREADS;
    const int64_t b0 = threadIdx.x * per, b1 = min(m, b0 + per);
    for (int64_t b = b0; b < b1; ++b) {
#pragma unroll
        for (int k = 0; k < K; ++k) v[k] += part[b * K + k];
    }
    block_tree_sum<T, K>(v, lds);
#pragma unroll
    for (int k = 0; k < K; ++k) out[k] = v[k];
}

} /* namespace pk */
