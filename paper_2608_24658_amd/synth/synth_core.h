/*
 * synth_core.h -- seeded synthetic reasoning-trajectory generator.
 *
 * Input generation only: this module holds none of the accounting or reward
 * arithmetic.  The same source is compiled for the device (hipcc, generator
 * kernels) and for the host (g++ with __host__/__device__ defined empty on the
 * command line), so a test can regenerate any row of a large device batch on
 * the CPU and get identical bits.  Everything is integer arithmetic.
 *
 * Random numbers: Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random
 * numbers: as easy as 1, 2, 3", SC'11), keyed by the 64-bit seed, with one
 * counter per draw: (row lo, row hi, purpose << 24 | index, 0).
 *
 * Shape of a row (modelled on the paper's workloads, see the design notes):
 *   <think> main_0 { <Parallel> <Outlines> (<X> entry </X>)^k </Outlines>
 *                    (<Thread> body </Thread>)^k </Parallel> main_j }^nb
 *   </think> answer
 * where a Subtask thread may hold one nested Trial block between two body
 * spans.  Text spans share a length budget by integer weights; each token id of
 * Text is drawn from the flat position in the batch, so the text fill is one
 * embarrassingly parallel pass and the tags are written by a second pass.
 */
#pragma once
#include <stdint.h>

#define SYNTH_MAX_TOP_BLOCKS 3
#define SYNTH_MAX_K 4

/* Tag classes in the order of tag_ids. */
enum {
    SY_THINK = 0, SY_END_THINK, SY_PAR, SY_END_PAR, SY_OUT, SY_END_OUT,
    SY_SUB, SY_END_SUB, SY_TRI, SY_END_TRI, SY_THR, SY_END_THR
};

/* Draw purposes (top byte of counter word 2). */
enum {
    D_LEN = 1, D_LEN2 /* unused */, D_CORRECT, D_TRUNC, D_TRUNC_POS, D_TRIGGER, D_NBLOCKS,
    D_KIND, D_K, D_NEST, D_NK, D_WEIGHT, D_OUTLIER, D_TEXT, D_LOGP
};

typedef struct synth_params {
    uint32_t seed_lo, seed_hi;
    int32_t vocab;           /* V: token ids are in [0, V) */
    int32_t tag_ids[12];     /* in SY_* order */
    int32_t sorted_tags[12]; /* tag_ids ascending (text ids skip them) */
    int32_t len_kind;        /* 0: uniform in [len_lo, len_hi]; 1: log-uniform (P(x) ~ 1/x) */
    int32_t len_lo, len_hi;
    uint32_t p_trigger;      /* probabilities in units of 2^-32 */
    uint32_t p_trial;
    uint32_t p_nest;
    uint32_t p_outlier;
    uint32_t p_trunc;
    uint32_t p_correct;
    uint32_t w_main, w_entry, w_body, w_answer; /* base span weights */
    int32_t outlier_mult;    /* length multiplier of an outlier thread body */
    int32_t max_blocks;      /* top-level blocks: 1 .. max_blocks */
} synth_params;

__host__ __device__ static inline void sy_mulhilo(uint32_t a, uint32_t b, uint32_t *hi, uint32_t *lo)
{
    uint64_t p = (uint64_t)a * (uint64_t)b;
    *hi = (uint32_t)(p >> 32);
    *lo = (uint32_t)p;
}

/* Philox4x32 with 10 rounds; returns the four output words in c. */
__host__ __device__ static inline void sy_philox(uint32_t c[4], uint32_t k0, uint32_t k1)
{
    for (int r = 0; r < 10; ++r) {
        uint32_t hi0, lo0, hi1, lo1;
        sy_mulhilo(0xD2511F53u, c[0], &hi0, &lo0);
        sy_mulhilo(0xCD9E8D57u, c[2], &hi1, &lo1);
        uint32_t n0 = hi1 ^ c[1] ^ k0;
        uint32_t n2 = hi0 ^ c[3] ^ k1;
        c[0] = n0;
        c[1] = lo1;
        c[2] = n2;
        c[3] = lo0;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
}

__host__ __device__ static inline uint32_t sy_draw(const synth_params *P, uint64_t row, uint32_t purpose, uint32_t idx)
{
    uint32_t c[4] = {(uint32_t)row, (uint32_t)(row >> 32), (purpose << 24) | (idx & 0xFFFFFFu), 0u};
    sy_philox(c, P->seed_lo, P->seed_hi);
    return c[0];
}

/* Uniform integer in [0, n) by multiply-shift. */
__host__ __device__ static inline uint32_t sy_below(uint32_t u, uint32_t n)
{
    return (uint32_t)(((uint64_t)u * (uint64_t)n) >> 32);
}

/* Four consecutive Text ids for flat positions 4q .. 4q+3. */
__host__ __device__ static inline void sy_text4(const synth_params *P, uint64_t q, int32_t out[4])
{
    uint32_t c[4] = {(uint32_t)q, (uint32_t)(q >> 32), (uint32_t)D_TEXT << 24, 0u};
    sy_philox(c, P->seed_lo, P->seed_hi);
    uint32_t n_text = (uint32_t)(P->vocab - 12);
    for (int j = 0; j < 4; ++j) {
        int32_t id = (int32_t)sy_below(c[j], n_text);
        for (int t = 0; t < 12; ++t) /* skip over the reserved ids, ascending */
            if (id >= P->sorted_tags[t]) ++id;
        out[j] = id;
    }
}

/* Row structure, drawn once per row. */
typedef struct {
    int32_t nb;                                   /* top-level blocks used */
    uint8_t kind[SYNTH_MAX_TOP_BLOCKS];           /* 0 Subtask, 1 Trial */
    uint8_t k[SYNTH_MAX_TOP_BLOCKS];
    uint8_t nk[SYNTH_MAX_TOP_BLOCKS][SYNTH_MAX_K]; /* nested Trial entries; 0 = none */
} sy_shape;

/* Tokens of a top-level block that do not depend on the text budget
 * (tags, plus one token of each entry's non-empty text). */
__host__ __device__ static inline int64_t sy_block_fixed(const sy_shape *s, int b)
{
    int64_t n = 4 + 3 * (int64_t)s->k[b] + 2 * (int64_t)s->k[b];
    for (int t = 0; t < s->k[b]; ++t)
        if (s->nk[b][t]) n += 4 + 5 * (int64_t)s->nk[b][t];
    return n;
}

__host__ __device__ static inline int64_t sy_target_len(const synth_params *P, uint64_t row)
{
    if (P->len_kind == 0)
        return (int64_t)P->len_lo + sy_below(sy_draw(P, row, D_LEN, 0), (uint32_t)(P->len_hi - P->len_lo + 1));
    /* Log-uniform: P(L = x) proportional to 1/x on [len_lo, len_hi], by
     * rejection in integer arithmetic.  Draw one of the J octaves
     * [lo 2^j, lo 2^(j+1)) that start inside the range, uniformly (the last
     * one as a whole octave), then x uniform in it; keep x when x <= len_hi,
     * with probability lo 2^j / x (u / 2^32 < lo 2^j / x).  A kept x has
     * probability (1/J) (1/(lo 2^j)) (lo 2^j / x) = 1/(J x) per attempt, for
     * every x of the range; about two attempts in three keep theirs. */
    const int64_t lo = P->len_lo, hi = P->len_hi;
    uint32_t J = 1;
    while ((lo << J) <= hi) ++J;
    for (uint32_t a = 0; a < 1024; ++a) {
        const int64_t base = lo << sy_below(sy_draw(P, row, D_LEN, 3 * a), J);
        const int64_t x = base + (int64_t)sy_below(sy_draw(P, row, D_LEN, 3 * a + 1), (uint32_t)base);
        if (x > hi) continue;
        const uint32_t u = sy_draw(P, row, D_LEN, 3 * a + 2);
        if ((uint64_t)u * (uint64_t)x < ((uint64_t)base << 32)) return x;
    }
    return lo; /* 1024 rejections in a row: probability below 2^-1500 */
}

__host__ __device__ static inline void sy_shape_of(const synth_params *P, uint64_t row, int64_t L, sy_shape *s)
{
    int nb = 0;
    if (sy_draw(P, row, D_TRIGGER, 0) < P->p_trigger)
        nb = 1 + (int)sy_below(sy_draw(P, row, D_NBLOCKS, 0), (uint32_t)P->max_blocks);
    for (int b = 0; b < SYNTH_MAX_TOP_BLOCKS; ++b) {
        int trial = sy_draw(P, row, D_KIND, b) < P->p_trial;
        s->kind[b] = (uint8_t)trial;
        /* Trial blocks: 1..4 attempts; Subtask blocks: 2..4 parts */
        s->k[b] = (uint8_t)(trial ? 1 + sy_below(sy_draw(P, row, D_K, b), 4) : 2 + sy_below(sy_draw(P, row, D_K, b), 3));
        for (int t = 0; t < SYNTH_MAX_K; ++t) {
            int nest = !trial && t < s->k[b] && sy_draw(P, row, D_NEST, b * 8 + t) < P->p_nest;
            s->nk[b][t] = (uint8_t)(nest ? 1 + sy_below(sy_draw(P, row, D_NK, b * 8 + t), 4) : 0);
        }
    }
    /* keep as many blocks as the target length holds */
    int64_t need = 2;
    int used = 0;
    for (int b = 0; b < nb; ++b) {
        int64_t f = sy_block_fixed(s, b);
        if (need + f > L) break;
        need += f;
        ++used;
    }
    s->nb = used;
}

/* Walk state: either measures the row (out == 0) or writes its tags (and,
 * on the host, its text) into out[0 .. limit). */
typedef struct {
    const synth_params *P;
    uint64_t row;
    int64_t pos;      /* next position in the row */
    int64_t limit;    /* positions >= limit are not written */
    int32_t *out;     /* row base, or 0 */
    int write_text;   /* host mirror fills Text too */
    uint64_t flat0;   /* flat index of position 0 (Text ids depend on it) */
    uint64_t R;       /* free text budget */
    uint64_t W;       /* total span weight */
    uint64_t cum;     /* cumulative weight of spans emitted so far */
    uint32_t span;    /* span index */
} sy_walk;

__host__ __device__ static inline void sy_put_text(sy_walk *w, int64_t n)
{
    if (w->out && w->write_text) {
        for (int64_t i = 0; i < n; ++i) {
            int64_t p = w->pos + i;
            if (p >= w->limit) break;
            int32_t t4[4];
            uint64_t q = w->flat0 + (uint64_t)p;
            sy_text4(w->P, q >> 2, t4);
            w->out[p] = t4[q & 3];
        }
    }
    w->pos += n;
}

__host__ __device__ static inline void sy_put_tag(sy_walk *w, int cls)
{
    if (w->out && w->pos < w->limit) w->out[w->pos] = w->P->tag_ids[cls];
    w->pos += 1;
}

/* Weight of span j of the given base weight: base * [0.5, 1.5). */
__host__ __device__ static inline uint64_t sy_weight(const sy_walk *w, uint32_t base, uint32_t j)
{
    return (uint64_t)base * (512u + (sy_draw(w->P, w->row, D_WEIGHT, j) & 1023u)) / 1024u;
}

/* A text span: its share of the budget is floor(R*C_j/W) - floor(R*C_{j-1}/W),
 * so the shares add up to R exactly.  Entry spans get one extra token (T is
 * non-empty).  An outlier body span is outlier_mult times longer. */
__host__ __device__ static inline void sy_span(sy_walk *w, uint32_t base, int is_entry, int is_body)
{
    uint32_t j = w->span++;
    uint64_t wt = sy_weight(w, base, j);
    uint64_t a = w->W ? (w->R * w->cum) / w->W : 0;
    w->cum += wt;
    uint64_t b = w->W ? (w->R * w->cum) / w->W : 0;
    int64_t n = (int64_t)(b - a) + (is_entry ? 1 : 0);
    if (is_body && sy_draw(w->P, w->row, D_OUTLIER, j) < w->P->p_outlier) n *= w->P->outlier_mult;
    sy_put_text(w, n);
}

__host__ __device__ static inline void sy_block(sy_walk *w, int trial, int k, const uint8_t *nk)
{
    int open = trial ? SY_TRI : SY_SUB, close = trial ? SY_END_TRI : SY_END_SUB;
    sy_put_tag(w, SY_PAR);
    sy_put_tag(w, SY_OUT);
    for (int e = 0; e < k; ++e) {
        sy_put_tag(w, open);
        sy_span(w, w->P->w_entry, 1, 0);
        sy_put_tag(w, close);
    }
    sy_put_tag(w, SY_END_OUT);
    for (int t = 0; t < k; ++t) {
        sy_put_tag(w, SY_THR);
        if (nk && nk[t]) {
            sy_span(w, w->P->w_body / 2, 0, 1);
            sy_block(w, 1, nk[t], 0);
            sy_span(w, w->P->w_body / 2, 0, 1);
        } else {
            sy_span(w, w->P->w_body, 0, 1);
        }
        sy_put_tag(w, SY_END_THR);
    }
    sy_put_tag(w, SY_END_PAR);
}

/* Emit (or measure) a complete row of the given shape. */
__host__ __device__ static inline void sy_row(sy_walk *w, const sy_shape *s)
{
    sy_put_tag(w, SY_THINK);
    sy_span(w, w->P->w_main, 0, 0);
    for (int b = 0; b < s->nb; ++b) {
        sy_block(w, s->kind[b], s->k[b], s->nk[b]);
        sy_span(w, w->P->w_main, 0, 0);
    }
    sy_put_tag(w, SY_END_THINK);
    sy_span(w, w->P->w_answer, 0, 0);
}

/* Total weight of the row's spans (a measuring walk with R = 0). */
__host__ __device__ static inline uint64_t sy_total_weight(const synth_params *P, uint64_t row, const sy_shape *s)
{
    sy_walk w = {P, row, 0, 0, 0, 0, 0, 0, 0, 0, 0};
    sy_row(&w, s);
    return w.cum;
}

typedef struct {
    sy_shape shape;
    int64_t target;   /* target length before outliers */
    uint64_t R, W;    /* text budget and total weight */
    int64_t full;     /* length of the complete row */
    int64_t len;      /* final length (after truncation) */
    uint8_t correct;
} sy_rowinfo;

/* Everything about a row except its tokens. */
__host__ __device__ static inline void sy_row_info(const synth_params *P, uint64_t row, sy_rowinfo *ri)
{
    int64_t L = sy_target_len(P, row);
    ri->target = L;
    sy_shape_of(P, row, L, &ri->shape);
    ri->correct = sy_draw(P, row, D_CORRECT, 0) < P->p_correct ? 1 : 0;
    if (L < 2) {
        /* too short for <think></think>: a prefix of it */
        ri->R = 0;
        ri->W = 0;
        ri->full = L;
        ri->len = L;
        return;
    }
    int64_t fixed = 2;
    for (int b = 0; b < ri->shape.nb; ++b) fixed += sy_block_fixed(&ri->shape, b);
    ri->R = (uint64_t)(L - fixed);
    ri->W = sy_total_weight(P, row, &ri->shape);
    sy_walk w = {P, row, 0, 0, 0, 0, 0, ri->R, ri->W, 0, 0};
    sy_row(&w, &ri->shape);
    ri->full = w.pos;
    ri->len = ri->full;
    if (sy_draw(P, row, D_TRUNC, 0) < P->p_trunc && ri->full > 0)
        ri->len = (int64_t)sy_below(sy_draw(P, row, D_TRUNC_POS, 0), (uint32_t)ri->full);
}

/* Write the row's tags (and its Text when write_text) into out[0 .. ri->len). */
__host__ __device__ static inline void sy_row_emit(const synth_params *P, uint64_t row, const sy_rowinfo *ri,
                                                   int32_t *out, uint64_t flat0, int write_text)
{
    if (ri->target < 2) {
        if (ri->len >= 1) out[0] = P->tag_ids[SY_THINK];
        return;
    }
    sy_walk w = {P, row, 0, ri->len, out, write_text, flat0, ri->R, ri->W, 0, 0};
    sy_row(&w, &ri->shape);
}

/* Log-probabilities of the generated tokens at flat positions 4q .. 4q+3, for
 * the policy-gradient step: logp_old uniform in (-8, 0], logp = logp_old +
 * delta with delta triangular on (-0.25, 0.25).  Both come from integers by
 * exact float operations (a conversion of an integer below 2^25 and power-of-
 * two scalings) and one float addition, so host and device agree bit for bit. */
__host__ __device__ static inline void sy_logp4(const synth_params *P, uint64_t q, float old4[4], float new4[4])
{
    uint32_t c[3][4];
    for (int k = 0; k < 3; ++k) {
        c[k][0] = (uint32_t)q;
        c[k][1] = (uint32_t)(q >> 32);
        c[k][2] = ((uint32_t)D_LOGP << 24) | (uint32_t)k;
        c[k][3] = 0u;
        sy_philox(c[k], P->seed_lo, P->seed_hi);
    }
    for (int j = 0; j < 4; ++j) {
        float o = (float)(int32_t)(c[0][j] >> 8) * (-8.0f / 16777216.0f);
        int32_t t = (int32_t)(c[1][j] >> 8) + (int32_t)(c[2][j] >> 8) - 16777216;
        float delta = (float)t * (1.0f / 67108864.0f);
        old4[j] = o;
        new4[j] = o + delta;
    }
}
