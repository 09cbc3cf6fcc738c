/*
 * parason_oracle.c -- CPU oracle for parallel-trajectory accounting and the
 * Parallelism-Aware GRPO reward.
 *
 * TEST INFRASTRUCTURE.  This file is the slow, obviously-correct reference that
 * the GPU path is checked against.  Only the test suite, the smoke check and the
 * CPU-baseline leg of the benchmark may load it.  It shares no code, header or
 * table with the GPU library: the tag order and the flag bit values below are
 * restated from the interface contract, not included from it.
 *
 * What it computes, and where the paper defines it:
 *   - Validity of a token stream against the grammar G = (V, Sigma, R, S) of the
 *     figure "Context-Free Grammar for Parason" (Sec. 3.2).  One parse function
 *     per production; each returns the synthesized attribute of its
 *     non-terminal.
 *   - Model latency T_i: the length of the longest generation path; sequential
 *     tokens count once, a <Parallel> block contributes its longest branch
 *     (Sec. 4, "Evaluation" paragraph; T_i and L_latency in Sec. 3.3).
 *   - Tokens placed in Subtask and in Trial branches (R_subtask, R_trial under
 *     Definition 3.1, Sec. 3.3).
 *   - eta(s) = 1 - L_latency / L_total (Sec. 3.3, list under Definition 3.1).
 *   - Group normalisation and the reward of Definition 3.1 (Eq. "Parallel RL
 *     Reward", Sec. 3.3) with f the identity, in IEEE double precision.
 *
 * Readings of points the paper leaves open (each one is listed in the design
 * notes of the repository):
 *   - every tag is one reserved token id; any other id is Text;
 *   - every token costs 1 on the path that emits it, tags included;
 *   - the outline (<Outlines> ... </Outlines>) is decoded by the main trajectory
 *     before the branches are dispatched (Sec. 3.4), so its tokens are on the
 *     main path of the block;
 *   - a token is a Subtask (Trial) token when its innermost enclosing <Thread>
 *     is paired with a Subtask (Trial) entry; thread k pairs with entry k, a
 *     surplus thread is untyped and the block is flagged COUNT_MISMATCH;
 *   - Text after </think> (the answer) is allowed and counted sequentially;
 *     nothing may precede <think>;
 *   - an invalid or truncated stream is sequential: latency = total, no branch
 *     tokens, no blocks; first_error_pos is the length of its longest prefix that
 *     is still a prefix of some valid stream;
 *   - mean and standard deviation are taken over the G rollouts of one prompt
 *     (population form); z = 0 when every member of the group has the same
 *     value (sigma = 0 in exact arithmetic) or the computed sigma is 0.
 *   - strict by default: no Text between the structural tags of a parallel
 *     region, as the grammar is printed.  With CFG_LENIENT_GAPS (the layout of
 *     Figure 3, which puts line breaks there) a run of Text may follow
 *     <Parallel>, <Outlines>, each outline entry, </Outlines> and each
 *     </Thread> of a region; those tokens are decoded by the enclosing path,
 *     like the outline, so they add to lat(P) and take the enclosing branch
 *     type.
 *
 * Deep nesting recurses; the batch entry point runs the parser on a worker
 * thread with a large stack so adversarial depth cannot overflow the C stack.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* Token classes: Text, then the twelve tags in the order of the tag_ids
 * argument: <think> </think> <Parallel> </Parallel> <Outlines> </Outlines>
 * <Subtask> </Subtask> <Trial> </Trial> <Thread> </Thread>. */
enum {
    K_TEXT = 0,
    K_THINK, K_END_THINK, K_PAR, K_END_PAR, K_OUT, K_END_OUT,
    K_SUB, K_END_SUB, K_TRI, K_END_TRI, K_THR, K_END_THR,
    K_EOS = -1
};

/* Branch type of the innermost enclosing thread. */
enum { CTX_MAIN = 0, CTX_SUBTASK = 1, CTX_TRIAL = 2 };

/* Per-row flag bits (interface contract). */
#define F_VALID          (1u << 0)
#define F_TRUNCATED      (1u << 1)
#define F_COUNT_MISMATCH (1u << 2)
#define F_TRIGGERED      (1u << 3)

/* Configuration flag bits (interface contract). */
#define CFG_INVALID_KEEPS_CORRECTNESS (1u << 0)
#define CFG_LENIENT_GAPS (1u << 3)

typedef struct {
    int32_t total;
    int32_t latency;
    int32_t n_subtask;
    int32_t n_trial;
    int32_t n_blocks;
    int32_t max_depth;
    int32_t first_error_pos;
    uint32_t flags;
} oracle_row_t;

typedef struct {
    const int32_t *tok;
    int64_t len;
    int64_t pos;
    const int32_t *tag_ids;
    int failed;
    int64_t err_pos;
    int64_t n_by_ctx[3];
    int64_t n_blocks;
    int64_t depth, max_depth;
    int mismatch;
    int lenient; /* CFG_LENIENT_GAPS */
} parser_t;

static int class_at(const parser_t *p, int64_t i)
{
    int32_t t = p->tok[i];
    for (int k = 0; k < 12; ++k)
        if (p->tag_ids[k] == t) return k + 1;
    return K_TEXT;
}

static int peek(const parser_t *p)
{
    return p->pos < p->len ? class_at(p, p->pos) : K_EOS;
}

/* The first token that cannot extend the prefix is where parsing stops. */
static void fail(parser_t *p)
{
    if (!p->failed) {
        p->failed = 1;
        p->err_pos = p->pos;
    }
}

/* Consume one token and attribute it to the innermost enclosing thread type. */
static void take(parser_t *p, int ctx)
{
    p->n_by_ctx[ctx] += 1;
    p->pos += 1;
}

static int expect(parser_t *p, int cls, int ctx)
{
    if (p->failed) return 0;
    if (peek(p) != cls) {
        fail(p);
        return 0;
    }
    take(p, ctx);
    return 1;
}

static int64_t parse_P(parser_t *p, int ctx);

/* T -> non-empty free-form text.  Returns the number of tokens. */
static int64_t parse_T(parser_t *p, int ctx)
{
    int64_t n = 0;
    while (peek(p) == K_TEXT) {
        take(p, ctx);
        ++n;
    }
    if (n == 0) fail(p);
    return n;
}

/* A gap between structural tags of a parallel region: with CFG_LENIENT_GAPS
 * any run of Text (possibly empty), otherwise nothing.  Returns its length. */
static int64_t parse_gap(parser_t *p, int ctx)
{
    int64_t n = 0;
    if (!p->lenient || p->failed) return 0;
    while (peek(p) == K_TEXT) {
        take(p, ctx);
        ++n;
    }
    return n;
}

/* B -> T B | P B | epsilon.  Returns lat(B): text counts once per token, a
 * parallel region contributes lat(P). */
static int64_t parse_B(parser_t *p, int ctx)
{
    int64_t lat = 0;
    for (;;) {
        if (p->failed) return 0;
        int c = peek(p);
        if (c == K_TEXT)
            lat += parse_T(p, ctx);
        else if (c == K_PAR)
            lat += parse_P(p, ctx);
        else
            return lat; /* epsilon; the caller checks what follows */
    }
}

/* E -> <Subtask> T </Subtask> | <Trial> T </Trial>.  Returns the entry type. */
static int parse_E(parser_t *p, int ctx)
{
    int c = peek(p);
    if (c == K_SUB) {
        take(p, ctx);
        parse_T(p, ctx);
        expect(p, K_END_SUB, ctx);
        return CTX_SUBTASK;
    }
    if (c == K_TRI) {
        take(p, ctx);
        parse_T(p, ctx);
        expect(p, K_END_TRI, ctx);
        return CTX_TRIAL;
    }
    fail(p);
    return CTX_MAIN;
}

typedef struct {
    int *type;
    int64_t n, cap;
} entries_t;

static void entries_push(entries_t *e, int t)
{
    if (e->n == e->cap) {
        e->cap = e->cap ? 2 * e->cap : 8;
        e->type = (int *)realloc(e->type, (size_t)e->cap * sizeof(int));
        if (!e->type) abort();
    }
    e->type[e->n++] = t;
}

/* G -> E G | E  (each E followed by a gap when lenient) */
static void parse_G(parser_t *p, int ctx, entries_t *entries)
{
    do {
        int t = parse_E(p, ctx);
        if (p->failed) return;
        entries_push(entries, t);
        parse_gap(p, ctx);
    } while (peek(p) == K_SUB || peek(p) == K_TRI);
}

/* O -> <Outlines> G </Outlines>  (a gap after <Outlines> when lenient).
 * Entry types are returned in order. */
static void parse_O(parser_t *p, int ctx, entries_t *entries)
{
    if (!expect(p, K_OUT, ctx)) return;
    parse_gap(p, ctx);
    parse_G(p, ctx, entries);
    expect(p, K_END_OUT, ctx);
}

/* W -> <Thread> B </Thread>.  The thread's own tags and body belong to the
 * thread's branch type.  Returns lat(W) = 2 + lat(B). */
static int64_t parse_W(parser_t *p, int type)
{
    if (!expect(p, K_THR, type)) return 0;
    int64_t body = parse_B(p, type);
    if (!expect(p, K_END_THR, type)) return 0;
    return 2 + body;
}

/* H -> W H | W  (each W followed by a gap when lenient; the gap tokens are the
 * enclosing path's, added to *gaps).  Thread k is paired with entry k.
 * Returns max_k lat(W_k). */
static int64_t parse_H(parser_t *p, const entries_t *entries, int ctx, int64_t *gaps)
{
    int64_t k = 0, longest = 0;
    do {
        int type = k < entries->n ? entries->type[k] : CTX_MAIN;
        int64_t lat = parse_W(p, type);
        if (p->failed) return 0;
        if (lat > longest) longest = lat;
        *gaps += parse_gap(p, ctx);
        ++k;
    } while (peek(p) == K_THR);
    if (k != entries->n) p->mismatch = 1;
    return longest;
}

/* P -> <Parallel> O H </Parallel>.  <Parallel> and the outline are decoded on
 * the enclosing path before dispatch, the block then waits for its longest
 * thread, then </Parallel> follows:
 *   lat(P) = 1 + |O| + max_k lat(W_k) + 1
 * and, when lenient, + the gap tokens after <Parallel>, </Outlines> and each
 * thread (the gaps inside O are part of |O|). */
static int64_t parse_P(parser_t *p, int ctx)
{
    p->n_blocks += 1;
    p->depth += 1;
    if (p->depth > p->max_depth) p->max_depth = p->depth;

    if (!expect(p, K_PAR, ctx)) return 0;
    int64_t gaps = parse_gap(p, ctx);
    int64_t o_start = p->pos;
    entries_t entries = {0, 0, 0};
    parse_O(p, ctx, &entries);
    int64_t o_len = p->pos - o_start;
    gaps += parse_gap(p, ctx);
    int64_t longest = 0;
    if (!p->failed) longest = parse_H(p, &entries, ctx, &gaps);
    free(entries.type);
    if (!expect(p, K_END_PAR, ctx)) return 0;

    p->depth -= 1;
    return 1 + gaps + o_len + longest + 1;
}

/* S -> <think> B </think>, followed by free text (the answer). */
static void parse_row(parser_t *p, oracle_row_t *out)
{
    int64_t lat = 0;
    if (expect(p, K_THINK, CTX_MAIN)) {
        int64_t body = parse_B(p, CTX_MAIN);
        if (expect(p, K_END_THINK, CTX_MAIN)) {
            int64_t tail = 0;
            while (peek(p) == K_TEXT) {
                take(p, CTX_MAIN);
                ++tail;
            }
            if (p->pos < p->len) fail(p); /* a tag after </think> */
            lat = 1 + body + 1 + tail;
        }
    }

    out->total = (int32_t)p->len;
    if (!p->failed) {
        out->latency = (int32_t)lat;
        out->n_subtask = (int32_t)p->n_by_ctx[CTX_SUBTASK];
        out->n_trial = (int32_t)p->n_by_ctx[CTX_TRIAL];
        out->n_blocks = (int32_t)p->n_blocks;
        out->max_depth = (int32_t)p->max_depth;
        out->first_error_pos = -1;
        out->flags = F_VALID;
        if (p->mismatch) out->flags |= F_COUNT_MISMATCH;
        if (p->n_blocks >= 1) out->flags |= F_TRIGGERED;
    } else {
        /* Invalid stream: accounted as purely sequential. */
        out->latency = (int32_t)p->len;
        out->n_subtask = 0;
        out->n_trial = 0;
        out->n_blocks = 0;
        out->max_depth = 0;
        out->first_error_pos = (int32_t)p->err_pos;
        out->flags = p->err_pos == p->len ? F_TRUNCATED : 0u;
    }
}

void oracle_eval_row(const int32_t *tok, int32_t len, const int32_t tag_ids[12],
                     uint32_t cfg_flags, oracle_row_t *out)
{
    parser_t p;
    memset(&p, 0, sizeof(p));
    p.tok = tok;
    p.len = len < 0 ? 0 : len;
    p.tag_ids = tag_ids;
    p.lenient = (cfg_flags & CFG_LENIENT_GAPS) != 0;
    parse_row(&p, out);
}

typedef struct {
    const int32_t *tokens;
    const int64_t *starts;
    const int32_t *lengths;
    int64_t n_rows;
    const int32_t *tag_ids;
    uint32_t cfg_flags;
    oracle_row_t *out;
} batch_t;

static void *batch_main(void *arg)
{
    batch_t *b = (batch_t *)arg;
    for (int64_t i = 0; i < b->n_rows; ++i)
        oracle_eval_row(b->tokens + b->starts[i], b->lengths[i], b->tag_ids, b->cfg_flags, &b->out[i]);
    return NULL;
}

/* Evaluate rows [0, n_rows); row i is tokens[starts[i] .. starts[i]+lengths[i]).
 * cfg_flags: CFG_LENIENT_GAPS or 0 (other bits are ignored here).
 * Runs single-threaded on one worker thread whose stack is large enough for
 * the deepest nesting any of the rows can reach.  Returns 0 on success. */
int oracle_eval_rows(const int32_t *tokens, const int64_t *starts, const int32_t *lengths,
                     int64_t n_rows, const int32_t tag_ids[12], uint32_t cfg_flags, oracle_row_t *out)
{
    batch_t b = {tokens, starts, lengths, n_rows, tag_ids, cfg_flags, out};
    /* The parser recurses once per <Parallel> it has consumed and not yet
     * closed, so a row's <Parallel> count bounds its depth; each level takes
     * at most a few hundred bytes of C stack across parse_B/parse_P/parse_H/
     * parse_W. */
    int64_t max_par = 0;
    for (int64_t i = 0; i < n_rows; ++i) {
        int64_t np = 0;
        for (int64_t j = 0; j < (int64_t)lengths[i]; ++j) np += tokens[starts[i] + j] == tag_ids[K_PAR - 1];
        if (np > max_par) max_par = np;
    }
    size_t stack = (size_t)64 << 20;
    size_t need = ((size_t)max_par + 64) * 640;
    if (need > stack) stack = need;
    pthread_attr_t attr;
    pthread_t th;
    if (pthread_attr_init(&attr)) return -1;
    if (pthread_attr_setstacksize(&attr, stack)) return -2;
    if (pthread_create(&th, &attr, batch_main, &b)) return -3;
    pthread_join(th, NULL);
    pthread_attr_destroy(&attr);
    return 0;
}

/* ---------------------------------------------------------------------------
 * Reward (Sec. 3.3, Definition 3.1), IEEE double, fixed summation order.
 *
 *   R_i = -1 + 2 * 1(correct_i) * ( 1 - alpha * z_T + beta_s * z_s
 *                                   + beta_r * z_r + min(rho * eta_i, rho_clip) )
 *   z_x = (x_i - mu_x) / sigma_x over the G rollouts of the prompt, f = identity.
 * ------------------------------------------------------------------------- */

/* The branch-token ratio N / L_total as an exact rational (0 when L_total = 0). */
static void ratio_of(int32_t n, int32_t total, int64_t *num, int64_t *den)
{
    if (total <= 0) {
        *num = 0;
        *den = 1;
    } else {
        *num = n;
        *den = total;
    }
}

static int ratios_all_equal(const oracle_row_t *r, int64_t G, int which)
{
    int64_t n0, d0;
    ratio_of(which ? r[0].n_trial : r[0].n_subtask, r[0].total, &n0, &d0);
    for (int64_t i = 1; i < G; ++i) {
        int64_t n, d;
        ratio_of(which ? r[i].n_trial : r[i].n_subtask, r[i].total, &n, &d);
        if (n * d0 != n0 * d) return 0;
    }
    return 1;
}

static int latency_all_equal(const oracle_row_t *r, int64_t G)
{
    for (int64_t i = 1; i < G; ++i)
        if (r[i].latency != r[0].latency) return 0;
    return 1;
}

/* mean and population standard deviation of x[0..G), then z-scores. */
static void zscores(const double *x, int64_t G, int all_equal, double *z)
{
    double sum = 0.0;
    for (int64_t i = 0; i < G; ++i) sum = sum + x[i];
    double mu = sum / (double)G;
    double ss = 0.0;
    for (int64_t i = 0; i < G; ++i) {
        double d = x[i] - mu;
        ss = ss + d * d;
    }
    double sigma = sqrt(ss / (double)G);
    for (int64_t i = 0; i < G; ++i)
        z[i] = (all_equal || sigma == 0.0) ? 0.0 : (x[i] - mu) / sigma;
}

static double frac_of(int32_t n, int32_t total)
{
    return total > 0 ? (double)n / (double)total : 0.0;
}

/* params = {alpha, beta_subtask, beta_trial, rho, rho_clip}.  Any of the
 * per-row outputs except reward may be NULL.  Returns 0 on success. */
int oracle_group_reward(const oracle_row_t *rows, const uint8_t *correct, int64_t n_rows,
                        int32_t G, const double params[5], uint32_t cfg_flags,
                        double *reward, double *r_sub, double *r_tri, double *eta)
{
    if (G <= 0 || n_rows % G != 0) return -1;
    const double alpha = params[0], beta_s = params[1], beta_r = params[2];
    const double rho = params[3], rho_clip = params[4];
    double *buf = (double *)malloc((size_t)G * 6 * sizeof(double));
    if (!buf) return -2;
    double *xT = buf, *xs = buf + G, *xr = buf + 2 * G;
    double *zT = buf + 3 * G, *zs = buf + 4 * G, *zr = buf + 5 * G;

    for (int64_t g0 = 0; g0 < n_rows; g0 += G) {
        const oracle_row_t *r = rows + g0;
        for (int64_t i = 0; i < G; ++i) {
            xT[i] = (double)r[i].latency;
            xs[i] = frac_of(r[i].n_subtask, r[i].total);
            xr[i] = frac_of(r[i].n_trial, r[i].total);
        }
        zscores(xT, G, latency_all_equal(r, G), zT);
        zscores(xs, G, ratios_all_equal(r, G, 0), zs);
        zscores(xr, G, ratios_all_equal(r, G, 1), zr);
        for (int64_t i = 0; i < G; ++i) {
            double e = r[i].total > 0 ? 1.0 - (double)r[i].latency / (double)r[i].total : 0.0;
            int valid = (r[i].flags & F_VALID) != 0;
            int c = correct[g0 + i] != 0 && (valid || (cfg_flags & CFG_INVALID_KEEPS_CORRECTNESS));
            double accel = rho * e;
            double clipped = accel < rho_clip ? accel : rho_clip;
            double inner = 1.0 - alpha * zT[i];
            inner = inner + beta_s * zs[i];
            inner = inner + beta_r * zr[i];
            inner = inner + clipped;
            reward[g0 + i] = -1.0 + 2.0 * (c ? 1.0 : 0.0) * inner;
            if (r_sub) r_sub[g0 + i] = xs[i];
            if (r_tri) r_tri[g0 + i] = xr[i];
            if (eta) eta[g0 + i] = e;
        }
    }
    free(buf);
    return 0;
}

/* ---------------------------------------------------------------------------
 * Batch metrics, as the paper reports them (Table 2, 4 and 5):
 *   trigger ratio      = share of samples with at least one <Parallel> block
 *                        (Table 4 caption);
 *   acceleration ratio = total tokens / longest-path tokens (Table 4 caption;
 *                        Table 5: generated / latency tokens);
 *   token latency      = mean longest-path tokens (Tables 2, 4);
 *   saved tokens       = generated - latency tokens (Table 5);
 * plus accuracy, validity and branch-token shares.  Index order is the
 * interface contract (PARASON_METRIC_* in the C-ABI).
 * ------------------------------------------------------------------------- */
enum {
    M_ROWS = 0, M_VALID, M_TRIGGERED, M_CORRECT, M_TRUNCATED, M_MISMATCH,
    M_SUM_TOTAL, M_SUM_LATENCY, M_SUM_SUBTASK, M_SUM_TRIAL,
    M_TRIGGER_RATIO, M_ACCELERATION, M_MEAN_LATENCY, M_MEAN_TOTAL, M_MEAN_SAVED,
    M_SUBTASK_SHARE, M_TRIAL_SHARE, M_ACCURACY, M_MEAN_REWARD, M_COUNT
};

int oracle_batch_metrics(const oracle_row_t *rows, const uint8_t *correct, const double *reward, int64_t n,
                         double *m)
{
    int64_t valid = 0, trig = 0, corr = 0, trunc = 0, mism = 0;
    int64_t st = 0, sl = 0, ss = 0, sr = 0;
    double rsum = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        valid += (rows[i].flags & F_VALID) != 0;
        trig += (rows[i].flags & F_TRIGGERED) != 0;
        trunc += (rows[i].flags & F_TRUNCATED) != 0;
        mism += (rows[i].flags & F_COUNT_MISMATCH) != 0;
        corr += correct[i] != 0;
        st += rows[i].total;
        sl += rows[i].latency;
        ss += rows[i].n_subtask;
        sr += rows[i].n_trial;
        rsum = rsum + reward[i];
    }
    for (int k = 0; k < M_COUNT; ++k) m[k] = 0.0;
    m[M_ROWS] = (double)n;
    m[M_VALID] = (double)valid;
    m[M_TRIGGERED] = (double)trig;
    m[M_CORRECT] = (double)corr;
    m[M_TRUNCATED] = (double)trunc;
    m[M_MISMATCH] = (double)mism;
    m[M_SUM_TOTAL] = (double)st;
    m[M_SUM_LATENCY] = (double)sl;
    m[M_SUM_SUBTASK] = (double)ss;
    m[M_SUM_TRIAL] = (double)sr;
    if (n > 0) {
        m[M_TRIGGER_RATIO] = (double)trig / (double)n;
        m[M_MEAN_LATENCY] = (double)sl / (double)n;
        m[M_MEAN_TOTAL] = (double)st / (double)n;
        m[M_MEAN_SAVED] = (double)(st - sl) / (double)n;
        m[M_ACCURACY] = (double)corr / (double)n;
        m[M_MEAN_REWARD] = rsum / (double)n;
    }
    if (sl > 0) m[M_ACCELERATION] = (double)st / (double)sl;
    if (st > 0) {
        m[M_SUBTASK_SHARE] = (double)ss / (double)st;
        m[M_TRIAL_SHARE] = (double)sr / (double)st;
    }
    return 0;
}
