/*
 * parason.h -- C-ABI of the MI355X (gfx950) hot path of Parason:
 * parallel-trajectory accounting and the Parallelism-Aware GRPO reward.
 *
 * For every generated token stream (a rollout) of a batch grouped G rollouts
 * per prompt, the library
 *   1. checks the stream against the grammar of the figure "Context-Free
 *      Grammar for Parason" (Sec. 3.2),
 *   2. computes its total tokens L_total and its model latency T_i, the length
 *      of the longest generation path, where each <Parallel> block contributes
 *      its longest branch (Sec. 4, "Evaluation"; T_i and L_latency in Sec. 3.3),
 *   3. counts the tokens placed in Subtask and in Trial branches (R_subtask and
 *      R_trial of Sec. 3.3),
 *   4. normalises latency and the two ratios within each group of G and
 *      evaluates the reward of Definition 3.1 ("Parallel RL Reward", Sec. 3.3)
 *      with the shaping function f the identity.
 *
 * Readings of points the paper leaves open (all implemented identically by the
 * test oracle):
 *   - each tag is one reserved token id; every other id is Text;
 *   - every token costs 1 on the path that emits it, tags included;
 *   - <Parallel> and its outline are on the enclosing path:
 *       lat(P) = 1 + |<Outlines> ... </Outlines>| + max_k lat(thread k) + 1,
 *       lat(thread) = 2 + lat(its body);
 *   - a token is a Subtask (Trial) token when its innermost enclosing <Thread>
 *     pairs with a Subtask (Trial) entry; thread k pairs with entry k; surplus
 *     threads are untyped and the row gets PARASON_FLAG_COUNT_MISMATCH;
 *   - free Text may follow </think> and counts sequentially; nothing may
 *     precede <think>;
 *   - strict by default: no Text between the structural tags of a parallel
 *     region, as the grammar is printed (PARASON_CFG_LENIENT_GAPS relaxes it);
 *   - an invalid or truncated stream is sequential (latency = total, no branch
 *     tokens, no blocks, depth 0); first_error_pos is the length of its longest
 *     prefix that is a prefix of some valid stream;
 *   - mu and sigma are over the G rollouts of one prompt, population form;
 *     z = 0 when all G values are equal (decided exactly) or sigma is 0;
 *   - the reward is evaluated in IEEE double precision in a fixed order with no
 *     fused multiply-add, then stored as float.
 *
 * Threading: a handle is immutable after parason_create; parason_run may be
 * called concurrently on different streams with different workspaces.
 * No function throws; every error is a negative status.
 */
#ifndef PARASON_H
#define PARASON_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------- */
#define PARASON_OK 0
#define PARASON_ERR_NULL (-1)      /* a required pointer argument is NULL */
#define PARASON_ERR_SIZE (-2)      /* negative or too large n_traj / total_tokens */
#define PARASON_ERR_GROUP (-3)     /* group_size < 1 or n_traj % group_size != 0 */
#define PARASON_ERR_WORKSPACE (-4) /* workspace smaller than parason_workspace_size */
#define PARASON_ERR_TAGS (-5)      /* a tag id is negative or two tag ids are equal */
#define PARASON_ERR_PARAM (-6)     /* a reward parameter is not finite */
#define PARASON_ERR_ALIGN (-7)     /* tokens not 4-byte aligned or workspace not 256-byte aligned */
#define PARASON_ERR_HIP (-8)       /* a HIP call or kernel launch failed */
#define PARASON_ERR_DEVICE (-9)    /* the current device is not gfx950 or cannot be queried (checked by
                                      every call that launches, before its first launch) */
#define PARASON_ERR_SCRATCH (-10)  /* parason_run_noalloc: the batch needs more than its static scratch */

/* ---- per-row flag bits (parason_outputs.flags) ------------------------- */
#define PARASON_FLAG_VALID (1u << 0)          /* the stream is in the language */
#define PARASON_FLAG_TRUNCATED (1u << 1)      /* invalid only because it ends early */
#define PARASON_FLAG_COUNT_MISMATCH (1u << 2) /* valid; some block has #threads != #entries */
#define PARASON_FLAG_TRIGGERED (1u << 3)      /* valid and holds >= 1 <Parallel> block (Table 4) */
/* The row was not evaluated; its counts are 0 (total is its length, 0 for a
 * bad row, and saved is 0), its float outputs (and those of its whole group)
 * are NaN: */
#define PARASON_FLAG_DEPTH_LIMIT (1u << 8)    /* nesting or entry count beyond the slow path's store */
#define PARASON_FLAG_WS_OVERFLOW (1u << 9)    /* the rows need more workspace than was passed */
#define PARASON_FLAG_BAD_ROW (1u << 10)       /* negative start or length */

/* ---- configuration flag bits (parason_config.flags) -------------------- */
/* An invalid stream keeps the caller's correctness bit (default: an invalid
 * stream counts as incorrect, reward -1). */
#define PARASON_CFG_INVALID_KEEPS_CORRECTNESS (1u << 0)
/* mu and sigma over the whole batch instead of each group of G rows (the
 * alternative reading of the normalisation population).  A batch holding any
 * row that was not evaluated gets NaN rewards throughout. */
#define PARASON_CFG_BATCH_STATS (1u << 1)
/* The token scan tests each token against the twelve tag ids one by one even
 * when a hash separates them (tag ids that are not twelve consecutive values
 * are otherwise looked up in a 64-slot table).  Same results, slower; there
 * for tag sets no hash of the scan separates, and for testing that path. */
#define PARASON_CFG_TAG_COMPARE (1u << 2)
/* Runs of Text may stand between the structural tags of a parallel region:
 * after <Parallel>, <Outlines>, each outline entry, </Outlines> and each
 * </Thread> of the region (the line breaks of Figure 3, which the grammar of
 * Figure 4 as printed does not allow).  Their tokens are decoded by the
 * enclosing path, like the outline: they add to the region's latency and count
 * toward the enclosing branch type.  Without the flag such Text is an error at
 * its first token.  Honoured by parason_run, parason_decode_step (Text becomes
 * allowed in those positions) and parason_fork (the outline check). */
#define PARASON_CFG_LENIENT_GAPS (1u << 3)

/* ---- batch metrics (parason_outputs.metrics, doubles) ------------------- */
/* As the paper reports them: trigger ratio = share of rows with >= 1
 * <Parallel> block (Table 4); acceleration = total tokens / longest-path
 * tokens (Tables 4 and 5); mean latency tokens (Tables 2 and 4); saved tokens
 * = generated - latency (Table 5).  Counts are exact; sums of token counts
 * are exact below 2^53. */
#define PARASON_METRIC_ROWS 0
#define PARASON_METRIC_VALID 1
#define PARASON_METRIC_TRIGGERED 2
#define PARASON_METRIC_CORRECT 3
#define PARASON_METRIC_TRUNCATED 4
#define PARASON_METRIC_COUNT_MISMATCH 5
#define PARASON_METRIC_SUM_TOTAL 6
#define PARASON_METRIC_SUM_LATENCY 7
#define PARASON_METRIC_SUM_SUBTASK 8
#define PARASON_METRIC_SUM_TRIAL 9
#define PARASON_METRIC_TRIGGER_RATIO 10
#define PARASON_METRIC_ACCELERATION 11
#define PARASON_METRIC_MEAN_LATENCY 12
#define PARASON_METRIC_MEAN_TOTAL 13
#define PARASON_METRIC_MEAN_SAVED 14
#define PARASON_METRIC_SUBTASK_SHARE 15
#define PARASON_METRIC_TRIAL_SHARE 16
#define PARASON_METRIC_ACCURACY 17
#define PARASON_METRIC_MEAN_REWARD 18
#define PARASON_METRIC_COUNT 19

/* Maximum nesting depth and number of outline entries of open blocks that the
 * library evaluates; a row beyond either is flagged PARASON_FLAG_DEPTH_LIMIT.
 * (A row needs at least 6 tokens per nesting level.) */
#define PARASON_MAX_DEPTH (1 << 20)
#define PARASON_MAX_OPEN_ENTRIES (1 << 24)

typedef struct parason_config {
    /* Token ids of the tags, in this order:
     *   <think> </think> <Parallel> </Parallel> <Outlines> </Outlines>
     *   <Subtask> </Subtask> <Trial> </Trial> <Thread> </Thread>
     * (the terminals of the grammar, Sec. 3.2).  Distinct and >= 0. */
    int32_t tag_ids[12];
    /* G: rollouts per prompt; rows [g*G, (g+1)*G) form group g (8 in Sec. 4). */
    int32_t group_size;
    /* Reward coefficients of Definition 3.1: alpha (latency penalty),
     * beta_subtask, beta_trial (parallelism incentives), rho and rho_clip
     * (clipped acceleration reward).  Must be finite. */
    double alpha, beta_subtask, beta_trial, rho, rho_clip;
    uint32_t flags; /* PARASON_CFG_* */
} parason_config;

/* Caller-owned device arrays of n_traj elements each.  All are required except
 * r_subtask, r_trial, eta, metrics, accel and saved, which may be NULL. */
typedef struct parason_outputs {
    int32_t *total;           /* L_total = length of the row */
    int32_t *latency;         /* T_i = L_latency (longest generation path) */
    int32_t *n_subtask;       /* tokens in Subtask branches */
    int32_t *n_trial;         /* tokens in Trial branches */
    int32_t *n_blocks;        /* number of <Parallel> blocks */
    int32_t *max_depth;       /* deepest <Parallel> nesting (1 = top level) */
    int32_t *first_error_pos; /* -1 if valid, else longest viable prefix length */
    uint32_t *flags;          /* PARASON_FLAG_* */
    float *reward;            /* R_i of Definition 3.1 */
    float *r_subtask;         /* optional: n_subtask / total (0 if total == 0) */
    float *r_trial;           /* optional: n_trial / total */
    float *eta;               /* optional: eta(s) = 1 - latency / total */
    double *metrics;          /* optional: PARASON_METRIC_COUNT batch metrics (mean reward
                                 over the stored float rewards) */
    float *accel;             /* optional: total / latency, the acceleration ratio of
                                 Tables 4 and 5 (1 if total == 0) */
    int32_t *saved;           /* optional: total - latency, the saved tokens of Table 5 */
} parason_outputs;

typedef struct parason_handle parason_handle;

/* Validate *cfg and create a handle (host memory only; no HIP call, so a
 * handle can be made and workspaces sized without a GPU).  On success *out
 * receives the handle.  Every call that launches kernels (parason_run and the
 * other steps below) first checks that the current HIP device is a gfx950 GPU
 * and returns PARASON_ERR_DEVICE, before any launch, when it is not. */
int parason_create(const parason_config *cfg, parason_handle **out);

/* Bytes of device workspace parason_run needs for n_traj rows whose lengths
 * add up to at most total_tokens: about 1.4 % of the token bytes for large
 * batches.  Batches beyond about 3.6e11 tokens (far more than one GPU holds)
 * return PARASON_ERR_SIZE. */
int parason_workspace_size(const parason_handle *h, int64_t n_traj, int64_t total_tokens, size_t *bytes);

/* Evaluate a batch, asynchronously on `stream` (a hipStream_t; NULL is the
 * default stream).  Device pointers:
 *   tokens   int32 token ids; row i is tokens[starts[i] .. starts[i]+lengths[i]).
 *            Rows may be in any order, may leave gaps (a padded [B, Lmax]
 *            layout is starts[i] = i*Lmax) and may overlap.  4-byte aligned.
 *   starts   int64[n_traj], element offsets into tokens
 *   lengths  int32[n_traj]
 *   correct  uint8[n_traj], nonzero = the final answer is correct
 *   out      per-row outputs (the struct itself is host memory)
 *   workspace, workspace_bytes: scratch from the caller, 256-byte aligned, at
 *            least parason_workspace_size(h, n_traj, sum of lengths) bytes; its
 *            contents need no initialisation and are meaningless afterwards.
 * Host-side argument errors return a negative status before any launch.
 * Device-side problems (bad rows, workspace too small for the actual lengths)
 * are reported per row in out->flags.  Nothing is synchronised inside. */
int parason_run(const parason_handle *h, const int32_t *tokens, const int64_t *starts, const int32_t *lengths,
                const uint8_t *correct, int64_t n_traj, const parason_outputs *out, void *workspace,
                size_t workspace_bytes, void *stream);

/* parason_run, plus hipEventRecord of scan_events[0] on `stream` just before
 * the token-scan kernel (the one whose HBM traffic bounds the path) and of
 * scan_events[1] just after it.  scan_events holds two hipEvent_t created by
 * the caller; a NULL array records nothing.  For measurement. */
int parason_run_timed(const parason_handle *h, const int32_t *tokens, const int64_t *starts, const int32_t *lengths,
                      const uint8_t *correct, int64_t n_traj, const parason_outputs *out, void *workspace,
                      size_t workspace_bytes, void *stream, void *const *scan_events);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): parason_run
 * with no workspace argument.  Its scratch is one static device array of
 * PARASON_NOALLOC_SCRATCH_BYTES per GPU the library runs on, held until the
 * process ends; nothing is allocated by this call, and nothing is freed.
 *   total_tokens: an upper bound of the sum of the row lengths, known on the
 *            host; a batch whose parason_workspace_size(h, n_traj,
 *            total_tokens) exceeds the scratch returns PARASON_ERR_SCRATCH
 *            before any launch (lengths beyond the bound are reported per row
 *            as PARASON_FLAG_WS_OVERFLOW, as for parason_run).
 * Every other argument and every result is as for parason_run.  All calls on
 * one GPU share that GPU's scratch, which keeps the last call's contents (no
 * call relies on them): calls that overlap on one GPU (on two streams, or from
 * two threads without ordering between them) race and give wrong results.
 * Serialise them, e.g. on one stream. */
#define PARASON_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)
int parason_run_noalloc(const parason_handle *h, const int32_t *tokens, const int64_t *starts, const int32_t *lengths,
                        const uint8_t *correct, int64_t n_traj, int64_t total_tokens, const parason_outputs *out,
                        void *stream);

void parason_destroy(parason_handle *h);

/* Measurement aid, not an operation of the paper: a plain streaming read of
 * data[0 .. bytes) with the token scan's loads, grid and work distribution
 * (an equal share per wave, then the rest in chunks through a counter) and
 * nothing else, the ceiling that a read of every token once reaches on this
 * GPU (the scan's roofline is reported against it and against the HBM peak).
 * data: device memory, 16-byte aligned, bytes a multiple of 4.  sink: device
 * uint32[sink_len], sink_len >= 1; each wave stores a checksum of what it read
 * to sink[wave % sink_len].  Asynchronous on `stream`; host-side argument
 * errors return a negative status before any launch.  The chunk counter is a
 * static variable of the library, one per GPU, cleared by a launch of its own
 * before the read: probes that overlap on one GPU read only part of their
 * data (never outside it).  Serialise them. */
int parason_read_probe(const void *data, size_t bytes, uint32_t *sink, int64_t sink_len, void *stream);

/* ---- policy-gradient step ------------------------------------------------
 * The update that consumes the rewards in PA-GRPO (Sec. 4 "Training
 * Framework": GRPO with 8 rollouts per prompt, lower clip ratio 0.2, upper
 * clip ratio 0.28).  The paper does not write the objective out; this is the
 * standard one:
 *   A_i   = (R_i - mean_g R) / std_g R over the G rollouts of a prompt
 *           (population std; A_i = 0 when all G rewards are equal);
 *   rho_t = exp(logp_t - logp_old_t);
 *   J     = (1 / N) sum_t min(rho_t A, clip(rho_t, 1 - eps_low, 1 + eps_high) A)
 *           over all N generated tokens of the batch (token-level mean);
 *   loss  = -J, and grad_t = d loss / d logp_t.
 * The clip decision compares the float log-ratio d = logp - logp_old with the
 * float thresholds ln(1 - eps_low) and ln(1 + eps_high) (rho > 1 + eps_high
 * exactly when d > ln(1 + eps_high)); values are float, the sum is double. */
#define PARASON_PG_STAT_LOSS 0
#define PARASON_PG_STAT_TOKENS 1
#define PARASON_PG_STAT_CLIP_HIGH 2 /* tokens with A > 0 held at 1 + eps_high */
#define PARASON_PG_STAT_CLIP_LOW 3  /* tokens with A < 0 held at 1 - eps_low */
#define PARASON_PG_STAT_COUNT 4

typedef struct parason_pg_config {
    int32_t group_size;         /* G, as for parason_run */
    double clip_low, clip_high; /* eps_low (0.2), eps_high (0.28); 0 <= eps_low < 1, eps_high >= 0 */
} parason_pg_config;

/* Bytes of device workspace parason_pg_run needs for n_traj rows. */
int parason_pg_workspace_size(int64_t n_traj, size_t *bytes);

/* One policy-gradient step, asynchronously on `stream`.  Device pointers:
 *   reward     float[n_traj] (the rewards of parason_run)
 *   logp, logp_old  float log-probabilities of the generated tokens; row i is
 *              [starts[i], starts[i] + lengths[i]) as for parason_run; the
 *              three float arrays must share their position modulo 16 bytes
 *   advantage  float[n_traj] out: A_i
 *   grad       float out, same layout as logp: d loss / d logp on every row
 *              position (other positions are not written)
 *   stats      double[PARASON_PG_STAT_COUNT] out
 * Returns a negative status on host-side argument errors, before any launch. */
int parason_pg_run(const parason_pg_config *cfg, const float *reward, const float *logp, const float *logp_old,
                   const int64_t *starts, const int32_t *lengths, int64_t n_traj, float *advantage, float *grad,
                   double *stats, void *workspace, size_t workspace_bytes, void *stream);

/* ---- grammar-constrained decode step ------------------------------------
 * During rollouts the tags are kept valid by grammar-constrained decoding
 * (Sec. 3.4) over the grammar of Figure 4 (Sec. 3.2).  A token may follow a
 * prefix when prefix + token is still a prefix of some valid stream; the
 * end-of-sequence token may follow a prefix that is itself a complete stream
 * (after </think>).  Text is every id that is neither a tag nor eos_id.
 *
 * Each sequence carries a 16-byte state in device memory.  One step
 *   1. advances the state by the token sampled last (tokens[i]; NULL, or a
 *      negative entry, advances nothing -- the first step of a rollout), then
 *   2. writes -inf into every logit of row i that the new state forbids.
 * Allowed logits are left untouched.  A sampled token that was not allowed
 * sets PARASON_DECODE_ERROR; a sampled eos_id that was allowed sets
 * PARASON_DECODE_DONE.  A state carrying either flag no longer changes and its
 * rows are not masked.  Thread and outline-entry counts are not forced to
 * match (as for parason_run, a mismatch is flagged, not invalid). */
#define PARASON_DECODE_ERROR (1u << 0)
#define PARASON_DECODE_DONE (1u << 1)

#define PARASON_DTYPE_F32 0
#define PARASON_DTYPE_BF16 1
#define PARASON_DTYPE_F16 2

typedef struct parason_decode_state {
    int32_t state;  /* position in the grammar (opaque) */
    int32_t depth;  /* open <Parallel> blocks */
    int32_t entry;  /* open outline entry (opaque) */
    uint32_t flags; /* PARASON_DECODE_* */
} parason_decode_state;

/* Set states[0 .. batch) to the start of a stream (device memory, 16-byte
 * aligned), asynchronously on `stream`. */
int parason_decode_init(parason_decode_state *states, int64_t batch, void *stream);

/* One decode step for `batch` sequences, asynchronously on `stream`, with the
 * tag ids of h.  Device pointers:
 *   states   parason_decode_state[batch], updated in place
 *   tokens   int32[batch] sampled last, or NULL
 *   logits   row i at logits + i * row_stride elements, vocab elements each,
 *            of type `dtype` (PARASON_DTYPE_*), aligned to the element size
 * eos_id: the end-of-sequence id (< vocab, not a tag), or -1 for none.  Every
 * tag id must be < vocab and row_stride >= vocab.  Host-side argument errors
 * return a negative status before any launch. */
int parason_decode_step(const parason_handle *h, parason_decode_state *states, const int32_t *tokens, int64_t batch,
                        void *logits, int64_t vocab, int64_t row_stride, int32_t dtype, int32_t eos_id, void *stream);

/* ---- fork/join packing for tool-call execution ---------------------------
 * At inference the runtime decodes a trajectory until the outline of a
 * <Parallel> region is complete, dispatches every <Subtask> / <Trial> entry as
 * an independent worker and returns the workers' <Thread> outputs to the main
 * trajectory (Sec. 3.4 "Inference"; format of Figure 4, Sec. 3.2).  These two
 * calls are that data movement on token ids (KV-cache handling is the
 * engine's).
 *
 * fork: row i must end with </Outlines>; its outline starts at the last
 * <Outlines> before that, which must directly follow <Parallel>, and must hold
 * one or more entries "<Subtask> text+ </Subtask>" or "<Trial> text+ </Trial>"
 * back to back.  Worker k of row i gets the context
 *     row i ++ <Thread> ++ (the text of entry k, with PARASON_FORK_SEED_ENTRY)
 * Workers are numbered row by row, entry by entry.
 *
 * join: worker w of row i hands back its whole sequence (its context followed
 * by what it generated, ending with its </Thread>).  Joined row i is
 *     row i ++ seq_w[len(row i):] for the row's workers in order
 *           ++ </Parallel> (with PARASON_JOIN_CLOSE_PARALLEL)
 * i.e. each worker's <Thread> ... </Thread> span as the worker saw it; with
 * PARASON_JOIN_APPEND_ONLY row i itself is left out of the output. */
#define PARASON_FORK_SEED_ENTRY (1u << 0)
#define PARASON_JOIN_CLOSE_PARALLEL (1u << 0)
#define PARASON_JOIN_APPEND_ONLY (1u << 1)

/* per-row status bits (row_status) */
#define PARASON_PACK_NO_OUTLINE_END (1u << 0) /* fork: the row does not end with </Outlines> */
#define PARASON_PACK_NO_OUTLINE (1u << 1)     /* fork: no <Outlines> before it, or not after <Parallel> */
#define PARASON_PACK_BAD_ENTRY (1u << 2)      /* fork: the outline is not a run of well-formed entries */
#define PARASON_PACK_BAD_THREAD (1u << 3)     /* join: a worker sequence is not <Thread> ... </Thread>
                                                 after the row (copied as it is) */
#define PARASON_PACK_TOO_LONG (1u << 4)       /* an output row would exceed INT32_MAX tokens (not written) */
#define PARASON_PACK_BAD_ROW (1u << 5)        /* negative start or length, or (join) worker_off out of
                                                 order or beyond n_workers (not written) */

typedef struct parason_fork_outputs {
    /* capacities: if the batch needs more, only worker_off, row_status and
     * totals are written (totals[2] = 1); allocate totals[0] workers and
     * totals[1] tokens and call again */
    int64_t max_workers;
    int64_t ctx_capacity;     /* int32 tokens */
    int32_t *ctx_tokens;      /* [ctx_capacity] contexts, packed in worker order */
    int64_t *ctx_starts;      /* [max_workers] */
    int32_t *ctx_lengths;     /* [max_workers] */
    int32_t *ctx_row;         /* [max_workers] the row a worker belongs to */
    int32_t *ctx_entry;       /* [max_workers] its entry index in the outline */
    int32_t *ctx_kind;        /* [max_workers] 1 = Subtask, 2 = Trial */
    int64_t *worker_off;      /* [n_rows + 1] first worker of each row; [n_rows] = workers */
    uint32_t *row_status;     /* [n_rows] PARASON_PACK_* (0: dispatched) */
    int64_t *totals;          /* [3] workers, context tokens, over capacity (0/1) */
} parason_fork_outputs;

typedef struct parason_join_outputs {
    int64_t capacity;         /* int32 tokens of out tokens; see parason_fork_outputs */
    int32_t *tokens;          /* [capacity] joined rows, packed */
    int64_t *starts;          /* [n_rows + 1]; [n_rows] = total tokens */
    int32_t *lengths;         /* [n_rows] */
    uint32_t *row_status;     /* [n_rows] PARASON_PACK_* */
    int64_t *totals;          /* [2] tokens, over capacity (0/1) */
} parason_join_outputs;

/* Bytes of device workspace parason_fork / parason_join need for n_rows rows. */
int parason_fork_workspace_size(int64_t n_rows, size_t *bytes);
int parason_join_workspace_size(int64_t n_rows, size_t *bytes);

/* Fork a batch of rows (device pointers as for parason_run; the output
 * struct itself is host memory, its arrays device memory), asynchronously on
 * `stream`.  The tag ids are those of h.  Host-side argument errors return a
 * negative status before any launch; per-row problems go to row_status. */
int parason_fork(const parason_handle *h, const int32_t *tokens, const int64_t *starts, const int32_t *lengths,
                 int64_t n_rows, uint32_t flags, const parason_fork_outputs *out, void *workspace,
                 size_t workspace_bytes, void *stream);

/* Join: rows as for parason_fork, worker_off[n_rows + 1] as parason_fork wrote
 * it, and the n_workers worker sequences (wtokens, wstarts, wlengths), each
 * beginning with its row (not checked) and continuing from its context. */
int parason_join(const parason_handle *h, const int32_t *tokens, const int64_t *starts, const int32_t *lengths,
                 int64_t n_rows, const int64_t *worker_off, const int32_t *wtokens, const int64_t *wstarts,
                 const int32_t *wlengths, int64_t n_workers, uint32_t flags, const parason_join_outputs *out,
                 void *workspace, size_t workspace_bytes, void *stream);

/* Static description of a status code. */
const char *parason_strerror(int status);

#ifdef __cplusplus
}
#endif
#endif /* PARASON_H */
