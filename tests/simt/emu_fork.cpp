/*
 * Driver of the CPU SIMT emulation build of fork/join packing.
 *
 * TEST INFRASTRUCTURE.  Compiled together with the library's own
 * csrc/parason.hip (the handle) and csrc/fork.hip for the host
 * (tests/simt/hip/hip_runtime.h stands in for the HIP runtime), under
 * AddressSanitizer and UndefinedBehaviorSanitizer.  Runs one fork or join
 * through the C-ABI as a caller would: a first call with no output capacity
 * returns the totals, a second with outputs of exactly that size writes them.
 * Every workspace and output buffer is sized exactly and filled with a byte
 * pattern first, so reliance on their contents or access past their ends
 * fails.
 *
 * Input (little endian): int32 mode (0 fork, 1 join), int32 tag_ids[12],
 * uint32 cfg_flags, uint32 call_flags, int32 cus, int64 n, int64 n_tok, then
 * int32 tokens[n_tok], int64 starts[n], int32 lengths[n]; for a join also
 * int64 n_workers, int64 n_wtok, int64 worker_off[n + 1], int32
 * wtokens[n_wtok], int64 wstarts[n_workers], int32 wlengths[n_workers].
 * Output: int32 status of the sizing call and of the writing call; fork:
 * int64 totals[3], uint32 row_status[n], int64 worker_off[n + 1], then for W
 * workers and T context tokens int64 ctx_starts[W], int32 ctx_lengths[W],
 * ctx_row[W], ctx_entry[W], ctx_kind[W], ctx_tokens[T]; join: int64
 * totals[2], uint32 row_status[n], int32 lengths[n], int64 starts[n + 1],
 * int32 tokens[totals[0]].
 */
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include <hip/hip_runtime.h>

#include "parason.h"

static void rd(FILE *f, void *p, size_t n)
{
    if (n && fread(p, 1, n, f) != n) {
        fprintf(stderr, "short read\n");
        exit(2);
    }
}

/* n elements of T in a buffer of exactly that size (at least one byte),
 * filled with a pattern; freed by the caller. */
template <class T>
static T *pattern(int64_t n)
{
    const size_t b = (size_t)(n > 0 ? n : 0) * sizeof(T);
    void *p = nullptr;
    if (posix_memalign(&p, 256, b ? b : 1) != 0) exit(2);
    memset(p, 0xA5, b ? b : 1);
    return (T *)p;
}

static void wr(FILE *o, const void *p, size_t n)
{
    if (n) fwrite(p, 1, n, o);
}

int main(int argc, char **argv)
{
    if (argc != 3) {
        fprintf(stderr, "usage: %s in out\n", argv[0]);
        return 2;
    }
    FILE *f = fopen(argv[1], "rb");
    if (!f) return 2;
    int32_t mode, tags[12], cus;
    uint32_t cfg_flags, call_flags;
    int64_t n, n_tok;
    rd(f, &mode, 4);
    rd(f, tags, sizeof tags);
    rd(f, &cfg_flags, 4);
    rd(f, &call_flags, 4);
    rd(f, &cus, 4);
    rd(f, &n, 8);
    rd(f, &n_tok, 8);
    int32_t *tokens = pattern<int32_t>(n_tok);
    int64_t *starts = pattern<int64_t>(n);
    int32_t *lengths = pattern<int32_t>(n);
    rd(f, tokens, (size_t)n_tok * 4);
    rd(f, starts, (size_t)n * 8);
    rd(f, lengths, (size_t)n * 4);
    int64_t n_workers = 0, n_wtok = 0;
    int64_t *worker_off = nullptr, *wstarts = nullptr;
    int32_t *wtokens = nullptr, *wlengths = nullptr;
    if (mode == 1) {
        rd(f, &n_workers, 8);
        rd(f, &n_wtok, 8);
        worker_off = pattern<int64_t>(n + 1);
        wtokens = pattern<int32_t>(n_wtok);
        wstarts = pattern<int64_t>(n_workers);
        wlengths = pattern<int32_t>(n_workers);
        rd(f, worker_off, (size_t)(n + 1) * 8);
        rd(f, wtokens, (size_t)n_wtok * 4);
        rd(f, wstarts, (size_t)n_workers * 8);
        rd(f, wlengths, (size_t)n_workers * 4);
    }
    fclose(f);
    simt::emulated_cus() = cus;

    parason_config cfg;
    memset(&cfg, 0, sizeof cfg);
    memcpy(cfg.tag_ids, tags, sizeof tags);
    cfg.group_size = 1;
    cfg.flags = cfg_flags;
    parason_handle *h = nullptr;
    int rc0 = parason_create(&cfg, &h), rc1 = rc0;
    FILE *o = fopen(argv[2], "wb");
    if (!o) return 2;
    if (rc0 == PARASON_OK && mode == 0) {
        size_t wsb = 0;
        rc0 = parason_fork_workspace_size(n, &wsb);
        int64_t totals[3] = {-1, -1, -1};
        uint32_t *status = pattern<uint32_t>(n);
        int64_t *woff = pattern<int64_t>(n + 1);
        int64_t W = 0, T = 0;
        parason_fork_outputs out;
        memset(&out, 0, sizeof out);
        out.row_status = status;
        out.worker_off = woff;
        out.totals = totals;
        if (rc0 == PARASON_OK) {
            void *ws = pattern<char>((int64_t)wsb);
            rc0 = parason_fork(h, tokens, starts, lengths, n, call_flags, &out, ws, wsb, nullptr);
            W = totals[0];
            T = totals[1];
            free(ws);
        }
        int64_t *cst = pattern<int64_t>(W);
        int32_t *cln = pattern<int32_t>(W), *crow = pattern<int32_t>(W), *cent = pattern<int32_t>(W),
                *ckind = pattern<int32_t>(W), *ctok = pattern<int32_t>(T);
        if (rc0 == PARASON_OK) {
            void *ws = pattern<char>((int64_t)wsb);
            out.max_workers = W;
            out.ctx_capacity = T;
            out.ctx_starts = W ? cst : nullptr;
            out.ctx_lengths = W ? cln : nullptr;
            out.ctx_row = W ? crow : nullptr;
            out.ctx_entry = W ? cent : nullptr;
            out.ctx_kind = W ? ckind : nullptr;
            out.ctx_tokens = T ? ctok : nullptr;
            rc1 = parason_fork(h, tokens, starts, lengths, n, call_flags, &out, ws, wsb, nullptr);
            free(ws);
        }
        wr(o, &rc0, 4);
        wr(o, &rc1, 4);
        wr(o, totals, sizeof totals);
        wr(o, status, (size_t)n * 4);
        wr(o, woff, (size_t)(n + 1) * 8);
        wr(o, cst, (size_t)W * 8);
        wr(o, cln, (size_t)W * 4);
        wr(o, crow, (size_t)W * 4);
        wr(o, cent, (size_t)W * 4);
        wr(o, ckind, (size_t)W * 4);
        wr(o, ctok, (size_t)T * 4);
        for (void *p : {(void *)status, (void *)woff, (void *)cst, (void *)cln, (void *)crow, (void *)cent,
                        (void *)ckind, (void *)ctok})
            free(p);
    } else if (rc0 == PARASON_OK) {
        size_t wsb = 0;
        rc0 = parason_join_workspace_size(n, &wsb);
        int64_t totals[2] = {-1, -1};
        uint32_t *status = pattern<uint32_t>(n);
        int32_t *olen = pattern<int32_t>(n);
        int64_t *ost = pattern<int64_t>(n + 1);
        int64_t T = 0;
        parason_join_outputs out;
        memset(&out, 0, sizeof out);
        out.row_status = status;
        out.lengths = olen;
        out.starts = ost;
        out.totals = totals;
        if (rc0 == PARASON_OK) {
            void *ws = pattern<char>((int64_t)wsb);
            rc0 = parason_join(h, tokens, starts, lengths, n, worker_off, wtokens, wstarts, wlengths, n_workers,
                               call_flags, &out, ws, wsb, nullptr);
            T = totals[0];
            free(ws);
        }
        int32_t *otok = pattern<int32_t>(T);
        if (rc0 == PARASON_OK) {
            void *ws = pattern<char>((int64_t)wsb);
            out.capacity = T;
            out.tokens = T ? otok : nullptr;
            rc1 = parason_join(h, tokens, starts, lengths, n, worker_off, wtokens, wstarts, wlengths, n_workers,
                               call_flags, &out, ws, wsb, nullptr);
            free(ws);
        }
        wr(o, &rc0, 4);
        wr(o, &rc1, 4);
        wr(o, totals, sizeof totals);
        wr(o, status, (size_t)n * 4);
        wr(o, olen, (size_t)n * 4);
        wr(o, ost, (size_t)(n + 1) * 8);
        wr(o, otok, (size_t)T * 4);
        for (void *p : {(void *)status, (void *)olen, (void *)ost, (void *)otok}) free(p);
    } else {
        wr(o, &rc0, 4);
        wr(o, &rc1, 4);
    }
    fclose(o);
    if (h) parason_destroy(h);
    for (void *p : {(void *)tokens, (void *)starts, (void *)lengths, (void *)worker_off, (void *)wtokens,
                    (void *)wstarts, (void *)wlengths})
        free(p);
    fprintf(stderr, "simt: %llu wave operations\n", (unsigned long long)simt::st().collectives);
    return 0;
}
