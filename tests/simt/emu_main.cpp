/*
 * Driver of the CPU SIMT emulation build of the accounting path.
 *
 * TEST INFRASTRUCTURE.  Compiled together with the library's own
 * csrc/parason.hip for the host (tests/simt/hip/hip_runtime.h stands in for
 * the HIP runtime), under AddressSanitizer and UndefinedBehaviorSanitizer.
 * Reads one batch from a binary file, runs it through the C-ABI exactly as a
 * caller would (host memory plays the device memory), writes the per-row
 * outputs to another file.
 *
 * Input (little endian): int64 n, int64 n_tok, int64 ws_tokens (the
 * total_tokens given to parason_workspace_size), int32 tag_ids[12],
 * int32 group_size, uint32 cfg_flags, int32 cus, int32 shift, int32 noalloc,
 * double coef[5], then int32 tokens[n_tok], int64 starts[n], int32
 * lengths[n], uint8 correct[n].
 * Output: int32 total, latency, n_subtask, n_trial, n_blocks, max_depth,
 * first_error_pos, flags [n each], float reward, r_subtask, r_trial, eta,
 * accel [n each], int32 saved [n], int32 status.
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

int main(int argc, char **argv)
{
    if (argc != 3) {
        fprintf(stderr, "usage: %s in out\n", argv[0]);
        return 2;
    }
    FILE *f = fopen(argv[1], "rb");
    if (!f) return 2;
    int64_t n, n_tok, ws_tokens;
    int32_t tags[12], G, cus, shift, noalloc;
    uint32_t flags;
    double coef[5];
    rd(f, &n, 8);
    rd(f, &n_tok, 8);
    rd(f, &ws_tokens, 8);
    rd(f, tags, sizeof tags);
    rd(f, &G, 4);
    rd(f, &flags, 4);
    rd(f, &cus, 4);
    rd(f, &shift, 4);
    rd(f, &noalloc, 4);
    rd(f, coef, sizeof coef);
    /* tokens at `shift` elements past a 256-byte boundary, in an allocation
     * that ends at the 16-byte vector holding the last token (the scan reads
     * whole vectors, which never cross a page), so any other read past the
     * buffer is caught */
    char *tok_mem = nullptr;
    if (posix_memalign((void **)&tok_mem, 256, ((size_t)(n_tok + shift) * 4 + 15) / 16 * 16 + 16) != 0) return 2;
    int32_t *tokens = (int32_t *)tok_mem + shift;
    std::vector<int64_t> starts(n);
    std::vector<int32_t> lengths(n);
    std::vector<uint8_t> correct(n);
    rd(f, tokens, (size_t)n_tok * 4);
    rd(f, starts.data(), (size_t)n * 8);
    rd(f, lengths.data(), (size_t)n * 4);
    rd(f, correct.data(), (size_t)n);
    fclose(f);
    simt::emulated_cus() = cus;

    parason_config cfg;
    memcpy(cfg.tag_ids, tags, sizeof tags);
    cfg.group_size = G;
    cfg.alpha = coef[0];
    cfg.beta_subtask = coef[1];
    cfg.beta_trial = coef[2];
    cfg.rho = coef[3];
    cfg.rho_clip = coef[4];
    cfg.flags = flags;
    parason_handle *h = nullptr;
    int rc = parason_create(&cfg, &h);
    std::vector<int32_t> I[8];
    std::vector<float> F[5];
    std::vector<int32_t> saved(n > 0 ? n : 1);
    for (auto &v : I) v.assign(n > 0 ? n : 1, -77);
    for (auto &v : F) v.assign(n > 0 ? n : 1, -77.0f);
    if (rc == PARASON_OK) {
        parason_outputs out;
        memset(&out, 0, sizeof out);
        out.total = I[0].data();
        out.latency = I[1].data();
        out.n_subtask = I[2].data();
        out.n_trial = I[3].data();
        out.n_blocks = I[4].data();
        out.max_depth = I[5].data();
        out.first_error_pos = I[6].data();
        out.flags = (uint32_t *)I[7].data();
        out.reward = F[0].data();
        out.r_subtask = F[1].data();
        out.r_trial = F[2].data();
        out.eta = F[3].data();
        out.accel = F[4].data();
        out.saved = saved.data();
        if (noalloc) {
            rc = parason_run_noalloc(h, tokens, starts.data(), lengths.data(), correct.data(), n, ws_tokens, &out,
                                     nullptr);
        } else {
            size_t ws = 0;
            rc = parason_workspace_size(h, n, ws_tokens, &ws);
            if (rc == PARASON_OK) {
                /* exact size, filled with a pattern: the path must not rely on
                 * the workspace's contents or read past its end */
                void *w = nullptr;
                if (posix_memalign(&w, 256, ws ? ws : 1) != 0) return 2;
                memset(w, 0xA5, ws);
                rc = parason_run(h, tokens, starts.data(), lengths.data(), correct.data(), n, &out, w, ws, nullptr);
                free(w);
            }
        }
        parason_destroy(h);
    }
    FILE *o = fopen(argv[2], "wb");
    if (!o) return 2;
    for (auto &v : I) fwrite(v.data(), 4, (size_t)n, o);
    for (auto &v : F) fwrite(v.data(), 4, (size_t)n, o);
    fwrite(saved.data(), 4, (size_t)n, o);
    fwrite(&rc, 4, 1, o);
    fclose(o);
    free(tok_mem);
    fprintf(stderr, "simt: %llu wave operations\n", (unsigned long long)simt::st().collectives);
    return 0;
}
