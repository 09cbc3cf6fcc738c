/*
 * synth_host.cpp -- host mirror of the seeded synthetic trajectory generator.
 * Built with g++ and -D__host__= -D__device__= so the portable core in
 * synth_core.h compiles as plain C++; rows match the device generator bit for
 * bit.  Input generation only.
 */
#include <stdint.h>
#include "synth_core.h"

extern "C" int synth_rows_host(const synth_params *P, uint64_t row0, int64_t n, int32_t *lengths, uint8_t *correct)
{
    if (!P || n < 0) return -1;
    for (int64_t i = 0; i < n; ++i) {
        sy_rowinfo ri;
        sy_row_info(P, row0 + (uint64_t)i, &ri);
        lengths[i] = (int32_t)ri.len;
        correct[i] = ri.correct;
    }
    return 0;
}

/* Tokens of one row whose first token sits at flat index flat0 of the batch.
 * Writes min(len, cap) tokens; returns the row length. */
extern "C" int64_t synth_row_tokens_host(const synth_params *P, uint64_t row, uint64_t flat0, int32_t *out, int64_t cap)
{
    sy_rowinfo ri;
    sy_row_info(P, row, &ri);
    if (ri.len > cap) return -1;
    if (ri.target < 2) {
        if (ri.len >= 1) out[0] = P->tag_ids[SY_THINK];
        return ri.len;
    }
    sy_row_emit(P, row, &ri, out, flat0, 1);
    return ri.len;
}

/* logp_old and logp for flat positions [p0, p0 + n). */
extern "C" int synth_logp_host(const synth_params *P, uint64_t p0, int64_t n, float *old_p, float *new_p)
{
    for (int64_t i = 0; i < n; ++i) {
        uint64_t pos = p0 + (uint64_t)i;
        float o[4], w[4];
        sy_logp4(P, pos >> 2, o, w);
        old_p[i] = o[pos & 3];
        new_p[i] = w[pos & 3];
    }
    return 0;
}
