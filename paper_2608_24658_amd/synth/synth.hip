/*
 * synth.hip -- device side of the seeded synthetic trajectory generator.
 * Input generation only (no accounting or reward arithmetic).  The row
 * structure code is the portable core in synth_core.h; the host mirror
 * (synth_host.cpp) compiles the same core, so rows match bit for bit.
 */
#include <hip/hip_runtime.h>
#include "synth_core.h"

__global__ void __launch_bounds__(256) synth_rows_kernel(synth_params P, uint64_t row0, int64_t n,
                                                         int32_t *lengths, uint8_t *correct)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    sy_rowinfo ri;
    sy_row_info(&P, row0 + (uint64_t)i, &ri);
    lengths[i] = (int32_t)ri.len;
    correct[i] = ri.correct;
}

/* Text ids for every position of the buffer: 4 per thread, 16-byte stores. */
__global__ void __launch_bounds__(256) synth_text_kernel(synth_params P, int32_t *tokens, int64_t n_tok)
{
    int64_t n4 = (n_tok + 3) >> 2;
    int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < n4; q += stride) {
        int32_t t[4];
        sy_text4(&P, (uint64_t)q, t);
        if (4 * q + 3 < n_tok) {
            *reinterpret_cast<int4 *>(tokens + 4 * q) = make_int4(t[0], t[1], t[2], t[3]);
        } else {
            for (int j = 0; j < 4; ++j)
                if (4 * q + j < n_tok) tokens[4 * q + j] = t[j];
        }
    }
}

/* Tags of every row, written over the Text fill. */
__global__ void __launch_bounds__(256) synth_tags_kernel(synth_params P, uint64_t row0, int64_t n,
                                                         const int64_t *starts, int32_t *tokens)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    sy_rowinfo ri;
    sy_row_info(&P, row0 + (uint64_t)i, &ri);
    sy_row_emit(&P, row0 + (uint64_t)i, &ri, tokens + starts[i], (uint64_t)starts[i], 0);
}

/* logp_old and logp for every position of two buffers of n floats. */
__global__ void __launch_bounds__(256) synth_logp_kernel(synth_params P, float *old_p, float *new_p, int64_t n)
{
    int64_t n4 = (n + 3) >> 2;
    int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < n4; q += stride) {
        float o[4], w[4];
        sy_logp4(&P, (uint64_t)q, o, w);
        if (4 * q + 3 < n) {
            *reinterpret_cast<float4 *>(old_p + 4 * q) = make_float4(o[0], o[1], o[2], o[3]);
            *reinterpret_cast<float4 *>(new_p + 4 * q) = make_float4(w[0], w[1], w[2], w[3]);
        } else {
            for (int j = 0; j < 4; ++j)
                if (4 * q + j < n) {
                    old_p[4 * q + j] = o[j];
                    new_p[4 * q + j] = w[j];
                }
        }
    }
}

static int launch_status() { return hipGetLastError() == hipSuccess ? 0 : -5; }

extern "C" int synth_rows_device(const synth_params *P, uint64_t row0, int64_t n, int32_t *lengths,
                                 uint8_t *correct, hipStream_t stream)
{
    if (!P || n < 0 || (n > 0 && (!lengths || !correct))) return -1;
    if (n == 0) return 0;
    int64_t blocks = (n + 255) / 256;
    synth_rows_kernel<<<dim3((unsigned)blocks), dim3(256), 0, stream>>>(*P, row0, n, lengths, correct);
    return launch_status();
}

extern "C" int synth_text_device(const synth_params *P, int32_t *tokens, int64_t n_tok, hipStream_t stream)
{
    if (!P || n_tok < 0 || (n_tok > 0 && !tokens)) return -1;
    if (((uintptr_t)tokens & 15u) != 0) return -2;
    if (n_tok == 0) return 0;
    int64_t n4 = (n_tok + 3) >> 2;
    int64_t blocks = (n4 + 255) / 256;
    if (blocks > 256 * 1024) blocks = 256 * 1024;
    synth_text_kernel<<<dim3((unsigned)blocks), dim3(256), 0, stream>>>(*P, tokens, n_tok);
    return launch_status();
}

extern "C" int synth_tags_device(const synth_params *P, uint64_t row0, int64_t n, const int64_t *starts,
                                 int32_t *tokens, hipStream_t stream)
{
    if (!P || n < 0 || (n > 0 && (!starts || !tokens))) return -1;
    if (n == 0) return 0;
    int64_t blocks = (n + 255) / 256;
    synth_tags_kernel<<<dim3((unsigned)blocks), dim3(256), 0, stream>>>(*P, row0, n, starts, tokens);
    return launch_status();
}

extern "C" int synth_logp_device(const synth_params *P, float *old_p, float *new_p, int64_t n, hipStream_t stream)
{
    if (!P || n < 0 || (n > 0 && (!old_p || !new_p))) return -1;
    if ((((uintptr_t)old_p | (uintptr_t)new_p) & 15u) != 0) return -2;
    if (n == 0) return 0;
    int64_t n4 = (n + 3) >> 2;
    int64_t blocks = (n4 + 255) / 256;
    if (blocks > 256 * 1024) blocks = 256 * 1024;
    synth_logp_kernel<<<dim3((unsigned)blocks), dim3(256), 0, stream>>>(*P, old_p, new_p, n);
    return launch_status();
}
