/*
 * decode.hip -- C-ABI of the grammar-constrained decode step (kernels in
 * decode_kernels.h).
 */
#include "abi_common.h"
#include "decode_kernels.h"

using abi::cu_count;

static_assert(sizeof(parason_decode_state) == sizeof(pk::DecodeState), "decode state layout");
static_assert(sizeof(parason_decode_state) == 16, "decode state is 16 bytes");

namespace {
#ifndef PARASON_DECODE_BLOCKS_PER_CU
#define PARASON_DECODE_BLOCKS_PER_CU 8
#endif
constexpr int DECODE_BLOCKS_PER_CU = PARASON_DECODE_BLOCKS_PER_CU;
}  // namespace

extern "C" {

int parason_decode_init(parason_decode_state *states, int64_t batch, void *stream_ptr)
{
    if (batch < 0 || batch > INT32_MAX) return PARASON_ERR_SIZE;
    if (batch == 0) return PARASON_OK;
    if (!states) return PARASON_ERR_NULL;
    if (((uintptr_t)states & 15u) != 0) return PARASON_ERR_ALIGN;
    if (cu_count() <= 0) return PARASON_ERR_DEVICE;
    hipStream_t stream = (hipStream_t)stream_ptr;
    pk::decode_init<<<dim3((unsigned)((batch + 255) / 256)), dim3(256), 0, stream>>>(
        reinterpret_cast<pk::DecodeState *>(states), batch);
    return hipGetLastError() == hipSuccess ? PARASON_OK : PARASON_ERR_HIP;
}

int parason_decode_step(const parason_handle *h, parason_decode_state *states, const int32_t *tokens, int64_t batch,
                        void *logits, int64_t vocab, int64_t row_stride, int32_t dtype, int32_t eos_id,
                        void *stream_ptr)
{
    if (!h) return PARASON_ERR_NULL;
    if (batch < 0 || batch > INT32_MAX || vocab < 1 || vocab > INT32_MAX || row_stride < vocab) return PARASON_ERR_SIZE;
    int32_t elem = 0;
    uint32_t ninf = 0;
    switch (dtype) {
    case PARASON_DTYPE_F32: elem = 4, ninf = 0xFF800000u; break;
    case PARASON_DTYPE_BF16: elem = 2, ninf = 0xFF80u; break;
    case PARASON_DTYPE_F16: elem = 2, ninf = 0xFC00u; break;
    default: return PARASON_ERR_PARAM;
    }
    for (int i = 0; i < 12; ++i)
        if (h->tm.ids[i] >= vocab || h->tm.ids[i] == eos_id) return PARASON_ERR_TAGS;
    if (eos_id < -1 || eos_id >= vocab) return PARASON_ERR_TAGS;
    if (row_stride > INT64_MAX / 4 / (batch > 0 ? batch : 1)) return PARASON_ERR_SIZE;
    if (batch == 0) return PARASON_OK;
    if (!states || !logits) return PARASON_ERR_NULL;
    if (((uintptr_t)states & 15u) != 0 || ((uintptr_t)logits & (uintptr_t)(elem - 1)) != 0 ||
        (tokens && ((uintptr_t)tokens & 3u) != 0))
        return PARASON_ERR_ALIGN;
    const int cus = cu_count();
    if (cus <= 0) return PARASON_ERR_DEVICE;
    hipStream_t stream = (hipStream_t)stream_ptr;

    pk::DecodeArgs da;
    da.states = reinterpret_cast<pk::DecodeState *>(states);
    da.tokens = tokens;
    da.batch = batch;
    da.logits = (char *)logits;
    da.vocab = vocab;
    da.row_bytes = row_stride * elem;
    da.elem = elem;
    da.ninf = ninf;
    da.eos_id = eos_id;
    da.tm = h->tm;
    da.lenient = (h->cfg.flags & PARASON_CFG_LENIENT_GAPS) != 0;
    const int64_t max_blocks = (int64_t)cus * DECODE_BLOCKS_PER_CU;
    const unsigned blocks = (unsigned)(batch < max_blocks ? batch : max_blocks);
    pk::decode_step<<<dim3(blocks), dim3(pk::DECODE_THREADS), 0, stream>>>(da);
    return hipGetLastError() == hipSuccess ? PARASON_OK : PARASON_ERR_HIP;
}

}  // extern "C"
