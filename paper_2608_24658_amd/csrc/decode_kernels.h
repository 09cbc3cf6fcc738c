/*
 * decode_kernels.h -- grammar-constrained decode step for gfx950.
 *
 * Rollouts keep the tags of the grammar of Figure 4 (Sec. 3.2) valid by
 * constrained decoding (Sec. 3.4).  Per sequence a 16-byte state holds the
 * position in the grammar; one step advances it by the token just sampled and
 * then masks the next-token logits to the tokens that keep the prefix viable:
 *
 *   state    allowed next tokens
 *   START    <think>
 *   BODY     Text, <Parallel>, and </think> (depth 0) or </Thread> (depth > 0)
 *   P_OPEN   <Outlines>
 *   O_OPEN   <Subtask>, <Trial>
 *   ENTRY    Text, and the matching close tag once the entry has text
 *   E_DONE   <Subtask>, <Trial>, </Outlines>
 *   O_DONE   <Thread>
 *   W_DONE   <Thread>, </Parallel>
 *   TRAIL    Text, end of sequence
 *
 * With PARASON_CFG_LENIENT_GAPS Text is also allowed in P_OPEN, O_OPEN,
 * E_DONE, O_DONE and W_DONE (a gap between the structural tags of a region)
 * and leaves the state unchanged.
 *
 * When Text is allowed only the (at most 13) tag and end-of-sequence logits
 * can change: a handful of scattered stores.  Otherwise the whole row becomes
 * -inf except the allowed tags: a full-row HBM write, 16 bytes per store.
 * A sequence that sampled a token its state does not allow is flagged and
 * left unmasked.
 */
#pragma once
#include "device_common.h"

namespace pk {

enum : int32_t { D_START = 0, D_BODY, D_P_OPEN, D_O_OPEN, D_ENTRY, D_E_DONE, D_O_DONE, D_W_DONE, D_TRAIL };

struct DecodeState {
    int32_t state;
    int32_t depth;      /* open <Parallel> blocks */
    int32_t entry;      /* ENTRY: class of the open entry tag | 0x100 once it has text */
    uint32_t flags;     /* PARASON_DECODE_ERROR, PARASON_DECODE_DONE */
};

constexpr uint32_t A_EOS = 1u << 13; /* allowed-set bit of the end-of-sequence token */
constexpr uint32_t A_ALL = 0xFFFFFFFFu;

__device__ __forceinline__ uint32_t bit(uint32_t c) { return 1u << c; }

__device__ __forceinline__ uint32_t allowed_set(const DecodeState &s, bool lenient)
{
    if (s.flags & (PARASON_DECODE_ERROR | PARASON_DECODE_DONE)) return A_ALL;
    const uint32_t gap = lenient ? bit(C_TEXT) : 0u;
    switch (s.state) {
    case D_START: return bit(C_THINK);
    case D_BODY: return bit(C_TEXT) | bit(C_PAR) | (s.depth == 0 ? bit(C_END_THINK) : bit(C_END_THR));
    case D_P_OPEN: return gap | bit(C_OUT);
    case D_O_OPEN: return gap | bit(C_SUB) | bit(C_TRI);
    case D_ENTRY: return bit(C_TEXT) | ((s.entry & 0x100) ? bit((uint32_t)(s.entry & 0xFF) + 1u) : 0u);
    case D_E_DONE: return gap | bit(C_SUB) | bit(C_TRI) | bit(C_END_OUT);
    case D_O_DONE: return gap | bit(C_THR);
    case D_W_DONE: return gap | bit(C_THR) | bit(C_END_PAR);
    default: return bit(C_TEXT) | A_EOS; /* D_TRAIL */
    }
}

/* Advance by one sampled token of class c (eos: it is the end-of-sequence id). */
__device__ __forceinline__ void advance(DecodeState &s, uint32_t c, bool eos, bool lenient)
{
    if (s.flags & (PARASON_DECODE_ERROR | PARASON_DECODE_DONE)) return;
    const uint32_t allow = allowed_set(s, lenient);
    const uint32_t want = eos ? A_EOS : bit(c);
    if (!(allow & want)) {
        s.flags |= PARASON_DECODE_ERROR;
        return;
    }
    if (eos) {
        s.flags |= PARASON_DECODE_DONE;
        return;
    }
    if (c == C_TEXT) { /* allowed Text changes nothing but an entry's has-text bit */
        if (s.state == D_ENTRY) s.entry |= 0x100;
        return;
    }
    switch (s.state) {
    case D_START: s.state = D_BODY; break;
    case D_BODY:
        if (c == C_PAR) {
            s.state = D_P_OPEN;
            s.depth += 1;
        } else if (c == C_END_THINK) {
            s.state = D_TRAIL;
        } else if (c == C_END_THR) {
            s.state = D_W_DONE;
        }
        break;
    case D_P_OPEN: s.state = D_O_OPEN; break;
    case D_O_OPEN:
    case D_E_DONE:
        if (c == C_END_OUT) {
            s.state = D_O_DONE;
        } else {
            s.state = D_ENTRY;
            s.entry = (int32_t)c;
        }
        break;
    case D_ENTRY: s.state = D_E_DONE; break;
    case D_O_DONE: s.state = D_BODY; break;
    case D_W_DONE:
        if (c == C_THR) {
            s.state = D_BODY;
        } else {
            s.state = D_BODY;
            s.depth -= 1;
        }
        break;
    default: break; /* D_TRAIL: Text */
    }
}

struct DecodeArgs {
    DecodeState *states;
    const int32_t *tokens; /* sampled token per row, NULL or < 0: no token */
    int64_t batch;
    char *logits;          /* row r at logits + r * row_bytes, elem-aligned */
    int64_t vocab;
    int64_t row_bytes;
    int32_t elem;          /* bytes per logit: 2 or 4 */
    uint32_t ninf;         /* bit pattern of -inf in the logit type (low elem bytes) */
    int32_t eos_id;        /* < 0: none */
    bool lenient;          /* PARASON_CFG_LENIENT_GAPS */
    TagMatch tm;
};

__device__ __forceinline__ void store_ninf(char *row, int64_t i, const DecodeArgs &a)
{
    if (a.elem == 2) reinterpret_cast<uint16_t *>(row)[i] = (uint16_t)a.ninf;
    else reinterpret_cast<uint32_t *>(row)[i] = a.ninf;
}

#ifndef PARASON_DECODE_THREADS
#define PARASON_DECODE_THREADS 256
#endif
constexpr int DECODE_THREADS = PARASON_DECODE_THREADS;

/* One block per row, grid-stride over the rows. */
__global__ void __launch_bounds__(DECODE_THREADS) decode_step(DecodeArgs a)
{
    __shared__ uint32_t allow_s;
    for (int64_t r = blockIdx.x; r < a.batch; r += gridDim.x) {
        if (threadIdx.x == 0) {
            DecodeState s = a.states[r];
            const int32_t t = a.tokens ? a.tokens[r] : -1;
            if (t >= 0) advance(s, classify(a.tm, t, a.tm.contiguous != 0), t == a.eos_id, a.lenient);
            a.states[r] = s;
            allow_s = allowed_set(s, a.lenient);
        }
        __syncthreads();
        const uint32_t allow = allow_s;
        __syncthreads();
        if (allow == A_ALL) continue;
        char *row = a.logits + r * a.row_bytes;
        if (allow & bit(C_TEXT)) {
            /* Text allowed: only tag and end-of-sequence logits can be disallowed */
            const int t = threadIdx.x;
            if (t < 12) {
                if (!(allow & bit((uint32_t)t + 1u))) store_ninf(row, a.tm.ids[t], a);
            } else if (t == 12 && a.eos_id >= 0 && !(allow & A_EOS)) {
                store_ninf(row, a.eos_id, a);
            }
            continue;
        }
        /* No Text: every logit but the (at most three) allowed tags becomes -inf. */
        int64_t keep0 = -1, keep1 = -1, keep2 = -1;
        for (int k = 0; k < 12; ++k) {
            if (!(allow & bit((uint32_t)k + 1u))) continue;
            if (keep0 < 0) keep0 = a.tm.ids[k];
            else if (keep1 < 0) keep1 = a.tm.ids[k];
            else keep2 = a.tm.ids[k];
        }
        const int64_t per = 16 / a.elem; /* logits per 16-byte store */
        /* head: logits before the first 16-byte boundary of the row */
        const int64_t head_bytes = (int64_t)((16u - ((uintptr_t)row & 15u)) & 15u);
        int64_t head = head_bytes / a.elem;
        head = head < a.vocab ? head : a.vocab;
        const int64_t n_vec = (a.vocab - head) / per;
        const int64_t tail0 = head + n_vec * per;
        const uint32_t w = a.elem == 2 ? (a.ninf | (a.ninf << 16)) : a.ninf;
        const uint4 ninf4 = make_uint4(w, w, w, w);
        uint4 *vrow = reinterpret_cast<uint4 *>(row + head * a.elem);
        /* the (at most three) vectors that hold a kept logit are written
         * elementwise below; every other vector is one 16-byte store */
        const int32_t nv = (int32_t)n_vec;
        const int32_t kv0 = keep0 >= head && keep0 < tail0 ? (int32_t)((keep0 - head) / per) : -1;
        const int32_t kv1 = keep1 >= head && keep1 < tail0 ? (int32_t)((keep1 - head) / per) : -1;
        const int32_t kv2 = keep2 >= head && keep2 < tail0 ? (int32_t)((keep2 - head) / per) : -1;
#ifndef PARASON_DECODE_UNROLL
#define PARASON_DECODE_UNROLL 4
#endif
        constexpr int U = PARASON_DECODE_UNROLL;
        int32_t v = (int32_t)threadIdx.x;
        for (; v + (U - 1) * DECODE_THREADS < nv; v += U * DECODE_THREADS) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int32_t vv = v + u * DECODE_THREADS;
                if (vv != kv0 && vv != kv1 && vv != kv2) vrow[vv] = ninf4;
            }
        }
        for (; v < nv; v += DECODE_THREADS)
            if (v != kv0 && v != kv1 && v != kv2) vrow[v] = ninf4;
        if (threadIdx.x < 3) {
            const int32_t kv = threadIdx.x == 0 ? kv0 : (threadIdx.x == 1 ? kv1 : kv2);
            /* a vector holding two kept logits is listed twice: only its first listing writes it */
            const bool first = kv >= 0 && !(threadIdx.x >= 1 && kv == kv0) && !(threadIdx.x == 2 && kv == kv1);
            if (first) {
                for (int64_t e = head + (int64_t)kv * per; e < head + (int64_t)(kv + 1) * per; ++e)
                    if (e != keep0 && e != keep1 && e != keep2) store_ninf(row, e, a);
            }
        }
        for (int64_t e = threadIdx.x; e < head; e += DECODE_THREADS)
            if (e != keep0 && e != keep1 && e != keep2) store_ninf(row, e, a);
        for (int64_t e = tail0 + threadIdx.x; e < a.vocab; e += DECODE_THREADS)
            if (e != keep0 && e != keep1 && e != keep2) store_ninf(row, e, a);
    }
}

__global__ void __launch_bounds__(256) decode_init(DecodeState *states, int64_t batch)
{
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r < batch) states[r] = DecodeState{D_START, 0, 0, 0u};
}

} /* namespace pk */
