/*
 * pg_kernels.h -- gfx950 kernels of the policy-gradient step that follows the
 * reward in every PA-GRPO update: group-normalised advantages and the
 * token-level clipped surrogate with separate lower and upper clip ratios
 * (the paper trains with clip ratios 0.2 and 0.28 and 8 rollouts per prompt,
 * Sec. 4 "Training Framework"; the objective itself is the standard GRPO one
 * with DAPO-style clip-higher and a token-level mean, which the paper does not
 * restate).
 *
 *   pg_advantage   one thread per group: A_i = (R_i - mean) / std over the
 *                  group's float rewards (population std, IEEE double, index
 *                  order; A = 0 when all rewards of the group are equal).
 *   sum_lengths_*  exact token count N (deterministic block sums).
 *   pg_surrogate   HBM-bound, one wave per segment of a row (the segment plan
 *                  of the accounting path, two segments in flight per wave):
 *                  d = logp - logp_old in float,
 *                  rho = exp(d) from the hardware exp2 (exp_ratio), the clip
 *                  decision on d against float thresholds ln(1 - eps_low),
 *                  ln(1 + eps_high), the objective term summed in double, the
 *                  gradient of the loss -J with respect to logp written in
 *                  float.  The row's advantage is uniform over a segment, so
 *                  its sign, and whether the segment holds a row end, are
 *                  wave-uniform branches rather than per-token selects.
 *   pg_final       loss, token count and clip counts in fixed order.
 */
#pragma once
#include "device_common.h"

namespace pk {

typedef float v4f __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float4 load_f4(const float4 *p)
{
    v4f v = __builtin_nontemporal_load(reinterpret_cast<const v4f *>(p));
    return make_float4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ void store_f4(float4 *p, float a, float b, float c, float d)
{
    v4f v = {a, b, c, d};
    __builtin_nontemporal_store(v, reinterpret_cast<v4f *>(p));
}

struct PgArgs {
    const float *logp_base;  /* 16-byte aligned bases: pointer - mis elements */
    const float *old_base;
    float *grad_base;
    int64_t mis;
    const int64_t *starts;
    const int32_t *lengths;
    int64_t n;
    const int64_t *seg_off;
    const float *adv;        /* per row */
    float thr_low, thr_high; /* ln(1 - eps_low), ln(1 + eps_high) */
    float lo_val, hi_val;    /* 1 - eps_low, 1 + eps_high */
    const int64_t *n_tokens; /* computed on the device */
    double *wsum;            /* [waves] sum of the objective terms */
    int64_t *wcnt;           /* [waves][2] clipped high, clipped low */
};

__global__ void __launch_bounds__(256) pg_advantage(const float *__restrict__ reward, int64_t n_groups, int32_t G,
                                                    float *__restrict__ adv)
{
    const int64_t grp = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (grp >= n_groups) return;
    const int64_t r0 = grp * G;
    bool equal = true;
    for (int32_t i = 1; i < G; ++i) equal = equal && reward[r0 + i] == reward[r0];
    if (equal) {
        for (int32_t i = 0; i < G; ++i) adv[r0 + i] = 0.0f;
        return;
    }
    double s = 0.0;
    for (int32_t i = 0; i < G; ++i) s = __dadd_rn(s, (double)reward[r0 + i]);
    const double mu = __ddiv_rn(s, (double)G);
    double ss = 0.0;
    for (int32_t i = 0; i < G; ++i) {
        const double d = __dsub_rn((double)reward[r0 + i], mu);
        ss = __dadd_rn(ss, __dmul_rn(d, d));
    }
    const double sigma = __dsqrt_rn(__ddiv_rn(ss, (double)G));
    for (int32_t i = 0; i < G; ++i)
        adv[r0 + i] = (float)__ddiv_rn(__dsub_rn((double)reward[r0 + i], mu), sigma);
}

/* part[b] = sum of max(lengths, 0) over rows [b*RED_TILE, (b+1)*RED_TILE). */
__global__ void __launch_bounds__(RED_THREADS) sum_lengths_tiles(const int32_t *__restrict__ lengths, int64_t n,
                                                                 int64_t *__restrict__ part)
{
    __shared__ int64_t il[RED_THREADS];
    const int64_t r0 = (int64_t)blockIdx.x * RED_TILE + (int64_t)threadIdx.x * ROWS_PER_THREAD;
    int64_t v[1] = {0};
    for (int j = 0; j < ROWS_PER_THREAD; ++j) {
        const int64_t r = r0 + j;
        if (r < n && lengths[r] > 0) v[0] += lengths[r];
    }
    block_tree_sum<int64_t, 1>(v, il);
    if (threadIdx.x == 0) part[blockIdx.x] = v[0];
}

__global__ void __launch_bounds__(RED_THREADS) sum_lengths_final(const int64_t *__restrict__ part, int64_t tiles,
                                                                 int64_t *__restrict__ n_tokens)
{
    __shared__ int64_t il[RED_THREADS];
    int64_t v[1];
    sum_partials<int64_t, 1>(part, tiles, v, il);
    if (threadIdx.x == 0) n_tokens[0] = v[0];
}

/* Wave-wide sums in a fixed order (butterfly over the 64 lanes). */
__device__ __forceinline__ double wave_sum(double v)
{
#pragma unroll
    for (int d = WAVE / 2; d > 0; d >>= 1) v += __shfl_xor(v, d, WAVE);
    return v;
}

__device__ __forceinline__ int64_t wave_sum(int64_t v)
{
#pragma unroll
    for (int d = WAVE / 2; d > 0; d >>= 1) v += __shfl_xor(v, d, WAVE);
    return v;
}

/* Loads of one segment: logp and logp_old vectors v0 + i*WAVE + lane. */
__device__ __forceinline__ void pg_loads(const PgArgs &a, const SegView &w, int lane, float4 (&xn)[LOADS],
                                         float4 (&xo)[LOADS])
{
    const float4 *pn = reinterpret_cast<const float4 *>(a.logp_base);
    const float4 *po = reinterpret_cast<const float4 *>(a.old_base);
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
        const int64_t v = w.v0 + i * WAVE + lane;
        if (!w.edge || v < w.v1) {
            xn[i] = load_f4(pn + v);
            xo[i] = load_f4(po + v);
        } else {
            xn[i] = make_float4(0.f, 0.f, 0.f, 0.f);
            xo[i] = make_float4(0.f, 0.f, 0.f, 0.f);
        }
    }
}

/* e^d for the policy ratio, from the hardware base-2 exponential with the
 * exponent split in the manner of Cody and Waite: d log2(e) = h + r with
 * h = fl(d * L2E_HI) and r = (d * L2E_HI - h) + d * L2E_LO, where the first
 * difference is exact by an fma and L2E_HI + L2E_LO equals log2(e) to 2^-51.
 * Then e^d = 2^h * 2^r, and 2^r = 1 + r ln 2 up to (r ln 2)^2 / 2 < 2^-35
 * because |r| < 2^-17 below the overflow threshold.  An exhaustive sweep of
 * every float d in [-87.33, 88.72) (normal results) on gfx950 measured at
 * most 2.2 ulp against e^d in double (the hardware exp2 itself: 0.79 ulp);
 * the result is +inf above 88.72, as expf's is, and below -87.33 it is
 * within 2^-126 of e^d.  Five float operations and one exp2, against about
 * a dozen for expf with its range checks. */
__device__ __forceinline__ float exp_ratio(float d)
{
    const float L2E_HI = 1.44269502162933349609375f;   /* log2(e) rounded to float */
    const float L2E_LO = 1.925963033500011079e-8f;      /* log2(e) - L2E_HI */
    const float LN2 = 0.693147182464599609375f;         /* ln 2 rounded to float */
    const float h = d * L2E_HI;
    float r = __builtin_fmaf(d, L2E_HI, -h);
    r = __builtin_fmaf(d, L2E_LO, r);
    return __builtin_amdgcn_exp2f(h) * __builtin_fmaf(r, LN2, 1.0f);
}

/* Objective terms, gradient stores and clipped-token count of one loaded
 * segment whose row has advantage A of sign SIGN (0 also stands for a NaN
 * advantage: nothing is clipped).  A token is kept (its unclipped term is the
 * minimum) when d <= ln(1 + eps_high) for A > 0 and d >= ln(1 - eps_low) for
 * A < 0; clipA is the clip bound times A.  EDGE segments hold the first or the
 * last vector of the row, where tokens outside the row are neither counted
 * nor stored. */
template <int SIGN, bool EDGE>
__device__ __forceinline__ void pg_tokens(const PgArgs &a, const SegView &w, int lane, const float4 (&xn)[LOADS],
                                          const float4 (&xo)[LOADS], float A, float thr, float clipA, float inv_n,
                                          double &acc, uint32_t &clipped)
{
    const uint32_t span = (uint32_t)(w.q_hi - w.q_lo);
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
        const int64_t v = w.v0 + i * WAVE + lane;
        const int32_t b = 4 * (i * WAVE + lane) - w.q_lo;
        const float nn[4] = {xn[i].x, xn[i].y, xn[i].z, xn[i].w};
        const float oo[4] = {xo[i].x, xo[i].y, xo[i].z, xo[i].w};
        float g[4];
        bool in[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            in[j] = !EDGE || (uint32_t)(b + j) < span;
            const float d = __fsub_rn(nn[j], oo[j]);
            const float p = A * exp_ratio(d);
            const bool keep = SIGN > 0 ? d <= thr : SIGN < 0 ? d >= thr : true;
            g[j] = keep ? -p * inv_n : 0.0f;
            const float L = keep ? p : clipA;
            if (EDGE) {
                acc += (double)(in[j] ? L : 0.0f);
                if (SIGN != 0) clipped += (!keep && in[j]) ? 1u : 0u;
            } else {
                acc += (double)L;
                if (SIGN != 0) clipped += keep ? 0u : 1u;
            }
        }
        float *dst = a.grad_base + 4 * v;
        if (!EDGE || (in[0] && in[3])) {
            store_f4(reinterpret_cast<float4 *>(dst), g[0], g[1], g[2], g[3]);
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (in[j]) dst[j] = g[j];
        }
    }
}

/* One loaded segment: the row's advantage decides the branch for the whole
 * wave. */
__device__ __forceinline__ void pg_segment(const PgArgs &a, const SegView &w, int lane, const float4 (&xn)[LOADS],
                                           const float4 (&xo)[LOADS], float inv_n, double &acc, uint32_t &clip_hi,
                                           uint32_t &clip_lo)
{
    const float A = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(a.adv[w.row])));
    if (A > 0.0f) {
        const float clipA = a.hi_val * A;
        if (w.edge) pg_tokens<1, true>(a, w, lane, xn, xo, A, a.thr_high, clipA, inv_n, acc, clip_hi);
        else pg_tokens<1, false>(a, w, lane, xn, xo, A, a.thr_high, clipA, inv_n, acc, clip_hi);
    } else if (A < 0.0f) {
        const float clipA = a.lo_val * A;
        if (w.edge) pg_tokens<-1, true>(a, w, lane, xn, xo, A, a.thr_low, clipA, inv_n, acc, clip_lo);
        else pg_tokens<-1, false>(a, w, lane, xn, xo, A, a.thr_low, clipA, inv_n, acc, clip_lo);
    } else {
        if (w.edge) pg_tokens<0, true>(a, w, lane, xn, xo, A, 0.0f, 0.0f, inv_n, acc, clip_hi);
        else pg_tokens<0, false>(a, w, lane, xn, xo, A, 0.0f, 0.0f, inv_n, acc, clip_hi);
    }
}

/* One wave per segment of the plan; the wave's segments are contiguous.  Two
 * register buffers alternate so that the next segment's loads are in flight
 * while the current one is evaluated. */
__global__ void __launch_bounds__(256, 4) pg_surrogate(PgArgs a)
{
    const int lane = threadIdx.x & (WAVE - 1);
    const int64_t wave = uniform64((int64_t)blockIdx.x * (blockDim.x / WAVE) + (threadIdx.x / WAVE));
    const int64_t n_waves = (int64_t)gridDim.x * (blockDim.x / WAVE);
    const int64_t S = a.seg_off[a.n];
    const int64_t s_begin = uniform64(S * wave / n_waves);
    const int64_t s_end = uniform64(S * (wave + 1) / n_waves);
    double acc = 0.0;
    /* per-lane clip counts: a lane sees at most a 64th of the batch's tokens */
    uint32_t clip_hi = 0, clip_lo = 0;
    if (s_begin < s_end) {
        const float inv_n = (float)__ddiv_rn(1.0, (double)a.n_tokens[0]);
        SegCursor cur;
        cur.seg_off = a.seg_off;
        cur.starts = a.starts;
        cur.lengths = a.lengths;
        cur.mis = a.mis;
        cur.s_begin = s_begin;
        cur.s_end = s_end;
        cur.seek(s_begin, a.n);
        float4 na[LOADS], oa[LOADS], nb[LOADS], ob[LOADS];
        SegView w = cur.view(s_begin);
        pg_loads(a, w, lane, na, oa);
        int64_t s = s_begin;
        while (true) {
            SegView wn;
            bool more = s + 1 < s_end;
            if (more) {
                wn = cur.view(s + 1);
                pg_loads(a, wn, lane, nb, ob);
            }
            pg_segment(a, w, lane, na, oa, inv_n, acc, clip_hi, clip_lo);
            if (!more) break;
            ++s;
            w = wn;
            more = s + 1 < s_end;
            if (more) {
                wn = cur.view(s + 1);
                pg_loads(a, wn, lane, na, oa);
            }
            pg_segment(a, w, lane, nb, ob, inv_n, acc, clip_hi, clip_lo);
            if (!more) break;
            ++s;
            w = wn;
        }
    }
    acc = wave_sum(acc);
    const int64_t hi_sum = wave_sum((int64_t)clip_hi);
    const int64_t lo_sum = wave_sum((int64_t)clip_lo);
    if (lane == 0) {
        a.wsum[wave] = acc;
        a.wcnt[2 * wave] = hi_sum;
        a.wcnt[2 * wave + 1] = lo_sum;
    }
}

/* stats = {loss, tokens, clipped high, clipped low}, sums over waves in order. */
__global__ void __launch_bounds__(RED_THREADS) pg_final(const double *__restrict__ wsum,
                                                        const int64_t *__restrict__ wcnt, int64_t waves,
                                                        const int64_t *__restrict__ n_tokens, double *__restrict__ stats)
{
    __shared__ double dl[RED_THREADS];
    __shared__ int64_t il[2 * RED_THREADS];
    double sv[1];
    int64_t cv[2];
    sum_partials<double, 1>(wsum, waves, sv, dl);
    sum_partials<int64_t, 2>(wcnt, waves, cv, il);
    if (threadIdx.x != 0) return;
    const int64_t N = n_tokens[0];
    stats[PARASON_PG_STAT_LOSS] = N > 0 ? -__ddiv_rn(sv[0], (double)N) : 0.0;
    stats[PARASON_PG_STAT_TOKENS] = (double)N;
    stats[PARASON_PG_STAT_CLIP_HIGH] = (double)cv[0];
    stats[PARASON_PG_STAT_CLIP_LOW] = (double)cv[1];
}

} /* namespace pk */
