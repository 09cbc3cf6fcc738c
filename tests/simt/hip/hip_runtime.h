/*
 * CPU SIMT emulation of the subset of HIP used by the accounting kernels.
 *
 * TEST INFRASTRUCTURE.  The test suite compiles the library's own sources
 * (csrc/parason.hip and the headers it includes) for the host with this file
 * in place of the HIP runtime header, so that the device code runs on the CPU
 * under AddressSanitizer and UndefinedBehaviorSanitizer.  Nothing in the
 * library includes or knows about this file.
 *
 * Memory: the lanes of a wave run one after another between two wave
 * operations, so what one lane writes to memory reaches another lane of its
 * wave only across a wave operation.  On the GPU the wave's accesses are
 * performed in program order; the kernels mark each place where a lane reads
 * (or overwrites) what another lane of its wave wrote with
 * __builtin_amdgcn_wave_barrier(), a wave operation here.
 *
 * Model: a kernel launch runs its blocks one after the other.  Every thread of
 * a block is a fiber with its own stack (switched by the few instructions of
 * simt_switch below: callee-saved registers and the stack pointer, x86-64); threads of a 64-wide wave
 * meet at every wave-level operation (ballot, shuffles, readlane,
 * readfirstlane, DPP row shifts, ds_bpermute) and threads of a block at
 * __syncthreads.  A thread that returns leaves its wave: later wave
 * operations include only the live lanes, as the exec mask does on the GPU.
 * The scheduler aborts with a message when the live lanes of a wave wait at
 * different wave operations (a collective in divergent control flow), when a
 * lane reads a lane that has exited, or when nothing can proceed.
 * __shared__ arrays become function-scope statics: one copy, which is what a
 * block sees since blocks never run at the same time.
 */
#pragma once
#include <stdint.h>
#include <string.h>

#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <functional>
#include <type_traits>
#include <vector>

#if defined(__has_feature)
#if __has_feature(address_sanitizer)
#define SIMT_ASAN 1
#include <sanitizer/asan_interface.h>
#endif
#endif

#define __global__
#define __device__
#define __host__
#define __forceinline__ inline
#define __launch_bounds__(...)
#define __shared__ static
#define __align__(n) __attribute__((aligned(n)))

struct dim3 {
    uint32_t x, y, z;
    dim3(uint32_t x_ = 1, uint32_t y_ = 1, uint32_t z_ = 1) : x(x_), y(y_), z(z_) {}
};

struct alignas(16) int4 {
    int x, y, z, w;
};
struct alignas(16) uint4 {
    unsigned x, y, z, w;
};
inline int4 make_int4(int x, int y, int z, int w) { return int4{x, y, z, w}; }
inline uint4 make_uint4(unsigned x, unsigned y, unsigned z, unsigned w) { return uint4{x, y, z, w}; }

template <class A, class B>
inline typename std::common_type<A, B>::type min(A a, B b)
{
    typedef typename std::common_type<A, B>::type C;
    return (C)a < (C)b ? (C)a : (C)b;
}
template <class A, class B>
inline typename std::common_type<A, B>::type max(A a, B b)
{
    typedef typename std::common_type<A, B>::type C;
    return (C)a > (C)b ? (C)a : (C)b;
}

/* Save the callee-saved registers on the current stack, store the stack
 * pointer to *save_sp, continue on new_sp (which holds the same frame). */
extern "C" void simt_switch(void **save_sp, void *new_sp);
__asm__(".text\n"
        ".weak simt_switch\n"
        ".type simt_switch,@function\n"
        "simt_switch:\n"
        "  pushq %rbp\n  pushq %rbx\n  pushq %r12\n  pushq %r13\n  pushq %r14\n  pushq %r15\n"
        "  movq %rsp, (%rdi)\n"
        "  movq %rsi, %rsp\n"
        "  popq %r15\n  popq %r14\n  popq %r13\n  popq %r12\n  popq %rbx\n  popq %rbp\n"
        "  ret\n"
        ".size simt_switch, .-simt_switch\n");

namespace simt {

constexpr int WAVE = 64;

enum Op : int { OP_NONE, OP_SYNC, OP_WAVE_BARRIER, OP_BALLOT, OP_SHFL, OP_SHFL_UP, OP_READFIRST, OP_READLANE, OP_DPP, OP_BPERMUTE };

struct Lane {
    void *sp = nullptr; /* saved stack pointer while switched out */
    char *stack = nullptr;
    bool alive = false, waiting = false;
    int op = OP_NONE;
    uintptr_t site = 0;
    uint64_t a = 0, b = 0, result = 0;
    void *fake_stack = nullptr;
};

struct State {
    dim3 grid, block, bidx;
    std::vector<Lane> lanes;
    size_t stack_size = 512 * 1024;
    std::vector<char> stacks;
    void *sched_sp = nullptr;
    const void *sched_bottom = nullptr;
    size_t sched_size = 0;
    void *sched_fake = nullptr;
    std::function<void()> body;
    int cur = -1;
    uint64_t collectives = 0;
};

inline State &st()
{
    static State s;
    return s;
}

[[noreturn]] inline void fail(const char *what, int lane)
{
    State &S = st();
    std::fprintf(stderr, "simt: %s (block %u, thread %d)\n", what, S.bidx.x, lane);
    std::abort();
}

inline void to_sched_from_lane(Lane &L, bool dying)
{
    State &S = st();
#ifdef SIMT_ASAN
    __sanitizer_start_switch_fiber(dying ? nullptr : &L.fake_stack, S.sched_bottom, S.sched_size);
#endif
    simt_switch(&L.sp, S.sched_sp);
#ifdef SIMT_ASAN
    __sanitizer_finish_switch_fiber(L.fake_stack, &S.sched_bottom, &S.sched_size);
#endif
}

extern "C" inline void simt_lane_entry()
{
    State &S = st();
    Lane &L = S.lanes[S.cur];
#ifdef SIMT_ASAN
    __sanitizer_finish_switch_fiber(nullptr, &S.sched_bottom, &S.sched_size);
#endif
    S.body();
    Lane &M = S.lanes[S.cur];
    M.alive = false;
    M.waiting = false;
    (void)L;
    to_sched_from_lane(M, true);
    fail("a finished thread was resumed", S.cur);
}

inline void run_lane(int i)
{
    State &S = st();
    Lane &L = S.lanes[i];
    S.cur = i;
#ifdef SIMT_ASAN
    __sanitizer_start_switch_fiber(&S.sched_fake, L.stack, S.stack_size);
#endif
    simt_switch(&S.sched_sp, L.sp);
#ifdef SIMT_ASAN
    __sanitizer_finish_switch_fiber(S.sched_fake, nullptr, nullptr);
#endif
    S.cur = -1;
}

/* A wave operation (or __syncthreads) of the current thread. */
inline uint64_t meet(int op, uintptr_t site, uint64_t a, uint64_t b)
{
    State &S = st();
    Lane &L = S.lanes[S.cur];
    L.op = op;
    L.site = site;
    L.a = a;
    L.b = b;
    L.waiting = true;
    to_sched_from_lane(L, false);
    return S.lanes[S.cur].result;
}

inline int lane_id() { return st().cur & (WAVE - 1); }

/* Resolve the wave [w0, w0 + 64) whose live lanes all wait at one wave operation. */
inline void resolve_wave(int w0, int nl)
{
    State &S = st();
    Lane *W = &S.lanes[w0];
    const int op = [&] {
        for (int i = 0; i < nl; ++i)
            if (W[i].alive) return W[i].op;
        return (int)OP_NONE;
    }();
    uint64_t mask = 0;
    for (int i = 0; i < nl; ++i)
        if (W[i].alive) mask |= 1ull << i;
    auto src = [&](int i, int j) -> uint64_t {
        if (j < 0 || j >= nl || !W[j].alive) fail("a wave operation reads a lane that has exited", w0 + i);
        return W[j].a;
    };
    int first = -1;
    for (int i = 0; i < nl && first < 0; ++i)
        if (W[i].alive) first = i;
    for (int i = 0; i < nl; ++i) {
        if (!W[i].alive) continue;
        Lane &L = W[i];
        switch (op) {
        case OP_WAVE_BARRIER: L.result = 0; break;
        case OP_BALLOT: {
            uint64_t m = 0;
            for (int j = 0; j < nl; ++j)
                if (W[j].alive && W[j].a) m |= 1ull << j;
            L.result = m;
            break;
        }
        case OP_SHFL: L.result = src(i, (int)(L.b & (WAVE - 1))); break;
        case OP_SHFL_UP: L.result = i >= (int)L.b ? src(i, i - (int)L.b) : L.a; break;
        case OP_READFIRST: L.result = W[first].a; break;
        case OP_READLANE: L.result = src(i, (int)L.b); break;
        case OP_BPERMUTE: L.result = src(i, (int)((L.b >> 2) & (WAVE - 1))); break;
        case OP_DPP: {
            /* b: old (32 bits) | ctrl << 32 | bound_ctrl << 48 */
            const uint32_t old = (uint32_t)L.b;
            const int ctrl = (int)((L.b >> 32) & 0xffff);
            int j = -1;
            if (ctrl > 0x110 && ctrl < 0x120) { /* row_shr:n within rows of 16 */
                const int n = ctrl - 0x110;
                j = (i & 15) >= n ? i - n : -1;
            } else if (ctrl == 0x138) { /* wave_shr:1 */
                j = i - 1;
            } else {
                fail("unsupported DPP control", w0 + i);
            }
            L.result = j >= 0 ? (uint32_t)src(i, j) : ((L.b >> 48) & 1 ? 0u : old);
            break;
        }
        default: fail("unknown wave operation", w0 + i);
        }
        L.waiting = false;
        L.op = OP_NONE;
    }
    (void)mask;
    ++S.collectives;
}

inline void run_block()
{
    State &S = st();
    const int n = (int)S.block.x;
    for (int i = 0; i < n; ++i) {
        Lane &L = S.lanes[i];
        L.alive = true;
        L.waiting = false;
        L.op = OP_NONE;
        L.stack = S.stacks.data() + (size_t)i * S.stack_size;
        /* a fresh stack that simt_switch "returns" into simt_lane_entry from:
         * six zero registers, then the entry as return address, placed so
         * that the entry starts with the stack aligned as after a call */
        uintptr_t top = ((uintptr_t)L.stack + S.stack_size) & ~(uintptr_t)15;
        void **sp = (void **)(top - 16);
        sp[0] = (void *)simt_lane_entry;
        sp[1] = nullptr;
        sp -= 6;
        for (int k = 0; k < 6; ++k) sp[k] = nullptr;
        L.sp = sp;
    }
    for (;;) {
        bool any_alive = false;
        for (int i = 0; i < n; ++i) {
            if (S.lanes[i].alive && !S.lanes[i].waiting) run_lane(i);
            any_alive = any_alive || S.lanes[i].alive;
        }
        if (!any_alive) return;
        /* every live thread now waits at a wave operation or at __syncthreads */
        bool progressed = false, at_sync_everywhere = true;
        for (int w0 = 0; w0 < n; w0 += WAVE) {
            const int nl = n - w0 < WAVE ? n - w0 : WAVE;
            int op = OP_NONE;
            uintptr_t site = 0;
            bool live = false, mixed = false;
            for (int i = 0; i < nl; ++i) {
                const Lane &L = S.lanes[w0 + i];
                if (!L.alive) continue;
                if (!live) {
                    op = L.op;
                    site = L.site;
                    live = true;
                } else if (L.op != op || L.site != site) {
                    mixed = true;
                }
            }
            if (!live) continue;
            if (mixed) fail("the live lanes of a wave wait at different wave operations", w0);
            if (op != OP_SYNC) {
                at_sync_everywhere = false;
                resolve_wave(w0, nl);
                progressed = true;
            }
        }
        if (!progressed) {
            if (!at_sync_everywhere) fail("no thread can proceed", -1);
            for (int i = 0; i < n; ++i)
                if (S.lanes[i].alive) {
                    S.lanes[i].waiting = false;
                    S.lanes[i].op = OP_NONE;
                }
        }
    }
}

/* Run `body` as a kernel over grid x block (x dimension only). */
inline void launch(dim3 grid, dim3 block, std::function<void()> body)
{
    State &S = st();
    if (grid.y != 1 || grid.z != 1 || block.y != 1 || block.z != 1 || block.x == 0 || block.x > 1024)
        fail("unsupported launch shape", -1);
    if (S.cur >= 0) fail("a launch from device code", S.cur);
    S.grid = grid;
    S.block = block;
    S.body = std::move(body);
    if (S.lanes.size() < block.x) S.lanes.resize(block.x);
    if (S.stacks.size() < (size_t)block.x * S.stack_size) S.stacks.assign((size_t)block.x * S.stack_size, 0);
    for (uint32_t b = 0; b < grid.x; ++b) {
        S.bidx = dim3(b);
        run_block();
    }
    S.body = nullptr;
}

inline dim3 thread_idx() { return dim3((uint32_t)st().cur); }

template <class T>
inline uint64_t bits(T v)
{
    static_assert(sizeof(T) <= 8, "64-bit values at most");
    uint64_t u = 0;
    memcpy(&u, &v, sizeof(T));
    return u;
}
template <class T>
inline T from_bits(uint64_t u)
{
    T v;
    memcpy(&v, &u, sizeof(T));
    return v;
}

inline uintptr_t site_of(const char *file, int line) { return (uintptr_t)file * 131u + (uintptr_t)line; }

template <class T>
inline T shfl(T v, int src, uintptr_t site)
{
    return from_bits<T>(meet(OP_SHFL, site, bits(v), (uint64_t)(uint32_t)src));
}
template <class T>
inline T shfl_up(T v, unsigned d, uintptr_t site)
{
    return from_bits<T>(meet(OP_SHFL_UP, site, bits(v), d));
}
inline uint64_t ballot(bool p, uintptr_t site) { return meet(OP_BALLOT, site, p ? 1 : 0, 0); }
inline int readfirstlane(int v, uintptr_t site) { return (int)(uint32_t)meet(OP_READFIRST, site, (uint32_t)v, 0); }
inline int readlane(int v, int l, uintptr_t site)
{
    return (int)(uint32_t)meet(OP_READLANE, site, (uint32_t)v, (uint64_t)(uint32_t)l);
}
inline int update_dpp(int old, int src, int ctrl, int row_mask, int bank_mask, bool bound_ctrl, uintptr_t site)
{
    if (row_mask != 0xf || bank_mask != 0xf) fail("unsupported DPP masks", st().cur);
    const uint64_t b = (uint64_t)(uint32_t)old | ((uint64_t)(uint32_t)ctrl << 32) | ((uint64_t)(bound_ctrl ? 1 : 0) << 48);
    return (int)(uint32_t)meet(OP_DPP, site, (uint32_t)src, b);
}
inline int bpermute(int addr, int v, uintptr_t site)
{
    return (int)(uint32_t)meet(OP_BPERMUTE, site, (uint32_t)v, (uint64_t)(uint32_t)addr);
}
inline uint32_t mbcnt_lo(uint32_t m, uint32_t acc)
{
    const int l = lane_id();
    const uint32_t below = l >= 32 ? 0xffffffffu : (l == 0 ? 0u : (0xffffffffu >> (32 - l)));
    return acc + (uint32_t)__builtin_popcount(m & below);
}
inline uint32_t mbcnt_hi(uint32_t m, uint32_t acc)
{
    const int l = lane_id() - 32;
    const uint32_t below = l <= 0 ? 0u : (0xffffffffu >> (32 - l));
    return acc + (uint32_t)__builtin_popcount(m & below);
}

} /* namespace simt */

#define threadIdx (simt::thread_idx())
#define blockIdx (simt::st().bidx)
#define blockDim (simt::st().block)
#define gridDim (simt::st().grid)

#define SIMT_SITE simt::site_of(__FILE__, __LINE__)
#define __syncthreads() ((void)simt::meet(simt::OP_SYNC, 0, 0, 0))
#define __ballot(p) simt::ballot((p), SIMT_SITE)
#define __shfl(v, src, ...) simt::shfl((v), (src), SIMT_SITE)
#define __shfl_up(v, d, ...) simt::shfl_up((v), (d), SIMT_SITE)
#define __builtin_amdgcn_readfirstlane(v) simt::readfirstlane((int)(v), SIMT_SITE)
#define __builtin_amdgcn_readlane(v, l) simt::readlane((int)(v), (l), SIMT_SITE)
#define __builtin_amdgcn_update_dpp(o, s, c, r, b, bc) simt::update_dpp((o), (s), (c), (r), (b), (bc), SIMT_SITE)
#define __builtin_amdgcn_ds_bpermute(a, v) simt::bpermute((a), (v), SIMT_SITE)
#define __builtin_amdgcn_wave_barrier() ((void)simt::meet(simt::OP_WAVE_BARRIER, SIMT_SITE, 0, 0))
/* the lanes of a wave meet only at wave operations, which the kernels place
 * next to each fence that orders memory within a wave */
#define __builtin_amdgcn_fence(order, scope) ((void)0)
#define __builtin_amdgcn_mbcnt_lo(m, a) simt::mbcnt_lo((m), (a))
#define __builtin_amdgcn_mbcnt_hi(m, a) simt::mbcnt_hi((m), (a))

inline int __popcll(unsigned long long x) { return __builtin_popcountll(x); }
inline float __int_as_float(int x) { return simt::from_bits<float>((uint32_t)x); }
inline double __dadd_rn(double a, double b) { return a + b; }
inline double __dsub_rn(double a, double b) { return a - b; }
inline double __dmul_rn(double a, double b) { return a * b; }
inline double __ddiv_rn(double a, double b) { return a / b; }
inline double __dsqrt_rn(double a) { return std::sqrt(a); }
template <class T>
inline T atomicAdd(T *p, T v)
{
    T o = *p;
    *p = o + v;
    return o;
}

/* ---- host API: one emulated gfx950 device ------------------------------- */
typedef enum hipError_t { hipSuccess = 0, hipErrorInvalidValue = 1, hipErrorNoDevice = 100 } hipError_t;
typedef void *hipStream_t;
typedef void *hipEvent_t;
typedef enum hipDeviceAttribute_t { hipDeviceAttributeMultiprocessorCount = 1 } hipDeviceAttribute_t;
struct hipDeviceProp_t {
    char gcnArchName[256];
    int multiProcessorCount;
};

namespace simt {
/* compute units the emulated device reports (the launch grids scale with it) */
inline int &emulated_cus()
{
    static int c = 2;
    return c;
}
} /* namespace simt */

inline hipError_t hipGetDevice(int *d)
{
    *d = 0;
    return hipSuccess;
}
inline hipError_t hipGetDeviceProperties(hipDeviceProp_t *p, int)
{
    memset(p, 0, sizeof(*p));
    strcpy(p->gcnArchName, "gfx950:sramecc+:xnack-");
    p->multiProcessorCount = simt::emulated_cus();
    return hipSuccess;
}
inline hipError_t hipDeviceGetAttribute(int *v, hipDeviceAttribute_t, int)
{
    *v = simt::emulated_cus();
    return hipSuccess;
}
inline hipError_t hipGetLastError() { return hipSuccess; }
inline hipError_t hipEventRecord(hipEvent_t, hipStream_t) { return hipSuccess; }
inline hipError_t hipGetSymbolAddress(void **p, const void *sym)
{
    *p = const_cast<void *>(sym);
    return hipSuccess;
}
#define HIP_SYMBOL(x) ((const void *)&(x))
#define hipLaunchKernelGGL(k, grid, block, shmem, stream, ...) \
    simt::launch(dim3(grid), dim3(block), [&]() { k(__VA_ARGS__); })
