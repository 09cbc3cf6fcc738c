/*
 * abi_common.h -- pieces shared by the C-ABI source files of libparason.so:
 * the handle, workspace alignment and the device's compute-unit count.
 */
#pragma once
#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstring>

#include "parason.h"
#include "device_common.h"

struct parason_handle {
    parason_config cfg;
    pk::TagMatch tm;
};

namespace abi {

constexpr size_t ALIGN = 256;

inline size_t align_up(size_t x) { return (x + ALIGN - 1) / ALIGN * ALIGN; }

/* Compute units of the current device (cached per device) when it is a
 * gfx950 GPU, the only target the kernels are built for; -1 when no device
 * can be queried, -2 when the current device is another GPU. */
inline int cu_count()
{
    static std::atomic<int> cached[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return -1;
    if (dev >= 0 && dev < 64) {
        int c = cached[dev].load(std::memory_order_relaxed);
        if (c != 0) return c;
    }
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return -1;
    /* gcnArchName is "gfx950" followed by nothing or by ":feature" suffixes */
    const bool gfx950 = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0 &&
                        (prop.gcnArchName[6] == '\0' || prop.gcnArchName[6] == ':');
    int cus = -2;
    if (gfx950) {
        cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
            return -1;
    }
    if (dev >= 0 && dev < 64) cached[dev].store(cus, std::memory_order_relaxed);
    return cus;
}

inline bool is_finite(double x) { return std::isfinite(x); }

/* The segment plan of n rows (three launches on `stream`, defined with the
 * plan kernels): seg_off[0 .. n] and mode[0 .. n) as the token scan uses them,
 * tile_sum/tile_off hold n_tiles partial counts. */
void launch_plan(const int64_t *starts, const int32_t *lengths, int64_t n, int64_t mis, int64_t n_tiles,
                 int64_t *tile_sum, int64_t *tile_off, int64_t *seg_off, int32_t *counters, uint8_t *mode,
                 hipStream_t stream);

}  // namespace abi
