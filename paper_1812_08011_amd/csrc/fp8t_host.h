// Host-side helpers shared by the library's entry points.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdlib.h>

#include <mutex>

#include "fp8train.h"

namespace fp8t {

// Largest M, N or K a GEMM entry point accepts: the kernels index rows,
// columns and k in 32 bits and form tile and slab ends (up to 4096 past an
// index) without overflow.
constexpr int64_t kMaxGemmDim = INT32_MAX - 4096;

// Blocks of a grid-stride launch over `total` items, `per_block` per block
// and pass: enough to fill the chip, never beyond the grid's limit.
inline unsigned stride_blocks(int64_t total, int per_block) {
    const int64_t b = (total + per_block - 1) / per_block;
    return (unsigned)(b < 65536 ? (b > 0 ? b : 1) : 65536);
}

inline bool aligned(const void* p, uintptr_t a) {
    return ((uintptr_t)p % a) == 0;
}

// Status of the launch just enqueued.
inline int launch_status() {
    return hipGetLastError() == hipSuccess ? FP8T_OK : FP8T_EHIP;
}

// Integer value of an environment variable (tests and tuning overrides).
inline int env_int(const char* name, int dflt) {
    const char* v = getenv(name);
    return v ? atoi(v) : dflt;
}

// Compute units of the current device (cached per device).
inline int device_cus() {
    static std::mutex mu;
    static int cached[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
    std::lock_guard<std::mutex> lk(mu);
    if (!cached[dev]) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
            return 0;
        cached[dev] = n;
    }
    return cached[dev];
}

// Resident workgroups per CU of a kernel (cached per device and kernel).
inline int kernel_occupancy(const void* fn, int threads) {
    static std::mutex mu;
    struct Ent { int dev; const void* fn; int occ; };
    static Ent cache[256];
    static int n = 0;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    std::lock_guard<std::mutex> lk(mu);
    for (int i = 0; i < n; ++i)
        if (cache[i].dev == dev && cache[i].fn == fn) return cache[i].occ;
    int occ = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, fn, threads, 0) != hipSuccess)
        return 0;
    if (n < 256) cache[n++] = Ent{dev, fn, occ};
    return occ;
}

}  // namespace fp8t
