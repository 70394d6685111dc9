// Host-side helpers shared by the library's entry points.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fp8train.h"

namespace fp8t {

inline bool aligned(const void* p, uintptr_t a) {
    return ((uintptr_t)p % a) == 0;
}

// Status of the launch just enqueued.
inline int launch_status() {
    return hipGetLastError() == hipSuccess ? FP8T_OK : FP8T_EHIP;
}

}  // namespace fp8t
