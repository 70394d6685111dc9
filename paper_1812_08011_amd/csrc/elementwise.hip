// Element-wise steps around the GEMMs of a training step in the paper's
// formats (Sec. 2.1: activations and errors enter the GEMMs in FP8; Sec. 3:
// the last layer in FP16, loss scaling).  All are HBM-bound streaming
// kernels: grid-strided, one element per thread per iteration.
#include "fp8t_device.h"
#include "fp8train.h"
#include "fp8t_host.h"

namespace fp8t {
namespace {

constexpr int kThreads = 256;

// ReLU on codes: negative values (sign bit set) become +0, NaN stays NaN.
__device__ __forceinline__ uint32_t relu8(uint32_t c) {
    return ((c & 0x7Fu) > 0x7Cu) ? kFp8NaN : ((c & 0x80u) ? 0u : c);
}
__device__ __forceinline__ uint32_t relu16(uint32_t c) {
    return ((c & 0x7FFFu) > 0x7E00u) ? kFp16NaN : ((c & 0x8000u) ? 0u : c);
}

__global__ __launch_bounds__(kThreads) void relu8_kernel(const uint8_t* __restrict__ x,
                                                         uint8_t* __restrict__ y, int64_t n) {
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += stride)
        y[i] = (uint8_t)relu8(x[i]);
}

__global__ __launch_bounds__(kThreads) void relu16_kernel(const uint16_t* __restrict__ x,
                                                          uint16_t* __restrict__ y, int64_t n) {
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += stride)
        y[i] = (uint16_t)relu16(x[i]);
}

// e8 = Q8(RN32(value(d) * scale)) where value(z) > 0, else +0.
__global__ __launch_bounds__(kThreads) void relu_bwd_kernel(const uint16_t* __restrict__ d,
                                                            const uint16_t* __restrict__ z,
                                                            uint8_t* __restrict__ e, int64_t n,
                                                            float scale) {
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += stride) {
        const float zv = fp16_to_f32(z[i]);
        const float dv = zv > 0.0f ? fp16_to_f32(d[i]) : 0.0f;
        e[i] = (uint8_t)f32_to_fp8(dv * scale);
    }
}

// e = RN16(RN32(RN32(value(y) - value(t)) * scale)).
__global__ __launch_bounds__(kThreads) void mse_grad_kernel(const uint16_t* __restrict__ y,
                                                            const uint16_t* __restrict__ t,
                                                            uint16_t* __restrict__ e, int64_t n,
                                                            float scale) {
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += stride) {
        const float diff = __fsub_rn(fp16_to_f32(y[i]), fp16_to_f32(t[i]));
        e[i] = f32_to_fp16_rn(__fmul_rn(diff, scale));
    }
}

unsigned grid_for(int64_t n) {
    int64_t g = (n + kThreads - 1) / kThreads;
    if (g > 256 * 64) g = 256 * 64;
    return (unsigned)g;
}

}  // namespace
}  // namespace fp8t

using namespace fp8t;

extern "C" int relu_codes(const void* x, int format, void* y, int64_t n, hipStream_t stream) {
    if (n < 0 || (format != 8 && format != 16)) return FP8T_EINVAL;
    if (n == 0) return FP8T_OK;
    if (!x || !y) return FP8T_EINVAL;
    if (format == 8)
        hipLaunchKernelGGL(relu8_kernel, dim3(grid_for(n)), dim3(kThreads), 0, stream,
                           static_cast<const uint8_t*>(x), static_cast<uint8_t*>(y), n);
    else
        hipLaunchKernelGGL(relu16_kernel, dim3(grid_for(n)), dim3(kThreads), 0, stream,
                           static_cast<const uint16_t*>(x), static_cast<uint16_t*>(y), n);
    return launch_status();
}

extern "C" int relu_backward_fp8(const uint16_t* d, const uint16_t* z, uint8_t* e, int64_t n,
                                 float scale, hipStream_t stream) {
    if (n < 0) return FP8T_EINVAL;
    if (n == 0) return FP8T_OK;
    if (!d || !z || !e) return FP8T_EINVAL;
    hipLaunchKernelGGL(relu_bwd_kernel, dim3(grid_for(n)), dim3(kThreads), 0, stream, d, z, e, n,
                       scale);
    return launch_status();
}

extern "C" int mse_grad_fp16(const uint16_t* y, const uint16_t* t, uint16_t* e, int64_t n,
                             float scale, hipStream_t stream) {
    if (n < 0) return FP8T_EINVAL;
    if (n == 0) return FP8T_OK;
    if (!y || !t || !e) return FP8T_EINVAL;
    hipLaunchKernelGGL(mse_grad_kernel, dim3(grid_for(n)), dim3(kThreads), 0, stream, y, t, e, n,
                       scale);
    return launch_status();
}
