// fp8_quantize and fp16_quantize: element-wise rounding into the paper's
// formats (Sec. 2.1, 2.2).  Both are HBM-bound streaming kernels: each thread
// handles four elements per iteration with one vector load and one vector
// store, grid-striding over the array; a scalar tail loop finishes the
// elements a vector iteration cannot cover.
#include "fp8t_device.h"
#include "fp8train.h"
#include "fp8t_host.h"

namespace fp8t {
namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void q8_from_f32_kernel(
    const float* __restrict__ src, float scale, uint8_t* __restrict__ dst,
    int64_t n, int vec_ok) {
    const int64_t tid = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    int64_t nvec = vec_ok ? n / 4 : 0;
    const float4* s4 = reinterpret_cast<const float4*>(src);
    uint32_t* d4 = reinterpret_cast<uint32_t*>(dst);
    for (int64_t i = tid; i < nvec; i += stride) {
        float4 x = s4[i];
        const uint32_t lo = f32x2_to_fp8x2<false>(x.x * scale, x.y * scale, 0u);
        d4[i] = f32x2_to_fp8x2<true>(x.z * scale, x.w * scale, lo);
    }
    for (int64_t i = nvec * 4 + tid; i < n; i += stride)
        dst[i] = (uint8_t)f32_to_fp8(src[i] * scale);
}

__global__ __launch_bounds__(kThreads) void q8_from_fp16_kernel(
    const uint16_t* __restrict__ src, float scale, uint8_t* __restrict__ dst,
    int64_t n, int vec_ok) {
    const int64_t tid = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    int64_t nvec = vec_ok ? n / 4 : 0;
    const uint2* s4 = reinterpret_cast<const uint2*>(src);
    uint32_t* d4 = reinterpret_cast<uint32_t*>(dst);
    for (int64_t i = tid; i < nvec; i += stride) {
        uint2 c = s4[i];
        const uint32_t lo = f32x2_to_fp8x2<false>(fp16_to_f32(c.x & 0xFFFFu) * scale,
                                                  fp16_to_f32(c.x >> 16) * scale, 0u);
        d4[i] = f32x2_to_fp8x2<true>(fp16_to_f32(c.y & 0xFFFFu) * scale,
                                     fp16_to_f32(c.y >> 16) * scale, lo);
    }
    for (int64_t i = nvec * 4 + tid; i < n; i += stride)
        dst[i] = (uint8_t)f32_to_fp8(fp16_to_f32(src[i]) * scale);
}

__global__ __launch_bounds__(kThreads) void fp16_from_f32_kernel(
    const float* __restrict__ src, uint16_t* __restrict__ dst, int64_t n,
    int vec_ok) {
    const int64_t tid = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    int64_t nvec = vec_ok ? n / 4 : 0;
    const float4* s4 = reinterpret_cast<const float4*>(src);
    uint2* d4 = reinterpret_cast<uint2*>(dst);
    for (int64_t i = tid; i < nvec; i += stride) {
        float4 x = s4[i];
        uint2 o;
        o.x = (uint32_t)f32_to_fp16_rn(x.x) | ((uint32_t)f32_to_fp16_rn(x.y) << 16);
        o.y = (uint32_t)f32_to_fp16_rn(x.z) | ((uint32_t)f32_to_fp16_rn(x.w) << 16);
        d4[i] = o;
    }
    for (int64_t i = nvec * 4 + tid; i < n; i += stride)
        dst[i] = f32_to_fp16_rn(src[i]);
}

// Enough workgroups to fill all 256 CUs several times over, capped so that
// each thread still loops over a few vectors.
unsigned grid_for(int64_t n) {
    int64_t groups = (n / 4 + kThreads - 1) / kThreads;
    if (groups > 256 * 16) groups = 256 * 16;
    if (groups < 1) groups = 1;
    return (unsigned)groups;
}

}  // namespace
}  // namespace fp8t

using namespace fp8t;

extern "C" int fp8_quantize(const void* src, int src_format, float scale,
                            uint8_t* dst, int64_t n, hipStream_t stream) {
    if (n < 0) return FP8T_EINVAL;
    if (src_format != FP8T_SRC_F32 && src_format != FP8T_SRC_FP16) return FP8T_EINVAL;
    if (n == 0) return FP8T_OK;
    if (!src || !dst) return FP8T_EINVAL;
    const unsigned grid = grid_for(n);
    if (src_format == FP8T_SRC_F32) {
        int vec_ok = aligned(src, 16) && aligned(dst, 4);
        hipLaunchKernelGGL(q8_from_f32_kernel, dim3(grid), dim3(kThreads), 0, stream,
                           (const float*)src, scale, dst, n, vec_ok);
    } else {
        int vec_ok = aligned(src, 8) && aligned(dst, 4);
        hipLaunchKernelGGL(q8_from_fp16_kernel, dim3(grid), dim3(kThreads), 0, stream,
                           (const uint16_t*)src, scale, dst, n, vec_ok);
    }
    return launch_status();
}

extern "C" int fp16_quantize(const float* src, uint16_t* dst, int64_t n,
                             hipStream_t stream) {
    if (n < 0) return FP8T_EINVAL;
    if (n == 0) return FP8T_OK;
    if (!src || !dst) return FP8T_EINVAL;
    int vec_ok = aligned(src, 16) && aligned(dst, 8);
    hipLaunchKernelGGL(fp16_from_f32_kernel, dim3(grid_for(n)), dim3(kThreads), 0,
                       stream, src, dst, n, vec_ok);
    return launch_status();
}
