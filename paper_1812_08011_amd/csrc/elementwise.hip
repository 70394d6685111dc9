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

// col2im: dX[n, ih, iw, c] = the FP16 sum, in ascending (kh, kw) order and
// rounded to nearest after every addition, of the lowered-matrix entries
// cols[(n, oh, ow), (kh, kw, c)] of the output positions whose window covers
// (ih, iw).  One thread per element of dX, channels fastest (coalesced).
struct Col2imGeom {
    int64_t total;                     // N H W C
    int H, W, C, KH, KW, OH, OW, pad, stride;
    int64_t K;                         // KH KW C
};

__global__ __launch_bounds__(kThreads) void col2im_kernel(const uint16_t* __restrict__ cols,
                                                          uint16_t* __restrict__ dx,
                                                          Col2imGeom q) {
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < q.total; i += stride) {
        const int c = (int)(i % q.C);
        const int64_t pix = i / q.C;
        const int iw = (int)(pix % q.W);
        const int64_t t = pix / q.W;
        const int ih = (int)(t % q.H);
        const int64_t n = t / q.H;
        float S = 0.0f;
        for (int kh = 0; kh < q.KH; ++kh) {
            const int yh = ih + q.pad - kh;
            if (yh < 0 || yh % q.stride) continue;
            const int oh = yh / q.stride;
            if (oh >= q.OH) continue;
            for (int kw = 0; kw < q.KW; ++kw) {
                const int yw = iw + q.pad - kw;
                if (yw < 0 || yw % q.stride) continue;
                const int ow = yw / q.stride;
                if (ow >= q.OW) continue;
                const int64_t row = (n * q.OH + oh) * q.OW + ow;
                const uint16_t v = cols[row * q.K + ((int64_t)kh * q.KW + kw) * q.C + c];
                S = rn16s(S + fp16_to_f32s(v));
            }
        }
        dx[i] = f32s_to_fp16(S);
    }
}

// The same with 8 consecutive channels per thread (C % 8 == 0, 16-byte
// aligned arrays): one 16-byte load per covering entry, one 16-byte store.
__global__ __launch_bounds__(kThreads) void col2im8_kernel(const uint16_t* __restrict__ cols,
                                                           uint16_t* __restrict__ dx,
                                                           Col2imGeom q) {
    const int64_t groups = q.total / 8;
    const int cg = q.C / 8;
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < groups; i += stride) {
        const int c = (int)(i % cg) * 8;
        const int64_t pix = i / cg;
        const int iw = (int)(pix % q.W);
        const int64_t t = pix / q.W;
        const int ih = (int)(t % q.H);
        const int64_t n = t / q.H;
        float S[8];
#pragma unroll
        for (int v = 0; v < 8; ++v) S[v] = 0.0f;
        for (int kh = 0; kh < q.KH; ++kh) {
            const int yh = ih + q.pad - kh;
            if (yh < 0 || yh % q.stride) continue;
            const int oh = yh / q.stride;
            if (oh >= q.OH) continue;
            for (int kw = 0; kw < q.KW; ++kw) {
                const int yw = iw + q.pad - kw;
                if (yw < 0 || yw % q.stride) continue;
                const int ow = yw / q.stride;
                if (ow >= q.OW) continue;
                const int64_t row = (n * q.OH + oh) * q.OW + ow;
                const uint4 w = *reinterpret_cast<const uint4*>(
                    cols + row * q.K + ((int64_t)kh * q.KW + kw) * q.C + c);
                const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
                for (int v = 0; v < 8; ++v)
                    S[v] = rn16s(S[v] + fp16_to_f32s((ws[v / 2] >> (16 * (v % 2))) & 0xFFFFu));
            }
        }
        uint32_t o[4];
#pragma unroll
        for (int v = 0; v < 4; ++v)
            o[v] = (uint32_t)f32s_to_fp16(S[2 * v]) | ((uint32_t)f32s_to_fp16(S[2 * v + 1]) << 16);
        *reinterpret_cast<uint4*>(dx + i * 8) = make_uint4(o[0], o[1], o[2], o[3]);
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

extern "C" int col2im_fp16(const uint16_t* cols, int64_t N, int64_t H, int64_t W, int64_t C,
                           int64_t KH, int64_t KW, int64_t pad, int64_t stride, uint16_t* dX,
                           hipStream_t stream) {
    if (N < 0 || H < 1 || W < 1 || C < 1 || KH < 1 || KW < 1 || pad < 0 || stride < 1)
        return FP8T_EINVAL;
    if (H + 2 * pad < KH || W + 2 * pad < KW) return FP8T_EINVAL;
    if (H > INT32_MAX || W > INT32_MAX || C > INT32_MAX || KH * KW * C > INT32_MAX)
        return FP8T_EINVAL;
    Col2imGeom q;
    q.total = N * H * W * C;
    if (q.total == 0) return FP8T_OK;
    if (!cols || !dX) return FP8T_EINVAL;
    q.H = (int)H;
    q.W = (int)W;
    q.C = (int)C;
    q.KH = (int)KH;
    q.KW = (int)KW;
    q.pad = (int)pad;
    q.stride = (int)stride;
    q.OH = (int)((H + 2 * pad - KH) / stride + 1);
    q.OW = (int)((W + 2 * pad - KW) / stride + 1);
    q.K = KH * KW * C;
    if (C % 8 == 0 && aligned(cols, 16) && aligned(dX, 16))
        hipLaunchKernelGGL(col2im8_kernel, dim3(grid_for(q.total / 8)), dim3(kThreads), 0, stream,
                           cols, dX, q);
    else
        hipLaunchKernelGGL(col2im_kernel, dim3(grid_for(q.total)), dim3(kThreads), 0, stream,
                           cols, dX, q);
    return launch_status();
}
