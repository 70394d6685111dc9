// sr_weight_update: the SGD step of Sec. 2.2 / Fig. 2(b) (L2-Reg,
// Momentum-Acc, Weight-Upd) entirely in FP16 with floating-point stochastic
// rounding (Sec. 2.3 Eq. (1), Sec. 4.3), fused with the FP8 copy of the new
// weights (Sec. 3).
//
// One thread handles one element pair, which is exactly one Philox4x32-10
// block of random bits (8 x 16-bit uniforms, 6 used).  The kernel streams
// 11 bytes per parameter (read w, g, v; write w, v, w8): at full size it is
// HBM-bound, with Philox's 32-bit multiplies as the largest ALU cost.
#include "fp8t_device.h"
#include "fp8train.h"
#include "fp8t_host.h"

namespace fp8t {
namespace {

constexpr int kThreads = 256;

struct upd_params {
    float lr, momentum, weight_decay;
    uint32_t k0, k1;          // Philox key = seed
    uint32_t off_lo, off_hi;  // counter words 2, 3 = offset
};

// Update one element with the three 16-bit uniforms h0, h1, h2.
template <bool HAS_V>
__device__ __forceinline__ void update_one(uint32_t wc, uint32_t gc, uint32_t vc,
                                           uint32_t h0, uint32_t h1, uint32_t h2,
                                           const upd_params& p, uint16_t& w_out,
                                           uint16_t& v_out, uint32_t& w8_out) {
    const float w = fp16_to_f32(wc);
    const float g = fp16_to_f32(gc);
    sr_result g1 = sr16(__builtin_fmaf(p.weight_decay, w, g), h0);
    float step = g1.value;
    if (HAS_V) {
        const float v = fp16_to_f32(vc);
        sr_result v1 = sr16(__builtin_fmaf(p.momentum, v, step), h1);
        v_out = v1.code;
        step = v1.value;
    }
    sr_result w1 = sr16(__builtin_fmaf(-p.lr, step, w), h2);
    w_out = w1.code;
    w8_out = f32_to_fp8(w1.value);
}

template <bool HAS_V, bool HAS_W8>
__global__ __launch_bounds__(kThreads) void sr_update_kernel(
    uint16_t* __restrict__ w, const uint16_t* __restrict__ g, uint16_t* __restrict__ v,
    uint8_t* __restrict__ w8, int64_t n, upd_params p, int vec_ok) {
    const int64_t npairs = (n + 1) / 2;
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t pr = (int64_t)blockIdx.x * kThreads + threadIdx.x; pr < npairs;
         pr += stride) {
        u32x4 ctr = {(uint32_t)pr, (uint32_t)((uint64_t)pr >> 32), p.off_lo, p.off_hi};
        u32x4 rnd = philox4x32_10(ctr, p.k0, p.k1);
        const int64_t i = 2 * pr;
        const bool both = i + 1 < n;
        uint32_t wc0, wc1, gc0, gc1, vc0 = 0, vc1 = 0;
        if (both && vec_ok) {
            const uint32_t wp = reinterpret_cast<const uint32_t*>(w)[pr];
            const uint32_t gp = reinterpret_cast<const uint32_t*>(g)[pr];
            wc0 = wp & 0xFFFFu; wc1 = wp >> 16;
            gc0 = gp & 0xFFFFu; gc1 = gp >> 16;
            if (HAS_V) {
                const uint32_t vp = reinterpret_cast<const uint32_t*>(v)[pr];
                vc0 = vp & 0xFFFFu; vc1 = vp >> 16;
            }
        } else {
            wc0 = w[i]; gc0 = g[i];
            if (HAS_V) vc0 = v[i];
            wc1 = both ? w[i + 1] : 0u;
            gc1 = both ? g[i + 1] : 0u;
            if (HAS_V) vc1 = both ? v[i + 1] : 0u;
        }
        uint16_t wo0, wo1, vo0 = 0, vo1 = 0;
        uint32_t q0, q1;
        // element 2p uses uniforms 0,1,2; element 2p+1 uses 3,4,5
        update_one<HAS_V>(wc0, gc0, vc0, rnd.x & 0xFFFFu, rnd.x >> 16, rnd.y & 0xFFFFu,
                          p, wo0, vo0, q0);
        update_one<HAS_V>(wc1, gc1, vc1, rnd.y >> 16, rnd.z & 0xFFFFu, rnd.z >> 16,
                          p, wo1, vo1, q1);
        if (both && vec_ok) {
            reinterpret_cast<uint32_t*>(w)[pr] = (uint32_t)wo0 | ((uint32_t)wo1 << 16);
            if (HAS_V)
                reinterpret_cast<uint32_t*>(v)[pr] = (uint32_t)vo0 | ((uint32_t)vo1 << 16);
            if (HAS_W8)
                reinterpret_cast<uint16_t*>(w8)[pr] = (uint16_t)(q0 | (q1 << 8));
        } else {
            w[i] = wo0;
            if (HAS_V) v[i] = vo0;
            if (HAS_W8) w8[i] = (uint8_t)q0;
            if (both) {
                w[i + 1] = wo1;
                if (HAS_V) v[i + 1] = vo1;
                if (HAS_W8) w8[i + 1] = (uint8_t)q1;
            }
        }
    }
}

}  // namespace
}  // namespace fp8t

using namespace fp8t;

extern "C" int sr_weight_update(uint16_t* w, const uint16_t* g, uint16_t* v, uint8_t* w8,
                                int64_t n, float lr, float momentum, float weight_decay,
                                uint64_t seed, uint64_t offset, hipStream_t stream) {
    if (n < 0) return FP8T_EINVAL;
    if (momentum != 0.0f && !v) return FP8T_EINVAL;
    if (n == 0) return FP8T_OK;
    if (!w || !g) return FP8T_EINVAL;
    upd_params p;
    p.lr = lr;
    p.momentum = momentum;
    p.weight_decay = weight_decay;
    p.k0 = (uint32_t)seed;
    p.k1 = (uint32_t)(seed >> 32);
    p.off_lo = (uint32_t)offset;
    p.off_hi = (uint32_t)(offset >> 32);
    const int vec_ok = aligned(w, 4) && aligned(g, 4) && (!v || aligned(v, 4)) &&
                       (!w8 || aligned(w8, 2));
    const int64_t npairs = (n + 1) / 2;
    int64_t groups = (npairs + kThreads - 1) / kThreads;
    if (groups > 256 * 32) groups = 256 * 32;
    const dim3 grid((unsigned)groups), block(kThreads);
#define FP8T_LAUNCH(HV, HW)                                                       \
    hipLaunchKernelGGL((sr_update_kernel<HV, HW>), grid, block, 0, stream, w, g, v, \
                       w8, n, p, vec_ok)
    if (v && w8) FP8T_LAUNCH(true, true);
    else if (v) FP8T_LAUNCH(true, false);
    else if (w8) FP8T_LAUNCH(false, true);
    else FP8T_LAUNCH(false, false);
#undef FP8T_LAUNCH
    return launch_status();
}
