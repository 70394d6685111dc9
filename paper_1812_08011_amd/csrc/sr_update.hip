// sr_weight_update: the SGD step of Sec. 2.2 / Fig. 2(b) (L2-Reg,
// Momentum-Acc, Weight-Upd) entirely in FP16 with floating-point stochastic
// rounding (Sec. 2.3 Eq. (1), Sec. 4.3), fused with the FP8 copy of the new
// weights (Sec. 3).
//
// An element pair takes exactly one Philox4x32-10 block of random bits
// (8 x 16-bit uniforms, 6 used); a thread handles 4 consecutive pairs.  The
// kernel streams
// 11 bytes per parameter (read w, g, v; write w, v, w8): at full size it is
// HBM-bound, with Philox's 32-bit multiplies as the largest ALU cost.
#include <cmath>

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
    int finite;               // lr, momentum and weight decay are finite
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

// The element pair pr (elements 2 pr, 2 pr + 1) takes Philox block pr:
// element 2 pr uses uniforms 0, 1, 2 and element 2 pr + 1 uses 3, 4, 5.
__device__ __forceinline__ u32x4 pair_bits(uint64_t pr, const upd_params& p) {
    const u32x4 ctr = {(uint32_t)pr, (uint32_t)(pr >> 32), p.off_lo, p.off_hi};
    return philox4x32_10(ctr, p.k0, p.k1);
}

template <bool HAS_V>
__device__ __forceinline__ void update_pair(const u32x4& rnd, uint32_t wp, uint32_t gp,
                                            uint32_t vp, const upd_params& p, uint32_t& w_out,
                                            uint32_t& v_out, uint32_t& w8_out) {
    uint16_t wo0, wo1, vo0 = 0, vo1 = 0;
    uint32_t q0, q1;
    update_one<HAS_V>(wp & 0xFFFFu, gp & 0xFFFFu, vp & 0xFFFFu, rnd.x & 0xFFFFu, rnd.x >> 16,
                      rnd.y & 0xFFFFu, p, wo0, vo0, q0);
    update_one<HAS_V>(wp >> 16, gp >> 16, vp >> 16, rnd.y >> 16, rnd.z & 0xFFFFu, rnd.z >> 16,
                      p, wo1, vo1, q1);
    w_out = (uint32_t)wo0 | ((uint32_t)wo1 << 16);
    v_out = (uint32_t)vo0 | ((uint32_t)vo1 << 16);
    w8_out = q0 | (q1 << 8);
}

// The same pair when every value involved is in FP16's normal range: the
// input codes, and the three FMA results in [2^-30, 2^31).  Then decoding is
// exponent rebiasing, SR16 is "carry one step into the kept bits with
// probability F / 2^16" on the raw float bits with no overflow, and encoding
// is rebiasing back.  The caller checks `ok` (false when anything left that
// range -- zeros, subnormals, Inf, NaN, overflow) and falls back to
// update_pair.
__device__ __forceinline__ float dec_lo(uint32_t w) {        // code in bits 0..15
    const uint32_t t = ((w & 0x7FFFu) << 14) + (96u << 23);
    return __uint_as_float(__builtin_amdgcn_ubfe(w, 15, 1) ? t | 0x80000000u : t);
}
__device__ __forceinline__ float dec_hi(uint32_t w) {        // code in bits 16..31
    const uint32_t t = (((w >> 16) & 0x7FFFu) << 14) + (96u << 23);
    return __uint_as_float((w & 0x80000000u) | t);
}
// SR16 of a float in [2^-30, 2^31) in magnitude; r14 = the 16-bit uniform >> 2
// (u < 4 D exactly when (u >> 2) < D for the 14 discarded bits D).
__device__ __forceinline__ float sr16_normal(float x, uint32_t r14) {
    const uint32_t u = __float_as_uint(x);
    const uint32_t up = (u & 0x3FFFu) > r14 ? 0x4000u : 0u;
    return __uint_as_float((u & 0xFFFFC000u) + up);
}
__device__ __forceinline__ uint32_t enc_normal(float v) {   // FP16 code
    const uint32_t u = __float_as_uint(v);
    return ((u >> 16) & 0x8000u) | (__builtin_amdgcn_ubfe(u, 14, 17) - (96u << 9));
}

template <bool HAS_V>
__device__ __forceinline__ bool update_pair_normal(const u32x4& rnd, uint32_t wp, uint32_t gp,
                                                   uint32_t vp, const upd_params& p,
                                                   uint32_t& w_out, uint32_t& v_out,
                                                   float (&w1)[2]) {
    const uint32_t r[6] = {__builtin_amdgcn_ubfe(rnd.x, 2, 14), __builtin_amdgcn_ubfe(rnd.x, 18, 14),
                           __builtin_amdgcn_ubfe(rnd.y, 2, 14), __builtin_amdgcn_ubfe(rnd.y, 18, 14),
                           __builtin_amdgcn_ubfe(rnd.z, 2, 14), __builtin_amdgcn_ubfe(rnd.z, 18, 14)};
    const float w[2] = {dec_lo(wp), dec_hi(wp)};
    const float g[2] = {dec_lo(gp), dec_hi(gp)};
    float lo = 0x1p31f, hi = 0.0f;
    uint32_t wc[2], vc[2] = {0u, 0u};
#pragma unroll
    for (int e = 0; e < 2; ++e) {
        const float x1 = __builtin_fmaf(p.weight_decay, w[e], g[e]);
        float step = sr16_normal(x1, r[3 * e]);
        lo = fminf(lo, fminf(fabsf(w[e]), fabsf(g[e])));
        hi = fmaxf(hi, fmaxf(fabsf(w[e]), fabsf(g[e])));
        lo = fminf(lo, fabsf(x1));
        hi = fmaxf(hi, fabsf(x1));
        if (HAS_V) {
            const float v = e ? dec_hi(vp) : dec_lo(vp);
            const float x2 = __builtin_fmaf(p.momentum, v, step);
            step = sr16_normal(x2, r[3 * e + 1]);
            vc[e] = enc_normal(step);
            lo = fminf(lo, fminf(fabsf(v), fabsf(x2)));
            hi = fmaxf(hi, fmaxf(fabsf(v), fabsf(x2)));
        }
        const float x3 = __builtin_fmaf(-p.lr, step, w[e]);
        w1[e] = sr16_normal(x3, r[3 * e + 2]);
        wc[e] = enc_normal(w1[e]);
        lo = fminf(lo, fabsf(x3));
        hi = fmaxf(hi, fabsf(x3));
    }
    w_out = wc[0] | (wc[1] << 16);
    v_out = vc[0] | (vc[1] << 16);
    // NaN never arises from values in range; comparisons are false for it
    return lo >= 0x1p-30f && hi < 0x1p31f;
}

// One thread updates kPairs consecutive element pairs.  When the tensors
// allow it, that is one 16-byte load of each of w, g, v and 16-byte stores of
// w, v plus an 8-byte store of w8; pairs at the ragged end, or all pairs when
// a pointer is not aligned for those widths, are handled element by element.
constexpr int kPairs = 4;

template <bool HAS_V, bool HAS_W8>
__global__ __launch_bounds__(kThreads) void sr_update_kernel(
    uint16_t* __restrict__ w, const uint16_t* __restrict__ g, uint16_t* __restrict__ v,
    uint8_t* __restrict__ w8, int64_t n, upd_params p, int vec_ok) {
    const int64_t npairs = (n + 1) / 2;
    const int64_t ngroups = (npairs + kPairs - 1) / kPairs;
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t q = (int64_t)blockIdx.x * kThreads + threadIdx.x; q < ngroups; q += stride) {
        const int64_t pr0 = q * kPairs;
        if (vec_ok && 2 * (pr0 + kPairs) <= n) {
            const uint4 wv = reinterpret_cast<const uint4*>(w)[q];
            const uint4 gv = reinterpret_cast<const uint4*>(g)[q];
            uint4 vv = {0u, 0u, 0u, 0u};
            if (HAS_V) vv = reinterpret_cast<const uint4*>(v)[q];
            const uint32_t wa[4] = {wv.x, wv.y, wv.z, wv.w};
            const uint32_t ga[4] = {gv.x, gv.y, gv.z, gv.w};
            const uint32_t va[4] = {vv.x, vv.y, vv.z, vv.w};
            uint32_t wo[4], vo[4], qo[2];
            float w1[4][2];
            bool ok = p.finite;
#pragma unroll
            for (int j = 0; j < kPairs; ++j)
                ok &= update_pair_normal<HAS_V>(pair_bits((uint64_t)(pr0 + j), p), wa[j], ga[j],
                                                va[j], p, wo[j], vo[j], w1[j]);
            if (__builtin_expect(ok, 1)) {
                qo[0] = f32x2_to_fp8x2<true>(w1[1][0], w1[1][1],
                                             f32x2_to_fp8x2<false>(w1[0][0], w1[0][1], 0u));
                qo[1] = f32x2_to_fp8x2<true>(w1[3][0], w1[3][1],
                                             f32x2_to_fp8x2<false>(w1[2][0], w1[2][1], 0u));
            } else {
                uint32_t q8[4];
                for (int j = 0; j < kPairs; ++j)
                    update_pair<HAS_V>(pair_bits((uint64_t)(pr0 + j), p), wa[j], ga[j], va[j], p,
                                       wo[j], vo[j], q8[j]);
                qo[0] = q8[0] | (q8[1] << 16);
                qo[1] = q8[2] | (q8[3] << 16);
            }
            reinterpret_cast<uint4*>(w)[q] = make_uint4(wo[0], wo[1], wo[2], wo[3]);
            if (HAS_V) reinterpret_cast<uint4*>(v)[q] = make_uint4(vo[0], vo[1], vo[2], vo[3]);
            if (HAS_W8)
                reinterpret_cast<uint2*>(w8)[q] = make_uint2(qo[0], qo[1]);
            continue;
        }
        for (int j = 0; j < kPairs; ++j) {
            const int64_t pr = pr0 + j;
            if (pr >= npairs) break;
            const int64_t i = 2 * pr;
            const bool both = i + 1 < n;
            const uint32_t wp = w[i] | (both ? (uint32_t)w[i + 1] << 16 : 0u);
            const uint32_t gp = g[i] | (both ? (uint32_t)g[i + 1] << 16 : 0u);
            uint32_t vp = 0;
            if (HAS_V) vp = v[i] | (both ? (uint32_t)v[i + 1] << 16 : 0u);
            uint32_t wo, vo, qo;
            update_pair<HAS_V>(pair_bits((uint64_t)pr, p), wp, gp, vp, p, wo, vo, qo);
            w[i] = (uint16_t)wo;
            if (HAS_V) v[i] = (uint16_t)vo;
            if (HAS_W8) w8[i] = (uint8_t)qo;
            if (both) {
                w[i + 1] = (uint16_t)(wo >> 16);
                if (HAS_V) v[i + 1] = (uint16_t)(vo >> 16);
                if (HAS_W8) w8[i + 1] = (uint8_t)(qo >> 8);
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
    p.finite = std::isfinite(lr) && std::isfinite(momentum) && std::isfinite(weight_decay);
    const int vec_ok = aligned(w, 16) && aligned(g, 16) && (!v || aligned(v, 16)) &&
                       (!w8 || aligned(w8, 8));
    const int64_t npairs = (n + 1) / 2;
    const int64_t nthreads = (npairs + kPairs - 1) / kPairs;
    int64_t groups = (nthreads + kThreads - 1) / kThreads;
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
