// Device-side number-format helpers for gfx950.
//
// FP8 = (1,5,2) bias 15 and FP16 = (1,6,9) bias 31 (Sec. 2.2), both with
// gradual underflow; the all-ones exponent holds Inf/NaN.
//
// The GEMM kernels work in a *scaled FP32 domain*: every FP16 quantity x is
// held as the IEEE float x * 2^96.  In that domain
//   - every FP16 value (2^-39 .. 2^32) maps to a normal float (2^57 .. 2^128),
//     so FP32 denormals never occur;
//   - the FP16 overflow threshold 2^32 maps onto FP32's own 2^128, so the
//     carry out of rounding the largest values lands exactly on the FP32 Inf
//     encoding and FP16 overflow needs no extra instruction.
// Rounding to FP16 is then "round the FP32 significand to 10 bits, ties to
// even" on the raw bits.  FP32 addition first rounds the exact sum to 24 bits;
// because 24 >= 2*10 + 1 that double rounding is innocuous (Figueroa 1995),
// and below 2^-30 (FP16 subnormals) sums of FP16 values are exact in FP32.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fp8t {

constexpr uint32_t kF32Inf = 0x7F800000u;
constexpr uint32_t kF32NaN = 0x7FC00000u;
constexpr uint16_t kFp16NaN = 0x7F00u;
constexpr uint16_t kFp16Inf = 0x7E00u;
constexpr uint32_t kFp8NaN = 0x7Fu;

// Round a scaled-domain float to the FP16 grid: keep 9 of the 23 stored
// mantissa bits, ties to even (bfe + add3 + and).
__device__ __forceinline__ float rn16s(float x) {
    uint32_t u = __float_as_uint(x);
    u = (u + 0x1FFFu + ((u >> 14) & 1u)) & 0xFFFFC000u;
    return __uint_as_float(u);
}

// FP8 code -> float times 2^SHIFT (exact).  SHIFT = 96 gives the scaled
// domain for one GEMM operand, 0 the plain value.
template <int SHIFT>
__device__ __forceinline__ float fp8_to_f32(uint32_t c) {
    uint32_t mag = c & 0x7Fu;
    uint32_t bits;
    if (mag >= 0x7Cu) {
        bits = (mag == 0x7Cu) ? kF32Inf : kF32NaN;
    } else if (mag >= 4u) {
        // normal: exponent field e (1..30), value (1 + m/4) 2^(e-15)
        bits = (mag << 21) + ((uint32_t)(112 + SHIFT) << 23);
    } else {
        // subnormal: m * 2^-16
        bits = __float_as_uint((float)mag * __builtin_ldexpf(1.0f, SHIFT - 16));
    }
    return __uint_as_float(bits | ((c & 0x80u) << 24));
}

// FP16 code -> value times 2^S (exact): a normal code's exponent and
// significand go into the FP32 fields (an FP16 value 2^(e-31) (1 + m/512)
// has FP32 exponent field e + 96 + S), a subnormal's significand m is
// converted and scaled (m 2^-39), Inf/NaN map to Inf/NaN.  S = 0 gives the
// plain value (every FP16 value is an FP32 value), S = 96 the scaled domain.
template <int S>
__device__ __forceinline__ float fp16_to_f32_pow2(uint32_t c) {
    const uint32_t e = (c >> 9) & 63u, m = c & 511u;
    uint32_t bits;
    if (e == 63u) {
        bits = m ? kF32NaN : kF32Inf;
    } else if (e == 0u) {
        bits = __float_as_uint((float)m * __builtin_ldexpf(1.0f, S - 39));
    } else {
        bits = ((c & 0x7FFFu) << 14) + ((uint32_t)(96 + S) << 23);
    }
    return __uint_as_float(bits | ((c & 0x8000u) << 16));
}

// FP16 code -> plain float.
__device__ __forceinline__ float fp16_to_f32(uint32_t c) { return fp16_to_f32_pow2<0>(c); }

// FP16 code -> scaled-domain float (value * 2^96).
__device__ __forceinline__ float fp16_to_f32s(uint32_t c) { return fp16_to_f32_pow2<96>(c); }

// Scaled-domain float already on the FP16 grid (low 14 bits zero) -> code.
__device__ __forceinline__ uint16_t f32s_to_fp16(float x) {
    uint32_t u = __float_as_uint(x);
    uint32_t s = (u >> 16) & 0x8000u;
    uint32_t a = u & 0x7FFFFFFFu;
    if (a > kF32Inf) return kFp16NaN;
    if (a >= (193u << 23))                       // >= 2^-30 (scaled 2^66)
        return (uint16_t)(s | ((a >> 14) - (192u << 9)));
    uint32_t k = (uint32_t)(__uint_as_float(a) * 0x1p-57f);   // subnormal
    return (uint16_t)(s | k);
}

// Float in the domain scaled by 2^S, already on the FP16 grid -> code
// (S = 96: the scaled domain above; S = 0: plain values).  An FP16 value 2^(e-31) (1 + m/512) has FP32 exponent
// field e + S + 96 there.
template <int S>
__device__ __forceinline__ uint16_t f32d_to_fp16(float x) {
    uint32_t u = __float_as_uint(x);
    uint32_t s = (u >> 16) & 0x8000u;
    uint32_t a = u & 0x7FFFFFFFu;
    if (a > kF32Inf) return kFp16NaN;
    if (a >= (uint32_t)(S + 159) << 23) return (uint16_t)(s | kFp16Inf);   // >= 2^(32+S)
    if (a >= (uint32_t)(S + 97) << 23)                                      // >= 2^(S-30)
        return (uint16_t)(s | ((a >> 14) - ((uint32_t)(S + 96) << 9)));
    uint32_t k = (uint32_t)(__uint_as_float(a) * __builtin_ldexpf(1.0f, 39 - S));
    return (uint16_t)(s | k);
}

// FP16 code of a plain value that is already on the FP16 grid and below
// 2^32 in magnitude -- what the exact mode's guarded path holds; a piece in
// which a value left that range fails the guard and is recomputed on the
// safe path, which overwrites whatever this wrote.  x 2^-96 is exact in
// FP32 (FP32's exponent bias exceeds FP16's by 96): for normal FP16 values
// (from 2^-30) its exponent field is the FP16 one (1 .. 62 below 2^32) and
// its top 9 significand bits the FP16 ones; for subnormal ones (m 2^-39) it
// is the FP32 subnormal m 2^14 2^-149 (denormals are kept).  Either way its
// bits 14 .. 28 are the code's exponent and significand and bit 31 its sign:
// the same codes as f32d_to_fp16<0> in that range, without its
// Inf/NaN/overflow cases, in 4 instructions.  The code comes in the low 16
// bits of a 32-bit word whose upper bits are zero (callers pack two codes
// without masking).
__device__ __forceinline__ uint32_t f32g_to_fp16(float x) {
    const uint32_t b = __float_as_uint(x * 0x1p-96f);
    return ((b >> 14) & 0x7FFFu) | ((b >> 16) & 0xFFFF8000u);
}

// FP16 code of a GEMM result in the domain scaled by 2^DOM: 0 is the
// guarded epilogues' plain domain, whose values are on the FP16 grid and
// below 2^32 wherever they are kept (f32g_to_fp16), 96 the safe path's.
template <int DOM>
__device__ __forceinline__ uint32_t fp16_code(float x) {
    if constexpr (DOM == 0) return f32g_to_fp16(x);
    else return f32d_to_fp16<DOM>(x);
}

// Round to a 10-bit significand, ties to even, by Veltkamp splitting
// (c = x (2^14 + 1), hi = c - (c - x)): three full-rate VALU operations.
// Valid when x (2^14 + 1) neither overflows nor leaves the normal range --
// for the GEMM's guarded path (|x| in [2^-39, 2^31] or 0) it always holds.
// Equality with integer round-to-nearest-even is checked exhaustively over
// whole binades of both signs in the tests.
__device__ __forceinline__ float rn16v(float x) {
    const float c = x * 16385.0f;
    const float d = c - x;
    return c - d;
}

// A product of two FP16 values rounded to FP16, nearest even (Sec. 2.3 /
// Fig. 3(a) with FP16 multiplication).  The exact product has at most 20
// significant bits, so the float product p is exact.  Plain values: adding
// 1.5 x 2^(E + 14), E the exponent of p clamped below at -30, puts the last
// kept bit of p at float's last bit (10 significant bits, or the fixed step
// 2^-39 of FP16's subnormal range below 2^-30), and subtracting it again is
// exact.  Valid for |p| < 2^100.
__device__ __forceinline__ float rn16_product(float p) {
    uint32_t e = __float_as_uint(p) & 0x7F800000u;
    e = e > (97u << 23) ? e : (97u << 23);
    const float magic = __uint_as_float(e + (14u << 23) + 0x00400000u);
    return (p + magic) - magic;
}

// The same for a product held scaled by 2^64 (operands scaled by 2^48 and
// 2^16), returned in the 2^96 domain.  The exponent that sets the magic
// number is clamped to [34, 113]: 34 is FP16's 2^-30 there, and a product
// above 2^113 (2^49 unscaled) overflows FP16 anyway -- the clamp only keeps
// the magic number finite.  Zero, Inf and NaN pass through, and FP16
// overflow becomes FP32 overflow in the final exact scaling by 2^32.
// Compare-free: a select per product would hold a lane mask per output.
__device__ __forceinline__ float rn16_product_s(float p) {
    uint32_t e = __float_as_uint(p) & 0x7F800000u;
    e = min(max(e, 161u << 23), 240u << 23);
    const float magic = __uint_as_float(e + (14u << 23) + 0x00400000u);
    return ((p + magic) - magic) * 0x1p32f;
}

// max(m, |a|, |b|) in one instruction (the compiler splits the fmaxf form
// into two or three).  For the GEMM guards: a NaN operand may or may not reach
// the result, and either way the guarded and safe paths give the same bits.
__device__ __forceinline__ float max3_abs(float m, float a, float b) {
    float r;
    asm("v_max3_f32 %0, %1, |%2|, |%3|" : "=v"(r) : "v"(m), "v"(a), "v"(b));
    return r;
}

// Plain float -> nearest FP16 code, ties to even; overflow -> Inf.
__device__ __forceinline__ uint16_t f32_to_fp16_rn(float x) {
    uint32_t u = __float_as_uint(x);
    uint32_t s = (u >> 16) & 0x8000u;
    uint32_t a = u & 0x7FFFFFFFu;
    if (a > kF32Inf) return kFp16NaN;
    if (a >= (97u << 23)) {                      // >= 2^-30: normal range
        uint32_t b = (a + 0x1FFFu + ((a >> 14) & 1u)) & 0xFFFFC000u;
        if (b >= (159u << 23)) return (uint16_t)(s | kFp16Inf);   // >= 2^32
        return (uint16_t)(s | ((b >> 14) - (96u << 9)));
    }
    // below 2^-30 the step is 2^-39: round |x| * 2^39 to an integer (<= 512)
    float t = __builtin_rintf(__uint_as_float(a) * 0x1p39f);
    return (uint16_t)(s | (uint32_t)t);
}

// Plain float -> nearest FP8 code, ties to even, gradual underflow below
// 2^-14, finite overflow saturating at 57344, Inf -> Inf, NaN -> 0x7F.
// The E5M2 conversion instruction rounds to nearest even with gradual
// underflow but turns finite overflow into Inf, so finite values are first
// clamped to +-57344 (magnitudes in [57344, 61440) round to 57344 anyway, and
// larger ones saturate there) and Inf / NaN get their codes explicitly.  This
// equals the integer definition (bias-15 exponent, mantissa rounded at bit
// 21, subnormal quantum 2^-16) on every one of the 2^32 float inputs; the
// tests compare it with the oracle over every exponent and sign.
__device__ __forceinline__ uint32_t fp8_special(uint32_t u) {
    const uint32_t a = u & 0x7FFFFFFFu;
    return a > kF32Inf ? kFp8NaN : (0x7Cu | ((u >> 24) & 0x80u));
}

__device__ __forceinline__ uint32_t f32_to_fp8(float x) {
    const float y = __builtin_amdgcn_fmed3f(x, -57344.0f, 57344.0f);
    const uint32_t r = __builtin_amdgcn_cvt_pk_bf8_f32(y, y, 0, false) & 0xFFu;
    const uint32_t u = __float_as_uint(x);
    return (u & 0x7FFFFFFFu) >= kF32Inf ? fp8_special(u) : r;
}

// Codes of x0, x1 into bytes 0, 1 (HI = false) or 2, 3 (HI = true) of old,
// whose other half is kept: one conversion instruction for two values.
template <bool HI>
__device__ __forceinline__ uint32_t f32x2_to_fp8x2(float x0, float x1, uint32_t old) {
    const float y0 = __builtin_amdgcn_fmed3f(x0, -57344.0f, 57344.0f);
    const float y1 = __builtin_amdgcn_fmed3f(x1, -57344.0f, 57344.0f);
    uint32_t r = __builtin_amdgcn_cvt_pk_bf8_f32(y0, y1, old, HI);
    const uint32_t u0 = __float_as_uint(x0), u1 = __float_as_uint(x1);
    if (__builtin_expect(((u0 & 0x7FFFFFFFu) >= kF32Inf) | ((u1 & 0x7FFFFFFFu) >= kF32Inf), 0)) {
        constexpr int sh = HI ? 16 : 0;
        const uint32_t c0 = (u0 & 0x7FFFFFFFu) >= kF32Inf ? fp8_special(u0) : (r >> sh) & 0xFFu;
        const uint32_t c1 = (u1 & 0x7FFFFFFFu) >= kF32Inf ? fp8_special(u1) : (r >> (sh + 8)) & 0xFFu;
        r = (r & ~(0xFFFFu << sh)) | (c0 << sh) | (c1 << (sh + 8));
    }
    return r;
}

// FP8 code of an FP16 result held as a float on the FP16 grid scaled by 2^S:
// Q8(RN32(value * scale)), the same as quantizing the result's FP16 code.
template <int S>
__device__ __forceinline__ uint32_t f32d_to_fp8_scaled(float x, float scale) {
    const float v = S ? x * __builtin_ldexpf(1.0f, -S) : x;     // exact
    return f32_to_fp8(v * scale);
}

// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11).
struct u32x4 { uint32_t x, y, z, w; };

// a ^ b ^ k in one instruction (gfx950's three-input bit operation; 0x96 is
// the truth table of a three-way exclusive or), k wave-uniform.
__device__ __forceinline__ uint32_t xor3_vvs(uint32_t a, uint32_t b, uint32_t k) {
    uint32_t r;
    asm("v_bitop3_b32 %0, %1, %2, %3 bitop3:0x96" : "=v"(r) : "v"(a), "v"(b), "s"(k));
    return r;
}

__device__ __forceinline__ u32x4 philox4x32_10(u32x4 c, uint32_t k0, uint32_t k1) {
    const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
    const uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        // one 32 x 32 -> 64-bit multiply gives both halves of each product
        const uint64_t p0 = (uint64_t)M0 * c.x;
        const uint64_t p1 = (uint64_t)M1 * c.z;
        u32x4 n;
        n.x = xor3_vvs((uint32_t)(p1 >> 32), c.y, k0);
        n.y = (uint32_t)p1;
        n.z = xor3_vvs((uint32_t)(p0 >> 32), c.w, k1);
        n.w = (uint32_t)p0;
        c = n;
        k0 += W0;
        k1 += W1;
    }
    return c;
}

// Stochastic rounding of a plain float into FP16 (Eq. (1), k' = 23, k = 9):
// round the magnitude up by one step with probability F / 2^16, where F is
// the discarded fraction of a step scaled to 16 bits; u16 is uniform on
// [0, 2^16).  Returns the rounded value as a float and its code.
struct sr_result { float value; uint16_t code; };

__device__ __forceinline__ sr_result sr16(float x, uint32_t u16) {
    uint32_t u = __float_as_uint(x);
    uint32_t s = u & 0x80000000u;
    uint32_t a = u & 0x7FFFFFFFu;
    sr_result r;
    if (a > kF32Inf) { r.value = __uint_as_float(kF32NaN); r.code = kFp16NaN; return r; }
    if (a >= (97u << 23)) {
        // normal FP16 range: 14 discarded bits D; F = 4 * D
        uint32_t up = (u16 < ((a & 0x3FFFu) << 2)) ? 0x4000u : 0u;
        uint32_t b = (a & 0xFFFFC000u) + up;
        if (b >= (159u << 23)) {
            r.value = __uint_as_float(s | kF32Inf);
            r.code = (uint16_t)((s >> 16) | kFp16Inf);
        } else {
            r.value = __uint_as_float(s | b);
            r.code = (uint16_t)((s >> 16) | ((b >> 14) - (96u << 9)));
        }
        return r;
    }
    // below 2^-30: fixed step 2^-39
    float t = __uint_as_float(a) * 0x1p39f;      // exact, < 512
    float n = __builtin_floorf(t);
    uint32_t F = (uint32_t)((t - n) * 65536.0f); // exact, floor
    uint32_t k = (uint32_t)n + ((u16 < F) ? 1u : 0u);
    r.value = __uint_as_float(s | __float_as_uint((float)k * 0x1p-39f));
    r.code = (uint16_t)((s >> 16) | k);
    return r;
}

}  // namespace fp8t
