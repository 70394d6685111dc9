/*
 * Oracle: the P8 and P16 number formats and their rounding rules.
 * TEST INFRASTRUCTURE ONLY (see oracle.h).
 *
 * Sec. 2.2 fixes only the bit split: P8 = (1, 5, 2), P16 = (1, 6, 9).
 * Readings taken where the paper is silent:
 *   - exponent bias 2^(e-1) - 1: 15 for P8, 31 for P16;
 *   - gradual underflow (subnormals) in both formats;
 *   - the all-ones exponent field is reserved for Inf (mantissa 0) and NaN;
 *   - "nearest" rounding (Sec. 2.2, last sentence) breaks ties to even;
 *   - quantizing into P8 saturates finite overflow at the largest finite
 *     value 57344 instead of producing Inf;
 *   - a P16 result beyond the largest finite value becomes +-Inf;
 *   - NaN results use one canonical code: 0x7F (P8), 0x7F00 (P16).
 *
 * Exact values are held as (class, sign, magnitude) with the magnitude an
 * unsigned 128-bit integer in units of 2^-39, the smallest P16 step: every
 * P8 value, every P16 value and every P8 x P8 product is an integer multiple
 * of 2^-39, so sums of them are exact.
 */
#include "oracle.h"
#include "oracle_internal.h"

#include <math.h>

/* ---- exact numbers ------------------------------------------------------ */

xnum xn_zero(int sign) { xnum r = {XN_FIN, sign, 0}; return r; }

/* Decode a P8 code: value = (1 + m/4) * 2^(e - 15) for 1 <= e <= 30,
 * m * 2^-16 for e = 0, Inf/NaN for e = 31. */
xnum xn_from_p8(uint8_t c) {
    xnum r;
    unsigned e = (c >> 2) & 31u, m = c & 3u;
    r.sign = c >> 7;
    r.mag = 0;
    if (e == 31) { r.cls = m ? XN_NAN : XN_INF; return r; }
    r.cls = XN_FIN;
    if (e == 0)
        r.mag = (u128)m << 23;                 /* m * 2^-16 = m * 2^23 units */
    else
        r.mag = (u128)(4u + m) << (e + 22);    /* (4+m) * 2^(e-17)          */
    return r;
}

/* Decode a P16 code: value = (1 + m/512) * 2^(e - 31) for 1 <= e <= 62,
 * m * 2^-39 for e = 0, Inf/NaN for e = 63. */
xnum xn_from_p16(uint16_t c) {
    xnum r;
    unsigned e = (c >> 9) & 63u, m = c & 511u;
    r.sign = c >> 15;
    r.mag = 0;
    if (e == 63) { r.cls = m ? XN_NAN : XN_INF; return r; }
    r.cls = XN_FIN;
    if (e == 0)
        r.mag = (u128)m;
    else
        r.mag = (u128)(512u + m) << (e - 1);
    return r;
}

static int bitlen128(u128 x) {
    int n = 0;
    while (x) { x >>= 1; n++; }
    return n;
}

/* Round an exact number to the nearest P16 value, ties to even (the
 * round-to-nearest applied after every P16 addition, Sec. 2.2 and 2.3). */
uint16_t xn_round_p16(xnum x) {
    uint16_t s = (uint16_t)(x.sign ? 0x8000u : 0u);
    if (x.cls == XN_NAN) return 0x7F00u;
    if (x.cls == XN_INF) return (uint16_t)(s | 0x7E00u);
    if (x.mag < 512) return (uint16_t)(s | (uint16_t)x.mag);   /* subnormal */
    int L = bitlen128(x.mag);
    int sh = L - 10;                   /* keep a 10-bit significand */
    u128 q = x.mag >> sh;
    if (sh > 0) {
        u128 rem = x.mag - (q << sh);
        u128 half = (u128)1 << (sh - 1);
        if (rem > half || (rem == half && (q & 1))) q++;
        if (q == 1024) { q = 512; sh++; }
    }
    int field = sh + 1;                /* q * 2^sh units = q/512 * 2^(sh-30) */
    if (field >= 63) return (uint16_t)(s | 0x7E00u);
    return (uint16_t)(s | (field << 9) | (unsigned)(q - 512));
}

/* Exact sum; the sign of an exact zero follows IEEE round-to-nearest:
 * +0 unless both addends are -0. */
xnum xn_add(xnum x, xnum y) {
    xnum r;
    if (x.cls == XN_NAN || y.cls == XN_NAN) { r.cls = XN_NAN; r.sign = 0; r.mag = 0; return r; }
    if (x.cls == XN_INF && y.cls == XN_INF) {
        if (x.sign == y.sign) return x;
        r.cls = XN_NAN; r.sign = 0; r.mag = 0; return r;
    }
    if (x.cls == XN_INF) return x;
    if (y.cls == XN_INF) return y;
    r.cls = XN_FIN;
    if (x.sign == y.sign) {
        r.sign = x.sign;
        r.mag = x.mag + y.mag;
        return r;
    }
    if (x.mag == y.mag) { r.sign = 0; r.mag = 0; return r; }
    if (x.mag > y.mag) { r.sign = x.sign; r.mag = x.mag - y.mag; }
    else               { r.sign = y.sign; r.mag = y.mag - x.mag; }
    return r;
}

/* Exact product of two P8 values (Sec. 2.3: the operands are multiplied in
 * FP8 and the products are accumulated in FP16; every product of two P8
 * values is exactly representable, so no rounding happens here). */
xnum xn_mul_p8(uint8_t a, uint8_t b) {
    xnum x = xn_from_p8(a), y = xn_from_p8(b), r;
    r.sign = x.sign ^ y.sign;
    r.mag = 0;
    if (x.cls == XN_NAN || y.cls == XN_NAN) { r.cls = XN_NAN; r.sign = 0; return r; }
    if (x.cls == XN_INF || y.cls == XN_INF) {
        if ((x.cls == XN_FIN && x.mag == 0) || (y.cls == XN_FIN && y.mag == 0)) {
            r.cls = XN_NAN; r.sign = 0; return r;          /* Inf * 0 */
        }
        r.cls = XN_INF; return r;
    }
    r.cls = XN_FIN;
    /* both magnitudes are multiples of 2^23 units; the product in units of
     * 2^-78 is shifted back to units of 2^-39 without loss. */
    r.mag = (x.mag * y.mag) >> 39;
    return r;
}

/* Exact conversion of a double (finite or not) to an exact number.  Only
 * used for values that are integer multiples of 2^-39 and below 2^89. */
xnum xn_from_double(double d) {
    xnum r;
    r.sign = signbit(d) ? 1 : 0;
    r.mag = 0;
    if (isnan(d)) { r.cls = XN_NAN; r.sign = 0; return r; }
    if (isinf(d)) { r.cls = XN_INF; return r; }
    r.cls = XN_FIN;
    double a = fabs(d);
    if (a == 0.0) return r;
    /* a * 2^39 is an integer below 2^128; split it into two 64-bit halves */
    double s = ldexp(a, 39);
    double hi = floor(ldexp(s, -64));
    double lo = s - ldexp(hi, 64);
    r.mag = ((u128)(uint64_t)hi << 64) + (u128)(uint64_t)lo;
    return r;
}

/* ---- public format functions ------------------------------------------- */

double orc_p8_value(uint8_t code) {
    unsigned e = (code >> 2) & 31u, m = code & 3u;
    double v;
    if (e == 31) v = m ? NAN : INFINITY;
    else if (e == 0) v = ldexp((double)m, -16);
    else v = ldexp(1.0 + m / 4.0, (int)e - 15);
    return (code & 0x80) ? -v : v;
}

double orc_p16_value(uint16_t code) {
    unsigned e = (code >> 9) & 63u, m = code & 511u;
    double v;
    if (e == 63) v = m ? NAN : INFINITY;
    else if (e == 0) v = ldexp((double)m, -39);
    else v = ldexp(1.0 + m / 512.0, (int)e - 31);
    return (code & 0x8000) ? -v : v;
}

/* Round-half-even of a non-negative double t to an integer (t < 2^52). */
static double rne_int(double t) {
    double n = floor(t);
    double f = t - n;
    if (f > 0.5 || (f == 0.5 && fmod(n, 2.0) != 0.0)) n += 1.0;
    return n;
}

/* Q8: round a (finite or not) value to P8, ties to even, gradual underflow
 * below 2^-14 with step 2^-16, finite overflow saturating at 57344. */
uint8_t orc_q8(double x) {
    if (isnan(x)) return 0x7F;
    uint8_t s = signbit(x) ? 0x80 : 0x00;
    if (isinf(x)) return (uint8_t)(s | 0x7C);
    double a = fabs(x);
    /* 61440 is the midpoint between 57344 = 1.75 * 2^15 (odd significand)
     * and 2^16; from there on RNE leaves the finite range. */
    if (a >= 61440.0) return (uint8_t)(s | 0x7B);
    if (a < ldexp(1.0, -14)) {
        double n = rne_int(ldexp(a, 16));   /* 0..4; 4 is 2^-14 = code 0x04 */
        return (uint8_t)(s | (uint8_t)n);
    }
    int E;
    (void)frexp(a, &E);                    /* a = f * 2^E, f in [0.5, 1) */
    int e = E - 1;                         /* a in [2^e, 2^(e+1))        */
    double n = rne_int(ldexp(a, 2 - e));   /* significand * 4, in [4, 8] */
    if (n == 8.0) { n = 4.0; e++; }
    return (uint8_t)(s | ((e + 15) << 2) | ((int)n - 4));
}

/* RN16: round any double to the nearest P16 value, ties to even, gradual
 * underflow below 2^-30 with step 2^-39, overflow to +-Inf. */
uint16_t orc_rn16(double x) {
    if (isnan(x)) return 0x7F00u;
    uint16_t s = (uint16_t)(signbit(x) ? 0x8000u : 0u);
    if (isinf(x)) return (uint16_t)(s | 0x7E00u);
    double a = fabs(x);
    if (a < ldexp(1.0, -30)) {
        double n = rne_int(ldexp(a, 39));   /* 0..512; 512 is 2^-30 = 0x0200 */
        return (uint16_t)(s | (uint16_t)n);
    }
    int E;
    (void)frexp(a, &E);
    int e = E - 1;                          /* a in [2^e, 2^(e+1))          */
    if (e > 31) return (uint16_t)(s | 0x7E00u);
    double n = rne_int(ldexp(a, 9 - e));    /* significand * 512, [512,1024] */
    if (n == 1024.0) { n = 512.0; e++; }
    if (e > 31) return (uint16_t)(s | 0x7E00u);
    return (uint16_t)(s | ((e + 31) << 9) | ((int)n - 512));
}

uint16_t orc_add16(uint16_t x, uint16_t y) {
    return xn_round_p16(xn_add(xn_from_p16(x), xn_from_p16(y)));
}

uint16_t orc_mul8(uint8_t a, uint8_t b) {
    return xn_round_p16(xn_mul_p8(a, b));
}

/* Floating-point stochastic rounding into P16, Eq. (1) of Sec. 2.3.
 * x = s * 2^e * (1 + m) holds k' = 23 mantissa bits (an FP32 value); it is
 * rounded to k = 9 bits.  The magnitude is rounded up by one step
 * eps * 2^e = 2^(e-9) with probability (m - floor(m)) / eps, realised with a
 * 16-bit uniform u: up iff u < F, F = floor(fraction * 2^16).  Below the
 * smallest normal P16 value 2^-30 the step is the fixed subnormal step
 * 2^-39.  A result beyond the largest finite P16 value is +-Inf. */
uint16_t orc_sr16(float xf, uint32_t u16) {
    double x = (double)xf;
    if (isnan(x)) return 0x7F00u;
    uint16_t s = (uint16_t)(signbit(x) ? 0x8000u : 0u);
    if (isinf(x)) return (uint16_t)(s | 0x7E00u);
    double a = fabs(x);
    if (a == 0.0) return s;
    int E;
    (void)frexp(a, &E);                       /* floor(log2 a) = E - 1 */
    int qexp = (a < ldexp(1.0, -30)) ? -39 : (E - 1 - 9);
    double t = ldexp(a, -qexp);               /* a / step, exact        */
    double n = floor(t);
    double F = floor((t - n) * 65536.0);
    double up = ((double)u16 < F) ? 1.0 : 0.0;
    double r = ldexp(n + up, qexp);
    if (r >= ldexp(1.0, 32)) return (uint16_t)(s | 0x7E00u);
    xnum xr = xn_from_double(r);
    xr.sign = s ? 1 : 0;
    return xn_round_p16(xr);                  /* exact: r is a P16 value */
}
