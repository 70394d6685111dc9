/*
 * Oracle internals: exact numbers.  TEST INFRASTRUCTURE ONLY (see oracle.h).
 */
#ifndef FP8T_ORACLE_INTERNAL_H
#define FP8T_ORACLE_INTERNAL_H

#include <stdint.h>

typedef unsigned __int128 u128;

enum { XN_FIN = 0, XN_INF = 1, XN_NAN = 2 };

/* value = (-1)^sign * mag * 2^-39 when cls == XN_FIN */
typedef struct {
    int cls;
    int sign;
    u128 mag;
} xnum;

xnum     xn_zero(int sign);
xnum     xn_from_p8(uint8_t c);
xnum     xn_from_p16(uint16_t c);
xnum     xn_from_double(double d);
xnum     xn_add(xnum x, xnum y);
xnum     xn_mul_p8(uint8_t a, uint8_t b);
uint16_t xn_round_p16(xnum x);

#endif
