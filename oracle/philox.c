/*
 * Oracle: Philox4x32-10 counter-based random numbers.
 * TEST INFRASTRUCTURE ONLY (see oracle.h).
 *
 * The paper does not say where the random bits of stochastic rounding come
 * from (Sec. 2.3 gives only the probabilities of Eq. (1)).  The random source
 * chosen here is Philox4x32 with 10 rounds as published by Salmon, Moraes,
 * Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC'11: a
 * 128-bit counter and a 64-bit key; each round multiplies counter words 0 and
 * 2 by fixed 32-bit constants, mixes the high and low product halves with the
 * other two words and the key, and the key is bumped by two Weyl constants
 * between rounds.
 */
#include "oracle.h"

static const uint32_t PHILOX_M0 = 0xD2511F53u;
static const uint32_t PHILOX_M1 = 0xCD9E8D57u;
static const uint32_t PHILOX_W0 = 0x9E3779B9u;   /* golden ratio          */
static const uint32_t PHILOX_W1 = 0xBB67AE85u;   /* sqrt(3) - 1           */

void orc_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2],
                       uint32_t out[4]) {
    uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; round++) {
        if (round > 0) { k0 += PHILOX_W0; k1 += PHILOX_W1; }
        uint64_t p0 = (uint64_t)PHILOX_M0 * c0;
        uint64_t p1 = (uint64_t)PHILOX_M1 * c2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t n0 = hi1 ^ c1 ^ k0;
        uint32_t n1 = lo1;
        uint32_t n2 = hi0 ^ c3 ^ k1;
        uint32_t n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}
