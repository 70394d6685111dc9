"""The bound behind the overflow guard of the exact-mode kernels (the chunked
dot product of Sec. 2.3, Fig. 3(a), with the paper's FP16 (1,6,9) rounding to
nearest after every addition).

The guarded kernels add FP8 products in plain FP32 registers and round with
Veltkamp splitting, which is only right while no partial sum can reach FP16's
overflow threshold.  They keep a result of the guarded path when
3 CL max|a| max|b| < 2^31 (every chunk's partial sums) and the running sums,
tracked at chunk ends, stay below 2^31 (an overflow would leave one at 2^32 or
more), which rests on three facts, pinned here:

1. one rounded addition of a non-negative x raises a non-negative FP16 sum T
   by at most 3x: RN16(T + x) - T <= 3x, checked exhaustively over every pair
   of finite non-negative FP16 values whose rounded sum is finite (a small C
   program with its own integer rounding; 1.04e9 pairs);
2. rounding is monotone and odd, so every partial sum of a chain of signed
   terms is bounded in magnitude by the same chain over the absolute values;
   with (1) each chunk's partial sum is at most 3 sum_chunk |p| (and the
   running sum at most 3 sum_c P_c <= 9 sum_k |p_k|; checked on adversarial
   and random chains through the oracle's addition);
3. Veltkamp splitting leaves FP16 subnormal sums unchanged: every partial sum
   of FP8 products is a multiple of 2^-39, so one below 2^-30 is m 2^-39 with
   m < 512 -- exact in FP32 and already an FP16 value.
"""
import os
import shutil
import subprocess
import tempfile

import numpy as np
import pytest

import oracle
from tests.helpers import p16_fraction

PAIRS_C = r"""
#include <stdint.h>
#include <stdio.h>
typedef unsigned __int128 u128;

/* value of a finite non-negative FP16 (1,6,9) code in units of 2^-39 */
static u128 units(unsigned c) {
    unsigned e = c >> 9, m = c & 511u;
    return e == 0 ? (u128)m : (u128)(512u + m) << (e - 1);
}

static int bitlen(u128 x) { int n = 0; while (x) { x >>= 1; n++; } return n; }

/* round an integer number of units to FP16: 10 significant bits, ties to
 * even; below 512 units (2^-30) the grid is one unit. Returns 0 on overflow
 * (a result of 2^32 = 2^71 units or more). */
static int rn16_units(u128 s, u128* out) {
    if (s < 512) { *out = s; return 1; }
    int sh = bitlen(s) - 10;
    u128 q = s >> sh, rem = s - (q << sh);
    if (sh > 0) {
        u128 half = (u128)1 << (sh - 1);
        if (rem > half || (rem == half && (q & 1))) q++;
    }
    u128 r = q << sh;
    if (r >= ((u128)1 << 71)) return 0;
    *out = r;
    return 1;
}

int main(void) {
    /* finite non-negative codes: exponent field 0..62 */
    const unsigned ncodes = 63u * 512u;
    unsigned long long pairs = 0, overflow = 0, bad = 0;
    double worst = 0.0;
    unsigned wt = 0, wx = 0;
    #pragma omp parallel for schedule(dynamic, 64) reduction(+:pairs, overflow, bad)
    for (unsigned t = 0; t < ncodes; t++) {
        u128 T = units(t);
        for (unsigned x = 1; x < ncodes; x++) {
            u128 X = units(x), R;
            if (!rn16_units(T + X, &R)) { overflow++; continue; }
            pairs++;
            if (R < T) { bad++; continue; }        /* never: x >= 0 */
            u128 d = R - T;
            if (d > 3 * X) bad++;
            double ratio = (double)d / (double)X;
            if (ratio > worst) {
                #pragma omp critical
                if (ratio > worst) { worst = ratio; wt = t; wx = x; }
            }
        }
    }
    printf("%llu %llu %llu %.17g %u %u\n", pairs, overflow, bad, worst, wt, wx);
    return 0;
}
"""


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc needed")
def test_one_rounded_step_adds_at_most_3x():
    with tempfile.TemporaryDirectory() as d:
        src, exe = os.path.join(d, "pairs.c"), os.path.join(d, "pairs")
        with open(src, "w") as f:
            f.write(PAIRS_C)
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-o", exe, src])
        out = subprocess.run([exe], capture_output=True, text=True, check=True,
                             timeout=300).stdout.split()
    pairs, overflow, bad = int(out[0]), int(out[1]), int(out[2])
    worst, wt, wx = float(out[3]), int(out[4]), int(out[5])
    assert pairs + overflow == (63 * 512) * (63 * 512 - 1)
    assert bad == 0
    # the bound is not loose by much: rounding up to the next grid point
    # after a term just above half a step nearly doubles the term
    assert 1.9 < worst <= 3.0, (worst, hex(wt), hex(wx))
    # the worst pair, re-evaluated with the oracle's addition
    r = oracle.add16(np.uint16(wt), np.uint16(wx))
    assert (p16_fraction(int(r)) - p16_fraction(wt)) / p16_fraction(wx) == worst


def _abs_chain_bounds(p_codes, CL):
    """Run the chunked chain on signed terms and on their magnitudes with the
    oracle's FP16 addition; return the largest |P| / T_P and |S| / T_S seen
    (T the chain over magnitudes), and the largest T_P / sum_chunk|p| and
    T_S / sum|p|."""
    val = lambda c: float(p16_fraction(int(c)))
    S, TS, sum_all = np.uint16(0), np.uint16(0), 0.0
    worst = [0.0, 0.0, 0.0, 0.0]
    for c0 in range(0, len(p_codes), CL):
        P, TP, sum_c = np.uint16(0), np.uint16(0), 0.0
        for c in p_codes[c0:c0 + CL]:
            a = np.uint16(int(c) & 0x7FFF)
            P = oracle.add16(P, np.uint16(c))
            TP = oracle.add16(TP, a)
            sum_c += val(a)
            if val(TP):
                worst[0] = max(worst[0], abs(val(P)) / val(TP))
            if sum_c:
                worst[2] = max(worst[2], val(TP) / sum_c)
        S = oracle.add16(S, P)
        TS = oracle.add16(TS, TP)
        sum_all += sum_c
        if val(TS):
            worst[1] = max(worst[1], abs(val(S)) / val(TS))
        if sum_all:
            worst[3] = max(worst[3], val(TS) / sum_all)
    return worst


def test_chains_stay_within_9x_the_sum_of_magnitudes():
    rng = np.random.default_rng(990)
    codes = []
    # random FP8 products of both signs
    # (magnitudes below 2^9, so the chains of up to 4000 terms stay finite)
    a = (rng.integers(0, 0x60, 4000) | (rng.integers(0, 2, 4000) << 7)).astype(np.uint8)
    b = (rng.integers(0, 0x60, 4000) | (rng.integers(0, 2, 4000) << 7)).astype(np.uint8)
    codes.append(oracle.mul8(a, b))
    # adversarial: each term just above half a step of the running sum, so
    # every addition rounds up (the most a rounding can add)
    T, adv = 1.0, []
    for _ in range(600):
        half = 2.0 ** (np.floor(np.log2(T)) - 10)
        x = oracle.rn16(half * 1.001)
        adv.append(int(x))
        T = float(p16_fraction(int(oracle.add16(oracle.rn16(T), x))))
    codes.append(np.array(adv, np.uint16))
    for p in codes:
        for CL in (1, 8, 64, len(p)):
            w = _abs_chain_bounds(p, CL)
            assert w[0] <= 1.0 and w[1] <= 1.0, w      # |partial| <= magnitude chain
            assert w[2] <= 3.0 and w[3] <= 9.0, w      # the 3x and 9x bounds


def veltkamp10(x):
    """The guarded kernels' rounding: c = x (2^14 + 1); hi = c - (c - x), in
    float32 arithmetic (numpy rounds to nearest even, as the VALU does)."""
    c = (x * np.float32(16385.0)).astype(np.float32)
    d = (c - x).astype(np.float32)
    return (c - d).astype(np.float32)


def test_veltkamp_keeps_fp16_subnormal_sums():
    m = np.arange(512, dtype=np.float64)
    x = (m * 2.0 ** -39).astype(np.float32)
    assert np.array_equal((x.astype(np.float64) / 2.0 ** -39), m)   # exact in FP32
    for s in (1.0, -1.0):
        y = np.float32(s) * x
        assert np.array_equal(veltkamp10(y).view(np.uint32), y.view(np.uint32))
    # and they are FP16 values: RN16 leaves them alone
    assert np.array_equal(oracle.p16_value(oracle.rn16(x.astype(np.float64))),
                          x.astype(np.float64))
