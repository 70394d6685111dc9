"""Pins for the oracle's stochastic rounding (Sec. 2.3, Eq. (1)) and the FP16
SGD weight update (Sec. 2.2, Sec. 4.3).

* SR counting: for a fixed x, over all 2^16 uniforms exactly F round up,
  where F is computed from the two FP16 neighbours found by brute-force search
  (Eq. (1): round up with probability (m - floor(m)) / eps);
* the exact mean over all uniforms equals x (unbiasedness);
* Philox4x32-10 blocks agree with rocRAND's independent implementation;
* the update's mean over many offsets converges to the exact SGD step, while
  round-to-nearest loses small updates (the effect behind Table 4);
* special cases: lr = 0, no weight decay -> weights unchanged.
"""
import os
import shutil
import subprocess
import tempfile
from fractions import Fraction

import numpy as np
import pytest

import oracle
from tests import helpers as H

ALL_U = np.arange(65536, dtype=np.uint32)


def _neighbours(x):
    t = H.p16_table()
    a = abs(Fraction(float(x)))
    i, j = t.neighbours(a)
    return t.values[i], t.values[j] if j < len(t.values) else None


@pytest.mark.parametrize("x", [1.0 + 2.0 ** -11, 1.0 + 2.0 ** -12 + 2.0 ** -20,
                               -3.14159, 2.0 ** -40, 2.0 ** -31 + 2.0 ** -45,
                               -(2.0 ** -35) * 1.7, 123456.789, 0.1, -1e-7])
def test_sr_counts_match_eq1(x):
    x32 = np.float32(x)
    codes = oracle.sr16(np.full(65536, x32), ALL_U)
    lo, hi = _neighbours(x32)
    a = abs(Fraction(float(x32)))
    vals = [abs(H.to_fraction16(c)) for c in np.unique(codes)]
    assert set(vals) <= {lo, hi}
    frac = (a - lo) / (hi - lo)
    F = int(frac * 65536)                      # floor
    ups = int(np.sum(np.array([abs(H.to_fraction16(c)) for c in codes]) == hi)) if hi != lo else 0
    assert ups == F
    if lo != hi and (frac * 65536).denominator == 1:
        # exact mean over the whole uniform space is x itself
        total = sum((hi if abs(H.to_fraction16(c)) == hi else lo) for c in codes)
        assert total / 65536 == a
    # sign is kept
    assert np.all((codes & 0x8000) == (0x8000 if x32 < 0 else 0))


def test_sr_deterministic_on_representable_values():
    rng = np.random.default_rng(400)
    c = rng.integers(0, 0x7E00, 3000).astype(np.uint16)
    c |= (rng.integers(0, 2, 3000) << 15).astype(np.uint16)
    vals = oracle.p16_value(c).astype(np.float32)
    u = rng.integers(0, 65536, 3000)
    out = oracle.sr16(vals, u)
    nz = (c & 0x7FFF) != 0
    assert np.array_equal(out[nz], c[nz])


def test_sr_unbiased_across_ranges():
    """For FP32 inputs in the normal FP16 range the 14 discarded mantissa bits
    make F exact, so the mean over all 2^16 uniforms equals x exactly."""
    rng = np.random.default_rng(401)
    for x in (rng.standard_normal(20) * np.exp2(rng.uniform(-25, 25, 20))).astype(np.float32):
        codes = oracle.sr16(np.full(65536, x), ALL_U)
        vals = oracle.p16_value(codes)
        assert Fraction(float(np.sum(vals))) / 65536 == Fraction(float(x))


def test_sr_overflow_and_specials():
    big = np.float32(4290772992.0 * 1.0009)
    codes = oracle.sr16(np.full(65536, big), ALL_U)
    assert set(np.unique(codes).tolist()) <= {0x7DFF, 0x7E00}
    assert int(oracle.sr16(np.float32(1e20), 0)) == 0x7E00
    assert int(oracle.sr16(np.float32(-np.inf), 0)) == 0xFE00
    assert int(oracle.sr16(np.float32(np.nan), 0)) == 0x7F00
    assert int(oracle.sr16(np.float32(-0.0), 7)) == 0x8000


ROCRAND_REF = r"""
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>
int main() {
  unsigned long long seed, pair, off;
  while (scanf("%llu %llu %llu", &seed, &pair, &off) == 3) {
    rocrand_device::philox4x32_10_engine e(seed, off, 4ull * pair);
    uint4 r = e.next4();
    printf("%u %u %u %u\n", r.x, r.y, r.z, r.w);
  }
  return 0;
}
"""


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="hipcc needed to build the rocRAND reference")
def test_philox_matches_rocrand_header():
    """rocRAND's header-only Philox4x32-10 engine, seeded with (seed,
    subsequence = offset, skip = 4 * pair), produces the raw block for
    counter (pair, offset) and key seed -- an independent implementation."""
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    rng = np.random.default_rng(402)
    cases = [(0, 0, 0), (1, 0, 0), (7, 12345, 3), (2 ** 64 - 1, 2 ** 40 + 5, 2 ** 63 + 9)]
    cases += [(int(rng.integers(0, 2 ** 63)), int(rng.integers(0, 2 ** 60)),
               int(rng.integers(0, 2 ** 63))) for _ in range(200)]
    with tempfile.TemporaryDirectory() as d:
        src = os.path.join(d, "ref.cpp")
        exe = os.path.join(d, "ref")
        with open(src, "w") as f:
            f.write(ROCRAND_REF)
        subprocess.check_call([hipcc, "-O1", "--offload-arch=gfx950", src, "-o", exe],
                              stdout=subprocess.DEVNULL, stderr=subprocess.DEVNULL)
        inp = "".join(f"{s} {p} {o}\n" for s, p, o in cases)
        out = subprocess.run([exe], input=inp, capture_output=True, text=True, check=True).stdout
    ref = [list(map(int, line.split())) for line in out.strip().splitlines()]
    assert len(ref) == len(cases)
    for (s, p, o), r in zip(cases, ref):
        ctr = [p & 0xFFFFFFFF, p >> 32, o & 0xFFFFFFFF, o >> 32]
        key = [s & 0xFFFFFFFF, s >> 32]
        assert oracle.philox4x32_10(ctr, key).tolist() == r


def test_update_identity_cases():
    rng = np.random.default_rng(403)
    w = oracle.rn16(rng.standard_normal(1000) * 0.05)
    g = oracle.rn16(rng.standard_normal(1000) * 1e-3)
    w1, v1, w8 = oracle.sr_weight_update(w, g, lr=0.0, seed=3)
    assert np.array_equal(w1, w) and v1 is None
    assert np.array_equal(w8, oracle.fp8_quantize(w))
    # momentum 0 with a buffer: v' = g' = g (deterministic: g is FP16)
    v = oracle.rn16(rng.standard_normal(1000) * 1e-3)
    w1, v1, _ = oracle.sr_weight_update(w, g, v, lr=0.0, momentum=0.0, seed=3)
    assert np.array_equal(v1, g) and np.array_equal(w1, w)
    with pytest.raises(ValueError):
        oracle.sr_weight_update(w, g, None, lr=0.1, momentum=0.9)


def test_update_mean_converges_to_exact_step():
    """The mean of the stochastically rounded update over independent offsets
    approaches the exact SGD step (within 5 standard errors)."""
    rng = np.random.default_rng(404)
    n, reps = 64, 4000
    w = oracle.rn16(rng.standard_normal(n) * 0.05)
    g = oracle.rn16(rng.standard_normal(n) * 1e-3)
    v = oracle.rn16(rng.standard_normal(n) * 1e-3)
    lr, mu, wd = 0.1, 0.9, 1e-4
    wf, gf, vf = (oracle.p16_value(t) for t in (w, g, v))
    exact_v = mu * vf + (gf + wd * wf)
    exact_w = wf - lr * exact_v
    acc_w = np.zeros(n)
    acc_v = np.zeros(n)
    sq = np.zeros(n)
    for o in range(reps):
        w1, v1, _ = oracle.sr_weight_update(w, g, v, lr=lr, momentum=mu, weight_decay=wd,
                                            seed=11, offset=o, want_w8=False)
        x = oracle.p16_value(w1)
        acc_w += x
        sq += x * x
        acc_v += oracle.p16_value(v1)
    mean = acc_w / reps
    sd = np.sqrt(np.maximum(sq / reps - mean ** 2, 0)) + 1e-30
    ulp = np.abs(exact_w) * 2.0 ** -9
    assert np.all(np.abs(mean - exact_w) <= 5 * sd / np.sqrt(reps) + 1e-3 * ulp)
    assert np.all(np.abs(acc_v / reps - exact_v) <= np.abs(exact_v) * 2.0 ** -9)


def test_small_updates_survive_sr_but_vanish_under_nearest():
    """Sec. 4.3 / Table 4: gradients far below half a step of the weights are
    lost by round-to-nearest FP16 updates but kept on average by SR."""
    w = oracle.rn16(np.full(256, 1.0))
    g = oracle.rn16(np.full(256, 2.0 ** -9 * 0.1 / 0.1))   # lr*g = 0.1 step
    lr = 0.1
    # nearest rounding: 1 - 0.1 * 2^-9 rounds back to 1 every time
    nr = oracle.rn16(np.float64(1.0) - lr * 2.0 ** -9)
    assert int(nr) == int(w[0])
    cur = w.copy()
    for step in range(40):
        cur, _, _ = oracle.sr_weight_update(cur, g, lr=lr, seed=5, offset=step, want_w8=False)
    moved = 1.0 - oracle.p16_value(cur).mean()
    expect = 40 * lr * 2.0 ** -9
    assert abs(moved - expect) < 0.35 * expect


def test_update_is_a_pure_function_of_offset():
    """Restarting from a saved state reproduces the same trajectory."""
    rng = np.random.default_rng(405)
    w = oracle.rn16(rng.standard_normal(300) * 0.05)
    g = oracle.rn16(rng.standard_normal(300) * 1e-3)
    v = oracle.rn16(np.zeros(300))
    traj = []
    cw, cv = w, v
    for s in range(6):
        cw, cv, _ = oracle.sr_weight_update(cw, g, cv, lr=0.1, momentum=0.9, seed=9, offset=s)
        traj.append(cw)
    cw, cv = traj[2], None
    # rebuild v at step 3 by replaying the first three steps
    rw, rv = w, v
    for s in range(3):
        rw, rv, _ = oracle.sr_weight_update(rw, g, rv, lr=0.1, momentum=0.9, seed=9, offset=s)
    for s in range(3, 6):
        rw, rv, _ = oracle.sr_weight_update(rw, g, rv, lr=0.1, momentum=0.9, seed=9, offset=s)
        assert np.array_equal(rw, traj[s])
