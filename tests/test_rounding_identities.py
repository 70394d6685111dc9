"""Rounding identities the GPU kernels rely on, checked on the host in IEEE
single precision (numpy float32 arithmetic rounds to nearest even, as the
VALU does).  These pin the device algorithms, not the oracle."""
import numpy as np


def rne_significand10(u):
    """Integer round-to-nearest-even of float32 bit patterns to 10 significant
    bits: add half an ulp minus one plus the kept LSB, clear 14 bits."""
    return (u + np.uint32(0x1FFF) + ((u >> 14) & np.uint32(1))) & np.uint32(0xFFFFC000)


def veltkamp10(x):
    """c = x (2^14 + 1); hi = c - (c - x), each step rounded to float32."""
    c = (x * np.float32(16385.0)).astype(np.float32)
    d = (c - x).astype(np.float32)
    return (c - d).astype(np.float32)


def test_veltkamp_split_is_round_to_nearest_even_on_whole_binades():
    """Exhaustive over every significand of binades spanning the exact GEMM's
    guarded domain (unscaled FP16 values: normal from 2^-30 up to the 2^31
    bound of the guard), both signs; ties (frequent for sums of FP8 products)
    must go to even."""
    m = np.arange(1 << 23, dtype=np.uint32)
    for e in (127 - 30, 127 - 1, 127, 127 + 30):
        for sign in (0, 1):
            u = (np.uint32(sign) << np.uint32(31)) | (np.uint32(e) << np.uint32(23)) | m
            x = u.view(np.float32)
            assert np.array_equal(veltkamp10(x).view(np.uint32), rne_significand10(u)), e


def test_veltkamp_split_keeps_short_values():
    """Values with at most 10 significant bits (e.g. FP16 subnormal sums,
    k * 2^-39 with k < 512) pass through unchanged."""
    k = np.arange(1, 1 << 10, dtype=np.float64)
    for scale in (2.0 ** -39, 2.0 ** -20, 2.0 ** 10):
        x = (k * scale).astype(np.float32)
        assert np.array_equal(veltkamp10(x), x)
        assert np.array_equal(veltkamp10(-x), -x)
    assert veltkamp10(np.float32([0.0]))[0] == 0.0
