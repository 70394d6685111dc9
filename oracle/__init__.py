"""CPU oracle for the FP8-training hot path (Wang et al., NeurIPS 2018).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import this package.  The product
path (``paper_1812_08011_amd``) never imports it, and the two share no code.

The oracle is plain C (``oracle/*.c``) doing exact integer arithmetic; this
module builds it with gcc and wraps it with ctypes over numpy arrays.
"""
import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liboracle.so")
SOURCES = ["formats.c", "philox.c", "ops.c"]

SRC_F32, SRC_P16 = 0, 1
EXACT, FAST = 0, 1

_lib = None


def build():
    """Compile the oracle into ``oracle/liboracle.so`` (always recompiles)."""
    tmp = LIB_PATH + ".tmp"
    cmd = ["gcc", "-O2", "-std=gnu11", "-fopenmp", "-fPIC", "-shared",
           "-ffp-contract=off", "-Wall", "-Wextra", "-o", tmp]
    cmd += [os.path.join(HERE, s) for s in SOURCES] + ["-lm"]
    subprocess.check_call(cmd)
    os.replace(tmp, LIB_PATH)


def lib():
    """Load the built oracle, building it first only if nothing is built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build()
        L = ctypes.CDLL(LIB_PATH)
        i64, u64, f32, vp = ctypes.c_int64, ctypes.c_uint64, ctypes.c_float, ctypes.c_void_p
        L.orc_p8_value.restype = ctypes.c_double
        L.orc_p8_value.argtypes = [ctypes.c_uint8]
        L.orc_p16_value.restype = ctypes.c_double
        L.orc_p16_value.argtypes = [ctypes.c_uint16]
        L.orc_q8.restype = ctypes.c_uint8
        L.orc_q8.argtypes = [ctypes.c_double]
        L.orc_rn16.restype = ctypes.c_uint16
        L.orc_rn16.argtypes = [ctypes.c_double]
        L.orc_add16.restype = ctypes.c_uint16
        L.orc_add16.argtypes = [ctypes.c_uint16, ctypes.c_uint16]
        L.orc_mul8.restype = ctypes.c_uint16
        L.orc_mul8.argtypes = [ctypes.c_uint8, ctypes.c_uint8]
        L.orc_sr16.restype = ctypes.c_uint16
        L.orc_sr16.argtypes = [f32, ctypes.c_uint32]
        L.orc_philox4x32_10.restype = None
        L.orc_philox4x32_10.argtypes = [vp, vp, vp]
        L.cpu_fp8_quantize.restype = ctypes.c_int
        L.cpu_fp8_quantize.argtypes = [vp, ctypes.c_int, f32, vp, i64]
        L.cpu_fp16_quantize.restype = ctypes.c_int
        L.cpu_fp16_quantize.argtypes = [vp, vp, i64]
        L.cpu_chunk_gemm.restype = ctypes.c_int
        L.cpu_chunk_gemm.argtypes = [ctypes.c_int, ctypes.c_int, i64, i64, i64, i64,
                                     vp, i64, vp, i64, vp, i64, ctypes.c_int]
        L.cpu_chunk_gemm_points.restype = ctypes.c_int
        L.cpu_chunk_gemm_points.argtypes = [ctypes.c_int, ctypes.c_int, i64, i64, i64,
                                            i64, vp, i64, vp, i64, ctypes.c_int,
                                            vp, vp, i64, vp]
        L.cpu_chunk_gemm_fast_bounds_points.restype = ctypes.c_int
        L.cpu_chunk_gemm_fast_bounds_points.argtypes = [ctypes.c_int, ctypes.c_int, i64, i64,
                                                        i64, i64, vp, i64, vp, i64,
                                                        ctypes.c_int, vp, vp, i64, vp, vp]
        u32 = ctypes.c_uint32
        L.cpu_chunk_gemm_sr.restype = ctypes.c_int
        L.cpu_chunk_gemm_sr.argtypes = [ctypes.c_int, ctypes.c_int, i64, i64, i64, i64,
                                        vp, i64, vp, i64, vp, i64, u64, u32]
        L.cpu_chunk_gemm_sr_points.restype = ctypes.c_int
        L.cpu_chunk_gemm_sr_points.argtypes = [ctypes.c_int, ctypes.c_int, i64, i64, i64,
                                               i64, vp, i64, vp, i64, u64, u32,
                                               vp, vp, i64, vp]
        L.cpu_sr_weight_update.restype = ctypes.c_int
        L.cpu_sr_weight_update.argtypes = [vp, vp, vp, vp, i64, f32, f32, f32, u64, u64]
        L.cpu_chunk_gemm_p16.restype = ctypes.c_int
        L.cpu_chunk_gemm_p16.argtypes = [ctypes.c_int, ctypes.c_int, i64, i64, i64, i64,
                                         vp, i64, vp, i64, vp, i64]
        L.cpu_chunk_gemm_p16_points.restype = ctypes.c_int
        L.cpu_chunk_gemm_p16_points.argtypes = [ctypes.c_int, ctypes.c_int, i64, i64, i64,
                                                i64, vp, i64, vp, i64, vp, vp, i64, vp]
        L.cpu_col2im.restype = ctypes.c_int
        L.cpu_col2im.argtypes = [vp, i64, i64, i64, i64, i64, i64, i64, i64, vp]
        L.cpu_adam_update.restype = ctypes.c_int
        L.cpu_adam_update.argtypes = [vp, vp, vp, vp, vp, i64, f32, f32, f32, f32, f32, u64,
                                      u64, u64]
        L.orc_adam_step_size.restype = f32
        L.orc_adam_step_size.argtypes = [f32, f32, f32, u64]
        L.orc_num_threads.restype = ctypes.c_int
        L.orc_num_threads.argtypes = []
        L.orc_set_threads.restype = None
        L.orc_set_threads.argtypes = [ctypes.c_int]
        _lib = L
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _check(status, what):
    if status != 0:
        raise ValueError(f"oracle {what} rejected its arguments (status {status})")


# ---- scalar helpers (vectorised over numpy arrays) -------------------------

def p8_value(codes):
    codes = np.asarray(codes, dtype=np.uint8)
    f = np.frompyfunc(lambda c: lib().orc_p8_value(int(c)), 1, 1)
    return np.asarray(f(codes)).astype(np.float64)


def p16_value(codes):
    codes = np.asarray(codes, dtype=np.uint16)
    f = np.frompyfunc(lambda c: lib().orc_p16_value(int(c)), 1, 1)
    return np.asarray(f(codes)).astype(np.float64)


def q8(x):
    x = np.asarray(x, dtype=np.float64)
    f = np.frompyfunc(lambda v: lib().orc_q8(float(v)), 1, 1)
    return np.asarray(f(x)).astype(np.uint8)


def rn16(x):
    x = np.asarray(x, dtype=np.float64)
    f = np.frompyfunc(lambda v: lib().orc_rn16(float(v)), 1, 1)
    return np.asarray(f(x)).astype(np.uint16)


def add16(x, y):
    x, y = np.broadcast_arrays(np.asarray(x, np.uint16), np.asarray(y, np.uint16))
    f = np.frompyfunc(lambda a, b: lib().orc_add16(int(a), int(b)), 2, 1)
    return np.asarray(f(x, y)).astype(np.uint16)


def mul8(a, b):
    a, b = np.broadcast_arrays(np.asarray(a, np.uint8), np.asarray(b, np.uint8))
    f = np.frompyfunc(lambda p, q: lib().orc_mul8(int(p), int(q)), 2, 1)
    return np.asarray(f(a, b)).astype(np.uint16)


def sr16(x, u):
    x, u = np.broadcast_arrays(np.asarray(x, np.float32), np.asarray(u, np.uint32))
    f = np.frompyfunc(lambda a, b: lib().orc_sr16(float(a), int(b)), 2, 1)
    return np.asarray(f(x, u)).astype(np.uint16)


def philox4x32_10(ctr, key):
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib().orc_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


# ---- the three operations ---------------------------------------------------

def fp8_quantize(src, scale=1.0):
    """FP32 (float32 array) or P16 (uint16 array) -> P8 codes (uint8)."""
    src = np.ascontiguousarray(src)
    if src.dtype == np.float32:
        fmt = SRC_F32
    elif src.dtype == np.uint16:
        fmt = SRC_P16
    else:
        raise TypeError("fp8_quantize takes float32 or uint16 (P16 codes)")
    dst = np.empty(src.shape, dtype=np.uint8)
    _check(lib().cpu_fp8_quantize(_ptr(src), fmt, float(scale), _ptr(dst), src.size),
           "fp8_quantize")
    return dst


def fp16_quantize(src):
    """float32 array -> P16 codes (uint16), round to nearest even."""
    src = np.ascontiguousarray(src, dtype=np.float32)
    dst = np.empty(src.shape, dtype=np.uint16)
    _check(lib().cpu_fp16_quantize(_ptr(src), _ptr(dst), src.size), "fp16_quantize")
    return dst


def _gemm_dims(trans_a, trans_b, A, B):
    M = A.shape[1] if trans_a else A.shape[0]
    K = A.shape[0] if trans_a else A.shape[1]
    Kb = B.shape[1] if trans_b else B.shape[0]
    N = B.shape[0] if trans_b else B.shape[1]
    if K != Kb:
        raise ValueError("inner dimensions differ")
    return M, N, K


def chunk_gemm(A, B, CL, trans_a=0, trans_b=0, mode=EXACT):
    """C = op(A) op(B) with chunk-based P16 accumulation; returns P16 codes."""
    A = np.ascontiguousarray(A, dtype=np.uint8)
    B = np.ascontiguousarray(B, dtype=np.uint8)
    M, N, K = _gemm_dims(trans_a, trans_b, A, B)
    C = np.zeros((M, N), dtype=np.uint16)
    lda = A.shape[1] if A.ndim == 2 and A.shape[1] > 0 else 1
    ldb = B.shape[1] if B.ndim == 2 and B.shape[1] > 0 else 1
    _check(lib().cpu_chunk_gemm(int(trans_a), int(trans_b), M, N, K, int(CL),
                                _ptr(A), lda, _ptr(B), ldb, _ptr(C), max(N, 1),
                                int(mode)), "chunk_gemm")
    return C


def chunk_gemm_points(A, B, CL, rows, cols, trans_a=0, trans_b=0, mode=EXACT):
    """Outputs C[rows[p], cols[p]] only."""
    A = np.ascontiguousarray(A, dtype=np.uint8)
    B = np.ascontiguousarray(B, dtype=np.uint8)
    M, N, K = _gemm_dims(trans_a, trans_b, A, B)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    cols = np.ascontiguousarray(cols, dtype=np.int64)
    out = np.zeros(rows.shape, dtype=np.uint16)
    lda = A.shape[1] if A.shape[1] > 0 else 1
    ldb = B.shape[1] if B.shape[1] > 0 else 1
    _check(lib().cpu_chunk_gemm_points(int(trans_a), int(trans_b), M, N, K, int(CL),
                                       _ptr(A), lda, _ptr(B), ldb, int(mode),
                                       _ptr(rows), _ptr(cols), rows.size, _ptr(out)),
           "chunk_gemm_points")
    return out


def chunk_gemm_fast_bounds(A, B, CL, trans_a=0, trans_b=0, rows=None, cols=None, *,
                           matrix_core):
    """(lo, hi) P16 codes bounding the fast mode's result at every output
    (rows, cols None: the whole M x N matrix, else the listed outputs), for
    chunk sums on the FP8 matrix cores (matrix_core=True) or in FP32 on the
    vector ALUs."""
    A = np.ascontiguousarray(A, dtype=np.uint8)
    B = np.ascontiguousarray(B, dtype=np.uint8)
    M, N, K = _gemm_dims(trans_a, trans_b, A, B)
    shape = (M, N) if rows is None else np.shape(rows)
    if rows is None:
        rows, cols = np.meshgrid(np.arange(M), np.arange(N), indexing="ij")
    rows = np.ascontiguousarray(rows, dtype=np.int64).ravel()
    cols = np.ascontiguousarray(cols, dtype=np.int64).ravel()
    lo = np.zeros(rows.size, dtype=np.uint16)
    hi = np.zeros(rows.size, dtype=np.uint16)
    lda = A.shape[1] if A.shape[1] > 0 else 1
    ldb = B.shape[1] if B.shape[1] > 0 else 1
    _check(lib().cpu_chunk_gemm_fast_bounds_points(int(trans_a), int(trans_b), M, N, K,
                                                   int(CL), _ptr(A), lda, _ptr(B), ldb,
                                                   int(bool(matrix_core)), _ptr(rows),
                                                   _ptr(cols), rows.size,
                                                   _ptr(lo), _ptr(hi)),
           "chunk_gemm_fast_bounds")
    return lo.reshape(shape), hi.reshape(shape)


def chunk_gemm_sr(A, B, CL, trans_a=0, trans_b=0, *, seed, offset=0):
    """chunk_gemm with stochastic rounding after every P16 addition."""
    A = np.ascontiguousarray(A, dtype=np.uint8)
    B = np.ascontiguousarray(B, dtype=np.uint8)
    M, N, K = _gemm_dims(trans_a, trans_b, A, B)
    C = np.zeros((M, N), dtype=np.uint16)
    lda = A.shape[1] if A.shape[1] > 0 else 1
    ldb = B.shape[1] if B.shape[1] > 0 else 1
    _check(lib().cpu_chunk_gemm_sr(int(trans_a), int(trans_b), M, N, K, int(CL), _ptr(A), lda,
                                   _ptr(B), ldb, _ptr(C), max(N, 1), int(seed), int(offset)),
           "chunk_gemm_sr")
    return C


def chunk_gemm_sr_points(A, B, CL, rows, cols, trans_a=0, trans_b=0, *, seed, offset=0):
    """chunk_gemm_sr at the outputs (rows[p], cols[p]) only."""
    A = np.ascontiguousarray(A, dtype=np.uint8)
    B = np.ascontiguousarray(B, dtype=np.uint8)
    M, N, K = _gemm_dims(trans_a, trans_b, A, B)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    cols = np.ascontiguousarray(cols, dtype=np.int64)
    out = np.zeros(rows.size, dtype=np.uint16)
    lda = A.shape[1] if A.shape[1] > 0 else 1
    ldb = B.shape[1] if B.shape[1] > 0 else 1
    _check(lib().cpu_chunk_gemm_sr_points(int(trans_a), int(trans_b), M, N, K, int(CL),
                                          _ptr(A), lda, _ptr(B), ldb, int(seed), int(offset),
                                          _ptr(rows), _ptr(cols), rows.size, _ptr(out)),
           "chunk_gemm_sr_points")
    return out


def chunk_gemm_p16(A, B, CL, trans_a=0, trans_b=0):
    """C = op(A) op(B) with P16 operands (uint16 codes): products rounded to
    P16, chunk-based P16 accumulation."""
    A = np.ascontiguousarray(A, dtype=np.uint16)
    B = np.ascontiguousarray(B, dtype=np.uint16)
    M, N, K = _gemm_dims(trans_a, trans_b, A, B)
    C = np.zeros((M, N), dtype=np.uint16)
    lda = A.shape[1] if A.shape[1] > 0 else 1
    ldb = B.shape[1] if B.shape[1] > 0 else 1
    _check(lib().cpu_chunk_gemm_p16(int(trans_a), int(trans_b), M, N, K, int(CL), _ptr(A), lda,
                                    _ptr(B), ldb, _ptr(C), max(N, 1)), "chunk_gemm_p16")
    return C


def chunk_gemm_p16_points(A, B, CL, rows, cols, trans_a=0, trans_b=0):
    A = np.ascontiguousarray(A, dtype=np.uint16)
    B = np.ascontiguousarray(B, dtype=np.uint16)
    M, N, K = _gemm_dims(trans_a, trans_b, A, B)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    cols = np.ascontiguousarray(cols, dtype=np.int64)
    out = np.zeros(rows.size, dtype=np.uint16)
    lda = A.shape[1] if A.shape[1] > 0 else 1
    ldb = B.shape[1] if B.shape[1] > 0 else 1
    _check(lib().cpu_chunk_gemm_p16_points(int(trans_a), int(trans_b), M, N, K, int(CL),
                                           _ptr(A), lda, _ptr(B), ldb, _ptr(rows), _ptr(cols),
                                           rows.size, _ptr(out)), "chunk_gemm_p16_points")
    return out


def sr_weight_update(w, g, v=None, *, lr, momentum=0.0, weight_decay=0.0,
                     seed=0, offset=0, want_w8=True):
    """Returns (w', v' or None, w8 or None); inputs are not modified."""
    w = np.array(w, dtype=np.uint16, copy=True)
    g = np.ascontiguousarray(g, dtype=np.uint16)
    v = None if v is None else np.array(v, dtype=np.uint16, copy=True)
    w8 = np.zeros(w.shape, dtype=np.uint8) if want_w8 else None
    _check(lib().cpu_sr_weight_update(_ptr(w), _ptr(g), _ptr(v), _ptr(w8), w.size,
                                      float(lr), float(momentum), float(weight_decay),
                                      int(seed), int(offset)), "sr_weight_update")
    return w, v, w8


def adam_update(w, g, m, v, *, lr, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0,
                t=1, seed=0, offset=0, want_w8=True):
    """Returns (w', m', v', w8 or None); inputs are not modified."""
    w = np.array(w, dtype=np.uint16, copy=True)
    g = np.ascontiguousarray(g, dtype=np.uint16)
    m = np.array(m, dtype=np.uint16, copy=True)
    v = np.array(v, dtype=np.uint16, copy=True)
    w8 = np.zeros(w.shape, dtype=np.uint8) if want_w8 else None
    _check(lib().cpu_adam_update(_ptr(w), _ptr(g), _ptr(m), _ptr(v), _ptr(w8), w.size,
                                 float(lr), float(beta1), float(beta2), float(eps),
                                 float(weight_decay), int(t), int(seed), int(offset)),
           "adam_update")
    return w, m, v, w8


def adam_step_size(lr, beta1, beta2, t):
    return float(lib().orc_adam_step_size(float(lr), float(beta1), float(beta2), int(t)))


def num_threads():
    return lib().orc_num_threads()


def set_threads(n):
    """Threads of the oracle's OpenMP loops from now on (n >= 1)."""
    lib().orc_set_threads(int(n))
