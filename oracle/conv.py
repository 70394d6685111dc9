"""Oracle for convolutions computed through a lowering and a GEMM (Sec. 2.2:
the convolution is implemented by first lowering the input data, followed by
the GEMM), and for col2im, the adjoint of the lowering.

TEST INFRASTRUCTURE ONLY, like the rest of this package.  Layouts: input X
NHWC (N, H, W, C); weights (KH KW C) x Cout, rows in (kh, kw, c) order; the
lowered matrix Xcol has rows (n, oh, ow) and columns (kh, kw, c):
    Xcol[(n, oh, ow), (kh, kw, c)] = X[n, oh*stride - pad + kh, ow*stride - pad + kw, c]
(0 outside the input).
"""
import numpy as np

from . import _check, _ptr, chunk_gemm, chunk_gemm_points, lib


def out_size(H, W, KH, KW, pad, stride):
    return (H + 2 * pad - KH) // stride + 1, (W + 2 * pad - KW) // stride + 1


def im2col(X, KH, KW, pad, stride):
    """Lowered matrix of the NHWC array X (any dtype; zeros outside)."""
    N, H, W, C = X.shape
    OH, OW = out_size(H, W, KH, KW, pad, stride)
    Xp = np.zeros((N, H + 2 * pad, W + 2 * pad, C), dtype=X.dtype)
    Xp[:, pad:pad + H, pad:pad + W, :] = X
    cols = np.zeros((N, OH, OW, KH, KW, C), dtype=X.dtype)
    for kh in range(KH):
        for kw in range(KW):
            cols[:, :, :, kh, kw, :] = Xp[:, kh:kh + stride * (OH - 1) + 1:stride,
                                          kw:kw + stride * (OW - 1) + 1:stride, :]
    return cols.reshape(N * OH * OW, KH * KW * C)


def conv2d_fwd(X8, Wt8, KH, KW, pad, stride, CL):
    """Y = Xcol W with chunk_gemm's exact mode (P16 codes, N OH OW x Cout)."""
    return chunk_gemm(im2col(X8, KH, KW, pad, stride), Wt8, CL)


def conv2d_wgrad(X8, dY8, KH, KW, pad, stride, CL):
    """dW = Xcol^T dY with chunk_gemm's exact mode (P16 codes, KH KW C x Cout)."""
    return chunk_gemm(im2col(X8, KH, KW, pad, stride), dY8, CL, 1, 0)


def conv2d_points(which, X8, B8, KH, KW, pad, stride, CL, rows, cols):
    Xcol = im2col(X8, KH, KW, pad, stride)
    if which == "fwd":
        return chunk_gemm_points(Xcol, B8, CL, rows, cols)
    return chunk_gemm_points(Xcol, B8, CL, rows, cols, 1, 0)


def col2im(cols16, N, H, W, C, KH, KW, pad, stride):
    """NHWC P16 codes: the P16 sum (ascending kh, kw) of the lowered entries of
    every input position."""
    cols16 = np.ascontiguousarray(cols16, dtype=np.uint16)
    dX = np.zeros((N, H, W, C), dtype=np.uint16)
    _check(lib().cpu_col2im(_ptr(cols16), N, H, W, C, KH, KW, pad, stride, _ptr(dX)), "col2im")
    return dX
