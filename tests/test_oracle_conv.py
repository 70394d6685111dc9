"""Pins for the oracle's convolution lowering (Sec. 2.2: a convolution is a
lowering of the input followed by a GEMM) and col2im:

* the lowered matrix equals the definition written as loops on tiny inputs,
  for strides 1 and 2 and paddings 0 and 1;
* on integer data whose sums FP16 holds exactly, the lowered Forward and
  Gradient GEMMs equal the directly computed convolution and correlation;
* col2im is the adjoint of the lowering (<col2im(G), X> = <G, Xcol>) on exact
  integer data, and adds in ascending (kh, kw) order with FP16 rounding (a
  case where the order changes the sum).
"""
import numpy as np
import pytest

import oracle
from oracle import conv


def _loops_im2col(X, KH, KW, pad, stride):
    N, H, W, C = X.shape
    OH, OW = conv.out_size(H, W, KH, KW, pad, stride)
    out = np.zeros((N * OH * OW, KH * KW * C), X.dtype)
    for n in range(N):
        for oh in range(OH):
            for ow in range(OW):
                for kh in range(KH):
                    for kw in range(KW):
                        for c in range(C):
                            ih, iw = oh * stride - pad + kh, ow * stride - pad + kw
                            if 0 <= ih < H and 0 <= iw < W:
                                out[(n * OH + oh) * OW + ow, (kh * KW + kw) * C + c] = \
                                    X[n, ih, iw, c]
    return out


@pytest.mark.parametrize("pad,stride", [(1, 1), (0, 1), (1, 2), (0, 2)])
def test_im2col_definition(pad, stride):
    rng = np.random.default_rng(1000 + 2 * pad + stride)
    X = rng.integers(0, 255, size=(2, 5, 6, 3)).astype(np.uint8)
    for KH, KW in ((3, 3), (1, 1), (2, 3)):
        assert np.array_equal(conv.im2col(X, KH, KW, pad, stride),
                              _loops_im2col(X, KH, KW, pad, stride))


def test_exact_region_convolution_and_gradient():
    rng = np.random.default_rng(1001)
    N, H, W, C, Cout, KH, KW, pad, stride = 2, 6, 5, 4, 3, 3, 3, 1, 1
    x = rng.integers(-2, 3, size=(N, H, W, C)).astype(np.float32)
    w = rng.integers(-2, 3, size=(KH * KW * C, Cout)).astype(np.float32)
    X8, W8 = oracle.fp8_quantize(x), oracle.fp8_quantize(w)
    Y = oracle.p16_value(conv.conv2d_fwd(X8, W8, KH, KW, pad, stride, 64))
    # direct convolution (cross-correlation, as the lowering defines it)
    xp = np.pad(x, ((0, 0), (pad, pad), (pad, pad), (0, 0)))
    wk = w.reshape(KH, KW, C, Cout)
    direct = np.zeros((N, H, W, Cout))
    for kh in range(KH):
        for kw in range(KW):
            direct += np.einsum("nhwc,cd->nhwd", xp[:, kh:kh + H, kw:kw + W, :], wk[kh, kw])
    assert np.array_equal(Y, direct.reshape(N * H * W, Cout))
    dy = rng.integers(-2, 3, size=(N * H * W, Cout)).astype(np.float32)
    dW = oracle.p16_value(conv.conv2d_wgrad(X8, oracle.fp8_quantize(dy), KH, KW, pad, stride, 7))
    direct_w = np.zeros((KH, KW, C, Cout))
    g = dy.reshape(N, H, W, Cout)
    for kh in range(KH):
        for kw in range(KW):
            direct_w[kh, kw] = np.einsum("nhwc,nhwd->cd", xp[:, kh:kh + H, kw:kw + W, :], g)
    assert np.array_equal(dW, direct_w.reshape(KH * KW * C, Cout))


@pytest.mark.parametrize("pad,stride", [(1, 1), (0, 2), (1, 2)])
def test_col2im_is_the_adjoint(pad, stride):
    rng = np.random.default_rng(1002 + stride)
    N, H, W, C, KH, KW = 2, 7, 6, 3, 3, 3
    OH, OW = conv.out_size(H, W, KH, KW, pad, stride)
    x = rng.integers(-3, 4, size=(N, H, W, C)).astype(np.float32)
    g = rng.integers(-3, 4, size=(N * OH * OW, KH * KW * C)).astype(np.float32)
    G16 = oracle.fp16_quantize(g)
    dX = oracle.p16_value(conv.col2im(G16, N, H, W, C, KH, KW, pad, stride))
    lhs = float(np.sum(dX * x))
    rhs = float(np.sum(g * conv.im2col(x, KH, KW, pad, stride)))
    assert lhs == rhs
    # and element by element: the sum of the entries that map to a position
    back = np.zeros((N, H, W, C))
    xp_idx = np.arange(N * H * W * C, dtype=np.float64).reshape(N, H, W, C) + 1
    where = conv.im2col(xp_idx, KH, KW, pad, stride)
    np.add.at(back.reshape(-1), (where[where > 0] - 1).astype(np.int64), g[where > 0])
    assert np.array_equal(dX, back)


def test_col2im_order():
    """Three windows cover input position (0, 1, 1) of a 1-channel 3 x 3
    image with a 3 x 1 kernel (pad 1): entries 1, 1, 1024 in ascending kh
    give 1026; the other order would give 1024 (1024 + 1 is a tie)."""
    N, H, W, C, KH, KW, pad = 1, 3, 3, 1, 3, 1, 1
    OH, OW = conv.out_size(H, W, KH, KW, pad, 1)
    g = np.zeros((OH * OW, KH * KW * C), np.float32)
    # position (1, 1) is covered by oh = 2 (kh = 0), oh = 1 (kh = 1), oh = 0
    # (kh = 2), all at ow = iw + pad = 2
    ow = 2
    g[2 * OW + ow, 0] = 1.0
    g[1 * OW + ow, 1] = 1.0
    g[0 * OW + ow, 2] = 1024.0
    dX = oracle.p16_value(conv.col2im(oracle.fp16_quantize(g), N, H, W, C, KH, KW, pad, 1))
    assert dX[0, 1, 1, 0] == 1026.0
    assert oracle.p16_value(oracle.add16(oracle.add16(oracle.rn16(1024.0), oracle.rn16(1.0)),
                                         oracle.rn16(1.0)))[()] == 1024.0
