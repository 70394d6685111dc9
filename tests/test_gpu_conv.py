"""GPU parity of the implicitly lowered convolutions and col2im with the
oracle, bit for bit: paddings, strides, kernel sizes, channel counts that
take the 4-channel loads and those that do not, whole and shared-out tiles,
and the conv stage of the benchmark (batch 256, 14 x 14, 256 -> 256) on
sampled outputs; col2im at small sizes and on the full 50176 x 2304 lowered
error of that stage."""
import numpy as np
import pytest
import torch

import oracle
import paper_1812_08011_amd as fp8t
import workloads
from oracle import conv as oconv
from tests.gpu_util import DEV, dev, host, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fp8t.lib()
    yield


def run_conv(which, X8, B8, geom, Cout, CL):
    N, H, W, C, KH, KW, pad, stride = geom
    OH, OW = oconv.out_size(H, W, KH, KW, pad, stride)
    rows = KH * KW * C if which == "wgrad" else N * OH * OW
    wb = fp8t.conv2d_workspace_size(which == "wgrad", N, H, W, C, KH, KW, pad, stride, Cout, CL)
    ws = torch.empty(wb, dtype=torch.uint8, device=DEV) if wb else None
    out = torch.full((rows, Cout), 0xABCD, dtype=torch.uint16, device=DEV)
    f = fp8t.conv2d_wgrad_fp8 if which == "wgrad" else fp8t.conv2d_fwd_fp8
    f(X8, N, H, W, C, KH, KW, pad, stride, B8, Cout, CL, out, Cout, ws, wb)
    return host(out)


CASES = [
    # N, H, W, C, KH, KW, pad, stride, Cout, CL
    (2, 9, 7, 8, 3, 3, 1, 1, 24, 64),
    (3, 8, 8, 4, 3, 3, 1, 2, 40, 16),
    (2, 6, 11, 6, 3, 3, 0, 1, 12, 7),       # C % 4 != 0: byte loads
    (1, 5, 5, 3, 5, 5, 2, 1, 9, 13),
    (4, 7, 7, 16, 1, 1, 0, 1, 70, 64),
    (2, 10, 9, 12, 2, 3, 1, 3, 5, 5),
]


@pytest.mark.parametrize("plan", ["auto", "shared", "tile4", "tile7", "tile7-shared"])
def test_conv_fwd_and_wgrad_match_oracle(plan, monkeypatch):
    if plan.endswith("shared"):
        monkeypatch.setenv("FP8T_GEMM_SPLIT", "1")
        monkeypatch.setenv("FP8T_GEMM_WGS", "5")
    if plan.startswith("tile"):
        # the two register-tile shapes the lowered-input kernels are built for
        monkeypatch.setenv("FP8T_VALU_TILE", plan[4])
    rng = np.random.default_rng(1010)
    for (N, H, W, C, KH, KW, pad, stride, Cout, CL) in CASES:
        geom = (N, H, W, C, KH, KW, pad, stride)
        OH, OW = oconv.out_size(H, W, KH, KW, pad, stride)
        X8 = oracle.fp8_quantize(np.maximum(rng.standard_normal((N, H, W, C)), 0)
                                 .astype(np.float32))
        W8 = oracle.fp8_quantize((rng.standard_normal((KH * KW * C, Cout)) * 0.3)
                                 .astype(np.float32))
        D8 = oracle.fp8_quantize(rng.standard_normal((N * OH * OW, Cout)).astype(np.float32))
        say(f"conv2d plan={plan} geom={geom} Cout={Cout} CL={CL}")
        got = run_conv("fwd", dev(X8), dev(W8), geom, Cout, CL)
        assert np.array_equal(got, oconv.conv2d_fwd(X8, W8, KH, KW, pad, stride, CL)), geom
        got = run_conv("wgrad", dev(X8), dev(D8), geom, Cout, CL)
        assert np.array_equal(got, oconv.conv2d_wgrad(X8, D8, KH, KW, pad, stride, CL)), geom


def test_conv_misaligned_input_takes_byte_loads():
    rng = np.random.default_rng(1011)
    N, H, W, C, KH, KW, pad, stride, Cout, CL = 2, 6, 6, 8, 3, 3, 1, 1, 16, 64
    X8 = oracle.fp8_quantize(rng.standard_normal((N, H, W, C)).astype(np.float32))
    W8 = oracle.fp8_quantize(rng.standard_normal((KH * KW * C, Cout)).astype(np.float32))
    buf = torch.zeros(X8.size + 1, dtype=torch.uint8, device=DEV)
    buf[1:] = dev(X8.ravel())
    Y = torch.zeros((N * H * W, Cout), dtype=torch.uint16, device=DEV)
    say("conv2d misaligned input")
    fp8t.lib().conv2d_fwd_fp8(buf.data_ptr() + 1, N, H, W, C, KH, KW, pad, stride,
                              dev(W8).data_ptr(), Cout, CL, Y.data_ptr(), Cout, None, 0,
                              torch.cuda.current_stream().cuda_stream)
    assert np.array_equal(host(Y), oconv.conv2d_fwd(X8, W8, KH, KW, pad, stride, CL))


def test_col2im_small():
    rng = np.random.default_rng(1012)
    for (N, H, W, C, KH, KW, pad, stride) in ((2, 7, 6, 5, 3, 3, 1, 1), (1, 9, 9, 4, 3, 3, 1, 2),
                                               (3, 5, 8, 2, 2, 3, 0, 1), (2, 6, 7, 16, 3, 3, 1, 1),
                                               (1, 8, 8, 24, 3, 2, 1, 2)):
        OH, OW = oconv.out_size(H, W, KH, KW, pad, stride)
        g = oracle.fp16_quantize((rng.standard_normal((N * OH * OW, KH * KW * C)) * 100)
                                 .astype(np.float32))
        g[rng.random(g.shape) < 0.01] = 0x7E00
        dX = torch.full((N, H, W, C), 0x1111, dtype=torch.uint16, device=DEV)
        say(f"col2im {N, H, W, C, KH, KW, pad, stride}")
        fp8t.col2im_fp16(dev(g), N, H, W, C, KH, KW, pad, stride, dX)
        assert np.array_equal(host(dX), oconv.col2im(g, N, H, W, C, KH, KW, pad, stride))


@pytest.fixture(scope="module")
def stage():
    say("generating the conv-stage workload")
    return workloads.conv_stage_input()


def test_conv_stage_sampled(stage):
    X8 = oracle.fp8_quantize(stage["X"])
    W8 = oracle.fp8_quantize(stage["W"])
    D8 = oracle.fp8_quantize(stage["dY"], stage["dy_scale"])
    N, H, W, C = stage["X"].shape
    Cout = stage["W"].shape[1]
    geom = (N, H, W, C, 3, 3, 1, 1)
    Xd = dev(X8)
    rng = np.random.default_rng(1013)
    for which, B8, rows in (("fwd", W8, N * H * W), ("wgrad", D8, 9 * C)):
        say(f"conv stage {which}")
        got = run_conv(which, Xd, dev(B8), geom, Cout, 64)
        r = np.concatenate([rng.integers(0, rows, 160), [0, rows - 1]])
        c = np.concatenate([rng.integers(0, Cout, 160), [Cout - 1, 0]])
        ref = oconv.conv2d_points(which, X8, B8, 3, 3, 1, 1, 64, r, c)
        assert np.array_equal(got[r, c], ref), which


def test_col2im_conv_stage():
    rng = np.random.default_rng(1014)
    N, H, W, C = 256, 14, 14, 256
    g = oracle.fp16_quantize((rng.standard_normal((N * H * W, 9 * C)) * 1e-2)
                             .astype(np.float32))
    dX = torch.empty((N, H, W, C), dtype=torch.uint16, device=DEV)
    say("col2im conv stage")
    fp8t.col2im_fp16(dev(g), N, H, W, C, 3, 3, 1, 1, dX)
    assert np.array_equal(host(dX), oconv.col2im(g, N, H, W, C, 3, 3, 1, 1))
