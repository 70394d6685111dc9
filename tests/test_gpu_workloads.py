"""GPU parity at the full sizes of the paper-shaped workloads, in the launch
configuration the benchmark times.  The oracle computes sampled outputs one
by one: every output of the small GEMM; otherwise two outputs in every
16 x 16 block of the output -- the smallest workgroup tile of any plan, so
every tile of the plan that ran is checked, and with it every piece of a
tile whose chunks were shared out over workgroups (each output's chain runs
through all of them) -- plus the corners and a sample of the last row and
column.  Quantization and the weight updates are compared in full."""
import numpy as np
import pytest
import torch

import oracle
import paper_1812_08011_amd as fp8t
import workloads
from tests.gpu_util import DEV, dev, gemm, host, q8, q16, say
from tests.test_gpu_kernels import abs_dot, check_fast

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fp8t.lib()
    yield


def sample_points(M, N, n, seed):
    rng = np.random.default_rng(seed)
    r = list(rng.integers(0, M, n)) + [0, 0, M - 1, M - 1, M // 2]
    c = list(rng.integers(0, N, n)) + [0, N - 1, 0, N - 1, N // 2]
    r += list(rng.integers(0, M, 16)) + [M - 1] * 16
    c += [N - 1] * 16 + list(rng.integers(0, N, 16))
    return np.array(r, np.int64), np.array(c, np.int64)


def tile_points(M, N, seed, block=16, per=2):
    """`per` random outputs inside every block x block block of the M x N
    output (clipped at the ragged edges), plus the sample of sample_points."""
    rng = np.random.default_rng(seed)
    bi, bj = np.meshgrid(np.arange(0, M, block), np.arange(0, N, block), indexing="ij")
    bi, bj = bi.ravel(), bj.ravel()
    hm, hn = np.minimum(block, M - bi), np.minimum(block, N - bj)
    r = [bi + (rng.random(bi.size) * hm).astype(np.int64) for _ in range(per)]
    c = [bj + (rng.random(bj.size) * hn).astype(np.int64) for _ in range(per)]
    r0, c0 = sample_points(M, N, 0, seed)
    return np.concatenate(r + [r0]), np.concatenate(c + [c0])


def quantize_both(x32, scale=1.0):
    """GPU fp8_quantize and the oracle's must agree bit for bit."""
    say(f"fp8_quantize {x32.shape} scale={scale}")
    g = q8(dev(x32), scale)
    o = oracle.fp8_quantize(x32, scale)
    assert np.array_equal(host(g), o)
    return g, o


def check_gemm_points(Ad, Bd, Ao, Bo, M, N, K, CL, ta, tb, seed, what):
    r, c = tile_points(M, N, seed)
    absum = None
    if r.size * K <= 30_000_000:
        # the looser sum|p| tolerance as a second check where it is cheap
        table = oracle.p8_value(np.arange(256, dtype=np.uint8)).astype(np.float32)
        va_rows = np.abs(table[(Ao.T if ta else Ao)[r, :]])          # npts x K
        vb_cols = np.abs(table[(Bo.T if tb else Bo)[:, c]])          # K x npts
        absum = np.einsum("pk,kp->p", va_rows.astype(np.float64), vb_cols.astype(np.float64))
    for mode in (fp8t.EXACT, fp8t.FAST):
        say(f"{what} chunk_gemm mode={mode} M={M} N={N} K={K} CL={CL} ta={ta} tb={tb} "
            f"({r.size} outputs checked)")
        C = host(gemm(Ad, Bd, M, N, K, CL, ta, tb, mode=mode))
        got = C[r, c]
        ref = oracle.chunk_gemm_points(Ao, Bo, CL, r, c, ta, tb, mode=mode)
        if mode == fp8t.EXACT:
            assert np.array_equal(got, ref), (what, np.flatnonzero(got != ref)[:5])
        else:
            check_fast(got, Ao, Bo, CL, ta, tb, f"{what} fast", rows=r, cols=c, Co=ref,
                       absum=absum, K=K)


def test_small_workload_full():
    A32, B32, s = workloads.small_gemm()
    Ad, Ao = quantize_both(A32, s)
    Bd, Bo = quantize_both(B32, s)
    for mode in (fp8t.EXACT, fp8t.FAST):
        say(f"small chunk_gemm mode={mode}")
        Cg = host(gemm(Ad, Bd, 128, 128, 1024, 64, mode=mode))
        Co = oracle.chunk_gemm(Ao, Bo, 64, mode=mode)
        if mode == fp8t.EXACT:
            assert np.array_equal(Cg, Co)
        else:
            check_fast(Cg, Ao, Bo, 64, 0, 0, "small fast", Co=Co,
                       absum=abs_dot(oracle.p8_value(Ao), oracle.p8_value(Bo)), K=1024)
    u = workloads.small_update()
    w16g, g16g = q16(dev(u["w"])), q16(dev(u["g"]))
    w16o, g16o = oracle.fp16_quantize(u["w"]), oracle.fp16_quantize(u["g"])
    assert np.array_equal(host(w16g), w16o) and np.array_equal(host(g16g), g16o)
    w8 = torch.zeros(4096, dtype=torch.uint8, device=DEV)
    say("small sr_weight_update")
    fp8t.sr_weight_update(w16g, g16g, None, w8, 4096, u["lr"], 0.0, 0.0, u["seed"], 0)
    ow, _, ow8 = oracle.sr_weight_update(w16o, g16o, None, lr=u["lr"], seed=u["seed"])
    assert np.array_equal(host(w16g), ow) and np.array_equal(host(w8), ow8)


@pytest.fixture(scope="module")
def conv():
    say("generating the conv-stage workload")
    return workloads.conv_gemms()


def test_conv_stage_gemms(conv):
    Xd, Xo = quantize_both(conv["Xcol"])
    Wd, Wo = quantize_both(conv["W"])
    Dd, Do = quantize_both(conv["dY"], conv["dy_scale"])
    M, K = conv["Xcol"].shape
    N = conv["W"].shape[1]
    check_gemm_points(Xd, Wd, Xo, Wo, M, N, K, 64, 0, 0, 600, "conv fwd")
    check_gemm_points(Dd, Wd, Do, Wo, M, K, N, 64, 0, 1, 601, "conv dgrad")
    check_gemm_points(Xd, Dd, Xo, Do, K, N, M, 64, 1, 0, 602, "conv wgrad")


def test_conv_stage_sr_gemms(conv):
    """chunk_gemm_sr at the conv-stage shapes, in the launch configuration the
    benchmark times (workspace from the query), on sampled outputs."""
    Xd, Xo = quantize_both(conv["Xcol"])
    Wd, Wo = quantize_both(conv["W"])
    Dd, Do = quantize_both(conv["dY"], conv["dy_scale"])
    M, K = conv["Xcol"].shape
    N = conv["W"].shape[1]
    for (Ad, Bd, Ao, Bo, m, n, k, ta, tb, what) in (
            (Xd, Wd, Xo, Wo, M, N, K, 0, 0, "fwd"),
            (Xd, Dd, Xo, Do, K, N, M, 1, 0, "wgrad")):
        wb = fp8t.chunk_gemm_sr_workspace_size(ta, tb, m, n, k, 64)
        ws = torch.empty(wb, dtype=torch.uint8, device=DEV) if wb else None
        C = torch.empty((m, n), dtype=torch.uint16, device=DEV)
        say(f"conv {what} chunk_gemm_sr {m}x{n}x{k} ws={wb}")
        fp8t.chunk_gemm_sr(ta, tb, m, n, k, 64, Ad, Ad.shape[1], Bd, Bd.shape[1], C, n, 17, 0,
                           ws, wb)
        # one output in every 64 x 64 tile (the SR kernel's tile)
        r, c = tile_points(m, n, 650 + ta, block=64, per=1)
        say(f"conv {what} chunk_gemm_sr: {r.size} outputs checked")
        ref = oracle.chunk_gemm_sr_points(Ao, Bo, 64, r, c, ta, tb, seed=17, offset=0)
        got = host(C)[r, c]
        assert np.array_equal(got, ref), (what, np.flatnonzero(got != ref)[:5])


@pytest.mark.parametrize("K", workloads.SWEEP_K)
def test_long_accumulation_sweep(K):
    A32, B32 = workloads.sweep_gemm(K)
    Ad, Ao = quantize_both(A32)
    Bd, Bo = quantize_both(B32)
    for CL in (1, 8, 64, 256, K):
        check_gemm_points(Ad, Bd, Ao, Bo, 512, 512, K, CL, 1, 0, 610 + CL % 97,
                          f"sweep K={K} CL={CL}")


@pytest.mark.parametrize("layer", range(len(workloads.SPEECH_LAYERS)))
def test_speech_dnn_layers(layer):
    d = workloads.speech_layer(layer)
    Xd, Xo = quantize_both(d["X"])
    Wd, Wo = quantize_both(d["W"])
    Ed, Eo = quantize_both(d["E"], d["e_scale"])
    fi, fo = workloads.SPEECH_LAYERS[layer]
    B = d["X"].shape[0]
    check_gemm_points(Xd, Wd, Xo, Wo, B, fo, fi, 64, 0, 0, 620 + layer, "speech fwd")
    check_gemm_points(Ed, Wd, Eo, Wo, B, fi, fo, 64, 0, 1, 630 + layer, "speech dgrad")
    check_gemm_points(Xd, Ed, Xo, Eo, fi, fo, B, 64, 1, 0, 640 + layer, "speech wgrad")


def test_big_update_full():
    u = workloads.big_update()
    n = u["w"].size
    say(f"big update: quantize n={n}")
    wg, gg, vg = q16(dev(u["w"])), q16(dev(u["g"])), q16(dev(u["v"]))
    wo, go, vo = (oracle.fp16_quantize(u[k]) for k in ("w", "g", "v"))
    assert np.array_equal(host(wg), wo) and np.array_equal(host(gg), go)
    assert np.array_equal(host(vg), vo)
    w8 = torch.zeros(n, dtype=torch.uint8, device=DEV)
    say("big sr_weight_update")
    fp8t.sr_weight_update(wg, gg, vg, w8, n, u["lr"], u["momentum"], u["weight_decay"],
                          u["seed"], u["offset"])
    ow, ov, ow8 = oracle.sr_weight_update(wo, go, vo, lr=u["lr"], momentum=u["momentum"],
                                          weight_decay=u["weight_decay"], seed=u["seed"],
                                          offset=u["offset"])
    assert np.array_equal(host(wg), ow)
    assert np.array_equal(host(vg), ov)
    assert np.array_equal(host(w8), ow8)
