"""Benchmark of the FP8-training hot path on one MI355X.

One step = one training pass of a 3x3 convolution stage of a 50-layer
residual CNN (batch 256, 14x14, 256 -> 256 channels) lowered to GEMMs:

  1. fp8_quantize the lowered activations (50176 x 2304) and the loss-scaled
     errors (50176 x 256, scale 1024) from FP32;
  2. chunk_gemm, exact mode, CL = 64: Forward Y = X W (50176x256x2304),
     Backward dX = dY W^T (50176x2304x256), Gradient dW = X^T dY
     (2304x256x50176);
  3. the same three GEMMs in fast mode (FP8 matrix cores within a chunk);
  4. sr_weight_update of the 2304 x 256 FP16 master weights with the exact
     Gradient GEMM's FP16 output, momentum 0.9, weight decay 1e-4, writing
     the FP8 weight copy used by the next step's GEMMs.

Inputs are seeded synthetic data (workloads.conv_gemms), resident in HBM
before timing.  `value` = all chunk_gemm multiply-accumulates of a step
(3 exact + 3 fast GEMMs) / step time, in GMAC/s.  Per-kernel times come from
HIP events recorded on the stream the library launches on.

    python bench.py [--steps K] [--warmup W] [--no-cpu-baseline] [--no-extras]
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

CL = 64
METRIC = "chunk_gemm GMAC/s (exact & fast mode) + % VALU/MFMA peak; SR update GB/s"

# MI355X published figures
CUS, CLOCK_HZ = 256, 2.4e9
# FP32 vector peak 157.3 TFLOP/s = 78.6e12 lane-instructions/s (an FMA counts
# as 2 flops): 128 lanes per clock per CU for single-issue 32-bit VALU ops.
VALU_LANE_OPS = 157.3e12 / 2
HBM_BYTES_S = 8.0e12
FP8_MFMA_MAC_S = 5.0e15 / 2                             # dense FP8 5.0 PFLOP/s


# HBM traffic of the exact-mode chunk_gemm calls of one step, from two
# rocprofv3 counter passes (FETCH_SIZE, WRITE_SIZE) over this benchmark,
# calibrated by the counters of a plain device copy of known size (fetch x2.0,
# write x1.0); average calibrated bytes per call (forward 189.9 MB,
# backward-data 300.0 MB, weight-gradient 2402.6 MB including the chunk sums
# of its shared tiles and the fold pass).  Valid only for the kernel sources
# they were measured on (EXACT_KERNEL_SOURCES): any change to them reports null.
TRAFFIC_SOURCES_SHA256 = "db50901dabab05030d5d7fa646f332cc0669e2180f3c2ded13dbd31be5b5c982"
EXACT_TRAFFIC_BYTES_PER_CALL = 963.8e6


# The sources that decide what an exact-mode chunk_gemm call runs: the VALU
# kernel, its instantiations, the planner and fold pass, the shared device code.
EXACT_KERNEL_SOURCES = ("chunk_gemm.hip", "fp8t_device.h", "fp8t_host.h", "gemm_plan.h",
                        "gemm_chain.hip", "gemm_valu.h", "gemm_valu.hip", "gemm_valu_impl.h",
                        "gemm_valu_nn.hip", "gemm_valu_nt.hip", "gemm_valu_tn.hip",
                        "gemm_valu_tt.hip")


def kernel_sources_sha256():
    import hashlib
    d = os.path.join(ROOT, "paper_1812_08011_amd", "csrc")
    h = hashlib.sha256()
    for f in sorted(os.listdir(d)):
        if f in EXACT_KERNEL_SOURCES:
            h.update(f.encode())
            with open(os.path.join(d, f), "rb") as fh:
                h.update(fh.read())
    return h.hexdigest()


def exact_peak_mac_s(cl):
    """Emulation ceiling of one exact-mode multiply-accumulate: gfx950 has no
    adder for the paper's FP16, so a MAC costs at least one FP32 FMA plus
    three more VALU ops that round the result to a 10-bit significand, and
    each chunk end adds one more add + rounding (4 ops) per output.  Priced at
    the chip's full VALU rate."""
    return VALU_LANE_OPS / (4.0 + 4.0 / cl)


def fast_peak_mac_s(cl):
    """Fast mode: min(FP8 MFMA peak, VALU epilogue of 8 ops per output per
    chunk: scale, round, add, round)."""
    return min(FP8_MFMA_MAC_S, VALU_LANE_OPS * cl / 8.0)


def sr_gemm_peak_mac_s():
    """ALU ceiling of chunk_gemm_sr: per multiply-accumulate one FP32 FMA, the
    stochastic rounding (an add and an and on the raw bits) and the uniform's
    extraction (a shift, or a half-rate bit-field extract: 1.5 on average), plus
    1/8 of a Philox4x32-10 block (20 64-bit multiplies at half rate, 20
    three-input xors, 4 complements = 64 full-rate slots): 12.5 full-rate VALU
    slots per MAC."""
    return VALU_LANE_OPS / 12.5


def p16_peak_mac_s(cl):
    """ALU ceiling of chunk_gemm_p16 (FP16 operands): per multiply-accumulate
    the product's Veltkamp rounding to FP16 (a multiply by the pre-split
    operand, an FMA and an add), the add into the chunk sum and its rounding
    (multiply, subtract, subtract): 7 VALU ops, plus the chunk end's 4 per
    output.  Priced at the chip's full VALU rate."""
    return VALU_LANE_OPS / (7.0 + 4.0 / cl)


def parse():
    p = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-extras", action="store_true",
                   help="skip the measurements outside the timed step (profiling runs)")
    p.add_argument("--cpu-seconds", type=float, default=20.0,
                   help="target wall time of the oracle sample")
    p.add_argument("--only", choices=sorted(ONLY),
                   help="run one of the measurements outside the timed step by itself and "
                        "print its JSON (profiling runs); no timed step")
    return p.parse_args()


def cpu_baseline(work, target_s):
    """The oracle, as it stands, on a bounded sample of the same workload:
    exact-mode outputs of the three GEMMs at sampled positions."""
    import oracle
    Xo = oracle.fp8_quantize(work["Xcol"])
    Wo = oracle.fp8_quantize(work["W"])
    Do = oracle.fp8_quantize(work["dY"], work["dy_scale"])
    M, K = work["Xcol"].shape
    N = work["W"].shape[1]
    gemms = [("fwd", Xo, Wo, M, N, K, 0, 0), ("dgrad", Do, Wo, M, K, N, 0, 1),
             ("wgrad", Xo, Do, K, N, M, 1, 0)]
    rng = np.random.default_rng(99)

    def run(npts):
        macs, t = 0, 0.0
        for _, A, B, m, n, k, ta, tb in gemms:
            r = rng.integers(0, m, npts)
            c = rng.integers(0, n, npts)
            t0 = time.perf_counter()
            oracle.chunk_gemm_points(A, B, CL, r, c, ta, tb)
            t += time.perf_counter() - t0
            macs += npts * k
        return macs, t

    macs, t = run(16)                                     # calibrate
    npts = int(max(16, min(400000, 16 * target_s / max(t, 1e-3))))
    macs, t = run(npts)
    cores = oracle.num_threads()
    # the same on one core, over a sample sized to take about half as long
    oracle.set_threads(1)
    try:
        n1 = int(max(16, npts * min(1.0, 0.5 / cores)))
        macs1, t1 = run(n1)
    finally:
        oracle.set_threads(cores)
    return {"value": macs / t / 1e9, "unit": "GMAC/s", "cores": cores,
            "kind": "oracle",
            "sample": f"exact mode, CL {CL}: {npts} sampled outputs of each of the forward, "
                      f"backward and gradient GEMMs ({macs / 1e6:.0f} M MAC, {t:.1f} s)",
            "single_core": {"value": macs1 / t1 / 1e9, "unit": "GMAC/s",
                            "sample": f"{n1} sampled outputs of each GEMM ({macs1 / 1e6:.0f} M MAC, "
                                      f"{t1:.1f} s)"},
            "host_cpu": host_cpu_model()}


def host_cpu_model():
    """Model name of the host CPU (from /proc/cpuinfo), for the oracle's
    timing."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def time_ms(torch, fn, reps, warm_s=0.03):
    """Average milliseconds of fn() over reps calls, from HIP events on the
    current stream (the one the library launches on), after warm-up calls
    for at least warm_s seconds (the first calls after host-side work or an
    idle gap run at lower clocks)."""
    fn()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < warm_s:
        fn()
        torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def extra_measurements(torch, fp8t, X8, D8, W8, M, N, K, u8, u16):
    """Measured outside the timed step:
    * the Backward-data GEMM (the step's largest result, 50176 x 2304) with its
      FP16 result rounded back to FP8 in the same pass (chunk_gemm_fp8, FP8
      result only) against chunk_gemm followed by fp8_quantize of the FP16
      result, both modes;
    * sr_weight_update at a 50-layer residual CNN's 25.6 M parameters
      (momentum 0.9, weight decay 1e-4, FP8 copy), against HBM;
    * chunk_gemm_sr (stochastic rounding after every FP16 addition) on the
      forward and weight-gradient shapes, against its ALU ceiling;
    * adam_update at 25.6 M parameters, against HBM;
    * one whole training step of the speech DNN (440 -> 1024 x 5 -> 6000,
      batch 256; FP8 hidden layers, FP16 last layer, loss scale 1000, SR
      update) in exact and fast mode;
    * the conv stage through the implicit lowering (Forward, Gradient) and
      col2im of its lowered error."""
    out = {}
    sr = {}
    for name, (ta, tb, m_, n_, k_, A, B) in (("fwd", (0, 0, M, N, K, X8, W8)),
                                             ("wgrad", (1, 0, K, N, M, X8, D8))):
        wb = fp8t.chunk_gemm_sr_workspace_size(ta, tb, m_, n_, k_, CL)
        ws = u8(wb) if wb else None
        C = u16(m_, n_)
        t = time_ms(torch, lambda: fp8t.chunk_gemm_sr(ta, tb, m_, n_, k_, CL, A, A.shape[1], B,
                                                      B.shape[1], C, n_, 7, 0, ws, wb), 2)
        sr[name] = {"ms": t, "tmac_s": m_ * n_ * k_ / (t * 1e-3) / 1e12,
                    "frac_of_alu_bound": m_ * n_ * k_ / (t * 1e-3) / sr_gemm_peak_mac_s(),
                    "workspace_mb": wb / 1e6}
        del ws, C
    out["sr_gemm"] = sr
    C16, C8 = u16(M, K), u8(M, K)
    for mode, tag in ((fp8t.EXACT, "exact"), (fp8t.FAST, "fast")):
        wb = fp8t.chunk_gemm_fp8_workspace_size(0, 1, M, K, N, CL, mode)
        w16b = fp8t.chunk_gemm_workspace_size(0, 1, M, K, N, CL, mode)
        ws8 = u8(wb) if wb else None
        ws16 = u8(w16b) if w16b else None
        def fused():
            fp8t.chunk_gemm_fp8(0, 1, M, K, N, CL, D8, N, W8, N, None, K, C8, K, 1.0, mode,
                                ws8, wb)

        def gemm():
            fp8t.chunk_gemm(0, 1, M, K, N, CL, D8, N, W8, N, C16, K, mode, ws16, w16b)

        def two_pass():
            gemm()
            fp8t.fp8_quantize(C16, C8)
        # the three side by side, interleaved twice, the faster of the two kept
        t = {"fused": [], "gemm_only": [], "gemm_then_quantize": []}
        for _ in range(2):
            for key, f in (("fused", fused), ("gemm_only", gemm), ("gemm_then_quantize", two_pass)):
                t[key].append(time_ms(torch, f, 10))
        out[f"dgrad_fp8_out_{tag}_ms"] = {k: min(v) for k, v in t.items()}
    n = 25_600_000
    g = torch.Generator(device="cuda")
    g.manual_seed(5)
    w16, g16, v16, w8 = u16(n), u16(n), u16(n), u8(n)
    fp8t.fp16_quantize(torch.randn(n, device="cuda", generator=g) * 0.02, w16)
    fp8t.fp16_quantize(torch.randn(n, device="cuda", generator=g) * 1e-4, g16)
    fp8t.fp16_quantize(torch.randn(n, device="cuda", generator=g) * 1e-4, v16)
    step = [0]

    def upd():
        step[0] += 1
        fp8t.sr_weight_update(w16, g16, v16, w8, n, 0.1, 0.9, 1e-4, 7, step[0])
    t = time_ms(torch, upd, 20)
    out["sr_update_25_6M"] = {"us": t * 1e3, "gb_s": 11 * n / (t * 1e-3) / 1e9,
                              "frac_of_hbm": 11 * n / (t * 1e-3) / HBM_BYTES_S}
    # ADAM: read w, g, m, v (8 B), write w, m, v (6 B) and w8 (1 B) per parameter
    m16, s16 = u16(n), u16(n)
    fp8t.fp16_quantize(torch.randn(n, device="cuda", generator=g) * 1e-4, m16)
    fp8t.fp16_quantize(torch.randn(n, device="cuda", generator=g).abs() * 1e-6, s16)
    t = time_ms(torch, lambda: fp8t.adam_update(w16, g16, m16, s16, w8, n, 1e-3, 0.9, 0.999,
                                                 1e-8, 1e-4, 10, 7, 0), 20)
    out["adam_update_25_6M"] = {"us": t * 1e3, "gb_s": 15 * n / (t * 1e-3) / 1e9,
                                "frac_of_hbm": 15 * n / (t * 1e-3) / HBM_BYTES_S}
    del w16, g16, v16, w8, m16, s16
    out["speech_dnn_step"] = mlp_measurement(torch, fp8t)
    out["conv_implicit"] = conv_measurement(torch, fp8t, W8, D8, u8, u16)
    return out


def valu_fast_peak_mac_s(cl):
    """Fast mode for chunks the matrix cores cannot split (CL not a multiple
    of 16): an FP32 FMA per MAC plus the 8-op epilogue per output per chunk."""
    return VALU_LANE_OPS / (1.0 + 8.0 / cl)


def mode_peak(mode_fast, cl, K=None):
    """Ceiling of a chunk_gemm call: CL = 1 is the single chain of CL = K in
    both modes (a one-product chunk is exact), priced as that."""
    if cl == 1 and K:
        return exact_peak_mac_s(K), "valu_emulation"
    if not mode_fast:
        return exact_peak_mac_s(cl), "valu_emulation"
    if cl % 16 == 0:
        return fast_peak_mac_s(cl), "min(fp8_mfma, valu_epilogue)"
    return valu_fast_peak_mac_s(cl), "valu_fp32"


def _p8_table():
    """FP8 (1,5,2) values of all 256 codes from the bit fields (bias 15,
    subnormals, Inf/NaN at exponent 31), for the error metric."""
    v = []
    for c in range(256):
        e, m = (c >> 2) & 31, c & 3
        x = float("nan") if e == 31 and m else float("inf") if e == 31 else \
            (m / 4.0) * 2.0 ** -14 if e == 0 else (1 + m / 4.0) * 2.0 ** (e - 15)
        v.append(-x if c & 0x80 else x)
    return v


def _p16_table():
    """FP16 (1,6,9) values of all 65536 codes from the bit fields (bias 31),
    for the error metric."""
    c = np.arange(65536, dtype=np.int64)
    e, m = (c >> 9) & 63, c & 511
    mag = np.where(e == 0, m * 2.0 ** -39, (512 + m) * np.exp2(np.maximum(e, 1) - 40.0))
    mag = np.where(e == 63, np.where(m == 0, np.inf, np.nan), mag)
    return np.where(c & 0x8000, -mag, mag)


def gemm_case(torch, fp8t, A, B, M, N, K, cl, ta, tb, reps):
    """ms, TMAC/s and fraction of each mode's ceiling of one GEMM shape."""
    C = torch.empty((M, N), dtype=torch.uint16, device="cuda")
    row = {}
    for mode, tag in ((0, "exact"), (1, "fast")):
        wb = fp8t.chunk_gemm_workspace_size(ta, tb, M, N, K, cl, mode)
        ws = torch.empty(wb, dtype=torch.uint8, device="cuda") if wb else None
        ms = time_ms(torch, lambda: fp8t.chunk_gemm(ta, tb, M, N, K, cl, A, A.shape[1], B,
                                                    B.shape[1], C, N, mode, ws, wb), reps)
        peak, kind = mode_peak(mode == 1, min(cl, K), K)
        rate = M * N * K / (ms * 1e-3)
        row[tag] = {"ms": ms, "tmac_s": rate / 1e12, "frac": rate / peak, "bound": kind,
                    "workspace_mb": wb / 1e6}
        del ws
    return row, C


def sweep_measurement(torch, fp8t):
    """The long-accumulation sweep (weight-gradient layout, 512 x 512 outputs,
    K in {4096, 16384, 65536} x CL in {1, 8, 64, 256, K}): per mode the time,
    rate and fraction of the mode's ceiling, and the normalized L2 error of
    the FP16 result against float64 dot products of the same FP8 operands
    (Sec. 2.3 Fig. 3(b), Sec. 4.2 Fig. 6: swamping at CL = 1 and CL = K,
    chunking in between)."""
    import workloads
    p8 = torch.tensor(_p8_table(), dtype=torch.float64, device="cuda")
    p16 = torch.tensor(_p16_table(), dtype=torch.float64, device="cuda")
    res = {}
    for K in workloads.SWEEP_K:
        A32, B32 = workloads.sweep_gemm(K)
        A8 = torch.empty(A32.shape, dtype=torch.uint8, device="cuda")
        B8 = torch.empty(B32.shape, dtype=torch.uint8, device="cuda")
        fp8t.fp8_quantize(torch.from_numpy(A32).cuda(), A8)
        fp8t.fp8_quantize(torch.from_numpy(B32).cuda(), B8)
        Af, Bf = p8[A8.long()], p8[B8.long()]
        ref = Af.t() @ Bf                  # float64: the products are exact
        del Af, Bf
        ref_norm = torch.linalg.vector_norm(ref).item()
        for cl in (1, 8, 64, 256, K):
            C = torch.empty((512, 512), dtype=torch.uint16, device="cuda")
            row = {}
            for mode, tag in ((0, "exact"), (1, "fast")):
                wb = fp8t.chunk_gemm_workspace_size(1, 0, 512, 512, K, cl, mode)
                ws = torch.empty(wb, dtype=torch.uint8, device="cuda") if wb else None
                ms = time_ms(torch, lambda: fp8t.chunk_gemm(1, 0, 512, 512, K, cl, A8, 512, B8,
                                                            512, C, 512, mode, ws, wb), 5)
                peak, kind = mode_peak(mode == 1, min(cl, K), K)
                rate = 512 * 512 * K / (ms * 1e-3)
                got = p16[C.view(torch.int16).long() & 0xFFFF]
                err = torch.linalg.vector_norm(got - ref).item() / ref_norm
                row[tag] = {"ms": ms, "tmac_s": rate / 1e12, "frac": rate / peak, "bound": kind,
                            "l2_err_vs_f64": err}
                del ws
            res[f"K{K}_CL{'K' if cl == K else cl}"] = row
        del ref
    return res


def small_measurement(torch, fp8t):
    """The small case: one 128 x 128 x 1024 GEMM (CL 64) and a 4096-element
    update -- launch-bound, so the time per call over many back-to-back calls
    (HIP events) is reported."""
    import workloads
    A32, B32, s = workloads.small_gemm()
    A8 = torch.empty(A32.shape, dtype=torch.uint8, device="cuda")
    B8 = torch.empty(B32.shape, dtype=torch.uint8, device="cuda")
    fp8t.fp8_quantize(torch.from_numpy(A32).cuda(), A8, s)
    fp8t.fp8_quantize(torch.from_numpy(B32).cuda(), B8, s)
    C = torch.empty((128, 128), dtype=torch.uint16, device="cuda")
    res = {}
    for mode, tag in ((0, "exact"), (1, "fast")):
        ms = time_ms(torch, lambda: fp8t.chunk_gemm(0, 0, 128, 128, 1024, CL, A8, 1024, B8, 128,
                                                    C, 128, mode), 200)
        res[f"gemm_{tag}_us"] = ms * 1e3
        res[f"gemm_{tag}_tmac_s"] = 128 * 128 * 1024 / (ms * 1e-3) / 1e12
    u = workloads.small_update()
    w16 = torch.empty(4096, dtype=torch.uint16, device="cuda")
    g16 = torch.empty(4096, dtype=torch.uint16, device="cuda")
    w8 = torch.empty(4096, dtype=torch.uint8, device="cuda")
    fp8t.fp16_quantize(torch.from_numpy(u["w"]).cuda(), w16)
    fp8t.fp16_quantize(torch.from_numpy(u["g"]).cuda(), g16)
    ms = time_ms(torch, lambda: fp8t.sr_weight_update(w16, g16, None, w8, 4096, u["lr"], 0.0,
                                                      0.0, u["seed"], 0), 200)
    res["sr_update_us"] = ms * 1e3
    return res


def speech_layers_measurement(torch, fp8t):
    """The speech DNN's 18 GEMMs at batch 256 (layers 440 -> 1024, four
    1024 -> 1024, 1024 -> 6000; forward, backward-data and weight-gradient
    each, CL 64) on their own, both modes."""
    import workloads
    res, macs = {}, 0
    for l, (fi, fo) in enumerate(workloads.SPEECH_LAYERS):
        d = workloads.speech_layer(l)
        X8 = torch.empty(d["X"].shape, dtype=torch.uint8, device="cuda")
        W8 = torch.empty(d["W"].shape, dtype=torch.uint8, device="cuda")
        E8 = torch.empty(d["E"].shape, dtype=torch.uint8, device="cuda")
        fp8t.fp8_quantize(torch.from_numpy(d["X"]).cuda(), X8)
        fp8t.fp8_quantize(torch.from_numpy(d["W"]).cuda(), W8)
        fp8t.fp8_quantize(torch.from_numpy(d["E"]).cuda(), E8, d["e_scale"])
        B = d["X"].shape[0]
        for g, (A, Bm, M, N, K, ta, tb) in (("fwd", (X8, W8, B, fo, fi, 0, 0)),
                                           ("dgrad", (E8, W8, B, fi, fo, 0, 1)),
                                           ("wgrad", (X8, E8, fi, fo, B, 1, 0))):
            res[f"L{l}_{fi}x{fo}_{g}"], _ = gemm_case(torch, fp8t, A, Bm, M, N, K, CL, ta, tb, 20)
            macs += M * N * K
    tot = {}
    for tag in ("exact", "fast"):
        ms = sum(r[tag]["ms"] for r in res.values())
        tot[tag] = {"ms": ms, "tmac_s": macs / (ms * 1e-3) / 1e12,
                    "frac": macs / (ms * 1e-3) / mode_peak(tag == "fast", CL)[0]}
    res["all_18"] = tot
    return res


def p16_last_layer_measurement(torch, fp8t):
    """chunk_gemm_p16 on the speech DNN's last layer (1024 -> 6000, batch
    256, FP16 operands as Sec. 3 keeps them): Forward, Backward (trans_b) and
    Gradient (trans_a) GEMMs, CL 64, each with its workspace."""
    import workloads
    d = workloads.speech_layer(5)

    def q16(x):
        t = torch.empty(x.shape, dtype=torch.uint16, device="cuda")
        fp8t.fp16_quantize(torch.from_numpy(x).cuda(), t)
        return t
    X16, W16, E16 = q16(d["X"]), q16(d["W"]), q16(d["E"] * np.float32(d["e_scale"]))
    res = {}
    B, (fi, fo) = d["X"].shape[0], workloads.SPEECH_LAYERS[5]
    for g, (A, Bm, M, N, K, ta, tb) in (("fwd", (X16, W16, B, fo, fi, 0, 0)),
                                       ("dgrad", (E16, W16, B, fi, fo, 0, 1)),
                                       ("wgrad", (X16, E16, fi, fo, B, 1, 0))):
        wb = fp8t.chunk_gemm_p16_workspace_size(ta, tb, M, N, K, CL)
        ws = torch.empty(wb, dtype=torch.uint8, device="cuda") if wb else None
        C = torch.empty((M, N), dtype=torch.uint16, device="cuda")
        ms = time_ms(torch, lambda: fp8t.chunk_gemm_p16(ta, tb, M, N, K, CL, A, A.shape[1], Bm,
                                                       Bm.shape[1], C, N, ws, wb), 20)
        rate = M * N * K / (ms * 1e-3)
        res[f"{M}x{N}x{K}_{g}"] = {"ms": ms, "tmac_s": rate / 1e12,
                                   "frac_of_alu_bound": rate / p16_peak_mac_s(CL),
                                   "workspace_mb": wb / 1e6}
    return res


def cpu_baseline_configs(target_s=2.0):
    """The oracle timed beside the other configurations (all host cores, a
    bounded sample each): the small GEMM and update in full, and sampled
    outputs of the sweep (K 16384, CL 64 and 1) and of the speech DNN's
    largest GEMMs (1024 -> 6000 layer)."""
    import oracle
    import workloads
    out = {}
    A32, B32, s = workloads.small_gemm()
    Ao, Bo = oracle.fp8_quantize(A32, s), oracle.fp8_quantize(B32, s)
    t0 = time.perf_counter()
    oracle.chunk_gemm(Ao, Bo, CL)
    t = time.perf_counter() - t0
    out["small_gemm_exact"] = {"us": t * 1e6, "gmac_s": 128 * 128 * 1024 / t / 1e9}
    u = workloads.small_update()
    wo, go = oracle.fp16_quantize(u["w"]), oracle.fp16_quantize(u["g"])
    t0 = time.perf_counter()
    oracle.sr_weight_update(wo, go, None, lr=u["lr"], seed=u["seed"])
    out["small_sr_update_us"] = (time.perf_counter() - t0) * 1e6

    def rate(name, A, B, M, N, K, cl, ta, tb, mode):
        rng = np.random.default_rng(98)
        npts = 4
        while True:
            r, c = rng.integers(0, M, npts), rng.integers(0, N, npts)
            t0 = time.perf_counter()
            oracle.chunk_gemm_points(A, B, cl, r, c, ta, tb, mode=mode)
            t = time.perf_counter() - t0
            if t > 0.25 * target_s or npts >= 1 << 16:
                break
            npts *= 4
        out[name] = {"gmac_s": npts * K / t / 1e9, "sample_outputs": npts}

    A32, B32 = workloads.sweep_gemm(16384)
    Ao, Bo = oracle.fp8_quantize(A32), oracle.fp8_quantize(B32)
    rate("sweep_K16384_CL64_exact", Ao, Bo, 512, 512, 16384, 64, 1, 0, oracle.EXACT)
    rate("sweep_K16384_CL1_exact", Ao, Bo, 512, 512, 16384, 1, 1, 0, oracle.EXACT)
    rate("sweep_K16384_CL64_fast", Ao, Bo, 512, 512, 16384, 64, 1, 0, oracle.FAST)
    d = workloads.speech_layer(5)
    Xo, Wo = oracle.fp8_quantize(d["X"]), oracle.fp8_quantize(d["W"])
    Eo = oracle.fp8_quantize(d["E"], d["e_scale"])
    rate("speech_L5_fwd_exact", Xo, Wo, 256, 6000, 1024, CL, 0, 0, oracle.EXACT)
    rate("speech_L5_wgrad_exact", Xo, Eo, 1024, 6000, 256, CL, 1, 0, oracle.EXACT)
    return out


def conv_measurement(torch, fp8t, W8, D8, u8, u16):
    """The conv stage's Forward and Gradient GEMMs reading the NHWC input
    directly (no lowered matrix in memory), and col2im of the lowered error."""
    import workloads
    st = workloads.conv_stage_input()
    N, H, W, C = st["X"].shape
    Cout = st["W"].shape[1]
    X8 = u8(N, H, W, C)
    fp8t.fp8_quantize(torch.from_numpy(st["X"]).cuda(), X8)
    M, K = N * H * W, 9 * C
    res = {}
    for wg, name, B, rows in ((0, "fwd", W8, M), (1, "wgrad", D8, K)):
        wb = fp8t.conv2d_workspace_size(wg, N, H, W, C, 3, 3, 1, 1, Cout, CL)
        ws = u8(wb) if wb else None
        out = u16(rows, Cout)
        f = fp8t.conv2d_wgrad_fp8 if wg else fp8t.conv2d_fwd_fp8
        t = time_ms(torch, lambda: f(X8, N, H, W, C, 3, 3, 1, 1, B, Cout, CL, out, Cout, ws, wb),
                    10)
        res[name] = {"ms": t, "tmac_s": M * K * Cout / (t * 1e-3) / 1e12,
                     "frac_of_valu_emulation_peak": M * K * Cout / (t * 1e-3) /
                     exact_peak_mac_s(CL)}
        del ws, out
    cols = u16(M, K)
    fp8t.fp16_quantize(torch.randn(M, K, device="cuda") * 1e-2, cols)
    dX = u16(N, H, W, C)
    t = time_ms(torch, lambda: fp8t.col2im_fp16(cols, N, H, W, C, 3, 3, 1, 1, dX), 5)
    res["col2im"] = {"us": t * 1e3, "gb_s": 2 * (M * K + N * H * W * C) / (t * 1e-3) / 1e9}
    return res


def mlp_measurement(torch, fp8t):
    import workloads
    from paper_1812_08011_amd.mlp import SPEECH_DNN, Fp8Mlp
    d = workloads.speech_mlp()
    res = {}
    for mode, tag in ((fp8t.EXACT, "exact"), (fp8t.FAST, "fast")):
        net = Fp8Mlp(SPEECH_DNN, 256, mode=mode)
        W16 = []
        for w in d["W"]:
            t16 = torch.empty(w.shape, dtype=torch.uint16, device="cuda")
            fp8t.fp16_quantize(torch.from_numpy(w).cuda(), t16)
            W16.append(t16.cpu().view(torch.int16).numpy().view(np.uint16))
        net.set_weights(W16)
        X8 = torch.empty(d["X"].shape, dtype=torch.uint8, device="cuda")
        fp8t.fp8_quantize(torch.from_numpy(d["X"]).cuda(), X8)
        T16 = torch.empty(d["T"].shape, dtype=torch.uint16, device="cuda")
        fp8t.fp16_quantize(torch.from_numpy(d["T"]).cuda(), T16)
        step = [0]

        def f():
            step[0] += 1
            net.step(X8, T16, d["lr"], d["momentum"], d["weight_decay"], d["loss_scale"],
                     d["seed"], step[0])
        ms = time_ms(torch, f, 10)
        res[tag] = {"ms": ms, "tmac_s": net.macs() / (ms * 1e-3) / 1e12}
        del net
    return res


# the measurements outside the timed step that --only runs by themselves
ONLY = {"sweep": lambda torch, fp8t: sweep_measurement(torch, fp8t),
        "small": lambda torch, fp8t: small_measurement(torch, fp8t),
        "speech_layers": lambda torch, fp8t: speech_layers_measurement(torch, fp8t),
        "p16_last_layer": lambda torch, fp8t: p16_last_layer_measurement(torch, fp8t)}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the path is "
              "single-GPU by design", file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_1812_08011_amd as fp8t
    import workloads

    if args.only:
        torch.cuda.set_device(0)
        fp8t.lib()
        print(json.dumps({"only": args.only, "kernels": {args.only: ONLY[args.only](torch, fp8t)}}),
              flush=True)
        return

    dev = "cuda:0"
    torch.cuda.set_device(0)
    fp8t.lib()
    work = workloads.conv_gemms()
    X32 = torch.from_numpy(work["Xcol"]).to(dev)
    W32 = torch.from_numpy(work["W"]).to(dev)
    D32 = torch.from_numpy(work["dY"]).to(dev)
    M, K = X32.shape
    N = W32.shape[1]
    u8 = lambda *s: torch.empty(*s, dtype=torch.uint8, device=dev)
    u16 = lambda *s: torch.empty(*s, dtype=torch.uint16, device=dev)
    X8, D8 = u8(M, K), u8(M, N)
    W16, V16, W8 = u16(K, N), u16(K, N), u8(K, N)
    fp8t.fp16_quantize(W32, W16)
    fp8t.fp16_quantize(torch.zeros_like(W32), V16)
    fp8t.fp8_quantize(W16, W8)
    outs = {m: (u16(M, N), u16(M, K), u16(K, N)) for m in (fp8t.EXACT, fp8t.FAST)}
    # each GEMM's workspace (chunk sums of tiles shared out over workgroups)
    shapes = {"fwd": (0, 0, M, N, K), "dgrad": (0, 1, M, K, N), "wgrad": (1, 0, K, N, M)}
    wss = {}
    for mode in (fp8t.EXACT, fp8t.FAST):
        for g, (ta, tb, m_, n_, k_) in shapes.items():
            b = fp8t.chunk_gemm_workspace_size(ta, tb, m_, n_, k_, CL, mode)
            wss[mode, g] = (u8(b) if b else None, b)
    # A plain device copy of known size (X32, read once and written once):
    # its FETCH_SIZE / WRITE_SIZE counters calibrate the traffic counters of
    # the other kernels in a profiled run.  Not part of the timed step.
    X32.clone()
    n_w = K * N
    gemm_macs = M * N * K

    names = ["quantize", "exact_fwd", "exact_dgrad", "exact_wgrad", "fast_fwd", "fast_dgrad",
             "fast_wgrad", "sr_update"]

    def step(i, ev=None):
        def mark(j):
            if ev is not None:
                ev[j].record()
        mark(0)
        fp8t.fp8_quantize(X32, X8)
        fp8t.fp8_quantize(D32, D8, work["dy_scale"])
        mark(1)
        j = 1
        for mode in (fp8t.EXACT, fp8t.FAST):
            Y, dX, dW = outs[mode]
            fp8t.chunk_gemm(0, 0, M, N, K, CL, X8, K, W8, N, Y, N, mode, *wss[mode, "fwd"])
            j += 1; mark(j)
            fp8t.chunk_gemm(0, 1, M, K, N, CL, D8, N, W8, N, dX, K, mode, *wss[mode, "dgrad"])
            j += 1; mark(j)
            fp8t.chunk_gemm(1, 0, K, N, M, CL, X8, K, D8, N, dW, N, mode, *wss[mode, "wgrad"])
            j += 1; mark(j)
        fp8t.sr_weight_update(W16, outs[fp8t.EXACT][2], V16, W8, n_w, 0.1, 0.9, 1e-4,
                              7, i)
        mark(8)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(9)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        step(args.warmup + s, evs[s])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per = {k: 0.0 for k in names}
    for s in range(args.steps):
        for j, k in enumerate(names):
            per[k] += evs[s][j].elapsed_time(evs[s][j + 1]) / 1e3
    per = {k: v / args.steps for k, v in per.items()}       # seconds per step

    step_s = wall / args.steps
    total_macs = 6 * gemm_macs
    exact_s = per["exact_fwd"] + per["exact_dgrad"] + per["exact_wgrad"]
    fast_s = per["fast_fwd"] + per["fast_dgrad"] + per["fast_wgrad"]
    upd_bytes = 11 * n_w
    q_bytes = 5 * (M * K + M * N)
    exact_avg = exact_s / 3
    exact_achieved = gemm_macs / exact_avg
    peak = exact_peak_mac_s(CL)

    result = {
        "metric": METRIC,
        "value": total_macs / step_s / 1e9,
        "unit": "GMAC/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": step_s * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp8(1,5,2) products, fp16(1,6,9) accumulation (emulated in f32+int)",
        "data": "synthetic",
        "config": {
            "workload": "resnet50-like 3x3 conv stage lowered to GEMMs: batch 256, 14x14, "
                        "256->256 ch; fwd 50176x256x2304, dgrad 50176x2304x256, wgrad "
                        "2304x256x50176; CL 64; exact + fast; SR update of 2304x256 weights",
            "global_batch": 256,
            "chunk_len": CL,
            "parallelism": "single GPU",
        },
        "roofline": {
            "kernel": "chunk_gemm exact mode (VALU kernel + fold pass), mean of the "
                      "forward, backward-data and weight-gradient calls",
            "bound": "alu",
            "achieved": exact_achieved / 1e12,
            "peak": peak / 1e12,
            "unit": "TMAC/s",
            "frac": exact_achieved / peak,
            "traffic": (EXACT_TRAFFIC_BYTES_PER_CALL
                        if kernel_sources_sha256() == TRAFFIC_SOURCES_SHA256 else None),
            "traffic_unit": "bytes per call",
        },
        "kernels": {
            "exact_gemm_gmac_s": 3 * gemm_macs / exact_s / 1e9,
            "exact_frac_of_valu_emulation_peak": 3 * gemm_macs / exact_s / peak,
            "exact_ms": {k: per[k] * 1e3 for k in ("exact_fwd", "exact_dgrad", "exact_wgrad")},
            "fast_gemm_gmac_s": 3 * gemm_macs / fast_s / 1e9,
            "fast_frac_of_fp8_mfma_peak": 3 * gemm_macs / fast_s / FP8_MFMA_MAC_S,
            "fast_frac_of_fast_bound": 3 * gemm_macs / fast_s / fast_peak_mac_s(CL),
            "fast_ms": {k: per[k] * 1e3 for k in ("fast_fwd", "fast_dgrad", "fast_wgrad")},
            "sr_update_gb_s": upd_bytes / per["sr_update"] / 1e9,
            "sr_update_us": per["sr_update"] * 1e6,
            "quantize_gb_s": q_bytes / per["quantize"] / 1e9,
        },
    }
    if not args.no_extras:
        result["kernels"].update(extra_measurements(torch, fp8t, X8, D8, W8, M, N, K, u8, u16))
        result["kernels"]["small"] = small_measurement(torch, fp8t)
        result["kernels"]["sweep"] = sweep_measurement(torch, fp8t)
        result["kernels"]["speech_layers"] = speech_layers_measurement(torch, fp8t)
        result["kernels"]["p16_last_layer"] = p16_last_layer_measurement(torch, fp8t)
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(work, args.cpu_seconds)
        if not args.no_extras:
            result["cpu_baseline"]["configs"] = cpu_baseline_configs()
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
