// chunk_gemm: FP8 x FP8 GEMM with chunk-based FP16 accumulation
// (Sec. 2.3 "Chunk-based Accumulation", dot-product algorithm of Fig. 3(a)).
//
// This file holds the C-ABI entry points, the planner that picks a kernel
// configuration and work decomposition (gemm_plan.h), and the fold kernel
// that finishes tiles whose chunks were shared out.  The kernels:
//
// * chunk_gemm_valu (gemm_valu_impl.h) -- the exact mode, and the fast mode
//   for chunk lengths the matrix cores cannot split;
// * chunk_gemm_mfma (gemm_mfma.hip) -- the fast mode for CL a multiple of the
//   MFMA instruction's K (16);
// * chunk_gemm_mfma_stream (gemm_mfma_stream.hip) -- the fast mode for CL a
//   multiple of 64, whole tiles streamed slab after slab;
// * chunk_gemm_mfma_kx, chunk_gemm_mfma_kx16 (gemm_mfma_kx.hip) -- the fast
//   mode for CL = 64 on GEMMs with few outputs and a long K: a 64 x 64 tile
//   per 16-wave workgroup, a step's chunks spread over the waves, or (kx16,
//   the one the planner picks) a 16 x 16 block per wave over the whole K.
#include <type_traits>

#include "fp8t_device.h"
#include "fp8train.h"
#include "fp8t_host.h"
#include "gemm_plan.h"
#include "gemm_mfma.h"
#include "gemm_valu.h"

#include <mutex>
#include <stdio.h>
#include <stdlib.h>

namespace fp8t {
namespace {

// ---------------------------------------------------------------------------
// fold: finish the shared tiles
// ---------------------------------------------------------------------------

// FP16 code -> value * 2^96 without branches (the fold pass decodes one code
// per output per chunk).  Normal, Inf and NaN codes by placing the code's
// fields in FP32's: the code sign-extended to 32 bits and shifted left by 14
// has the sign in bits 29-31, the exponent in 23-28 and the significand in
// 14-22, so setting bits 29 and 30 adds the scaled domain's 192 to the
// exponent (63, Inf and NaN, lands on 255).  Zero and subnormal codes
// (exponent 0) come out as +-(2^65 + m 2^56), whose value is +-m 2^57: the
// magnitude 2 |x| - 2^66, one exact FMA.  For every other code that FMA gives
// a magnitude >= |x|, so the result is the operand of smaller magnitude: with
// x's sign put on the FMA's (non-negative) result, the smaller of the two bit
// patterns as unsigned integers (both NaN for a NaN code; -0 stays -0).
__device__ __forceinline__ float fold_decode(int32_t code_sx) {
    const uint32_t u = ((uint32_t)code_sx << 14) | 0x60000000u;
    const float y = fmaf(fabsf(__uint_as_float(u)), 2.0f, -0x1p66f);
    const uint32_t ys = __float_as_uint(y) | (u & 0x80000000u);
    return __uint_as_float(min(u, ys));
}
// the code in bits 0-15 / 16-31 of w
__device__ __forceinline__ float fold_decode_lo(uint32_t w) {
    return fold_decode(__builtin_amdgcn_sbfe((int32_t)w, 0, 16));
}
__device__ __forceinline__ float fold_decode_hi(uint32_t w) {
    return fold_decode(__builtin_amdgcn_sbfe((int32_t)w, 16, 16));
}

// Each thread takes kFoldV consecutive outputs of one row of a shared tile and
// continues their running sums, held in C (the FP16 sums of the tile's first
// piece), over the chunk sums the other pieces left in the workspace, in
// ascending chunk order -- the same additions a whole-tile pass makes after
// its first piece.  The chunk sums of kFoldV outputs are one 2 kFoldV-byte
// load per chunk, in batches of kFoldU chunks with the next batch in flight
// while one is added (a split GEMM has few shared outputs and many chunks, so
// the pass needs many loads in flight per thread; 4 outputs x 16 chunks was
// the fastest of 4/8 x 16/32 on the conv stage's weight-gradient GEMM).  In
// the workspace's banded layout (ws_index) the threads of a band of 4 rows
// read one contiguous run per chunk, and its successive chunks are adjacent.
#ifndef FP8T_FOLD_V
#define FP8T_FOLD_V 4
#endif
#ifndef FP8T_FOLD_U
#define FP8T_FOLD_U 16
#endif
#ifndef FP8T_FOLD_T
#define FP8T_FOLD_T 64
#endif
// kFoldT threads per workgroup: one-wave workgroups spread evenly over the CUs
// (the conv stage's weight-gradient fold is 2304 waves: 9 per CU, where
// 256-thread workgroups left some CUs three and others two)
constexpr int kFoldV = FP8T_FOLD_V, kFoldU = FP8T_FOLD_U, kFoldT = FP8T_FOLD_T;
static_assert(kFoldV == 2 || kFoldV == 4 || kFoldV == 8, "2, 4 or 8 outputs per thread");
typedef std::conditional<kFoldV == 8, uint4,
                         std::conditional<kFoldV == 4, uint2, uint32_t>::type>::type FoldVec;

// A workspace vector loaded non-temporally (each chunk sum is read once).
__device__ __forceinline__ uint32_t nt_load(const uint32_t* q) { return __builtin_nontemporal_load(q); }
__device__ __forceinline__ uint2 nt_load(const uint2* q) {
    typedef uint32_t v2 __attribute__((ext_vector_type(2)));
    const v2 v = __builtin_nontemporal_load(reinterpret_cast<const v2*>(q));
    return make_uint2(v.x, v.y);
}
__device__ __forceinline__ uint4 nt_load(const uint4* q) {
    typedef uint32_t v4 __attribute__((ext_vector_type(4)));
    const v4 v = __builtin_nontemporal_load(reinterpret_cast<const v4*>(q));
    return make_uint4(v.x, v.y, v.z, v.w);
}

__global__ __launch_bounds__(kFoldT) void chunk_fold(GemmArgs g, Plan p, int BM, int BN) {
    const int64_t per = (int64_t)BM * BN;
    const int64_t idx = ((int64_t)blockIdx.x * kFoldT + threadIdx.x) * kFoldV;
    const int64_t lt = idx / per;
    if (lt * p.nch >= p.L) return;
    // thread index -> band of 4 rows (ws_index), then row-major inside it
    const int local = (int)(idx - lt * per);
    const int band = local / (4 * BN), pos = local % (4 * BN);
    const int r = 4 * band + pos / BN, c = pos % BN;
    const int64_t tile = p.t_whole + lt;
    int tr, tc;
    tile_rc(p, tile, tr, tc);
    const int m = tr * BM + r;
    const int n0 = tc * BN + c;
    if (m >= g.M || n0 >= g.N) return;
    const int a = first_piece_end(p, lt);
    // a tile whose first piece took every chunk needs only its FP8 result
    if (a >= p.nch && !g.C8) return;
    // the running sum of the first piece: in C, or in s_ws (FP8 result only)
    uint16_t* cp = g.C ? g.C + (int64_t)m * g.ldc + n0 : nullptr;
    const uint16_t* sp = g.C ? cp : g.s_ws + lt * per + r * BN + c;
    const int nv = min(kFoldV, g.N - n0);
    float S[kFoldV];
#pragma unroll
    for (int v = 0; v < kFoldV; ++v) S[v] = v < nv ? fold_decode_lo(sp[v]) : 0.0f;
    const FoldVec* src = reinterpret_cast<const FoldVec*>(g.ws + ws_index(p, BM, BN, lt, 0, r, c));
    const int step = 4 * BN / kFoldV;           // vectors per chunk of a band
    auto add = [&](FoldVec q) __attribute__((always_inline)) {
        uint32_t w[kFoldV / 2];
        __builtin_memcpy(w, &q, sizeof(q));
#pragma unroll
        for (int v = 0; v < kFoldV; ++v)
            S[v] = rn16s(S[v] + (v % 2 ? fold_decode_hi(w[v / 2]) : fold_decode_lo(w[v / 2])));
    };
    // two batches of kFoldU chunks: one in flight while the other is added.
    // Every batch load is unconditional (chunk indices clamped to the last
    // chunk, the extra values never added), so the compiler waits for the
    // older batch only; a conditional load makes it wait for both.
    // A batch that lies inside the tile's chunks loads from one base pointer
    // at uniform offsets; only the last one clamps each index.
    const int last = p.nch - 1;
    auto load = [&](FoldVec (&q)[kFoldU], int c0) __attribute__((always_inline)) {
        if (c0 + kFoldU <= p.nch) {
            const FoldVec* b = src + (int64_t)c0 * step;
#pragma unroll
            for (int u = 0; u < kFoldU; ++u) q[u] = nt_load(&b[u * step]);
        } else {
#pragma unroll
            for (int u = 0; u < kFoldU; ++u) q[u] = src[(int64_t)min(c0 + u, last) * step];
        }
    };
    auto fold_all = [&](const FoldVec (&q)[kFoldU]) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < kFoldU; ++u) add(q[u]);
    };
    auto fold_part = [&](const FoldVec (&q)[kFoldU], int n) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < kFoldU; ++u)
            if (u < n) add(q[u]);
    };
    if (a < p.nch) {
        FoldVec q0[kFoldU], q1[kFoldU];
        int c = a;
        load(q0, c);
        for (;;) {
            // q0 holds chunks c ..
            if (c + kFoldU > p.nch) {
                fold_part(q0, p.nch - c);
                break;
            }
            load(q1, c + kFoldU);
            fold_all(q0);
            c += kFoldU;
            // q1 holds chunks c ..
            if (c + kFoldU > p.nch) {
                fold_part(q1, p.nch - c);
                break;
            }
            load(q0, c + kFoldU);
            fold_all(q1);
            c += kFoldU;
        }
    }
#pragma unroll
    for (int v = 0; v < kFoldV; ++v) {
        if (v >= nv) continue;
        if (cp) cp[v] = f32s_to_fp16(S[v]);
        if (g.C8) g.C8[(int64_t)m * g.ldc8 + n0 + v] = (uint8_t)f32d_to_fp8_scaled<96>(S[v], g.q_scale);
    }
}

// K = 0: every result is +0 (FP16 code 0, FP8 code of 0 * scale).
__global__ void fill_empty(uint16_t* __restrict__ C, int64_t ldc, uint8_t* __restrict__ C8,
                           int64_t ldc8, float scale, int M, int N) {
    const int64_t total = (int64_t)M * N;
    const int64_t step = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += step) {
        const int64_t r = i / N, c = i % N;
        if (C) C[r * ldc + c] = 0;
        if (C8) C8[r * ldc8 + c] = (uint8_t)f32_to_fp8(0.0f * scale);
    }
}

// ---------------------------------------------------------------------------
// planner
// ---------------------------------------------------------------------------

constexpr double kClockHz = 2.4e9;      // MI355X peak engine clock
constexpr double kLanesPerCU = 128.0;   // 32-bit VALU lane-ops per clock per CU
constexpr double kFoldBytesPerS = 5e12; // effective HBM rate of the fold pass

// Relative cost per multiply-accumulate of each register tile on a CU with
// enough waves resident (see valu_efficiency), in VALU instructions (4 for
// the rounded FMA of the guarded path, plus operand decode, LDS reads and
// loop overhead; measured on the conv-stage GEMMs for the large tiles, on
// the 512 x 512 long-accumulation GEMMs for the small ones).
double valu_ops_per_mac(int cfg) {
    switch (cfg) {
        case 4: return 4.6;     // 4 x 4, 4 waves per SIMD
        case 3: return 4.85;    // 4 x 8
        case 2: return 4.9;     // 8 x 4
        case 1: return 5.1;     // 8 x 8, 2 waves per SIMD
        case 0: return 5.2;
        case 7: return 4.3;     // 4 x 4 on 128 x 64 tiles, 8 waves per workgroup
        case 8: return 4.3;     // 4 x 4 on 64 x 128 tiles, 8 waves per workgroup
        case 5: return 7.0;     // 2 x 2
        case kChainConfig: return 6.0;       // chain kernel, 2 x 2
        case kChainConfig + 1: return 6.1;   // chain kernel, 1 x 2
        case kChainConfig + 2: return 9.0;   // chain kernel, 1 x 1
        default: return 10.8;   // 1 x 1
    }
}

// Fraction of a CU's VALU rate reached with w waves per SIMD resident: each
// multiply-accumulate is a chain of four dependent instructions, and on
// gfx950 about four waves per SIMD are needed to issue every cycle whatever
// the outputs per lane (measured: a 2 x 2 register tile at one wave per SIMD
// runs at a quarter of the rate a 1 x 1 tile reaches at four).
// VALU instructions per multiply-accumulate the fast chain kernel saves over
// the exact one (measured on 512 x 512 outputs, K 16384 and 65536, CL 8 and
// 12): the rounding after each FMA goes, worth more on the 2 x 2 tile than
// on the narrower ones.
double chain_fast_saving(int cfg) {
    return cfg == kChainConfig ? 3.0 : cfg == kChainConfig + 1 ? 2.3 : 2.6;
}

double valu_efficiency(double w) { return w >= 4.0 ? 1.0 : w / 4.0; }

// Extra VALU instructions per multiply-accumulate with FP16 operands: the
// product's multiplication and its rounding to FP16 (and, max, add and the
// magic-number add and subtract) replace the FMA's one.
constexpr double kP16ProductOps = 6.0;

// Matrix-core fast mode, CU time of one output-chunk (the VALU epilogue
// dominates; the matrix-core share grows with CL) and of the per-tile start
// (pipeline fill, C stores), measured on the conv-stage GEMMs: 64 x 64 tiles
// with 64-k slabs, 32 x 32 tiles with 128-k slabs, the streamed 64 x 64
// kernel and the 64 x 64 kernel with chunks spread over 16 waves (both
// fitted to their forward and backward-data times; the latter predicts its
// weight-gradient time within 5%); the 16 x 16 block-per-wave kernel scaled
// from it by their measured weight-gradient times (0.265 against 0.279 ms);
// the wave-independent 32 x 128 kernel fitted to its forward and
// backward-data times (one tile per workgroup).
double mfma_cost_per_output_chunk(int cfg, int64_t CL) {
    const double base = cfg == 0 ? 0.156e-9 : cfg == 1 ? 0.17e-9 : cfg == 2 ? 0.0856e-9
                      : cfg == 3 ? 0.0993e-9 : cfg == 4 ? 0.0942e-9 : 0.0557e-9;
    return base * (0.6 + 0.4 * (double)CL / 64.0);
}
double mfma_cost_per_tile(int cfg) {
    return cfg == 0 ? 1.1e-6 : cfg == 1 ? 0.66e-6 : cfg == 2 ? 0.67e-6 : cfg == 3 ? 0.93e-6
         : cfg == 4 ? 0.88e-6 : 0.33e-6;
}
constexpr size_t kWsAlignBt = 256;

// The k-contiguous copy of an operand B stored with n contiguous (the
// wave-independent kernel's second operand): its workspace bytes, and its
// cost (one small kernel reading and writing N x K bytes).
size_t wave_bt_bytes(int64_t N, int64_t K) {
    return (size_t)N * (size_t)((K + 15) / 16 * 16) + kWsAlignBt;
}
double wave_bt_cost(int64_t N, int64_t K) { return 2e-6 + 2.0 * (double)N * (double)K / 3e12; }

// VALU_P16: FP16 operands, products rounded to FP16 (chunk_gemm_p16)
enum Kind { VALU_EXACT = 0, VALU_FAST = 1, MFMA_FAST = 2, VALU_P16 = 3 };

struct Choice {
    int cfg = -1;
    const void* fn = nullptr;
    const void* fn_aligned = nullptr;    // variant taken when mfma_kx_aligned(args)
    int NT = 0, BM = 0, BN = 0;
    Plan plan{};
    size_t ws_bytes = 0;                 // chunk sums of the shared tiles
    size_t bt_bytes = 0;                 // the k-contiguous copy of B (configuration 5)
    double est_s = 0.0;
};

constexpr size_t kWsAlign = 256;

// The best kernel configuration and work decomposition for these sizes; with
// allow_ws false only plans that need no workspace are considered, otherwise
// only plans whose workspace is at most ws_cap bytes.  wave_ok: the operands
// allow the wave-independent kernel's 16-byte loads (configuration 5).
Choice plan_gemm(Kind kind, int ta, int tb, int64_t M, int64_t N, int64_t K, int64_t CL,
                 bool allow_ws, bool conv = false, size_t ws_cap = SIZE_MAX,
                 bool wave_ok = true) {
    Choice best;
    const int cus = device_cus();
    if (cus <= 0) return best;
    const bool mf = kind == MFMA_FAST;
    const bool p16 = kind == VALU_P16;
    const int fast = kind == VALU_FAST || kind == MFMA_FAST;
    const int ncfg = mf ? kMfmaConfigs : kValuConfigs;
    // Overrides for tests and tuning: the tile configuration, a cap on the
    // workgroups, and 1 / 0 to require / forbid shared tiles.
    int force_cfg = env_int(mf ? "FP8T_MFMA_TILE" : "FP8T_VALU_TILE", -1);
    if (force_cfg >= 0 && force_cfg >= ncfg) force_cfg = -1;
    const int force_g = env_int("FP8T_GEMM_WGS", 0);
    const int force_split = env_int("FP8T_GEMM_SPLIT", -1);
    const int verbose = env_int("FP8T_GEMM_VERBOSE", 0);
    const int64_t nch = (K + CL - 1) / CL;
    for (int pass = 0; pass < 2 && best.cfg < 0; ++pass) {
        for (int cfg = 0; cfg < ncfg; ++cfg) {
            if (pass == 0 && force_cfg >= 0 && cfg != force_cfg) continue;
            if (!mf && force_cfg < 0 && cfg == 0) continue;   // kept for comparison only
            const void* fn;
            int NT, BM, BN;
            double t_out;                        // CU time of one output-chunk
            double t_tile = 0.0;                 // CU time of a tile's start
            if (mf) {
                const MfmaShape sh = mfma_shape(cfg);
                if (CL % sh.kstep != 0) continue;
                if ((cfg == 3 || cfg == 4) && CL != 64) continue;   // 64-product chunks only
                if (cfg == 5 && (!wave_ok || (!tb && (!allow_ws || wave_bt_bytes(N, K) > ws_cap))))
                    continue;
                fn = mfma_kernel(cfg, ta, tb);
                NT = sh.NT, BM = sh.BM, BN = sh.BN;
                t_out = mfma_cost_per_output_chunk(cfg, CL);
                t_tile = mfma_cost_per_tile(cfg);
            } else {
                // the chain kernel: 4-k groups inside one chunk
                if (is_chain(cfg) && (conv || p16 || (CL % 4 != 0 && CL < K))) continue;
                const ValuShape sh = valu_shape(cfg);
                fn = conv ? valu_conv_kernel(cfg, ta)
                   : p16  ? valu_p16_kernel(cfg, ta, tb)
                          : valu_kernel(cfg, ta, tb, fast);
                NT = sh.NT, BM = sh.BM, BN = sh.BN;
                // the MACs of a chunk, and its end (an add and a rounding); an
                // FP16 product costs its multiplication and rounding on top,
                // and the fast chain kernel does without the rounding
                const double ops = valu_ops_per_mac(cfg) + (p16 ? kP16ProductOps : 0.0) -
                                   (fast && is_chain(cfg) ? chain_fast_saving(cfg) : 0.0);
                t_out = ((double)CL * ops + 4.0) / (kLanesPerCU * kClockHz);
            }
            if (!fn) continue;
            int occ = kernel_occupancy(fn, NT);
            if (occ <= 0) continue;
            if (occ > 8) occ = 8;
            const int64_t tiles_m = (M + BM - 1) / BM;
            const int64_t tiles_n = (N + BN - 1) / BN;
            const int64_t T = tiles_m * tiles_n;
            int64_t gmax = (int64_t)cus * occ;
            if (force_g > 0 && force_g < gmax) gmax = force_g;
            const double t_chunk = (double)BM * BN * t_out;     // one tile-chunk on a CU
            for (int split = 0; split < 2; ++split) {
                if (split && !allow_ws) continue;
                if (force_split == 0 && split) continue;
                Plan p{};
                p.tiles_n = tiles_n;
                p.nch = (int)nch;
                double est;
                size_t ws = 0;
                // the streamed kernel writes split tiles' chunk sums as scattered
                // 2-byte stores: the other kernels are faster there; the
                // chunk-per-wave and chain kernels have no shared tiles
                if (split && mf && cfg >= 2) continue;
                if (split && !mf && is_chain(cfg)) continue;
                if (!split && mf && cfg == 5) {
                    // one tile per workgroup (the hardware deals the next
                    // workgroup to whichever CU has room: measured a few %
                    // faster than a persistent grid on the conv stage)
                    const int64_t G = force_g > 0 && force_g < T ? force_g : T;
                    p.G = (int)G;
                    p.t_whole = T;
                    p.L = 0;
                    // fewer tiles than CUs: a lone tile is not done faster
                    // than 2.3 tiles' CU time (its waves wait on their own
                    // latency; measured on 64 tiles of K 6000)
                    const double per_cu = (double)T / cus;
                    est = (T < cus ? 2.3 : per_cu) * (nch * t_chunk + t_tile) +
                          (tb ? 0.0 : wave_bt_cost(N, K));
                } else if (!split) {
                    const int64_t G = T < gmax ? T : gmax;
                    p.G = (int)G;
                    p.t_whole = T;
                    p.L = 0;
                    // tiles on the busiest CU; the streamed kernel needs at least
                    // two workgroups on a CU to overlap its matrix-core, vector and
                    // memory work (a lone one runs at about half the CU rate)
                    int64_t per_cu = (T + cus - 1) / cus;
                    if (mf && cfg == 2 && per_cu < 2) per_cu = 2;
                    est = (double)per_cu * (nch * t_chunk + t_tile);
                    if (!mf) {
                        const int64_t res = per_cu < occ ? per_cu : occ;
                        est /= valu_efficiency((double)res * NT / 256.0);
                    }
                } else {
                    int64_t G = gmax;
                    if (G > T * nch) G = T * nch;
                    const int64_t q = T / G;
                    p.G = (int)G;
                    p.t_whole = q * G;
                    p.L = (T - p.t_whole) * nch;
                    if (p.L == 0) continue;                // same as the plain plan
                    const int64_t wg_per_cu = (G + cus - 1) / cus;
                    const int64_t per_wg = q * nch + (p.L + G - 1) / G;
                    ws = (size_t)(T - p.t_whole) * nch * BM * BN * sizeof(uint16_t) + kWsAlign;
                    if (ws > ws_cap) continue;
                    est = (double)wg_per_cu * (per_wg * t_chunk + (q + 2) * t_tile);
                    if (!mf) {
                        const int64_t res = wg_per_cu < occ ? wg_per_cu : occ;
                        est /= valu_efficiency((double)res * NT / 256.0);
                    }
                    est += 2.0 * (double)ws / kFoldBytesPerS + 4e-6;
                }
                p.xcd_remap = p.t_whole % 8 == 0 && p.G % 8 == 0;
                if (force_split == 1 && !split && allow_ws) est *= 1e6;   // any shared plan wins
                if (verbose)
                    fprintf(stderr, "[fp8t plan] kind %d cfg %d occ %d split %d G %d T %lld "
                            "t_whole %lld L %lld ws %zu est %.1f us\n", (int)kind, cfg, occ, split,
                            p.G, (long long)T, (long long)p.t_whole, (long long)p.L, ws, est * 1e6);
                if (best.cfg < 0 || est < best.est_s) {
                    best.cfg = cfg;
                    best.fn = fn;
                    best.fn_aligned = mf && cfg == 3 ? mfma_kx_kernel_aligned(ta, tb)
                                    : mf && cfg == 4 ? mfma_kx16_kernel_aligned(ta, tb)
                                                     : nullptr;
                    best.NT = NT;
                    best.BM = BM;
                    best.BN = BN;
                    best.plan = p;
                    best.ws_bytes = ws;
                    best.bt_bytes = mf && cfg == 5 && !tb ? wave_bt_bytes(N, K) : 0;
                    best.est_s = est;
                }
            }
        }
    }
    if (verbose)
        fprintf(stderr, "[fp8t plan] chose kind %d cfg %d G %d t_whole %lld L %lld\n", (int)kind,
                best.cfg, best.plan.G, (long long)best.plan.t_whole, (long long)best.plan.L);
    return best;
}

int launch_plan(const Choice& ch, GemmArgs g, hipStream_t stream) {
    void* args[] = {&g, const_cast<Plan*>(&ch.plan)};
    const void* fn = ch.fn_aligned && mfma_kx_aligned(g) ? ch.fn_aligned : ch.fn;
    if (hipLaunchKernel(fn, dim3(ch.plan.G), dim3(ch.NT), args, 0, stream) != hipSuccess)
        return FP8T_EHIP;
    if (ch.plan.L > 0) {
        const int64_t shared = ch.plan.L / ch.plan.nch;
        const int64_t threads = shared * ch.BM * ch.BN / kFoldV;
        hipLaunchKernelGGL(chunk_fold, dim3((unsigned)((threads + kFoldT - 1) / kFoldT)), dim3(kFoldT), 0,
                           stream, g, ch.plan, ch.BM, ch.BN);
    }
    return launch_status();
}

}  // namespace
}  // namespace fp8t

using namespace fp8t;

// ---------------------------------------------------------------------------
// scratch of chunk_gemm_noalloc
// ---------------------------------------------------------------------------

namespace {

// The chunk sums of shared tiles for chunk_gemm_noalloc: one array per GPU,
// held by the loaded code object until the process ends.  Nothing in it needs
// to start at zero: a call's fold reads only chunk sums its own GEMM kernel
// wrote before, in stream order.  Calls that overlap in time on one GPU
// share the array and race.
__device__ __align__(256) uint8_t scratch[FP8T_NOALLOC_SCRATCH_BYTES];

// The device address of `scratch` on each GPU, taken once per device with
// that device current.  In host code `scratch` names a host-side stand-in,
// so only this address may be handed to kernels.
void* scratch_address() {
    static std::mutex mu;
    static void* ptr[64] = {nullptr};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
    std::lock_guard<std::mutex> lk(mu);
    if (!ptr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
        ptr[dev] = p;
    }
    return ptr[dev];
}

}  // namespace

namespace {
bool gemm_args_ok(int ta, int tb, int64_t M, int64_t N, int64_t K, int64_t CL, int mode) {
    if (M < 0 || N < 0 || K < 0 || CL < 1) return false;
    if ((ta != 0 && ta != 1) || (tb != 0 && tb != 1)) return false;
    if (mode != FP8T_EXACT && mode != FP8T_FAST) return false;
    // indices inside the kernels are 32-bit per dimension
    if (M > kMaxGemmDim || N > kMaxGemmDim || K > kMaxGemmDim) return false;
    return true;
}

// CL = 1 is the plain sequential FP16 sum in both modes (a one-product chunk
// is exact, also when summed in FP32), the same chain as one chunk of K in
// exact mode: run it that way.
void normalize_chunking(int& mode, int64_t K, int64_t& CL) {
    if (CL == 1 && K > 1) {
        CL = K;
        mode = FP8T_EXACT;
    }
}

Kind kind_of(int mode, int64_t K, int64_t CL) {
    const int64_t cl = CL > K ? K : CL;
    if (mode == FP8T_EXACT) return VALU_EXACT;
    return cl % 16 == 0 ? MFMA_FAST : VALU_FAST;
}
// Workspace of a plan: the chunk sums of its shared tiles, and (entry points
// with an FP8 result) room for their first pieces' running sums.
size_t plan_workspace(const Choice& ch, bool fp8out) {
    if (ch.cfg < 0) return 0;
    size_t b = ch.bt_bytes;
    if (ch.plan.L == 0) return b;
    b += ch.ws_bytes;
    if (fp8out)
        b += (size_t)(ch.plan.L / ch.plan.nch) * ch.BM * ch.BN * sizeof(uint16_t) + kWsAlign;
    return b;
}

size_t workspace_query(int ta, int tb, int64_t M, int64_t N, int64_t K, int64_t CL, int mode,
                       bool fp8out, bool p16 = false) {
    if (!gemm_args_ok(ta, tb, M, N, K, CL, mode)) return 0;
    if (M == 0 || N == 0 || K == 0) return 0;
    normalize_chunking(mode, K, CL);
    const int64_t cl = CL > K ? K : CL;
    const Kind kind = p16 ? VALU_P16 : kind_of(mode, K, cl);
    return plan_workspace(plan_gemm(kind, ta, tb, M, N, K, cl, true), fp8out);
}

int gemm_call(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K, int64_t CL,
              const uint8_t* A, int64_t lda, const uint8_t* B, int64_t ldb, uint16_t* C,
              int64_t ldc, uint8_t* C8, int64_t ldc8, float scale, int mode, void* workspace,
              size_t workspace_bytes, hipStream_t stream, bool fp8out,
              bool use_scratch = false, bool p16 = false) {
    if (!gemm_args_ok(trans_a, trans_b, M, N, K, CL, mode)) return FP8T_EINVAL;
    if (M == 0 || N == 0) return FP8T_OK;
    if (!fp8out && !C) return FP8T_EINVAL;
    if (C && ldc < N) return FP8T_EINVAL;
    if (fp8out && (!C8 || ldc8 < N)) return FP8T_EINVAL;
    if (K > 0) {
        if (!A || !B) return FP8T_EINVAL;
        if (lda < (trans_a ? M : K) || ldb < (trans_b ? K : N)) return FP8T_EINVAL;
    }
    if (workspace_bytes > 0 && !workspace) return FP8T_EINVAL;
    if (use_scratch) {                    // after validation: nothing touched the GPU yet
        workspace = scratch_address();
        if (!workspace) return FP8T_EHIP;
        workspace_bytes = FP8T_NOALLOC_SCRATCH_BYTES;
    }
    normalize_chunking(mode, K, CL);
    if (CL > K && K > 0) CL = K;           // one chunk
    const int m = (int)M, n = (int)N, k = (int)K, cl = (int)(K > 0 ? CL : 1);
    if (K == 0) {
        const int64_t total = M * N;
        hipLaunchKernelGGL(fill_empty, dim3(stride_blocks(total, 256)), dim3(256), 0,
                           stream, C, ldc, C8, ldc8, scale, m, n);
        return launch_status();
    }
    // With no workspace, the best plan that needs none; with one, the best
    // plan overall, which must then fit; with the scratch, the best plan that
    // fits in it.  Operands that rule out the wave-independent kernel's
    // 16-byte loads (which the workspace query assumes) also take the best
    // plan that fits.
    // (and keep a block's 32 rows within 32-bit byte offsets)
    const bool wave_ok = !p16 && aligned(A, 16) && lda % 16 == 0 && lda < (1 << 26) &&
                         (trans_b ? aligned(B, 16) && ldb % 16 == 0 && ldb < (1 << 26)
                                  : K < (1 << 26));
    const Kind kind = p16 ? VALU_P16 : kind_of(mode, K, cl);
    const Choice ch = plan_gemm(kind, trans_a, trans_b, M, N, K, cl, workspace_bytes > 0, false,
                                use_scratch || !wave_ok ? workspace_bytes : SIZE_MAX, wave_ok);
    if (ch.cfg < 0) return FP8T_EHIP;
    if (plan_workspace(ch, fp8out) > workspace_bytes) return FP8T_EWORKSPACE;
    GemmArgs g{};
    g.A = A;
    g.B = B;
    g.C = C;
    g.C8 = C8;
    g.ldc8 = ldc8;
    g.q_scale = scale;
    if (ch.plan.L > 0) {
        const uintptr_t base = ((uintptr_t)workspace + kWsAlign - 1) & ~(uintptr_t)(kWsAlign - 1);
        g.ws = reinterpret_cast<uint16_t*>(base);
        const uintptr_t sbase = (base + ch.ws_bytes - kWsAlign + kWsAlign - 1) &
                                ~(uintptr_t)(kWsAlign - 1);
        g.s_ws = fp8out ? reinterpret_cast<uint16_t*>(sbase) : nullptr;
    }
    g.lda = lda;
    g.ldb = ldb;
    g.ldc = C ? ldc : 0;
    g.M = m;
    g.N = n;
    g.K = k;
    g.CL = cl;
    // 4-code loads (4 bytes, or 8 with FP16 codes) need aligned rows; the
    // matrix-core kernel's interior path also keeps per-thread offsets within
    // a slab in 32 bits
    const int eb = p16 ? 2 : 1;            // bytes per operand element
    g.a_vec = aligned(A, 4 * eb) && lda % 4 == 0 && lda < (1 << 24);
    g.b_vec = aligned(B, 4 * eb) && ldb % 4 == 0 && ldb < (1 << 24);
    g.a_vec16 = !p16 && aligned(A, 16) && lda % 16 == 0;
    g.b_vec16 = !p16 && aligned(B, 16) && ldb % 16 == 0;
    g.c_vec = C && aligned(C, 4) && ldc % 2 == 0;
    g.c_vec8 = C && aligned(C, 8) && ldc % 4 == 0;
    g.c_vec16 = C && aligned(C, 16) && ldc % 8 == 0;
    g.c8_vec8 = C8 && aligned(C8, 8) && ldc8 % 8 == 0;
    g.c8_vec4 = C8 && aligned(C8, 4) && ldc8 % 4 == 0;
    // FP8T_GEMM_GUARD=0 runs every piece on the safe path (tests, tuning).
    g.guarded = env_int("FP8T_GEMM_GUARD", 1) != 0;
    if (ch.bt_bytes > 0) {
        // the wave-independent kernel reads B k-contiguous: its copy, at the
        // start of the workspace (the plan has no shared tiles)
        const uintptr_t base = ((uintptr_t)workspace + kWsAlignBt - 1) & ~(uintptr_t)(kWsAlignBt - 1);
        uint8_t* bt = reinterpret_cast<uint8_t*>(base);
        const int64_t ldt = (K + 15) / 16 * 16;
        launch_transpose_bytes(B, ldb, k, n, bt, ldt, stream);
        g.B = bt;
        g.ldb = ldt;
        g.b_vec = 1;
        g.b_vec16 = 1;
    }
    return launch_plan(ch, g, stream);
}
}  // namespace

extern "C" size_t chunk_gemm_workspace_size(int trans_a, int trans_b, int64_t M,
                                            int64_t N, int64_t K, int64_t CL, int mode) {
    return workspace_query(trans_a, trans_b, M, N, K, CL, mode, false);
}

extern "C" int chunk_gemm(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K,
                          int64_t CL, const uint8_t* A, int64_t lda, const uint8_t* B,
                          int64_t ldb, uint16_t* C, int64_t ldc, int mode,
                          void* workspace, size_t workspace_bytes, hipStream_t stream) {
    return gemm_call(trans_a, trans_b, M, N, K, CL, A, lda, B, ldb, C, ldc, nullptr, 0, 1.0f,
                     mode, workspace, workspace_bytes, stream, false);
}

extern "C" int chunk_gemm_noalloc(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K,
                                  int64_t CL, const uint8_t* A, int64_t lda, const uint8_t* B,
                                  int64_t ldb, uint16_t* C, int64_t ldc, int mode,
                                  hipStream_t stream) {
    return gemm_call(trans_a, trans_b, M, N, K, CL, A, lda, B, ldb, C, ldc, nullptr, 0, 1.0f,
                     mode, nullptr, 0, stream, false, true);
}

extern "C" size_t chunk_gemm_p16_workspace_size(int trans_a, int trans_b, int64_t M, int64_t N,
                                                int64_t K, int64_t CL) {
    return workspace_query(trans_a, trans_b, M, N, K, CL, FP8T_EXACT, false, true);
}

extern "C" int chunk_gemm_p16(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K,
                              int64_t CL, const uint16_t* A, int64_t lda, const uint16_t* B,
                              int64_t ldb, uint16_t* C, int64_t ldc, void* workspace,
                              size_t workspace_bytes, hipStream_t stream) {
    return gemm_call(trans_a, trans_b, M, N, K, CL, reinterpret_cast<const uint8_t*>(A), lda,
                     reinterpret_cast<const uint8_t*>(B), ldb, C, ldc, nullptr, 0, 1.0f,
                     FP8T_EXACT, workspace, workspace_bytes, stream, false, false, true);
}

extern "C" size_t chunk_gemm_fp8_workspace_size(int trans_a, int trans_b, int64_t M,
                                                int64_t N, int64_t K, int64_t CL, int mode) {
    return workspace_query(trans_a, trans_b, M, N, K, CL, mode, true);
}

extern "C" int chunk_gemm_fp8(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K,
                              int64_t CL, const uint8_t* A, int64_t lda, const uint8_t* B,
                              int64_t ldb, uint16_t* C, int64_t ldc, uint8_t* C8,
                              int64_t ldc8, float scale, int mode, void* workspace,
                              size_t workspace_bytes, hipStream_t stream) {
    return gemm_call(trans_a, trans_b, M, N, K, CL, A, lda, B, ldb, C, ldc, C8, ldc8, scale,
                     mode, workspace, workspace_bytes, stream, true);
}

// ---------------------------------------------------------------------------
// convolutions lowered implicitly (Sec. 2.2)
// ---------------------------------------------------------------------------

namespace {

struct ConvShape {
    int64_t M, K, OH, OW;   // M = N OH OW output pixels, K = KH KW C
    bool ok;
};

ConvShape conv_shape(int64_t N, int64_t H, int64_t W, int64_t C, int64_t KH, int64_t KW,
                     int64_t pad, int64_t stride) {
    ConvShape r{0, 0, 0, 0, false};
    if (N < 0 || H < 1 || W < 1 || C < 1 || KH < 1 || KW < 1 || pad < 0 || stride < 1)
        return r;
    r.OH = (H + 2 * pad - KH) / stride + 1;
    r.OW = (W + 2 * pad - KW) / stride + 1;
    if (H + 2 * pad < KH || W + 2 * pad < KW) return r;
    r.M = N * r.OH * r.OW;
    r.K = KH * KW * C;
    // every index of X, Xcol and the GEMM in 32 bits
    if (r.M > kMaxGemmDim || r.K > kMaxGemmDim || N * H * W * C > ((int64_t)1 << 40)) return r;
    r.ok = true;
    return r;
}

// The exact-mode GEMM with A = Xcol (wgrad: Xcol^T) read from the NHWC input.
int conv_gemm_call(bool wgrad, const uint8_t* X, int64_t N, int64_t H, int64_t W, int64_t C,
                   int64_t KH, int64_t KW, int64_t pad, int64_t stride, const uint8_t* B,
                   int64_t Cout, int64_t CL, uint16_t* Out, int64_t ldo, void* workspace,
                   size_t workspace_bytes, hipStream_t stream, bool query, size_t* need) {
    const ConvShape cs = conv_shape(N, H, W, C, KH, KW, pad, stride);
    if (!cs.ok || Cout < 0 || Cout > kMaxGemmDim || CL < 1) return FP8T_EINVAL;
    // GEMM dimensions: fwd  Y (M x Cout) = Xcol (M x K) W (K x Cout);
    //                  wgrad dW (K x Cout) = Xcol^T (K x M) dY (M x Cout)
    const int64_t gM = wgrad ? cs.K : cs.M, gN = Cout, gK = wgrad ? cs.M : cs.K;
    const int ta = wgrad ? 1 : 0;
    if (query) {
        *need = 0;
        if (gM == 0 || gN == 0 || gK == 0) return FP8T_OK;
        const int64_t cl = CL > gK ? gK : CL;
        *need = plan_workspace(plan_gemm(VALU_EXACT, ta, 0, gM, gN, gK, cl, true, true), false);
        return FP8T_OK;
    }
    if (gM == 0 || gN == 0) return FP8T_OK;
    if (!Out || ldo < gN) return FP8T_EINVAL;
    if (gK > 0 && (!X || !B)) return FP8T_EINVAL;
    if (workspace_bytes > 0 && !workspace) return FP8T_EINVAL;
    if (gK == 0) {
        const int64_t total = gM * gN;
        hipLaunchKernelGGL(fill_empty, dim3(stride_blocks(total, 256)), dim3(256), 0,
                           stream, Out, ldo, (uint8_t*)nullptr, (int64_t)0, 1.0f, (int)gM,
                           (int)gN);
        return launch_status();
    }
    if (CL > gK) CL = gK;
    const Choice ch = plan_gemm(VALU_EXACT, ta, 0, gM, gN, gK, CL, workspace_bytes > 0, true);
    if (ch.cfg < 0) return FP8T_EHIP;
    if (plan_workspace(ch, false) > workspace_bytes) return FP8T_EWORKSPACE;
    GemmArgs g{};
    g.A = X;
    g.B = B;
    g.C = Out;
    if (ch.plan.L > 0) {
        const uintptr_t base = ((uintptr_t)workspace + kWsAlign - 1) & ~(uintptr_t)(kWsAlign - 1);
        g.ws = reinterpret_cast<uint16_t*>(base);
    }
    g.lda = wgrad ? cs.M : cs.K;          // not used: A is read through g.conv
    g.ldb = Cout;
    g.ldc = ldo;
    g.M = (int)gM;
    g.N = (int)gN;
    g.K = (int)gK;
    g.CL = (int)CL;
    g.a_vec = 0;
    g.b_vec = aligned(B, 4) && Cout % 4 == 0 && Cout < (1 << 24);
    g.c_vec = aligned(Out, 4) && ldo % 2 == 0;
    g.c_vec8 = aligned(Out, 8) && ldo % 4 == 0;
    g.c_vec16 = aligned(Out, 16) && ldo % 8 == 0;
    g.guarded = env_int("FP8T_GEMM_GUARD", 1) != 0;
    g.conv.H = (int)H;
    g.conv.W = (int)W;
    g.conv.C = (int)C;
    g.conv.KW = (int)KW;
    g.conv.KWC = (int)(KW * C);
    g.conv.OW = (int)cs.OW;
    g.conv.OHW = (int)(cs.OH * cs.OW);
    g.conv.pad = (int)pad;
    g.conv.stride = (int)stride;
    g.conv.vec = C % 4 == 0 && aligned(X, 4);
    return launch_plan(ch, g, stream);
}

}  // namespace

extern "C" int conv2d_fwd_fp8(const uint8_t* X, int64_t N, int64_t H, int64_t W, int64_t C,
                              int64_t KH, int64_t KW, int64_t pad, int64_t stride,
                              const uint8_t* Wt, int64_t Cout, int64_t CL, uint16_t* Y,
                              int64_t ldy, void* workspace, size_t workspace_bytes,
                              hipStream_t stream) {
    return conv_gemm_call(false, X, N, H, W, C, KH, KW, pad, stride, Wt, Cout, CL, Y, ldy,
                          workspace, workspace_bytes, stream, false, nullptr);
}

extern "C" int conv2d_wgrad_fp8(const uint8_t* X, int64_t N, int64_t H, int64_t W, int64_t C,
                                int64_t KH, int64_t KW, int64_t pad, int64_t stride,
                                const uint8_t* dY, int64_t Cout, int64_t CL, uint16_t* dW,
                                int64_t lddw, void* workspace, size_t workspace_bytes,
                                hipStream_t stream) {
    return conv_gemm_call(true, X, N, H, W, C, KH, KW, pad, stride, dY, Cout, CL, dW, lddw,
                          workspace, workspace_bytes, stream, false, nullptr);
}

extern "C" size_t conv2d_workspace_size(int wgrad, int64_t N, int64_t H, int64_t W, int64_t C,
                                        int64_t KH, int64_t KW, int64_t pad, int64_t stride,
                                        int64_t Cout, int64_t CL) {
    size_t need = 0;
    if (wgrad != 0 && wgrad != 1) return 0;
    if (conv_gemm_call(wgrad != 0, nullptr, N, H, W, C, KH, KW, pad, stride, nullptr, Cout, CL,
                       nullptr, 0, nullptr, 0, nullptr, true, &need) != FP8T_OK)
        return 0;
    return need;
}
