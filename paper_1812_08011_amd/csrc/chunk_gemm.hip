// chunk_gemm: FP8 x FP8 GEMM with chunk-based FP16 accumulation
// (Sec. 2.3 "Chunk-based Accumulation", dot-product algorithm of Fig. 3(a)).
//
// This file holds the C-ABI entry points, the planner that picks a kernel
// configuration and work decomposition (gemm_plan.h), the fold kernel that
// finishes tiles whose chunks were shared out, and the matrix-core kernel of
// the fast mode.  The vector-ALU kernels are in gemm_valu.hip.
//
// * chunk_gemm_valu (gemm_valu.hip) -- the exact mode, and the fast mode for
//   chunk lengths the matrix cores cannot split.
// * chunk_gemm_mfma -- the fast mode for CL a multiple of 16.  FP8 bytes are
//   the OCP E5M2 ("bf8") encoding (same bias, subnormals and specials), so
//   the FP8 codes feed v_mfma_f32_32x32x16_bf8_bf8 directly.  Each wave owns a
//   64x64 output tile (2x2 MFMA blocks); each chunk is accumulated on the
//   matrix cores from zero, then rounded to FP16 and added into S on the VALU.
#include "fp8t_device.h"
#include "fp8train.h"
#include "fp8t_host.h"
#include "gemm_plan.h"
#include "gemm_valu.h"

#include <mutex>
#include <stdio.h>
#include <stdlib.h>

namespace fp8t {
namespace {

// ---------------------------------------------------------------------------
// MFMA kernel (fast mode, CL % 16 == 0)
// ---------------------------------------------------------------------------

typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int MF_BM = 128, MF_BN = 128, MF_BK = 64, MF_NT = 256;
constexpr int MF_PITCH = MF_BK + 8;     // bytes per LDS row (k-contiguous)

// Load the 4 bytes (r, c..c+3) of a row-major byte matrix with `rows` x
// `cols` valid elements and leading dimension ld; bytes outside are 0.
template <bool ALIGN4>
__device__ __forceinline__ uint32_t load4(const uint8_t* __restrict__ p, int64_t ld,
                                          int r, int c, int rows, int cols) {
    if (r >= rows) return 0u;
    const uint8_t* row = p + (int64_t)r * ld;
    if (ALIGN4 && c + 3 < cols) return *reinterpret_cast<const uint32_t*>(row + c);
    uint32_t v = 0;
#pragma unroll
    for (int b = 0; b < 4; ++b)
        if (c + b < cols) v |= (uint32_t)row[c + b] << (8 * b);
    return v;
}

// 4x4 byte transpose: out[i] byte j = in[j] byte i.
__device__ __forceinline__ void transpose4x4(uint32_t d[4]) {
    uint32_t lo01 = __builtin_amdgcn_perm(d[1], d[0], 0x05010400u);
    uint32_t hi01 = __builtin_amdgcn_perm(d[1], d[0], 0x07030602u);
    uint32_t lo23 = __builtin_amdgcn_perm(d[3], d[2], 0x05010400u);
    uint32_t hi23 = __builtin_amdgcn_perm(d[3], d[2], 0x07030602u);
    d[0] = __builtin_amdgcn_perm(lo23, lo01, 0x05040100u);
    d[1] = __builtin_amdgcn_perm(lo23, lo01, 0x07060302u);
    d[2] = __builtin_amdgcn_perm(hi23, hi01, 0x05040100u);
    d[3] = __builtin_amdgcn_perm(hi23, hi01, 0x07060302u);
}

// Operand tile loader: a 128 x 64 slab (rows = M or N index, k = 0..63) of
// an operand whose k index is contiguous in memory (KC = true) or whose row
// index is contiguous (KC = false), written k-contiguous into LDS.
template <bool KC, bool ALIGN4>
struct SlabLoader {
    // KC: 128 rows x 16 dwords = 2048 dwords, 8 per thread.
    // !KC: 32 row-groups x 16 k-groups of 4x4 bytes = 512 blocks, 2 per thread.
    static constexpr int NREG = 8;
    uint32_t r[NREG];

    __device__ __forceinline__ void load(const uint8_t* __restrict__ p, int64_t ld,
                                         int row0, int k0, int rows, int K, int tid) {
        if (KC) {
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const int e = tid + MF_NT * q;
                const int rr = e / 16, kq = (e % 16) * 4;
                r[q] = load4<ALIGN4>(p, ld, row0 + rr, k0 + kq, rows, K);
            }
        } else {
            // memory is k-major: element (row, k) at p[k * ld + row]
#pragma unroll
            for (int q = 0; q < 2; ++q) {
                const int blk = tid + MF_NT * q;
                const int rg = blk % 32, kg = blk / 32;
#pragma unroll
                for (int b = 0; b < 4; ++b)
                    r[q * 4 + b] = load4<ALIGN4>(p, ld, k0 + kg * 4 + b, row0 + rg * 4,
                                                 K, rows);
            }
        }
    }

    __device__ __forceinline__ void store(uint8_t (*lds)[MF_PITCH], int tid) {
        if (KC) {
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const int e = tid + MF_NT * q;
                const int rr = e / 16, kq = (e % 16) * 4;
                *reinterpret_cast<uint32_t*>(&lds[rr][kq]) = r[q];
            }
        } else {
#pragma unroll
            for (int q = 0; q < 2; ++q) {
                const int blk = tid + MF_NT * q;
                const int rg = blk % 32, kg = blk / 32;
                uint32_t d[4] = {r[q * 4 + 0], r[q * 4 + 1], r[q * 4 + 2], r[q * 4 + 3]};
                transpose4x4(d);
#pragma unroll
                for (int b = 0; b < 4; ++b)
                    *reinterpret_cast<uint32_t*>(&lds[rg * 4 + b][kg * 4]) = d[b];
            }
        }
    }
};

template <bool TA, bool TB, bool ALIGN4>
__global__ __launch_bounds__(MF_NT) void chunk_gemm_mfma(
    int M, int N, int K, int CL, const uint8_t* __restrict__ A, int64_t lda,
    const uint8_t* __restrict__ B, int64_t ldb, uint16_t* __restrict__ C,
    int64_t ldc) {
    __shared__ __attribute__((aligned(16))) uint8_t As[2][MF_BM][MF_PITCH];
    __shared__ __attribute__((aligned(16))) uint8_t Bs[2][MF_BN][MF_PITCH];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wy = wave >> 1, wx = wave & 1;
    const int m0 = blockIdx.x * MF_BM, n0 = blockIdx.y * MF_BN;

    SlabLoader<!TA, ALIGN4> la;    // A is k-contiguous unless transposed
    SlabLoader<TB, ALIGN4> lb;     // B is k-contiguous only when transposed

    v16f acc[2][2];
    float S[2][2][16];
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int bj = 0; bj < 2; ++bj) {
#pragma unroll
            for (int r = 0; r < 16; ++r) { acc[bi][bj][r] = 0.0f; S[bi][bj][r] = 0.0f; }
        }

    auto flush = [&]() {
#pragma unroll
        for (int bi = 0; bi < 2; ++bi)
#pragma unroll
            for (int bj = 0; bj < 2; ++bj)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    float p = rn16s(acc[bi][bj][r] * 0x1p96f);
                    S[bi][bj][r] = rn16s(S[bi][bj][r] + p);
                    acc[bi][bj][r] = 0.0f;
                }
    };

    const int nslabs = (K + MF_BK - 1) / MF_BK;
    const int lrow = lane & 31, lk = (lane >> 5) * 8;
    int crem = CL;
    if (nslabs > 0) {
        la.load(A, lda, m0, 0, M, K, tid);
        lb.load(B, ldb, n0, 0, N, K, tid);
        la.store(As[0], tid);
        lb.store(Bs[0], tid);
        __syncthreads();
    }
    for (int s = 0; s < nslabs; ++s) {
        const int buf = s & 1;
        if (s + 1 < nslabs) {
            la.load(A, lda, m0, (s + 1) * MF_BK, M, K, tid);
            lb.load(B, ldb, n0, (s + 1) * MF_BK, N, K, tid);
        }
        const int ksteps = min(MF_BK, K - s * MF_BK + 15) / 16;   // 16-wide steps
        for (int ks = 0; ks < ksteps; ++ks) {
            long a[2], b[2];
#pragma unroll
            for (int bi = 0; bi < 2; ++bi)
                a[bi] = *reinterpret_cast<const long*>(
                    &As[buf][wy * 64 + bi * 32 + lrow][ks * 16 + lk]);
#pragma unroll
            for (int bj = 0; bj < 2; ++bj)
                b[bj] = *reinterpret_cast<const long*>(
                    &Bs[buf][wx * 64 + bj * 32 + lrow][ks * 16 + lk]);
#pragma unroll
            for (int bi = 0; bi < 2; ++bi)
#pragma unroll
                for (int bj = 0; bj < 2; ++bj)
                    acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x16_bf8_bf8(
                        a[bi], b[bj], acc[bi][bj], 0, 0, 0);
            crem -= 16;
            if (crem == 0) {
                flush();
                crem = CL;
            }
        }
        if (s + 1 < nslabs) {
            la.store(As[buf ^ 1], tid);
            lb.store(Bs[buf ^ 1], tid);
        }
        __syncthreads();
    }
    if (crem != CL) flush();

    // D layout of the 32x32 MFMA: lane l, register r -> row 8(r/4) + 4(l/32) +
    // r%4, column l%32.
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int bj = 0; bj < 2; ++bj)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int m = m0 + wy * 64 + bi * 32 + 8 * (r / 4) + 4 * (lane >> 5) + (r % 4);
                const int n = n0 + wx * 64 + bj * 32 + (lane & 31);
                if (m < M && n < N) C[(int64_t)m * ldc + n] = f32s_to_fp16(S[bi][bj][r]);
            }
}

// ---------------------------------------------------------------------------
// fold: finish the shared tiles
// ---------------------------------------------------------------------------

// One thread per output of a shared tile: continue the running sum held in C
// (the FP16 sum of the tile's first piece) over the chunk sums the other
// pieces left in the workspace, in ascending chunk order -- the same
// additions a whole-tile pass makes after its first piece.
__global__ __launch_bounds__(256) void chunk_fold(GemmArgs g, Plan p, int BM, int BN) {
    const int64_t per = (int64_t)BM * BN;
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t lt = idx / per;
    if (lt * p.nch >= p.L) return;
    const int local = (int)(idx - lt * per);
    const int64_t tile = p.t_whole + lt;
    const int m = (int)(tile / p.tiles_n) * BM + local / BN;
    const int n = (int)(tile % p.tiles_n) * BN + local % BN;
    if (m >= g.M || n >= g.N) return;
    const int a = first_piece_end(p, lt);
    if (a >= p.nch) return;
    uint16_t* cp = g.C + (int64_t)m * g.ldc + n;
    float S = fp16_to_f32s(*cp);
    const uint16_t* src = g.ws + lt * p.nch * per + local;
    int c = a;
    for (; c + 8 <= p.nch; c += 8) {
        uint32_t v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = src[(int64_t)(c + j) * per];
#pragma unroll
        for (int j = 0; j < 8; ++j) S = rn16s(S + fp16_to_f32s(v[j]));
    }
    for (; c < p.nch; ++c) S = rn16s(S + fp16_to_f32s(src[(int64_t)c * per]));
    *cp = f32s_to_fp16(S);
}

__global__ void fill_zero_u16(uint16_t* __restrict__ C, int M, int N, int64_t ldc) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t total = (int64_t)M * N;
    if (i < total) C[(i / N) * ldc + (i % N)] = 0;
}

// ---------------------------------------------------------------------------
// planner
// ---------------------------------------------------------------------------

constexpr double kClockHz = 2.4e9;      // MI355X peak engine clock
constexpr double kLanesPerCU = 128.0;   // 32-bit VALU lane-ops per clock per CU
constexpr double kFoldBytesPerS = 4e12; // effective HBM rate of the fold pass

int env_int(const char* name, int dflt) {
    const char* v = getenv(name);
    return v ? atoi(v) : dflt;
}

// Compute units of the current device (cached per device).
int device_cus() {
    static std::mutex mu;
    static int cached[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
    std::lock_guard<std::mutex> lk(mu);
    if (!cached[dev]) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
            return 0;
        cached[dev] = n;
    }
    return cached[dev];
}

// Resident workgroups per CU of a kernel (cached per device and kernel).
int kernel_occupancy(const void* fn, int threads) {
    static std::mutex mu;
    struct Ent { int dev; const void* fn; int occ; };
    static Ent cache[256];
    static int n = 0;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    std::lock_guard<std::mutex> lk(mu);
    for (int i = 0; i < n; ++i)
        if (cache[i].dev == dev && cache[i].fn == fn) return cache[i].occ;
    int occ = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, fn, threads, 0) != hipSuccess)
        return 0;
    if (n < 256) cache[n++] = Ent{dev, fn, occ};
    return occ;
}

// Relative cost per multiply-accumulate of each register tile on a fully
// loaded CU, in VALU instructions (4 for the rounded FMA of the guarded path,
// plus operand decode, LDS reads, loop overhead and lost occupancy; measured
// on the conv-stage GEMMs for the large tiles).
double valu_ops_per_mac(int cfg) {
    switch (cfg) {
        case 4: return 4.6;     // 4 x 4, 4 waves per SIMD
        case 3: return 4.85;    // 4 x 8
        case 2: return 4.9;     // 8 x 4
        case 1: return 5.1;     // 8 x 8, 2 waves per SIMD
        case 0: return 5.2;
        case 5: return 6.5;     // 2 x 2
        default: return 10.0;   // 1 x 1
    }
}

struct Choice {
    int cfg = -1;
    ValuShape shape{};
    Plan plan{};
    size_t ws_bytes = 0;
    double est_s = 0.0;
};

constexpr size_t kWsAlign = 256;

// The best configuration for these sizes; with allow_ws false only plans
// that need no workspace are considered.
Choice plan_valu(int ta, int tb, int fast, int64_t M, int64_t N, int64_t K, int64_t CL,
                 bool allow_ws) {
    Choice best;
    const int cus = device_cus();
    if (cus <= 0) return best;
    // Overrides for tests and tuning: the register tile, a cap on the
    // workgroups, and 1 / 0 to require / forbid shared tiles.
    int force_cfg = env_int("FP8T_VALU_TILE", -1);
    if (force_cfg >= 0 && (force_cfg >= kValuConfigs || !valu_kernel(force_cfg, ta, tb, fast)))
        force_cfg = -1;                      // not built for this mode: plan freely
    const int force_g = env_int("FP8T_GEMM_WGS", 0);
    const int force_split = env_int("FP8T_GEMM_SPLIT", -1);
    const int64_t nch = (K + CL - 1) / CL;
    for (int cfg = 0; cfg < kValuConfigs; ++cfg) {
        if (force_cfg >= 0 && cfg != force_cfg) continue;
        if (force_cfg < 0 && cfg == 0) continue;      // cfg 0 is kept for comparison only
        const ValuShape sh = valu_shape(cfg);
        const void* fn = valu_kernel(cfg, ta, tb, fast);
        if (!fn) continue;
        int occ = kernel_occupancy(fn, sh.NT);
        if (occ <= 0) continue;
        if (occ > 8) occ = 8;
        const int64_t tiles_m = (M + sh.BM - 1) / sh.BM;
        const int64_t tiles_n = (N + sh.BN - 1) / sh.BN;
        const int64_t T = tiles_m * tiles_n;
        int64_t gmax = (int64_t)cus * occ;
        if (force_g > 0 && force_g < gmax) gmax = force_g;
        // time of one tile-chunk on a CU
        const double t_chunk = (double)sh.BM * sh.BN * (double)CL * valu_ops_per_mac(cfg) /
                               (kLanesPerCU * kClockHz);
        for (int split = 0; split < 2; ++split) {
            if (split && !allow_ws) continue;
            if (force_split == 0 && split) continue;
            Plan p{};
            p.tiles_n = tiles_n;
            p.nch = (int)nch;
            double est;
            size_t ws = 0;
            if (!split) {
                const int64_t G = T < gmax ? T : gmax;
                p.G = (int)G;
                p.t_whole = T;
                p.L = 0;
                // tile-chunks on the busiest CU
                const int64_t per_cu = (T + cus - 1) / cus;
                est = (double)per_cu * nch * t_chunk;
            } else {
                int64_t G = gmax;
                if (G > T * nch) G = T * nch;
                const int64_t q = T / G;
                p.G = (int)G;
                p.t_whole = q * G;
                p.L = (T - p.t_whole) * nch;
                if (p.L == 0) continue;                    // same as the plain plan
                const int64_t wg_per_cu = (G + cus - 1) / cus;
                const int64_t per_wg = q * nch + (p.L + G - 1) / G;
                ws = (size_t)(T - p.t_whole) * nch * sh.BM * sh.BN * sizeof(uint16_t) + kWsAlign;
                est = (double)wg_per_cu * per_wg * t_chunk + 2.0 * (double)ws / kFoldBytesPerS +
                      4e-6;
            }
            if (force_split == 1 && !split && allow_ws) est *= 1e6;   // any shared plan wins
            if (env_int("FP8T_GEMM_VERBOSE", 0))
                fprintf(stderr, "[fp8t plan] cfg %d occ %d split %d G %d T %lld t_whole %lld L %lld "
                        "ws %zu est %.1f us\n", cfg, occ, split, p.G, (long long)T,
                        (long long)p.t_whole, (long long)p.L, ws, est * 1e6);
            if (best.cfg < 0 || est < best.est_s) {
                best.cfg = cfg;
                best.shape = sh;
                best.plan = p;
                best.ws_bytes = ws;
                best.est_s = est;
            }
        }
    }
    return best;
}

int launch_valu_plan(const Choice& ch, int ta, int tb, int fast, GemmArgs g,
                     hipStream_t stream) {
    void* args[] = {&g, const_cast<Plan*>(&ch.plan)};
    if (hipLaunchKernel(valu_kernel(ch.cfg, ta, tb, fast), dim3(ch.plan.G),
                        dim3(ch.shape.NT), args, 0, stream) != hipSuccess)
        return FP8T_EHIP;
    if (ch.plan.L > 0) {
        const int64_t shared = ch.plan.L / ch.plan.nch;
        const int64_t threads = shared * ch.shape.BM * ch.shape.BN;
        hipLaunchKernelGGL(chunk_fold, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0,
                           stream, g, ch.plan, ch.shape.BM, ch.shape.BN);
    }
    return launch_status();
}

int dispatch_mfma(int ta, int tb, int M, int N, int K, int CL, const uint8_t* A,
                  int64_t lda, const uint8_t* B, int64_t ldb, uint16_t* C, int64_t ldc,
                  hipStream_t stream) {
    const bool al = aligned(A, 4) && aligned(B, 4) && lda % 4 == 0 && ldb % 4 == 0;
    dim3 grid((M + MF_BM - 1) / MF_BM, (N + MF_BN - 1) / MF_BN);
    if (grid.y > 65535u) return FP8T_EINVAL;
#define FP8T_LAUNCH(TA_, TB_, AL_)                                                    \
    hipLaunchKernelGGL((chunk_gemm_mfma<TA_, TB_, AL_>), grid, dim3(MF_NT), 0, stream, \
                       M, N, K, CL, A, lda, B, ldb, C, ldc)
    if (al) {
        if (!ta && !tb) FP8T_LAUNCH(false, false, true);
        else if (!ta && tb) FP8T_LAUNCH(false, true, true);
        else if (ta && !tb) FP8T_LAUNCH(true, false, true);
        else FP8T_LAUNCH(true, true, true);
    } else {
        if (!ta && !tb) FP8T_LAUNCH(false, false, false);
        else if (!ta && tb) FP8T_LAUNCH(false, true, false);
        else if (ta && !tb) FP8T_LAUNCH(true, false, false);
        else FP8T_LAUNCH(true, true, false);
    }
#undef FP8T_LAUNCH
    return launch_status();
}


}  // namespace
}  // namespace fp8t

using namespace fp8t;

namespace {
bool gemm_args_ok(int ta, int tb, int64_t M, int64_t N, int64_t K, int64_t CL, int mode) {
    if (M < 0 || N < 0 || K < 0 || CL < 1) return false;
    if ((ta != 0 && ta != 1) || (tb != 0 && tb != 1)) return false;
    if (mode != FP8T_EXACT && mode != FP8T_FAST) return false;
    // indices inside the kernels are 32-bit per dimension
    if (M > INT32_MAX || N > INT32_MAX || K > INT32_MAX) return false;
    return true;
}

bool uses_mfma(int mode, int64_t K, int64_t CL) {
    const int64_t cl = CL > K ? K : CL;
    return mode == FP8T_FAST && cl % 16 == 0;
}
}  // namespace

extern "C" size_t chunk_gemm_workspace_size(int trans_a, int trans_b, int64_t M,
                                            int64_t N, int64_t K, int64_t CL, int mode) {
    if (!gemm_args_ok(trans_a, trans_b, M, N, K, CL, mode)) return 0;
    if (M == 0 || N == 0 || K == 0 || uses_mfma(mode, K, CL)) return 0;
    const int64_t cl = CL > K ? K : CL;
    const Choice ch = plan_valu(trans_a, trans_b, mode == FP8T_FAST, M, N, K, cl, true);
    return ch.cfg < 0 ? 0 : ch.ws_bytes;
}

extern "C" int chunk_gemm(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K,
                          int64_t CL, const uint8_t* A, int64_t lda, const uint8_t* B,
                          int64_t ldb, uint16_t* C, int64_t ldc, int mode,
                          void* workspace, size_t workspace_bytes, hipStream_t stream) {
    if (!gemm_args_ok(trans_a, trans_b, M, N, K, CL, mode)) return FP8T_EINVAL;
    if (M == 0 || N == 0) return FP8T_OK;
    if (!C || ldc < N) return FP8T_EINVAL;
    if (K > 0) {
        if (!A || !B) return FP8T_EINVAL;
        if (lda < (trans_a ? M : K) || ldb < (trans_b ? K : N)) return FP8T_EINVAL;
    }
    if (workspace_bytes > 0 && !workspace) return FP8T_EINVAL;
    if (CL > K && K > 0) CL = K;           // one chunk
    const int m = (int)M, n = (int)N, k = (int)K, cl = (int)(K > 0 ? CL : 1);
    if (K == 0) {
        const int64_t total = M * N;
        hipLaunchKernelGGL(fill_zero_u16, dim3((unsigned)((total + 255) / 256)), dim3(256),
                           0, stream, C, m, n, ldc);
        return launch_status();
    }
    if (uses_mfma(mode, K, cl))
        return dispatch_mfma(trans_a, trans_b, m, n, k, cl, A, lda, B, ldb, C, ldc, stream);

    const int fast = mode == FP8T_FAST;
    // With no workspace, the best plan that needs none; with one, the best
    // plan overall, which must then fit.
    Choice ch = plan_valu(trans_a, trans_b, fast, M, N, K, cl, workspace_bytes > 0);
    if (ch.cfg < 0) return FP8T_EHIP;
    if (ch.ws_bytes > workspace_bytes) return FP8T_EWORKSPACE;
    GemmArgs g{};
    g.A = A;
    g.B = B;
    g.C = C;
    g.ws = nullptr;
    if (ch.plan.L > 0) {
        const uintptr_t base = ((uintptr_t)workspace + kWsAlign - 1) & ~(uintptr_t)(kWsAlign - 1);
        g.ws = reinterpret_cast<uint16_t*>(base);
    }
    g.lda = lda;
    g.ldb = ldb;
    g.ldc = ldc;
    g.M = m;
    g.N = n;
    g.K = k;
    g.CL = cl;
    g.a_vec = aligned(A, 4) && lda % 4 == 0;
    g.b_vec = aligned(B, 4) && ldb % 4 == 0;
    g.c_vec = aligned(C, 4) && ldc % 2 == 0;
    // FP8T_GEMM_GUARD=0 runs every piece on the safe path (tests, tuning).
    g.guarded = env_int("FP8T_GEMM_GUARD", 1) != 0;
    return launch_valu_plan(ch, trans_a, trans_b, fast, g, stream);
}
