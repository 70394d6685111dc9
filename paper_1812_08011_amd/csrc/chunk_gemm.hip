// chunk_gemm: FP8 x FP8 GEMM with chunk-based FP16 accumulation
// (Sec. 2.3 "Chunk-based Accumulation", dot-product algorithm of Fig. 3(a)).
//
// Two kernels:
//
// * chunk_gemm_valu -- the exact mode (and the fast mode for chunk lengths
//   the matrix cores cannot split).  Every output keeps two registers, the
//   intra-chunk sum P and the running sum S, in the scaled FP32 domain of
//   fp8t_device.h.  One multiply-accumulate step is
//       P = rn16s(fma(a * 2^96, b, P))        (v_fma, v_bfe, v_add3, v_and)
//   -- the product of two FP8 values is exact in FP32, so the FMA's single
//   rounding is the rounding of the exact sum -- and at every chunk end
//       S = rn16s(S + P), P = +0.
//   This is VALU-bound by construction (gfx950 has no adder for the paper's
//   FP16), so the kernel is shaped to keep the VALU busy: a TM x TN register
//   tile per lane, operands staged through LDS already decoded to FP32 (one
//   decode per element per workgroup tile instead of per use), and a
//   double-buffered K loop that prefetches the next slab from HBM into
//   registers while the current slab is consumed.
//
// * chunk_gemm_mfma -- the fast mode for CL a multiple of 16.  FP8 bytes are
//   the OCP E5M2 ("bf8") encoding (same bias, subnormals and specials), so
//   the FP8 codes feed v_mfma_f32_32x32x16_bf8_bf8 directly.  Each wave owns a
//   64x64 output tile (2x2 MFMA blocks); each chunk is accumulated on the
//   matrix cores from zero, then rounded to FP16 and added into S on the VALU.
#include "fp8t_device.h"
#include "fp8train.h"
#include "fp8t_host.h"

#include <stdlib.h>

namespace fp8t {
namespace {

// ---------------------------------------------------------------------------
// VALU kernel
// ---------------------------------------------------------------------------

template <int TM, int TN, int LM, int LN, int BK, bool TA, bool TB, bool FAST>
__global__ __launch_bounds__(LM * LN) void chunk_gemm_valu(
    int M, int N, int K, int CL, const uint8_t* __restrict__ A, int64_t lda,
    const uint8_t* __restrict__ B, int64_t ldb, uint16_t* __restrict__ C,
    int64_t ldc) {
    constexpr int NT = LM * LN;
    constexpr int BM = TM * LM;
    constexpr int BN = TN * LN;
    constexpr int EA = BM * BK / NT;         // A bytes loaded per thread per slab
    constexpr int EB = BN * BK / NT;
    static_assert(EA * NT == BM * BK && EB * NT == BN * BK, "tile/threads mismatch");
    // pad rows written with a stride across lanes to spread LDS banks
    constexpr int PA = TA ? 0 : 4;
    constexpr int PB = TB ? 4 : 0;
    // A holds a * 2^96 in exact mode (the scaled domain); the fast VALU path
    // sums plain products in FP32 and scales once per chunk.
    constexpr int ASHIFT = FAST ? 0 : 96;

    __shared__ float As[2][BK][BM + PA];
    __shared__ float Bs[2][BK][BN + PB];

    const int tid = threadIdx.x;
    const int ly = tid / LN, lx = tid % LN;
    const int m0 = blockIdx.x * BM, n0 = blockIdx.y * BN;

    uint32_t ra[EA], rb[EB];

    auto load_slab = [&](int k0) {
#pragma unroll
        for (int r = 0; r < EA; ++r) {
            const int e = tid + NT * r;
            const int mm = TA ? (e % BM) : (e / BK);
            const int kk = TA ? (e / BM) : (e % BK);
            const int m = m0 + mm, k = k0 + kk;
            uint32_t v = 0;
            if (m < M && k < K)
                v = TA ? A[(int64_t)k * lda + m] : A[(int64_t)m * lda + k];
            ra[r] = v;
        }
#pragma unroll
        for (int r = 0; r < EB; ++r) {
            const int e = tid + NT * r;
            const int nn = TB ? (e / BK) : (e % BN);
            const int kk = TB ? (e % BK) : (e / BN);
            const int n = n0 + nn, k = k0 + kk;
            uint32_t v = 0;
            if (n < N && k < K)
                v = TB ? B[(int64_t)n * ldb + k] : B[(int64_t)k * ldb + n];
            rb[r] = v;
        }
    };
    auto store_slab = [&](int buf) {
#pragma unroll
        for (int r = 0; r < EA; ++r) {
            const int e = tid + NT * r;
            const int mm = TA ? (e % BM) : (e / BK);
            const int kk = TA ? (e / BM) : (e % BK);
            As[buf][kk][mm] = fp8_to_f32<ASHIFT>(ra[r]);
        }
#pragma unroll
        for (int r = 0; r < EB; ++r) {
            const int e = tid + NT * r;
            const int nn = TB ? (e / BK) : (e % BN);
            const int kk = TB ? (e % BK) : (e / BN);
            Bs[buf][kk][nn] = fp8_to_f32<0>(rb[r]);
        }
    };

    float P[TM][TN], S[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) { P[i][j] = 0.0f; S[i][j] = 0.0f; }

    auto mac = [&](int buf, int kk) {
        float a[TM], b[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i) a[i] = As[buf][kk][ly * TM + i];
#pragma unroll
        for (int j = 0; j < TN; ++j) b[j] = Bs[buf][kk][lx * TN + j];
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                float t = __builtin_fmaf(a[i], b[j], P[i][j]);
                P[i][j] = FAST ? t : rn16s(t);
            }
    };
    auto flush = [&]() {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                float p = FAST ? rn16s(P[i][j] * 0x1p96f) : P[i][j];
                S[i][j] = rn16s(S[i][j] + p);
                P[i][j] = 0.0f;
            }
    };

    const int nslabs = (K + BK - 1) / BK;
    int crem = CL;                  // products left in the current chunk
    if (nslabs > 0) {
        load_slab(0);
        store_slab(0);
        __syncthreads();
    }
    for (int s = 0; s < nslabs; ++s) {
        const int buf = s & 1;
        if (s + 1 < nslabs) load_slab((s + 1) * BK);
        const int kmax = min(BK, K - s * BK);
        int kk = 0;
        while (kk < kmax) {
            const int seg = min(kmax - kk, crem);
            if (seg == BK) {
#pragma unroll
                for (int q = 0; q < BK; ++q) mac(buf, q);
            } else {
                for (int q = kk; q < kk + seg; ++q) mac(buf, q);
            }
            kk += seg;
            crem -= seg;
            if (crem == 0) {
                flush();
                crem = CL;
            }
        }
        if (s + 1 < nslabs) store_slab(buf ^ 1);
        __syncthreads();
    }
    if (crem != CL) flush();        // the last, shorter chunk

#pragma unroll
    for (int i = 0; i < TM; ++i) {
        const int m = m0 + ly * TM + i;
        if (m >= M) continue;
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int n = n0 + lx * TN + j;
            if (n < N) C[(int64_t)m * ldc + n] = f32s_to_fp16(S[i][j]);
        }
    }
}

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
// host dispatch
// ---------------------------------------------------------------------------

template <int TM, int TN, int LM, int LN, int BK, bool FAST>
int launch_valu(int ta, int tb, int M, int N, int K, int CL, const uint8_t* A,
                int64_t lda, const uint8_t* B, int64_t ldb, uint16_t* C, int64_t ldc,
                hipStream_t stream) {
    constexpr int BM = TM * LM, BN = TN * LN;
    dim3 grid((M + BM - 1) / BM, (N + BN - 1) / BN);
    if (grid.y > 65535u) return FP8T_EINVAL;
    dim3 block(LM * LN);
#define FP8T_LAUNCH(TA_, TB_)                                                        \
    hipLaunchKernelGGL((chunk_gemm_valu<TM, TN, LM, LN, BK, TA_, TB_, FAST>), grid, \
                       block, 0, stream, M, N, K, CL, A, lda, B, ldb, C, ldc)
    if (!ta && !tb) FP8T_LAUNCH(false, false);
    else if (!ta && tb) FP8T_LAUNCH(false, true);
    else if (ta && !tb) FP8T_LAUNCH(true, false);
    else FP8T_LAUNCH(true, true);
#undef FP8T_LAUNCH
    return launch_status();
}

template <bool FAST>
int dispatch_valu(int ta, int tb, int M, int N, int K, int CL, const uint8_t* A,
                  int64_t lda, const uint8_t* B, int64_t ldb, uint16_t* C, int64_t ldc,
                  hipStream_t stream) {
    // FP8T_VALU_TILE = 1, 2, 4 or 8 forces the register tile (for tests and
    // tuning).  Otherwise: the largest square register tile that still gives
    // every SIMD (1024 on the chip) at least two waves.
    const char* force = getenv("FP8T_VALU_TILE");
    const int t = force ? atoi(force) : 0;
    if (t == 8)
        return launch_valu<8, 8, 16, 16, 16, FAST>(ta, tb, M, N, K, CL, A, lda, B, ldb, C, ldc, stream);
    if (t == 4)
        return launch_valu<4, 4, 16, 16, 32, FAST>(ta, tb, M, N, K, CL, A, lda, B, ldb, C, ldc, stream);
    if (t == 2)
        return launch_valu<2, 2, 16, 16, 32, FAST>(ta, tb, M, N, K, CL, A, lda, B, ldb, C, ldc, stream);
    if (t == 1)
        return launch_valu<1, 1, 16, 16, 64, FAST>(ta, tb, M, N, K, CL, A, lda, B, ldb, C, ldc, stream);
    const int64_t outs = (int64_t)M * N;
    if (outs / 64 >= 2048 * 64)
        return launch_valu<8, 8, 16, 16, 16, FAST>(ta, tb, M, N, K, CL, A, lda, B, ldb, C, ldc, stream);
    if (outs / 16 >= 2048 * 64)
        return launch_valu<4, 4, 16, 16, 32, FAST>(ta, tb, M, N, K, CL, A, lda, B, ldb, C, ldc, stream);
    if (outs / 4 >= 2048 * 64)
        return launch_valu<2, 2, 16, 16, 32, FAST>(ta, tb, M, N, K, CL, A, lda, B, ldb, C, ldc, stream);
    return launch_valu<1, 1, 16, 16, 64, FAST>(ta, tb, M, N, K, CL, A, lda, B, ldb, C, ldc, stream);
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

__global__ void fill_zero_u16(uint16_t* __restrict__ C, int M, int N, int64_t ldc) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t total = (int64_t)M * N;
    if (i < total) C[(i / N) * ldc + (i % N)] = 0;
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
}  // namespace

extern "C" size_t chunk_gemm_workspace_size(int trans_a, int trans_b, int64_t M,
                                            int64_t N, int64_t K, int64_t CL, int mode) {
    (void)trans_a; (void)trans_b; (void)M; (void)N; (void)K; (void)CL; (void)mode;
    return 0;
}

extern "C" int chunk_gemm(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K,
                          int64_t CL, const uint8_t* A, int64_t lda, const uint8_t* B,
                          int64_t ldb, uint16_t* C, int64_t ldc, int mode,
                          void* workspace, size_t workspace_bytes, hipStream_t stream) {
    (void)workspace;
    if (!gemm_args_ok(trans_a, trans_b, M, N, K, CL, mode)) return FP8T_EINVAL;
    if (M == 0 || N == 0) return FP8T_OK;
    if (!C || ldc < N) return FP8T_EINVAL;
    if (K > 0) {
        if (!A || !B) return FP8T_EINVAL;
        if (lda < (trans_a ? M : K) || ldb < (trans_b ? K : N)) return FP8T_EINVAL;
    }
    if (workspace_bytes < chunk_gemm_workspace_size(trans_a, trans_b, M, N, K, CL, mode))
        return FP8T_EWORKSPACE;
    if (CL > K && K > 0) CL = K;           // one chunk
    const int m = (int)M, n = (int)N, k = (int)K, cl = (int)(K > 0 ? CL : 1);
    if (K == 0) {
        const int64_t total = M * N;
        hipLaunchKernelGGL(fill_zero_u16, dim3((unsigned)((total + 255) / 256)), dim3(256),
                           0, stream, C, m, n, ldc);
        return launch_status();
    }
    if (mode == FP8T_FAST && cl % 16 == 0)
        return dispatch_mfma(trans_a, trans_b, m, n, k, cl, A, lda, B, ldb, C, ldc, stream);
    if (mode == FP8T_FAST)
        return dispatch_valu<true>(trans_a, trans_b, m, n, k, cl, A, lda, B, ldb, C, ldc, stream);
    return dispatch_valu<false>(trans_a, trans_b, m, n, k, cl, A, lda, B, ldb, C, ldc, stream);
}
