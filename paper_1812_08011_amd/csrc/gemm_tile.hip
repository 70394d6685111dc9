// chunk_gemm_sr: the chunk-based GEMM of Sec. 2.3 / Fig. 3(a) with FP8
// operands and every FP16 addition rounded stochastically (Eq. (1)) instead
// of to nearest -- the paper's second rounding mode after FP16 additions,
// whose behaviour on long accumulations Fig. 3(b) compares with nearest
// rounding.  A vector-ALU tile kernel.
//
// Each addition first forms the FP32 sum of the running value and the next
// product (a product of two FP8 values is exact in FP32) and then rounds it
// into FP16.  As in chunk_gemm's exact mode, FP16 quantities are held scaled
// by 2^96 (fp8t_device.h), so FP16 overflow is FP32 overflow and FP16
// subnormals are FP32 normals: operands enter as a(k) 2^96 and b(k).
// Stochastic rounding of the 14 discarded mantissa bits D with uniform u
// rounds the magnitude up iff D > (u >> 2); adding (2^14 - 1 - (u >> 2)) to
// the raw bits and clearing the low 14 bits does exactly that, with the carry
// running into the exponent (and to the Inf encoding past the largest FP16
// value).  Sums below 2^-30 are multiples of 2^-39 with at most 9 significant
// bits, so their discarded bits are zero and the rounding leaves them
// unchanged, as the fixed subnormal step requires.
//
// Random bits: Philox4x32-10, key = seed, eight 16-bit uniforms per block
// (word halves, low half first).  The addition of product k into output
// (i, j) takes uniform 4 (k mod 2) + (j mod 4) of block (i, j / 4, k / 2,
// 2 offset): a thread owning 4 x 4 outputs (four rows of four aligned
// columns) draws four blocks per two k.  The addition of chunk c into the
// running sum takes uniform j mod 8 of block (i, j / 8, c, 2 offset + 1).
//
// The work decomposition is the persistent plan of gemm_plan.h: whole tiles,
// then the chunks of the remaining tiles shared out as ranges; a piece that
// does not start at chunk 0 leaves each chunk's FP16 sum in the workspace and
// chunk_fold_sr continues the running sum over them in ascending order, with
// the same random bits -- the result does not depend on the plan.
#include "fp8t_device.h"
#include "fp8train.h"
#include "fp8t_host.h"
#include "gemm_plan.h"

#include <stdio.h>

namespace fp8t {
namespace {

constexpr int kT = 4;                 // outputs per thread in each direction
constexpr int kTiles = 16;            // threads per tile edge
constexpr int kBM = kT * kTiles, kBN = kT * kTiles;
constexpr int kNT = kTiles * kTiles;  // 256 threads
constexpr int kBK = 32;               // k per LDS slab (a multiple of 8)
constexpr int kPitch = kBM + 4;       // floats per LDS row
constexpr size_t kWsAlign = 256;

struct TileArgs {
    const uint8_t* A;
    const uint8_t* B;
    uint16_t* C;
    uint16_t* ws;                     // chunk sums of the shared tiles
    int64_t lda, ldb, ldc;
    int M, N, K, CL;
    uint32_t k0, k1;                  // Philox key (stochastic rounding)
    uint32_t w3;                      // 2 * offset
    int c_vec;                        // C rows allow 8-byte stores of 4 codes
    int a_vec, b_vec;                 // A / B rows allow 8-element loads
};

// Uniform-derived addend: (2^14 - 1) - (u >> 2) for the 16-bit uniform in
// bits [16 h, 16 h + 16) of word w, taken from the complemented word.
__device__ __forceinline__ uint32_t sr_addend(uint32_t nw, int h) {
    return __builtin_amdgcn_ubfe(nw, 16 * h + 2, 14);
}

// Stochastic rounding of a scaled-domain float given its addend.
__device__ __forceinline__ float sr16s(float x, uint32_t add) {
    return __uint_as_float((__float_as_uint(x) + add) & 0xFFFFC000u);
}

__device__ __forceinline__ u32x4 block_of(uint32_t i, uint32_t j, uint32_t q, uint32_t w3,
                                          const TileArgs& g) {
    const u32x4 c = {i, j, q, w3};
    return philox4x32_10(c, g.k0, g.k1);
}

// Stage a whole slab (64 rows x 32 k, all inside the matrix, aligned rows)
// with one 8-byte load per thread, A scaled by 2^96, B plain.  KC: k is
// contiguous in memory (element (r, k) at p[r * ld + k]); otherwise the row
// index is.
template <bool IS_A, bool KC>
__device__ __forceinline__ void stage_fast(const uint8_t* __restrict__ p, int64_t ld, int r0,
                                           int k0, float (*X)[kPitch], int tid) {
    uint32_t w[2];
    float f[8];
    int r, kq, k, rq;
    if (KC) {
        r = tid / (kBK / 8), kq = (tid % (kBK / 8)) * 8;
        const uint2 v = *reinterpret_cast<const uint2*>(p + (int64_t)(r0 + r) * ld + k0 + kq);
        w[0] = v.x, w[1] = v.y;
    } else {
        k = tid / (kBM / 8), rq = (tid % (kBM / 8)) * 8;
        const uint2 v = *reinterpret_cast<const uint2*>(p + (int64_t)(k0 + k) * ld + r0 + rq);
        w[0] = v.x, w[1] = v.y;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const uint32_t c = (w[e / 4] >> (8 * (e % 4))) & 0xFFu;
        f[e] = IS_A ? fp8_to_f32<96>(c) : fp8_to_f32<0>(c);
    }
    if (KC) {
#pragma unroll
        for (int e = 0; e < 8; ++e) X[kq + e][r] = f[e];
    } else {
        *reinterpret_cast<float4*>(&X[k][rq]) = make_float4(f[0], f[1], f[2], f[3]);
        *reinterpret_cast<float4*>(&X[k][rq + 4]) = make_float4(f[4], f[5], f[6], f[7]);
    }
}

// One launch of the persistent plan: workgroup w takes whole tiles w, w + G,
// ..., then its range of the shared tile-chunks.
template <bool TA, bool TB>
__global__ __launch_bounds__(kNT) void chunk_gemm_sr_kernel(TileArgs g, Plan p) {
    const uint8_t* __restrict__ A = g.A;
    const uint8_t* __restrict__ B = g.B;
    __shared__ __attribute__((aligned(16))) float As[kBK][kPitch];
    __shared__ __attribute__((aligned(16))) float Bs[kBK][kPitch];
    const int tid = threadIdx.x;
    const int tx = tid % kTiles, ty = tid / kTiles;

    // chunks [c0, c1) of tile; lt >= 0 for a shared tile
    auto piece = [&](int64_t tile, int c0, int c1, int64_t lt) __attribute__((always_inline)) {
        int tr, tc;
        tile_rc(p, tile, tr, tc);
        const int m0 = tr * kBM;
        const int n0 = tc * kBN;
        const int kbeg = (int)((int64_t)c0 * g.CL);
        const int64_t kend64 = (int64_t)c1 * g.CL;
        const int kend = kend64 < g.K ? (int)kend64 : g.K;
        const bool to_ws = c0 > 0;
        const uint32_t gi = (uint32_t)(m0 + ty * kT), gj = (uint32_t)(n0 + tx * kT);
        float P[kT][kT], S[kT][kT];
#pragma unroll
        for (int r = 0; r < kT; ++r)
#pragma unroll
            for (int c = 0; c < kT; ++c) P[r][c] = S[r][c] = 0.0f;
        int chunk = c0;
        int64_t cend = (int64_t)(c0 + 1) * g.CL;
        if (cend > g.K) cend = g.K;

        auto chunk_end = [&]() __attribute__((always_inline)) {
            if (to_ws) {
                uint16_t* dst = g.ws + (lt * p.nch + chunk) * (int64_t)(kBM * kBN) +
                                (ty * kT) * kBN + tx * kT;
#pragma unroll
                for (int r = 0; r < kT; ++r) {
                    uint2 v;
                    v.x = (uint32_t)f32s_to_fp16(P[r][0]) | ((uint32_t)f32s_to_fp16(P[r][1]) << 16);
                    v.y = (uint32_t)f32s_to_fp16(P[r][2]) | ((uint32_t)f32s_to_fp16(P[r][3]) << 16);
                    *reinterpret_cast<uint2*>(dst + r * kBN) = v;
                }
            } else {
                // uniforms 4 (tx mod 2) + c of block (i, j / 8, chunk)
                const bool odd = tx & 1;
#pragma unroll
                for (int r = 0; r < kT; ++r) {
                    const u32x4 b = block_of(gi + r, gj >> 3, (uint32_t)chunk, g.w3 + 1u, g);
                    const uint32_t w0 = ~(odd ? b.z : b.x), w1 = ~(odd ? b.w : b.y);
#pragma unroll
                    for (int c = 0; c < kT; ++c)
                        S[r][c] = sr16s(S[r][c] + P[r][c], sr_addend(c < 2 ? w0 : w1, c % 2));
                }
            }
#pragma unroll
            for (int r = 0; r < kT; ++r)
#pragma unroll
                for (int c = 0; c < kT; ++c) P[r][c] = 0.0f;
            ++chunk;
            cend += g.CL;
            if (cend > g.K) cend = g.K;
        };

        for (int sb = kbeg & ~(kBK - 1); sb < kend; sb += kBK) {
            const int lo = sb > kbeg ? sb : kbeg;
            const int hi = sb + kBK < kend ? sb + kBK : kend;
            __syncthreads();               // the previous slab is consumed
            // stage op(A)[m0.., lo..hi) and op(B)[lo..hi), n0..) as floats;
            // rows, columns and k outside are zero
            if (lo == sb && hi == sb + kBK && m0 + kBM <= g.M && g.a_vec) {
                stage_fast<true, !TA>(A, g.lda, m0, sb, As, tid);
            } else {
#pragma unroll
                for (int q = 0; q < kBM * kBK / kNT; ++q) {
                    const int e = tid + kNT * q;
                    int mm, kk;
                    if (TA) { kk = e / kBM; mm = e % kBM; } else { mm = e / kBK; kk = e % kBK; }
                    const int m = m0 + mm, k = sb + kk;
                    uint32_t code = 0;
                    if (m < g.M && k >= lo && k < hi)
                        code = TA ? A[(int64_t)k * g.lda + m] : A[(int64_t)m * g.lda + k];
                    As[kk][mm] = fp8_to_f32<96>(code);
                }
            }
            if (lo == sb && hi == sb + kBK && n0 + kBN <= g.N && g.b_vec) {
                stage_fast<false, TB>(B, g.ldb, n0, sb, Bs, tid);
            } else {
#pragma unroll
                for (int q = 0; q < kBN * kBK / kNT; ++q) {
                    const int e = tid + kNT * q;
                    int nn, kk;
                    if (TB) { nn = e / kBK; kk = e % kBK; } else { kk = e / kBN; nn = e % kBN; }
                    const int n = n0 + nn, k = sb + kk;
                    uint32_t code = 0;
                    if (n < g.N && k >= lo && k < hi)
                        code = TB ? B[(int64_t)n * g.ldb + k] : B[(int64_t)k * g.ldb + n];
                    Bs[kk][nn] = fp8_to_f32<0>(code);
                }
            }
            __syncthreads();
#pragma unroll 1
            for (int gq = lo & ~1; gq < hi; gq += 2) {
                // rows' blocks for k = gq, gq + 1 (complemented words)
                uint32_t nw[kT][4];
#pragma unroll
                for (int r = 0; r < kT; ++r) {
                    const u32x4 b = block_of(gi + r, gj >> 2, (uint32_t)(gq >> 1), g.w3, g);
                    nw[r][0] = ~b.x;
                    nw[r][1] = ~b.y;
                    nw[r][2] = ~b.z;
                    nw[r][3] = ~b.w;
                }
#pragma unroll
                for (int s = 0; s < 2; ++s) {
                    const int k = gq + s;
                    if (k < lo || k >= hi) continue;
                    const float4 a4 = *reinterpret_cast<const float4*>(&As[k - sb][ty * kT]);
                    const float4 b4 = *reinterpret_cast<const float4*>(&Bs[k - sb][tx * kT]);
                    const float av[4] = {a4.x, a4.y, a4.z, a4.w};
                    const float bv[4] = {b4.x, b4.y, b4.z, b4.w};
#pragma unroll
                    for (int r = 0; r < kT; ++r)
#pragma unroll
                        for (int c = 0; c < kT; ++c)
                            P[r][c] = sr16s(__builtin_fmaf(av[r], bv[c], P[r][c]),
                                            sr_addend(nw[r][2 * s + c / 2], c % 2));
                    if (k + 1 == cend) chunk_end();
                }
            }
        }
        if (to_ws) return;
        // the running sum: the result of a whole tile, or the start of a
        // shared tile's chain (continued by chunk_fold_sr)
#pragma unroll
        for (int r = 0; r < kT; ++r) {
            const int m = m0 + ty * kT + r, n = n0 + tx * kT;
            if (m >= g.M) continue;
            uint16_t* cp = g.C + (int64_t)m * g.ldc + n;
            if (g.c_vec && n + kT <= g.N) {
                uint2 v;
                v.x = (uint32_t)f32s_to_fp16(S[r][0]) | ((uint32_t)f32s_to_fp16(S[r][1]) << 16);
                v.y = (uint32_t)f32s_to_fp16(S[r][2]) | ((uint32_t)f32s_to_fp16(S[r][3]) << 16);
                *reinterpret_cast<uint2*>(cp) = v;
            } else {
#pragma unroll
                for (int c = 0; c < kT; ++c)
                    if (n + c < g.N) cp[c] = f32s_to_fp16(S[r][c]);
            }
        }
    };

    const int w = blockIdx.x;
    for (int64_t t = w; t < p.t_whole; t += p.G) piece(whole_tile(p, t), 0, p.nch, -1);
    if (p.L > 0) {
        int64_t s = (int64_t)w * p.L / p.G;
        const int64_t e = (int64_t)(w + 1) * p.L / p.G;
        while (s < e) {
            const int64_t lt = s / p.nch;
            const int c0 = (int)(s - lt * p.nch);
            const int64_t c1l = e - lt * p.nch;
            const int c1 = c1l < p.nch ? (int)c1l : p.nch;
            piece(p.t_whole + lt, c0, c1, lt);
            s = lt * p.nch + c1;
        }
    }
}

// Continue the running sums of the shared tiles (in C, from their first
// pieces) over the chunk sums in the workspace, in ascending chunk order --
// the additions a whole-tile pass makes, with the same inter-chunk uniforms.
// A thread takes 8 consecutive outputs of a row: one 16-byte load of chunk
// sums and one block of uniforms per chunk.
constexpr int kFoldV = 8, kFoldTU = 8;

__global__ __launch_bounds__(256) void chunk_fold_sr(TileArgs g, Plan p) {
    const int64_t per = (int64_t)kBM * kBN;
    const int64_t idx = ((int64_t)blockIdx.x * 256 + threadIdx.x) * kFoldV;
    const int64_t lt = idx / per;
    if (lt * p.nch >= p.L) return;
    const int local = (int)(idx - lt * per);
    const int64_t tile = p.t_whole + lt;
    int tr, tc;
    tile_rc(p, tile, tr, tc);
    const int m = tr * kBM + local / kBN;
    const int n0 = tc * kBN + local % kBN;
    if (m >= g.M || n0 >= g.N) return;
    const int a = first_piece_end(p, lt);
    if (a >= p.nch) return;
    const int nv = min(kFoldV, g.N - n0);
    uint16_t* cp = g.C + (int64_t)m * g.ldc + n0;
    float S[kFoldV];
#pragma unroll
    for (int v = 0; v < kFoldV; ++v) S[v] = v < nv ? fp16_to_f32s(cp[v]) : 0.0f;
    const uint4* src = reinterpret_cast<const uint4*>(g.ws + lt * p.nch * per + local);
    const int64_t step = per / kFoldV;
    auto add = [&](const uint4& q, int c) __attribute__((always_inline)) {
        const uint32_t cw[4] = {q.x, q.y, q.z, q.w};
        const u32x4 b = block_of((uint32_t)m, (uint32_t)(n0 >> 3), (uint32_t)c, g.w3 + 1u, g);
        const uint32_t nw[4] = {~b.x, ~b.y, ~b.z, ~b.w};
#pragma unroll
        for (int v = 0; v < kFoldV; ++v) {
            const float x = S[v] + fp16_to_f32s((cw[v / 2] >> (16 * (v % 2))) & 0xFFFFu);
            S[v] = sr16s(x, sr_addend(nw[v / 2], v % 2));
        }
    };
    // Batches of kFoldTU chunk loads, the next batch in flight while one is
    // added; every batch load is unconditional (indices clamped to the last
    // chunk, the extra values never added) so the compiler waits for the
    // older batch only.
    const int last = p.nch - 1;
    auto load = [&](uint4 (&q)[kFoldTU], int c0) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < kFoldTU; ++u) q[u] = src[(int64_t)min(c0 + u, last) * step];
    };
    auto fold = [&](const uint4 (&q)[kFoldTU], int c0) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < kFoldTU; ++u)
            if (c0 + u < p.nch) add(q[u], c0 + u);
    };
    uint4 q0[kFoldTU], q1[kFoldTU];
    int c = a;
    load(q0, c);
    for (;;) {
        if (c + kFoldTU >= p.nch) {
            fold(q0, c);
            break;
        }
        load(q1, c + kFoldTU);
        fold(q0, c);
        c += kFoldTU;
        if (c + kFoldTU >= p.nch) {
            fold(q1, c);
            break;
        }
        load(q0, c + kFoldTU);
        fold(q1, c);
        c += kFoldTU;
    }
#pragma unroll
    for (int v = 0; v < kFoldV; ++v)
        if (v < nv) cp[v] = f32s_to_fp16(S[v]);
}

__global__ void fill_zero16(uint16_t* __restrict__ C, int64_t ldc, int M, int N) {
    const int64_t total = (int64_t)M * N;
    const int64_t step = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += step)
        C[(i / N) * ldc + i % N] = 0;
}

const void* tile_kernel(int ta, int tb) {
    if (!ta && !tb) return reinterpret_cast<const void*>(&chunk_gemm_sr_kernel<false, false>);
    if (!ta && tb) return reinterpret_cast<const void*>(&chunk_gemm_sr_kernel<false, true>);
    if (ta && !tb) return reinterpret_cast<const void*>(&chunk_gemm_sr_kernel<true, false>);
    return reinterpret_cast<const void*>(&chunk_gemm_sr_kernel<true, true>);
}

struct TilePlan {
    Plan plan;
    size_t ws_bytes = 0;
    bool ok = false;
};

// One workgroup per resident slot; with a workspace allowed, tiles that do
// not divide evenly over the slots have their chunks shared out (every
// workgroup then ends with the same number of chunks).
TilePlan plan_tile(const void* fn, int64_t M, int64_t N, int64_t K, int64_t CL, bool allow_ws) {
    TilePlan r;
    const int cus = device_cus();
    const int occ = kernel_occupancy(fn, kNT);
    if (cus <= 0 || occ <= 0) return r;
    int64_t gmax = (int64_t)cus * occ;
    const int force_g = env_int("FP8T_GEMM_WGS", 0);
    if (force_g > 0 && force_g < gmax) gmax = force_g;
    const int force_split = env_int("FP8T_GEMM_SPLIT", -1);
    const int64_t tiles_m = (M + kBM - 1) / kBM, tiles_n = (N + kBN - 1) / kBN;
    const int64_t T = tiles_m * tiles_n;
    const int64_t nch = (K + CL - 1) / CL;
    Plan p{};
    p.tiles_n = tiles_n;
    p.nch = (int)nch;
    const int64_t G = T < gmax ? T : gmax;
    const int64_t q = T / gmax;
    // the plain plan leaves T % gmax tiles for a last, partly idle round
    const bool split = allow_ws && force_split != 0 && T % gmax != 0 &&
                       (force_split == 1 || q < 4) && nch > 1;
    if (!split) {
        p.G = (int)G;
        p.t_whole = T;
        p.L = 0;
    } else {
        int64_t Gs = gmax;
        if (Gs > T * nch) Gs = T * nch;
        p.G = (int)Gs;
        p.t_whole = (T / Gs) * Gs;
        p.L = (T - p.t_whole) * nch;
        r.ws_bytes = (size_t)(T - p.t_whole) * nch * kBM * kBN * sizeof(uint16_t) + kWsAlign;
    }
    p.xcd_remap = p.t_whole % 8 == 0 && p.G % 8 == 0;
    if (env_int("FP8T_GEMM_VERBOSE", 0))
        fprintf(stderr, "[fp8t tile plan] occ %d G %d T %lld t_whole %lld L %lld ws %zu\n", occ,
                p.G, (long long)T, (long long)p.t_whole, (long long)p.L, r.ws_bytes);
    r.plan = p;
    r.ok = true;
    return r;
}

bool tile_args_ok(int ta, int tb, int64_t M, int64_t N, int64_t K, int64_t CL) {
    if (M < 0 || N < 0 || K < 0 || CL < 1) return false;
    if ((ta != 0 && ta != 1) || (tb != 0 && tb != 1)) return false;
    // 32-bit indices inside the kernel (k also runs one slab past K)
    return M <= kMaxGemmDim && N <= kMaxGemmDim && K <= kMaxGemmDim;
}

// Validation, K = 0, planning and launch.
int tile_call(int ta, int tb, int64_t M, int64_t N, int64_t K, int64_t CL, const uint8_t* A,
              int64_t lda, const uint8_t* B, int64_t ldb, uint16_t* C, int64_t ldc, uint64_t seed,
              uint64_t offset, void* workspace, size_t workspace_bytes, hipStream_t stream) {
    if (!tile_args_ok(ta, tb, M, N, K, CL)) return FP8T_EINVAL;
    if (M == 0 || N == 0) return FP8T_OK;
    if (!C || ldc < N) return FP8T_EINVAL;
    if (K > 0) {
        if (!A || !B) return FP8T_EINVAL;
        if (lda < (ta ? M : K) || ldb < (tb ? K : N)) return FP8T_EINVAL;
    }
    if (workspace_bytes > 0 && !workspace) return FP8T_EINVAL;
    if (K == 0) {
        const int64_t total = M * N;
        hipLaunchKernelGGL(fill_zero16, dim3(stride_blocks(total, 256)), dim3(256), 0,
                           stream, C, ldc, (int)M, (int)N);
        return launch_status();
    }
    if (CL > K) CL = K;
    const void* fn = tile_kernel(ta, tb);
    const TilePlan tp = plan_tile(fn, M, N, K, CL, workspace_bytes > 0);
    if (!tp.ok) return FP8T_EHIP;
    if (tp.ws_bytes > workspace_bytes) return FP8T_EWORKSPACE;
    TileArgs g{};
    g.A = A;
    g.B = B;
    g.C = C;
    if (tp.plan.L > 0)
        g.ws = reinterpret_cast<uint16_t*>(((uintptr_t)workspace + kWsAlign - 1) &
                                           ~(uintptr_t)(kWsAlign - 1));
    g.lda = lda;
    g.ldb = ldb;
    g.ldc = ldc;
    g.M = (int)M;
    g.N = (int)N;
    g.K = (int)K;
    g.CL = (int)CL;
    g.k0 = (uint32_t)seed;
    g.k1 = (uint32_t)(seed >> 32);
    g.w3 = 2u * (uint32_t)offset;
    g.c_vec = aligned(C, 8) && ldc % 4 == 0;
    g.a_vec = aligned(A, 8) && lda % 8 == 0;
    g.b_vec = aligned(B, 8) && ldb % 8 == 0;
    Plan plan = tp.plan;
    void* args[] = {&g, &plan};
    if (hipLaunchKernel(fn, dim3(plan.G), dim3(kNT), args, 0, stream) != hipSuccess)
        return FP8T_EHIP;
    if (plan.L > 0) {
        const int64_t threads = (plan.L / plan.nch) * kBM * kBN / kFoldV;
        hipLaunchKernelGGL(chunk_fold_sr, dim3((unsigned)((threads + 255) / 256)),
                           dim3(256), 0, stream, g, plan);
    }
    return launch_status();
}

size_t tile_workspace(int ta, int tb, int64_t M, int64_t N, int64_t K, int64_t CL) {
    if (!tile_args_ok(ta, tb, M, N, K, CL)) return 0;
    if (M == 0 || N == 0 || K == 0) return 0;
    const TilePlan tp = plan_tile(tile_kernel(ta, tb), M, N, K, CL > K ? K : CL, true);
    return tp.ok ? tp.ws_bytes : 0;
}

}  // namespace
}  // namespace fp8t

using namespace fp8t;

extern "C" size_t chunk_gemm_sr_workspace_size(int trans_a, int trans_b, int64_t M, int64_t N,
                                               int64_t K, int64_t CL) {
    return tile_workspace(trans_a, trans_b, M, N, K, CL);
}

extern "C" int chunk_gemm_sr(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K,
                             int64_t CL, const uint8_t* A, int64_t lda, const uint8_t* B,
                             int64_t ldb, uint16_t* C, int64_t ldc, uint64_t seed,
                             uint64_t offset, void* workspace, size_t workspace_bytes,
                             hipStream_t stream) {
    if (offset >= 0x80000000ull) return FP8T_EINVAL;
    return tile_call(trans_a, trans_b, M, N, K, CL, A, lda, B, ldb, C, ldc, seed, offset,
                     workspace, workspace_bytes, stream);
}
