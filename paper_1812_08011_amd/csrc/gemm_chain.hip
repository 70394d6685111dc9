// chunk_gemm for GEMMs with few outputs and long dot products (the
// long-accumulation Gradient GEMMs of Sec. 4.2 / Fig. 6, and the sequential
// FP16 sums of Fig. 3(b)): the exact mode, and the fast mode for chunk
// lengths the matrix cores cannot split.
//
// Every output's chain of rounded FP16 additions (Sec. 2.3, Fig. 3(a)) is
// sequential in k; K can be shared out over workgroups only at chunk
// boundaries and only by writing every chunk sum for an ordered fold.  With
// short chunks (CL = 8: K/8 chunk sums per output) or one chunk (CL >= K)
// that is impossible or costs far more memory traffic than the arithmetic,
// so the chip's parallelism has to come from the outputs alone: a 512 x 512
// output is 262144 chains.  Each chain step is an FMA and a three-instruction
// rounding, each depending on the last, so a SIMD needs several waves (or
// several chains per lane) in flight to issue every cycle; with few outputs
// the kernel keeps few chains per lane -- TM x TN of 1 x 1, 1 x 2 or 2 x 2,
// on 16 x 16 lanes (rows ly + 16 i, columns lx + 16 j, which keeps the LDS
// reads free of bank conflicts) -- so that the outputs fill the chip with
// waves.  Operands are decoded once per tile into LDS with k contiguous, so
// one 16-byte read gives a lane 4 consecutive k of a row; the reads of the
// next 4 k are issued before the arithmetic of the current 4, and K slabs of
// 64 are double-buffered from HBM.  Per multiply-accumulate it issues the FMA
// and the rounding of the exact-mode kernels (guarded: plain values,
// Veltkamp; safe: scaled by 2^96, integer rounding, for tiles that fail the
// overflow guard), with the same bits.  FAST: a chunk is summed in plain FP32
// (one FMA per multiply-accumulate) and rounded to FP16 once at its end, then
// added into the running sum in the 2^96 domain -- the arithmetic of the
// fast-mode variant of the main VALU kernel, with no guard needed.
//
// Chunk lengths must be multiples of 4 (the 4-k groups never straddle a
// chunk boundary) or cover K; CL = 1 reaches this kernel as CL = K (the same
// chain: a one-product chunk is exact).
#include "fp8t_device.h"
#include "fp8train.h"
#include "gemm_plan.h"
#include "gemm_valu_impl.h"

namespace fp8t {
namespace {

constexpr int kNT = 256;            // 16 x 16 lanes
constexpr int kBK = 64;             // k per slab
constexpr int kPitch = kBK + 4;     // floats per LDS row (16-byte aligned rows)

// Decode a thread's words into an LDS slab of R rows laid out [row][k] (k
// contiguous), values times 2^SH; TRACK keeps the largest magnitude and flags
// Inf/NaN codes, as in the main exact kernel.
template <bool KC, int R, int W, int SH, bool TRACK>
__device__ __forceinline__ void store_rowk(float* lds, int tid, const uint32_t (&reg)[W],
                                           float& amax, uint32_t& special) {
    typedef float v2f __attribute__((ext_vector_type(2)));
#pragma unroll
    for (int w = 0; w < W; ++w) {
        const int d = tid + kNT * w;
        const uint32_t v = reg[w];
        const v2f lo = __builtin_amdgcn_cvt_pk_f32_bf8((int)v, false);
        const v2f hi = __builtin_amdgcn_cvt_pk_f32_bf8((int)v, true);
        float f[4] = {lo.x, lo.y, hi.x, hi.y};
        if (TRACK) {
            special |= ((v & 0x7C7C7C7Cu) + 0x04040404u) & 0x80808080u;
            amax = max3_abs(amax, f[0], f[1]);
            amax = max3_abs(amax, f[2], f[3]);
        }
        if (SH != 0) {
#pragma unroll
            for (int b = 0; b < 4; ++b) f[b] *= __builtin_ldexpf(1.0f, SH);   // exact
        }
        if (KC) {       // 4 consecutive k of one row
            const int r = d / (kBK / 4), k = (d % (kBK / 4)) * 4;
            *reinterpret_cast<float4*>(&lds[r * kPitch + k]) = make_float4(f[0], f[1], f[2], f[3]);
        } else {        // 4 consecutive rows at one k
            const int k = d / (R / 4), r = (d % (R / 4)) * 4;
#pragma unroll
            for (int b = 0; b < 4; ++b) lds[(r + b) * kPitch + k] = f[b];
        }
    }
}

template <int TM, int TN, bool TA, bool TB, bool FAST>
__global__ __launch_bounds__(kNT) void chunk_gemm_chain(GemmArgs g, Plan p) {
    constexpr int BM = 16 * TM, BN = 16 * TN;
    constexpr int WA = BM * kBK / 4 / kNT, WB = BN * kBK / 4 / kNT;   // words per thread
    static_assert(WA * kNT * 4 == BM * kBK && WB * kNT * 4 == BN * kBK, "tile/threads");
    constexpr bool KCA = !TA;      // A is k-contiguous unless transposed
    constexpr bool KCB = TB;       // B is k-contiguous only when transposed
    __shared__ __attribute__((aligned(16))) float As[2][BM * kPitch];
    __shared__ __attribute__((aligned(16))) float Bs[2][BN * kPitch];
    // |a| max, |b| max, specials, |S| max of the guarded tiles, two slots
    __shared__ uint32_t s_track[2][4];

    const int tid = threadIdx.x;
    const int ly = tid / 16, lx = tid % 16;
    if (tid < 8) (&s_track[0][0])[tid] = 0;    // ordered by the first slab's barrier
    int gslot = 0;
    uint32_t ra[WA], rb[WB];
    // chunk length in 4-k groups; one chunk for CL >= K
    const int K4 = (g.K + 3) / 4;
    const int clg = g.CL >= g.K ? K4 : g.CL / 4;

    // One whole tile on one path; the guarded path returns false, having
    // written nothing, when its check fails.
    auto tile_pass = [&](auto safe_tag, int64_t tile) __attribute__((always_inline)) -> bool {
        constexpr bool SAFE = decltype(safe_tag)::value;
        constexpr int DOM = SAFE ? 96 : 0;
        constexpr int ASHIFT = FAST ? 0 : DOM;   // the fast mode sums plain products
        constexpr bool TRACK = !SAFE;
        int tr, tc;
        tile_rc(p, tile, tr, tc);
        const int m0 = tr * BM, n0 = tc * BN;
        float amax_a = 0.0f, amax_b = 0.0f, smax = 0.0f;
        uint32_t special = 0;
        auto rnd = [&](float x) __attribute__((always_inline)) -> float {
            return SAFE ? rn16s(x) : rn16v(x);
        };
        float P[TM][TN], S[TM][TN];
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) { P[i][j] = 0.0f; S[i][j] = 0.0f; }

        // 4 k of one group; fresh: the group starts a chunk, whose first
        // product is exact and needs no rounding
        auto group = [&](const float4 (&a)[TM], const float4 (&b)[TN], bool fresh)
                         __attribute__((always_inline)) {
            float av[TM][4], bv[TN][4];
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                av[i][0] = a[i].x; av[i][1] = a[i].y; av[i][2] = a[i].z; av[i][3] = a[i].w;
            }
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                bv[j][0] = b[j].x; bv[j][1] = b[j].y; bv[j][2] = b[j].z; bv[j][3] = b[j].w;
            }
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j) {
                        if (q == 0 && fresh)
                            P[i][j] = __builtin_fmaf(av[i][q], bv[j][q], 0.0f);
                        else if (FAST)
                            P[i][j] = __builtin_fmaf(av[i][q], bv[j][q], P[i][j]);
                        else
                            P[i][j] = rnd(__builtin_fmaf(av[i][q], bv[j][q], P[i][j]));
                    }
        };
        auto flush = [&]() __attribute__((always_inline)) {
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    // fast: the FP32 chunk sum rounded to FP16 in the 2^96 domain
                    const float pv = FAST ? rn16s(P[i][j] * 0x1p96f) : P[i][j];
                    S[i][j] = rnd(S[i][j] + pv);
                    if (TRACK) smax = max3_abs(smax, S[i][j], S[i][j]);
                }
        };
        auto read = [&](float4 (&a)[TM], float4 (&b)[TN], int buf, int kk)
                        __attribute__((always_inline)) {
#pragma unroll
            for (int i = 0; i < TM; ++i)
                a[i] = *reinterpret_cast<const float4*>(&As[buf][(ly + 16 * i) * kPitch + kk]);
#pragma unroll
            for (int j = 0; j < TN; ++j)
                b[j] = *reinterpret_cast<const float4*>(&Bs[buf][(lx + 16 * j) * kPitch + kk]);
        };

        const int nslabs = (g.K + kBK - 1) / kBK;
        int crem = clg;                  // groups left in the current chunk
        valu_impl::slab_load<KCA, BM, kBK, kNT, WA>(g.A, g.lda, g.a_vec, m0, g.M, 0, g.K, tid, ra);
        valu_impl::slab_load<KCB, BN, kBK, kNT, WB>(g.B, g.ldb, g.b_vec, n0, g.N, 0, g.K, tid, rb);
        store_rowk<KCA, BM, WA, ASHIFT, TRACK>(As[0], tid, ra, amax_a, special);
        store_rowk<KCB, BN, WB, 0, TRACK>(Bs[0], tid, rb, amax_b, special);
        __syncthreads();
        for (int s = 0; s < nslabs; ++s) {
            const int buf = s & 1;
            const int ks = s * kBK;
            if (s + 1 < nslabs) {
                valu_impl::slab_load<KCA, BM, kBK, kNT, WA>(g.A, g.lda, g.a_vec, m0, g.M,
                                                             ks + kBK, g.K, tid, ra);
                valu_impl::slab_load<KCB, BN, kBK, kNT, WB>(g.B, g.ldb, g.b_vec, n0, g.N,
                                                             ks + kBK, g.K, tid, rb);
            }
            // groups of this slab (the last slab's beyond K4 are skipped; its
            // zero-filled k up to a multiple of 4 add exact zeros)
            const int ng = min(kBK / 4, K4 - ks / 4);
            if (ng == kBK / 4) {
                float4 a0[TM], b0[TN], a1[TM], b1[TN];
                read(a0, b0, buf, 0);
#pragma unroll
                for (int q = 0; q < kBK / 4; q += 2) {
                    read(a1, b1, buf, 4 * q + 4);
                    group(a0, b0, crem == clg);
                    if (--crem == 0) { flush(); crem = clg; }
                    if (q + 2 < kBK / 4) read(a0, b0, buf, 4 * q + 8);
                    group(a1, b1, crem == clg);
                    if (--crem == 0) { flush(); crem = clg; }
                }
            } else {
                for (int q = 0; q < ng; ++q) {
                    float4 a[TM], b[TN];
                    read(a, b, buf, 4 * q);
                    group(a, b, crem == clg);
                    if (--crem == 0) { flush(); crem = clg; }
                }
            }
            if (s + 1 < nslabs) {
                store_rowk<KCA, BM, WA, ASHIFT, TRACK>(As[buf ^ 1], tid, ra, amax_a, special);
                store_rowk<KCB, BN, WB, 0, TRACK>(Bs[buf ^ 1], tid, rb, amax_b, special);
            }
            __syncthreads();
        }
        if (crem != clg) flush();        // the last, shorter chunk

        if (!SAFE) {
            // the overflow guard of the exact-mode kernels: no Inf/NaN
            // operand; chunk partial sums at most 3 CL max|a| max|b| < 2^31;
            // running sums, tracked at chunk ends, below 2^31
            uint32_t* st = s_track[gslot];
            uint32_t ua = __float_as_uint(amax_a), ub = __float_as_uint(amax_b), us = special;
            uint32_t uS = __float_as_uint(smax);
#pragma unroll
            for (int o = 32; o > 0; o >>= 1) {
                ua = max(ua, (uint32_t)__shfl_xor((int)ua, o));
                ub = max(ub, (uint32_t)__shfl_xor((int)ub, o));
                us |= (uint32_t)__shfl_xor((int)us, o);
                uS = max(uS, (uint32_t)__shfl_xor((int)uS, o));
            }
            if ((tid & 63) == 0) {
                atomicMax(&st[0], ua);
                atomicMax(&st[1], ub);
                atomicOr(&st[2], us);
                atomicMax(&st[3], uS);
            }
            if (tid == 0) {
#pragma unroll
                for (int q = 0; q < 4; ++q) s_track[gslot ^ 1][q] = 0;
            }
            __syncthreads();
            const float ma = __uint_as_float(st[0]), mb = __uint_as_float(st[1]);
            const uint32_t sp = st[2];
            const float sm = __uint_as_float(st[3]);
            gslot ^= 1;
            if (sp) return false;
            const double bound = 3.0 * (double)min(g.CL, g.K) * (double)ma * (double)mb;
            if (!(bound < 2147483648.0)) return false;
            if (!(sm < 2147483648.0f)) return false;
        }
        // outputs (ly + 16 i, lx + 16 j): lanes of a row write 16 consecutive
        // codes
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            const int m = m0 + ly + 16 * i;
            if (m >= g.M) continue;
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int n = n0 + lx + 16 * j;
                if (n >= g.N) continue;
                if (g.C) g.C[(int64_t)m * g.ldc + n] = fp16_code<DOM>(S[i][j]);
                if (g.C8)
                    g.C8[(int64_t)m * g.ldc8 + n] =
                        (uint8_t)f32d_to_fp8_scaled<DOM>(S[i][j], g.q_scale);
            }
        }
        return true;
    };

    for (int64_t t = blockIdx.x; t < p.t_whole; t += p.G) {
        const int64_t tile = whole_tile(p, t);
        bool done = false;
        // the fast mode has the 2^96-domain path only
        if (!FAST && g.guarded) done = tile_pass(std::integral_constant<bool, false>{}, tile);
        if (!done) tile_pass(std::integral_constant<bool, true>{}, tile);
    }
}

template <int TM, int TN, bool FAST>
const void* chain_sel(int ta, int tb) {
    if (ta) return tb ? reinterpret_cast<const void*>(&chunk_gemm_chain<TM, TN, true, true, FAST>)
                      : reinterpret_cast<const void*>(&chunk_gemm_chain<TM, TN, true, false, FAST>);
    return tb ? reinterpret_cast<const void*>(&chunk_gemm_chain<TM, TN, false, true, FAST>)
              : reinterpret_cast<const void*>(&chunk_gemm_chain<TM, TN, false, false, FAST>);
}

template <bool FAST>
const void* chain_shape(int shape, int ta, int tb) {
    switch (shape) {
        case 0: return chain_sel<2, 2, FAST>(ta, tb);
        case 1: return chain_sel<1, 2, FAST>(ta, tb);
        default: return chain_sel<1, 1, FAST>(ta, tb);
    }
}

}  // namespace

const void* chain_kernel(int shape, int ta, int tb, int fast) {
    return fast ? chain_shape<true>(shape, ta, tb) : chain_shape<false>(shape, ta, tb);
}

}  // namespace fp8t
