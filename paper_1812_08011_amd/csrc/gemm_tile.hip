// Vector-ALU tile kernel for two variants of the chunk-based GEMM of
// Sec. 2.3 / Fig. 3(a):
//
// * chunk_gemm_sr -- FP8 operands, every FP16 addition rounded stochastically
//   (Eq. (1)) instead of to nearest: the paper's second rounding mode after
//   FP16 additions, whose behaviour on long accumulations Fig. 3(b) compares
//   with nearest rounding;
// * chunk_gemm_p16 -- FP16 operands (the last layer's GEMMs, which Sec. 3
//   keeps in FP16): each product is rounded to FP16 (the multiplication in
//   FP_mult = FP16 of Fig. 3(a)), then accumulated in chunks with rounding to
//   nearest, as in chunk_gemm's exact mode.
//
// Each addition first forms the FP32 sum of the running value and the next
// term (products of two FP8 values are exact in FP32; products of two FP16
// values, 20 significant bits, too) and then rounds it into FP16.  As in the
// exact mode, FP16 quantities are held scaled by 2^96 (fp8t_device.h), so FP16
// overflow is FP32 overflow and FP16 subnormals are FP32 normals: FP8 operands
// enter as a(k) 2^96 and b(k), FP16 operands as a(k) 2^48 and b(k) 2^48.
// Rounding to nearest is rn16s on the raw bits.  Stochastic rounding of the
// 14 discarded mantissa bits D with uniform u rounds the magnitude up iff
// D > (u >> 2); adding (2^14 - 1 - (u >> 2)) to the raw bits and clearing the
// low 14 bits does exactly that, with the carry running into the exponent
// (and to the Inf encoding past the largest FP16 value).  Sums below 2^-30
// are multiples of 2^-39 with at most 9 significant bits, so their discarded
// bits are zero and neither rounding changes them, as the fixed subnormal
// step requires.  A product of FP16 values below 2^-30 is rounded to a
// multiple of 2^-39 by adding and subtracting 1.5 x 2^-16 (2^80 scaled).
//
// Random bits (chunk_gemm_sr): Philox4x32-10, key = seed, eight 16-bit
// uniforms per block (word halves, low half first).  The addition of product
// k into output (i, j) takes uniform 4 (k mod 2) + (j mod 4) of block
// (i, j / 4, k / 2, 2 offset): a thread owning 4 x 4 outputs (four rows of
// four aligned columns) draws four blocks per two k.  The addition of chunk c
// into the running sum takes uniform j mod 8 of block (i, j / 8, c,
// 2 offset + 1).
//
// The work decomposition is the persistent plan of gemm_plan.h: whole tiles,
// then the chunks of the remaining tiles shared out as ranges; a piece that
// does not start at chunk 0 leaves each chunk's FP16 sum in the workspace and
// chunk_fold_tile continues the running sum over them in ascending order, with
// the same random bits -- the result does not depend on the plan.
#include "fp8t_device.h"
#include "fp8train.h"
#include "fp8t_host.h"
#include "gemm_plan.h"

#include <stdio.h>

#include <type_traits>

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
    const void* A;
    const void* B;
    uint16_t* C;
    uint16_t* ws;                     // chunk sums of the shared tiles
    int64_t lda, ldb, ldc;
    int M, N, K, CL;
    uint32_t k0, k1;                  // Philox key (stochastic rounding)
    uint32_t w3;                      // 2 * offset
    int c_vec;                        // C rows allow 8-byte stores of 4 codes
    int a_vec, b_vec;                 // A / B rows allow 8-element loads
    int guarded;                      // FP16 operands: try the guarded path first
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

// FP16 code -> value * 2^S (exact).
template <int S>
__device__ __forceinline__ float fp16_to_f32_shift(uint32_t c) {
    const uint32_t e = (c >> 9) & 63u, m = c & 511u;
    uint32_t bits;
    if (e == 63u)
        bits = m ? kF32NaN : kF32Inf;
    else if (e == 0u)
        bits = __float_as_uint((float)m * __builtin_ldexpf(1.0f, S - 39));
    else
        bits = ((c & 0x7FFFu) << 14) + ((uint32_t)(96 + S) << 23);
    return __uint_as_float(bits | ((c & 0x8000u) << 16));
}

// Operand element (code) -> float in the kernel's domain: FP8 A scaled by
// 2^96, FP8 B plain; FP16 A and B scaled by 2^48 each, or plain on the
// guarded path (PLAIN).
template <int FMT, bool IS_A, bool PLAIN = false>
__device__ __forceinline__ float decode(uint32_t c) {
    if (FMT == 8) return IS_A ? fp8_to_f32<96>(c) : fp8_to_f32<0>(c);
    return PLAIN ? fp16_to_f32(c) : fp16_to_f32_shift<48>(c);
}

// Operand statistics of a piece on the guarded path: largest magnitude
// decoded, and whether an Inf/NaN code was seen.
struct Track {
    float amax = 0.0f;
    uint32_t special = 0u;
    __device__ __forceinline__ void add(float f) { amax = fmaxf(amax, __builtin_fabsf(f)); }
};

template <int FMT> struct Elem;
template <> struct Elem<8> { typedef uint8_t t; typedef uint2 v8; };
template <> struct Elem<16> { typedef uint16_t t; typedef uint4 v8; };

// Stage a whole slab (64 rows x 32 k, all inside the matrix, aligned rows)
// with one 8-element load per thread.  KC: k is contiguous in memory
// (element (r, k) at p[r * ld + k]); otherwise the row index is.
template <int FMT, bool IS_A, bool KC, bool PLAIN = false>
__device__ __forceinline__ void stage_fast(const typename Elem<FMT>::t* __restrict__ p,
                                           int64_t ld, int r0, int k0, float (*X)[kPitch],
                                           int tid, Track& tr) {
    typedef typename Elem<FMT>::v8 V;
    uint32_t w[FMT / 4];
    float f[8];
    int r, kq, k, rq;
    if (KC) {
        r = tid / (kBK / 8), kq = (tid % (kBK / 8)) * 8;
        const V v = *reinterpret_cast<const V*>(p + (int64_t)(r0 + r) * ld + k0 + kq);
        __builtin_memcpy(w, &v, sizeof(v));
    } else {
        k = tid / (kBM / 8), rq = (tid % (kBM / 8)) * 8;
        const V v = *reinterpret_cast<const V*>(p + (int64_t)(k0 + k) * ld + r0 + rq);
        __builtin_memcpy(w, &v, sizeof(v));
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const uint32_t c = FMT == 8 ? (w[e / 4] >> (8 * (e % 4))) & 0xFFu
                                    : (w[e / 2] >> (16 * (e % 2))) & 0xFFFFu;
        f[e] = decode<FMT, IS_A, PLAIN>(c);
        if (PLAIN) {
            tr.add(f[e]);
            tr.special |= (FMT == 16 && ((c >> 9) & 63u) == 63u) ? 1u : 0u;
        }
    }
    if (KC) {
#pragma unroll
        for (int e = 0; e < 8; ++e) X[kq + e][r] = f[e];
    } else {
        *reinterpret_cast<float4*>(&X[k][rq]) = make_float4(f[0], f[1], f[2], f[3]);
        *reinterpret_cast<float4*>(&X[k][rq + 4]) = make_float4(f[4], f[5], f[6], f[7]);
    }
}

// FP16 product in the 2^96 domain rounded to FP16 (nearest even): raw-bit
// rounding of the significand, or a multiple of 2^-39 below 2^-30.
__device__ __forceinline__ float round_product16(float p) {
    const float kMagic = 0x1.8p80f;            // 1.5 x 2^80: step 2^57 there
    const float sub = (p + kMagic) - kMagic;
    return __builtin_fabsf(p) < 0x1p66f ? sub : rn16s(p);
}

// Plain product of two FP16 values (exact in float: at most 20 significant
// bits, far inside float's exponent range) rounded to FP16, nearest even:
// adding 1.5 x 2^(E + 14), E = max(exponent of p, -30), puts the last kept
// bit of p at float's last bit (10 significant bits; a fixed step of 2^-39
// below 2^-30, FP16's subnormal range), and subtracting it again is exact.
__device__ __forceinline__ float rn16_product_plain(float p) {
    uint32_t e = __float_as_uint(p) & 0x7F800000u;
    e = e > (97u << 23) ? e : (97u << 23);
    const float magic = __uint_as_float(e + (14u << 23) + 0x00400000u);
    return (p + magic) - magic;
}

// FMT: operand format (8 = FP8 codes, 16 = FP16 codes); SR: stochastic
// rounding of every addition (else nearest).  FP16 operands with nearest
// rounding first try a guarded path, like the exact mode of chunk_gemm: plain
// values, products rounded by rn16_product_plain and sums by Veltkamp
// splitting (rn16v), valid when no operand is Inf/NaN and no partial sum can
// reach FP16's overflow threshold (each is at most 9 (1 + 2^-10) K max|a|
// max|b|, the rounded products being at most (1 + 2^-10) |a b|).  Sums below
// 2^-30 need no subnormal step there: every term is a multiple of 2^-39, so
// such a sum is exact in float and already an FP16 value.  A piece that
// fails is recomputed in the 2^96 domain.
template <bool TA, bool TB, int FMT, bool SR>
__global__ __launch_bounds__(kNT) void chunk_gemm_tile_kernel(TileArgs g, Plan p) {
    constexpr bool HAS_GUARDED = FMT == 16 && !SR;
    // |a| max bits, |b| max bits, specials of the guarded pieces, in two slots
    // used by alternate pieces
    __shared__ uint32_t s_track[2][3];
    int gslot = 0;
    if (threadIdx.x < 6) (&s_track[0][0])[threadIdx.x] = 0;   // ordered by the first slab's barrier
    typedef typename Elem<FMT>::t E;
    const E* __restrict__ A = static_cast<const E*>(g.A);
    const E* __restrict__ B = static_cast<const E*>(g.B);
    __shared__ __attribute__((aligned(16))) float As[kBK][kPitch];
    __shared__ __attribute__((aligned(16))) float Bs[kBK][kPitch];
    const int tid = threadIdx.x;
    const int tx = tid % kTiles, ty = tid / kTiles;

    // chunks [c0, c1) of tile; lt >= 0 for a shared tile.  Returns false when
    // the guarded path's check fails (nothing has then been written to C).
    auto piece = [&](auto guard_tag, int64_t tile, int c0, int c1, int64_t lt)
                     __attribute__((always_inline)) -> bool {
        constexpr bool GUARDED = decltype(guard_tag)::value;
        constexpr int DOM = GUARDED ? 0 : 96;
        auto rnd = [&](float x) __attribute__((always_inline)) -> float {
            return GUARDED ? rn16v(x) : rn16s(x);
        };
        Track ta, tb;
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
                    v.x = (uint32_t)f32d_to_fp16<DOM>(P[r][0]) |
                          ((uint32_t)f32d_to_fp16<DOM>(P[r][1]) << 16);
                    v.y = (uint32_t)f32d_to_fp16<DOM>(P[r][2]) |
                          ((uint32_t)f32d_to_fp16<DOM>(P[r][3]) << 16);
                    *reinterpret_cast<uint2*>(dst + r * kBN) = v;
                }
            } else if (SR) {
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
            } else {
#pragma unroll
                for (int r = 0; r < kT; ++r)
#pragma unroll
                    for (int c = 0; c < kT; ++c) S[r][c] = rnd(S[r][c] + P[r][c]);
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
                stage_fast<FMT, true, !TA, GUARDED>(A, g.lda, m0, sb, As, tid, ta);
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
                    As[kk][mm] = decode<FMT, true, GUARDED>(code);
                    if (GUARDED) {
                        ta.add(As[kk][mm]);
                        ta.special |= ((code >> 9) & 63u) == 63u ? 1u : 0u;
                    }
                }
            }
            if (lo == sb && hi == sb + kBK && n0 + kBN <= g.N && g.b_vec) {
                stage_fast<FMT, false, TB, GUARDED>(B, g.ldb, n0, sb, Bs, tid, tb);
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
                    Bs[kk][nn] = decode<FMT, false, GUARDED>(code);
                    if (GUARDED) {
                        tb.add(Bs[kk][nn]);
                        tb.special |= ((code >> 9) & 63u) == 63u ? 1u : 0u;
                    }
                }
            }
            __syncthreads();
#pragma unroll 1
            for (int gq = lo & ~1; gq < hi; gq += 2) {
                // rows' blocks for k = gq, gq + 1 (complemented words)
                uint32_t nw[kT][4];
                if (SR) {
#pragma unroll
                    for (int r = 0; r < kT; ++r) {
                        const u32x4 b = block_of(gi + r, gj >> 2, (uint32_t)(gq >> 1), g.w3, g);
                        nw[r][0] = ~b.x;
                        nw[r][1] = ~b.y;
                        nw[r][2] = ~b.z;
                        nw[r][3] = ~b.w;
                    }
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
                        for (int c = 0; c < kT; ++c) {
                            float x;
                            if (FMT == 8) {
                                x = __builtin_fmaf(av[r], bv[c], P[r][c]);
                            } else {
                                x = P[r][c] + (GUARDED ? rn16_product_plain(av[r] * bv[c])
                                                       : round_product16(av[r] * bv[c]));
                            }
                            P[r][c] = SR ? sr16s(x, sr_addend(nw[r][2 * s + c / 2], c % 2))
                                         : rnd(x);
                        }
                    if (k + 1 == cend) chunk_end();
                }
            }
        }
        if (GUARDED) {
            // The workgroup's operand statistics of this piece, reduced within
            // each wave, then one LDS atomic per wave (non-negative floats
            // compare as their bit patterns).  Slot gslot was cleared during the
            // previous guarded piece and is read after the one barrier here;
            // the other slot, cleared now, is next written after at least one
            // more barrier (every piece has a slab).
            uint32_t* st = s_track[gslot];
            uint32_t ua = __float_as_uint(ta.amax), ub = __float_as_uint(tb.amax);
            uint32_t us = ta.special | tb.special;
#pragma unroll
            for (int o = 32; o > 0; o >>= 1) {
                ua = max(ua, (uint32_t)__shfl_xor((int)ua, o));
                ub = max(ub, (uint32_t)__shfl_xor((int)ub, o));
                us |= (uint32_t)__shfl_xor((int)us, o);
            }
            if ((tid & 63) == 0) {
                atomicMax(&st[0], ua);
                atomicMax(&st[1], ub);
                atomicOr(&st[2], us);
            }
            if (tid == 0) {
                s_track[gslot ^ 1][0] = 0;
                s_track[gslot ^ 1][1] = 0;
                s_track[gslot ^ 1][2] = 0;
            }
            __syncthreads();
            const float ma = __uint_as_float(st[0]), mb = __uint_as_float(st[1]);
            const uint32_t sp = st[2];
            gslot ^= 1;
            if (sp) return false;
            // the bound uses the full K, so that pieces of one tile that each
            // pass bound the whole chain together
            if (!(9.01 * (double)g.K * (double)ma * (double)mb < 2147483648.0)) return false;
        }
        if (to_ws) return true;
        // the running sum: the result of a whole tile, or the start of a
        // shared tile's chain (continued by chunk_fold_tile)
#pragma unroll
        for (int r = 0; r < kT; ++r) {
            const int m = m0 + ty * kT + r, n = n0 + tx * kT;
            if (m >= g.M) continue;
            uint16_t* cp = g.C + (int64_t)m * g.ldc + n;
            if (g.c_vec && n + kT <= g.N) {
                uint2 v;
                v.x = (uint32_t)f32d_to_fp16<DOM>(S[r][0]) |
                      ((uint32_t)f32d_to_fp16<DOM>(S[r][1]) << 16);
                v.y = (uint32_t)f32d_to_fp16<DOM>(S[r][2]) |
                      ((uint32_t)f32d_to_fp16<DOM>(S[r][3]) << 16);
                *reinterpret_cast<uint2*>(cp) = v;
            } else {
#pragma unroll
                for (int c = 0; c < kT; ++c)
                    if (n + c < g.N) cp[c] = f32d_to_fp16<DOM>(S[r][c]);
            }
        }
        return true;
    };

    auto run = [&](int64_t tile, int c0, int c1, int64_t lt) __attribute__((always_inline)) {
        bool done = false;
        if constexpr (HAS_GUARDED) {
            if (g.guarded) done = piece(std::integral_constant<bool, true>{}, tile, c0, c1, lt);
        }
        if (!done) piece(std::integral_constant<bool, false>{}, tile, c0, c1, lt);
    };

    const int w = blockIdx.x;
    for (int64_t t = w; t < p.t_whole; t += p.G) run(whole_tile(p, t), 0, p.nch, -1);
    if (p.L > 0) {
        int64_t s = (int64_t)w * p.L / p.G;
        const int64_t e = (int64_t)(w + 1) * p.L / p.G;
        while (s < e) {
            const int64_t lt = s / p.nch;
            const int c0 = (int)(s - lt * p.nch);
            const int64_t c1l = e - lt * p.nch;
            const int c1 = c1l < p.nch ? (int)c1l : p.nch;
            run(p.t_whole + lt, c0, c1, lt);
            s = lt * p.nch + c1;
        }
    }
}

// Continue the running sums of the shared tiles (in C, from their first
// pieces) over the chunk sums in the workspace, in ascending chunk order --
// the additions a whole-tile pass makes, with the same rounding (and, for
// SR, the same inter-chunk uniforms).  A thread takes 8 consecutive outputs
// of a row: one 16-byte load of chunk sums (and one block of uniforms) per
// chunk.
constexpr int kFoldV = 8, kFoldTU = 8;

template <bool SR>
__global__ __launch_bounds__(256) void chunk_fold_tile(TileArgs g, Plan p) {
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
        uint32_t nw[4] = {0u, 0u, 0u, 0u};
        if (SR) {
            const u32x4 b = block_of((uint32_t)m, (uint32_t)(n0 >> 3), (uint32_t)c, g.w3 + 1u, g);
            nw[0] = ~b.x;
            nw[1] = ~b.y;
            nw[2] = ~b.z;
            nw[3] = ~b.w;
        }
#pragma unroll
        for (int v = 0; v < kFoldV; ++v) {
            const float x = S[v] + fp16_to_f32s((cw[v / 2] >> (16 * (v % 2))) & 0xFFFFu);
            S[v] = SR ? sr16s(x, sr_addend(nw[v / 2], v % 2)) : rn16s(x);
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

template <int FMT, bool SR>
const void* tile_kernel(int ta, int tb) {
    if (!ta && !tb) return reinterpret_cast<const void*>(&chunk_gemm_tile_kernel<false, false, FMT, SR>);
    if (!ta && tb) return reinterpret_cast<const void*>(&chunk_gemm_tile_kernel<false, true, FMT, SR>);
    if (ta && !tb) return reinterpret_cast<const void*>(&chunk_gemm_tile_kernel<true, false, FMT, SR>);
    return reinterpret_cast<const void*>(&chunk_gemm_tile_kernel<true, true, FMT, SR>);
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

// Validation, K = 0, planning and launch shared by the two entry points.
template <int FMT, bool SR>
int tile_call(int ta, int tb, int64_t M, int64_t N, int64_t K, int64_t CL, const void* A,
              int64_t lda, const void* B, int64_t ldb, uint16_t* C, int64_t ldc, uint64_t seed,
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
    const void* fn = tile_kernel<FMT, SR>(ta, tb);
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
    const int eb = FMT / 8;                   // bytes per element
    g.a_vec = aligned(A, 8 * eb) && lda % 8 == 0;
    g.b_vec = aligned(B, 8 * eb) && ldb % 8 == 0;
    // FP8T_GEMM_GUARD=0 runs every piece on the 2^96-domain path (tests)
    g.guarded = env_int("FP8T_GEMM_GUARD", 1) != 0;
    Plan plan = tp.plan;
    void* args[] = {&g, &plan};
    if (hipLaunchKernel(fn, dim3(plan.G), dim3(kNT), args, 0, stream) != hipSuccess)
        return FP8T_EHIP;
    if (plan.L > 0) {
        const int64_t threads = (plan.L / plan.nch) * kBM * kBN / kFoldV;
        hipLaunchKernelGGL(chunk_fold_tile<SR>, dim3((unsigned)((threads + 255) / 256)),
                           dim3(256), 0, stream, g, plan);
    }
    return launch_status();
}

template <int FMT, bool SR>
size_t tile_workspace(int ta, int tb, int64_t M, int64_t N, int64_t K, int64_t CL) {
    if (!tile_args_ok(ta, tb, M, N, K, CL)) return 0;
    if (M == 0 || N == 0 || K == 0) return 0;
    const TilePlan tp = plan_tile(tile_kernel<FMT, SR>(ta, tb), M, N, K, CL > K ? K : CL, true);
    return tp.ok ? tp.ws_bytes : 0;
}

}  // namespace
}  // namespace fp8t

using namespace fp8t;

extern "C" size_t chunk_gemm_sr_workspace_size(int trans_a, int trans_b, int64_t M, int64_t N,
                                               int64_t K, int64_t CL) {
    return tile_workspace<8, true>(trans_a, trans_b, M, N, K, CL);
}

extern "C" int chunk_gemm_sr(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K,
                             int64_t CL, const uint8_t* A, int64_t lda, const uint8_t* B,
                             int64_t ldb, uint16_t* C, int64_t ldc, uint64_t seed,
                             uint64_t offset, void* workspace, size_t workspace_bytes,
                             hipStream_t stream) {
    if (offset >= 0x80000000ull) return FP8T_EINVAL;
    return tile_call<8, true>(trans_a, trans_b, M, N, K, CL, A, lda, B, ldb, C, ldc, seed,
                              offset, workspace, workspace_bytes, stream);
}

extern "C" size_t chunk_gemm_p16_workspace_size(int trans_a, int trans_b, int64_t M, int64_t N,
                                                int64_t K, int64_t CL) {
    return tile_workspace<16, false>(trans_a, trans_b, M, N, K, CL);
}

extern "C" int chunk_gemm_p16(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K,
                              int64_t CL, const uint16_t* A, int64_t lda, const uint16_t* B,
                              int64_t ldb, uint16_t* C, int64_t ldc, void* workspace,
                              size_t workspace_bytes, hipStream_t stream) {
    return tile_call<16, false>(trans_a, trans_b, M, N, K, CL, A, lda, B, ldb, C, ldc, 0, 0,
                                workspace, workspace_bytes, stream);
}
