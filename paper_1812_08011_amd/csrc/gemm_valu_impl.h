// chunk_gemm on the vector ALUs: the exact mode, and the fast mode for chunk
// lengths that are not a multiple of the matrix-core K step.
//
// Every output keeps two registers, the intra-chunk sum P and the running sum
// S, as FP32 values on the FP16 grid.  One multiply-accumulate of the dot
// product of Sec. 2.3 / Fig. 3(a) is one FMA -- an FP8 x FP8 product is exact
// in FP32, so its one rounding is the rounding of the exact sum -- followed
// by rounding to the 10-bit FP16 significand; at every chunk end
//     S = round(S + P), P = +0.
// The double rounding 24 -> 10 bits is innocuous since 24 >= 2*10 + 2.
// gfx950 has no adder for the paper's FP16, so this is bound by the VALU
// issue rate.  Two paths compute the same bits:
//   * guarded (default): plain values, rounding by Veltkamp splitting
//     (rn16v: v_mul, v_sub, v_sub) -- 4 full-rate instructions per
//     multiply-accumulate (FP16 subnormals are FP32-normal, so no scaling is
//     needed when nothing can overflow).  It holds when no operand is Inf/NaN
//     and no partial sum reaches the FP16 overflow threshold.  A chunk's
//     partial sums are at most 3 sum_chunk |a_k b_k| (an RN step adds at most
//     3x its non-negative addend), so 3 CL max|a| max|b| < 2^31 bounds them;
//     the running sum changes only at chunk ends, where its largest magnitude
//     is tracked (one max per output per chunk) and must stay below 2^31 --
//     an overflow would leave it at 2^32 or more.  Each workgroup tracks the
//     largest operand magnitude and any Inf/NaN code while decoding, and
//     checks both at the end of a piece;
//   * safe: values scaled by 2^96, which maps FP16 overflow onto FP32
//     overflow, rounding on the raw bits (rn16s: v_bfe, v_add3, v_and).  A
//     piece that fails the check is recomputed this way (chunk sums in the
//     workspace are simply rewritten; C is written only after the check).
// The kernel is shaped to issue little else:
//   * a TM x TN register tile per lane; operands are staged through LDS
//     already decoded to FP32 (one decode per element per workgroup tile);
//   * K slabs of BK are double-buffered in LDS, the next slab is fetched from
//     HBM (4-byte loads where alignment allows) while the current one is
//     consumed, and with PF the LDS reads of step k+1 are issued before the
//     arithmetic of step k so their latency is hidden;
//   * a persistent grid of exactly as many workgroups as fit on the chip,
//     sharing out tiles and chunks evenly (gemm_plan.h), so no CU idles in a
//     last partial wave of workgroups.
#pragma once

#include "fp8t_device.h"
#include "gemm_valu.h"

namespace fp8t {
namespace valu_impl {

// One operand slab of a workgroup: rows [r0, r0 + R) of the operand's row
// index (m for A, n for B) by k in [k0, k0 + BK), clipped to `rows` and
// `kend`.  KC: k is the contiguous index in memory (element (r, k) at
// p[r * ld + k]); otherwise the row index is (element at p[k * ld + r]).  Each
// of the NT threads holds W words of 4 consecutive bytes between the HBM load
// and the LDS store; `vec` allows 4-byte loads (aligned base and ld).
template <bool KC, int R, int BK, int NT, int W>
__device__ __forceinline__ void slab_load(const uint8_t* __restrict__ ptr, int64_t ld,
                                          int vec, int r0, int rows, int k0, int kend,
                                          int tid, uint32_t (&reg)[W]) {
#pragma unroll
    for (int w = 0; w < W; ++w) {
        const int d = tid + NT * w;
        int r, k;
        if (KC) { r = d / (BK / 4); k = (d % (BK / 4)) * 4; }
        else    { k = d / (R / 4);  r = (d % (R / 4)) * 4; }
        const int gr = r0 + r, gk = k0 + k;
        uint32_t v = 0;
        if (KC) {
            if (gr < rows && gk < kend) {
                const uint8_t* q = ptr + (int64_t)gr * ld + gk;
                if (vec && gk + 3 < kend) {
                    v = *reinterpret_cast<const uint32_t*>(q);
                } else {
                    for (int b = 0; b < 4; ++b)
                        if (gk + b < kend) v |= (uint32_t)q[b] << (8 * b);
                }
            }
        } else {
            if (gk < kend && gr < rows) {
                const uint8_t* q = ptr + (int64_t)gk * ld + gr;
                if (vec && gr + 3 < rows) {
                    v = *reinterpret_cast<const uint32_t*>(q);
                } else {
                    for (int b = 0; b < 4; ++b)
                        if (gr + b < rows) v |= (uint32_t)q[b] << (8 * b);
                }
            }
        }
        reg[w] = v;
    }
}

// The same for an implicitly lowered convolution input (ConvGeom): the
// operand is Xcol (KC: element (r, k) = Xcol(r, k), rows are output pixels)
// or Xcol^T (element (r, k) = Xcol(k, r)).  A word holds 4 consecutive Xcol
// columns of one pixel: 4 consecutive channels of one input position when
// C % 4 == 0 (one 4-byte load), otherwise gathered byte by byte.
__device__ __forceinline__ uint32_t xcol_byte(const uint8_t* __restrict__ X, const ConvGeom& cg,
                                              int pix, int col) {
    const int n = pix / cg.OHW, rem = pix - n * cg.OHW;
    const int oh = rem / cg.OW, ow = rem - oh * cg.OW;
    const int kh = col / cg.KWC, r2 = col - kh * cg.KWC;
    const int kw = r2 / cg.C, c = r2 - kw * cg.C;
    const int ih = oh * cg.stride - cg.pad + kh, iw = ow * cg.stride - cg.pad + kw;
    if ((unsigned)ih >= (unsigned)cg.H || (unsigned)iw >= (unsigned)cg.W) return 0u;
    return X[(((int64_t)n * cg.H + ih) * cg.W + iw) * cg.C + c];
}

template <bool KC, int R, int BK, int NT, int W>
__device__ __forceinline__ void slab_load_conv(const uint8_t* __restrict__ X, const ConvGeom& cg,
                                               int r0, int rows, int k0, int kend, int tid,
                                               uint32_t (&reg)[W]) {
#pragma unroll
    for (int w = 0; w < W; ++w) {
        const int d = tid + NT * w;
        int r, k;
        if (KC) { r = d / (BK / 4); k = (d % (BK / 4)) * 4; }
        else    { k = d / (R / 4);  r = (d % (R / 4)) * 4; }
        const int gr = r0 + r, gk = k0 + k;
        // pixel and first column of the word; valid columns [col, col + nb)
        const int pix = KC ? gr : gk, col = KC ? gk : gr;
        const bool in = gr < rows && gk < kend;
        const int lim = KC ? kend - gk : rows - gr;
        const int nb = lim < 4 ? lim : 4;
        uint32_t v = 0;
        if (in) {
            // one 4-byte load when the word is 4 aligned channels of one input
            // position (chunk ranges need not start at a multiple of 4)
            if (cg.vec && (col & 3) == 0) {
                const int n = pix / cg.OHW, rem = pix - n * cg.OHW;
                const int oh = rem / cg.OW, ow = rem - oh * cg.OW;
                const int kh = col / cg.KWC, r2 = col - kh * cg.KWC;
                const int kw = r2 / cg.C, c = r2 - kw * cg.C;
                const int ih = oh * cg.stride - cg.pad + kh, iw = ow * cg.stride - cg.pad + kw;
                if ((unsigned)ih < (unsigned)cg.H && (unsigned)iw < (unsigned)cg.W)
                    v = *reinterpret_cast<const uint32_t*>(
                        X + (((int64_t)n * cg.H + ih) * cg.W + iw) * cg.C + c);
                if (nb < 4) v &= (1u << (8 * nb)) - 1u;
            } else {
                for (int b = 0; b < nb; ++b) v |= xcol_byte(X, cg, pix, col + b) << (8 * b);
            }
        }
        reg[w] = v;
    }
}

// Decode a thread's words into the LDS slab, laid out [k][row] with `pitch`
// floats per k, each value times 2^SH.  The FP8 codes are the OCP E5M2
// ("bf8") encoding (bias 15, gradual underflow, exponent 31 for Inf/NaN), so
// the hardware conversion decodes two of them per instruction, exactly.
// TRACK keeps the largest magnitude decoded (amax) and flags any Inf/NaN
// code (special: nonzero iff some byte has an all-ones exponent field).
template <bool KC, int R, int BK, int NT, int W, int SH, bool TRACK>
__device__ __forceinline__ void slab_store(float* lds, int pitch, int tid,
                                           const uint32_t (&reg)[W], float& amax,
                                           uint32_t& special) {
    typedef float v2f __attribute__((ext_vector_type(2)));
#pragma unroll
    for (int w = 0; w < W; ++w) {
        const int d = tid + NT * w;
        const uint32_t v = reg[w];
        const v2f lo = __builtin_amdgcn_cvt_pk_f32_bf8((int)v, false);
        const v2f hi = __builtin_amdgcn_cvt_pk_f32_bf8((int)v, true);
        float f[4] = {lo.x, lo.y, hi.x, hi.y};
        if (TRACK) {
            // exponent field 0x7C in a byte: adding 0x04 sets its top bit,
            // and no smaller field carries into the next byte
            special |= ((v & 0x7C7C7C7Cu) + 0x04040404u) & 0x80808080u;
#pragma unroll
            for (int b = 0; b < 4; ++b) amax = fmaxf(amax, fabsf(f[b]));
        }
        if (SH != 0) {
#pragma unroll
            for (int b = 0; b < 4; ++b) f[b] *= __builtin_ldexpf(1.0f, SH);   // exact
        }
        if (KC) {
            const int r = d / (BK / 4), k = (d % (BK / 4)) * 4;
#pragma unroll
            for (int b = 0; b < 4; ++b) lds[(k + b) * pitch + r] = f[b];
        } else {
            const int k = d / (R / 4), r = (d % (R / 4)) * 4;
            *reinterpret_cast<float4*>(&lds[k * pitch + r]) = make_float4(f[0], f[1], f[2], f[3]);
        }
    }
}

// FP16 operands (chunk_gemm_p16): the same slab layout with each thread
// word holding 4 consecutive codes (8 bytes); `vec` allows 8-byte loads.
template <bool KC, int R, int BK, int NT, int W>
__device__ __forceinline__ void slab_load16(const uint16_t* __restrict__ ptr, int64_t ld,
                                            int vec, int r0, int rows, int k0, int kend,
                                            int tid, uint2 (&reg)[W]) {
#pragma unroll
    for (int w = 0; w < W; ++w) {
        const int d = tid + NT * w;
        int r, k;
        if (KC) { r = d / (BK / 4); k = (d % (BK / 4)) * 4; }
        else    { k = d / (R / 4);  r = (d % (R / 4)) * 4; }
        const int gr = r0 + r, gk = k0 + k;
        uint2 v = make_uint2(0u, 0u);
        if (gr < rows && gk < kend) {
            const uint16_t* q = KC ? ptr + (int64_t)gr * ld + gk : ptr + (int64_t)gk * ld + gr;
            const int lim = KC ? kend - gk : rows - gr;
            if (vec && lim >= 4) {
                v = *reinterpret_cast<const uint2*>(q);
            } else {
                uint32_t h[2] = {0u, 0u};
                for (int b = 0; b < 4; ++b)
                    if (b < lim) h[b / 2] |= (uint32_t)q[b] << (16 * (b % 2));
                v = make_uint2(h[0], h[1]);
            }
        }
        reg[w] = v;
    }
}

// Minimum of m over each 16-lane row, in every lane (DPP rotations by 8, 4,
// 2 and 1 within the row).
__device__ __forceinline__ uint32_t row_min(uint32_t m) {
    m = min(m, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)m, 0x128 /* row_ror:8 */, 0xF, 0xF, false));
    m = min(m, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)m, 0x124 /* row_ror:4 */, 0xF, 0xF, false));
    m = min(m, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)m, 0x122 /* row_ror:2 */, 0xF, 0xF, false));
    return min(m, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)m, 0x121 /* row_ror:1 */, 0xF, 0xF, false));
}

// op (max or or) over all 64 lanes of a wave, in every lane: DPP rotations
// within 16-lane rows, then the 16- and 32-lane swaps -- VALU steps instead
// of shuffles through the LDS crossbar (measured: Backward-data and Gradient
// GEMMs of the conv stage 1.5-2% faster, Forward 1% slower).
template <typename Op>
__device__ __forceinline__ uint32_t wave_reduce(uint32_t x, Op op) {
    x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x128 /* row_ror:8 */, 0xF, 0xF, false));
    x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x124 /* row_ror:4 */, 0xF, 0xF, false));
    x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x122 /* row_ror:2 */, 0xF, 0xF, false));
    x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x121 /* row_ror:1 */, 0xF, 0xF, false));
    const auto t16 = __builtin_amdgcn_permlane16_swap(x, x, false, false);
    x = op(x, op((uint32_t)t16[0], (uint32_t)t16[1]));
    const auto t32 = __builtin_amdgcn_permlane32_swap(x, x, false, false);
    return op(x, op((uint32_t)t32[0], (uint32_t)t32[1]));
}

// Minimum of m over the lanes of a wave equal modulo G (G 8 or 16: lane
// bits log2 G .. 5), in every lane: a DPP rotation by 8 within 16-lane rows,
// then gfx950's 16- and 32-lane swaps (each returns both registers' swapped
// halves; their minimum with m is the partner lane's value or m's own).
template <int G>
__device__ __forceinline__ uint32_t lanes_mod_min(uint32_t m) {
    static_assert(G == 8 || G == 16, "lanes equal modulo 8 or 16");
    if constexpr (G == 8)
        m = min(m, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)m, 0x128 /* row_ror:8 */, 0xF,
                                                         0xF, false));
    const auto t16 = __builtin_amdgcn_permlane16_swap(m, m, false, false);
    m = min(m, min((uint32_t)t16[0], (uint32_t)t16[1]));
    const auto t32 = __builtin_amdgcn_permlane32_swap(m, m, false, false);
    return min(m, min((uint32_t)t32[0], (uint32_t)t32[1]));
}

// Decode FP16 words into the LDS slab, each value times 2^SH; TRACK keeps the
// largest magnitude and flags Inf/NaN codes (exponent field 63: adding 0x200
// to the masked field sets bit 15 only then), and lowers kmin[k] to the
// smallest nonzero magnitude staged at k, held as its bit pattern minus one
// (a zero wraps to ~0, which never lowers the entry).  Where the lanes of a
// wave that stage the same k form groups of 8 or 16 (a k-contiguous operand
// of 64 or more rows: lanes equal modulo BK/4; a row-contiguous one of 64
// rows: 16-lane runs), they first take their minima across lanes and one of
// them updates kmin, instead of every lane's atomic on the same LDS address
// (FP16-operand GEMMs of the 1024 -> 6000 layer, Forward / Backward /
// Gradient: 0.292 / 0.333 / 0.220 -> 0.283 / 0.285 / 0.221 ms).  Elsewhere
// the reduction measured slower than the atomics (32-lane runs; tiles of 32
// rows, with 8 times less compute per staged word).
template <bool KC, int R, int BK, int NT, int W, int SH, bool TRACK>
__device__ __forceinline__ void slab_store16(float* lds, int pitch, int tid,
                                             const uint2 (&reg)[W], float& amax,
                                             uint32_t& special, uint32_t* kmin) {
    static_assert(NT % (BK / 4) == 0, "a thread's words share one k group");
    auto key = [](float f) __attribute__((always_inline)) -> uint32_t {
        return (__float_as_uint(f) & 0x7FFFFFFFu) - 1u;
    };
    uint32_t mk[4] = {~0u, ~0u, ~0u, ~0u};  // KC: minima of this thread's 4 k
#pragma unroll
    for (int w = 0; w < W; ++w) {
        const int d = tid + NT * w;
        const uint32_t v[2] = {reg[w].x, reg[w].y};
        float f[4];
#pragma unroll
        for (int b = 0; b < 4; ++b) f[b] = fp16_to_f32_pow2<SH>((v[b / 2] >> (16 * (b % 2))) & 0xFFFFu);
        if (TRACK) {
#pragma unroll
            for (int h = 0; h < 2; ++h)
                special |= ((v[h] & 0x7E007E00u) + 0x02000200u) & 0x80008000u;
#pragma unroll
            for (int b = 0; b < 4; ++b) amax = fmaxf(amax, fabsf(f[b]));
            if (KC) {
#pragma unroll
                for (int b = 0; b < 4; ++b) mk[b] = min(mk[b], key(f[b]));
            } else {
                const int k = d / (R / 4);
                uint32_t m = min(min(key(f[0]), key(f[1])), min(key(f[2]), key(f[3])));
                if constexpr (R / 4 == 16) {
                    // the 16 lanes of a row stage the same k
                    m = row_min(m);
                    if ((tid & 15) == 0) atomicMin(&kmin[k], m);
                } else {
                    atomicMin(&kmin[k], m);
                }
            }
        }
        if (KC) {
            const int r = d / (BK / 4), k = (d % (BK / 4)) * 4;
#pragma unroll
            for (int b = 0; b < 4; ++b) lds[(k + b) * pitch + r] = f[b];
        } else {
            const int k = d / (R / 4), r = (d % (R / 4)) * 4;
            *reinterpret_cast<float4*>(&lds[k * pitch + r]) = make_float4(f[0], f[1], f[2], f[3]);
        }
    }
    if (TRACK && KC) {
        const int k = (tid % (BK / 4)) * 4;
        if constexpr ((BK / 4 == 8 || BK / 4 == 16) && R >= 64) {
#pragma unroll
            for (int b = 0; b < 4; ++b) mk[b] = lanes_mod_min<BK / 4>(mk[b]);
            if ((tid & 63) < BK / 4) {
#pragma unroll
                for (int b = 0; b < 4; ++b) atomicMin(&kmin[k + b], mk[b]);
            }
        } else {
#pragma unroll
            for (int b = 0; b < 4; ++b) atomicMin(&kmin[k + b], mk[b]);
        }
    }
}

// CONV: the A operand is the implicit lowering of an NHWC input (g.conv).
// P16: A and B hold FP16 codes (chunk_gemm_p16, exact mode only).
template <int TM, int TN, int LM, int LN, int BK, bool PF, int WPE, bool TA, bool TB, bool FAST,
          bool CONV = false, bool P16 = false>
__global__ __launch_bounds__(LM * LN) __attribute__((amdgpu_waves_per_eu(WPE)))
void chunk_gemm_valu(GemmArgs g, Plan p) {
    constexpr int NT = LM * LN;
    constexpr int BM = TM * LM;
    constexpr int BN = TN * LN;
    // 4-byte words per thread per slab
    constexpr int WA = BM * BK / 4 / NT;
    constexpr int WB = BN * BK / 4 / NT;
    static_assert(WA * NT * 4 == BM * BK && WB * NT * 4 == BN * BK, "tile/threads mismatch");
    static_assert(BK % 4 == 0 && BM % 4 == 0 && BN % 4 == 0, "tile must hold whole words");
    static_assert(TN == 1 || TN % 2 == 0, "codes are stored in pairs");
    // padding of rows written with a stride across lanes (spreads LDS banks)
    constexpr int PA = TA ? 0 : 4;
    constexpr int PB = TB ? 4 : 0;
    constexpr bool KCA = !TA;      // A is k-contiguous unless transposed
    constexpr bool KCB = TB;       // B is k-contiguous only when transposed
    // The guarded path exists for the exact mode; the fast mode's VALU
    // variant (chunks summed in plain FP32, rounded once) always runs safe.
    constexpr bool HAS_GUARDED = !FAST;

    __shared__ __attribute__((aligned(16))) float As[2][BK][BM + PA];
    __shared__ __attribute__((aligned(16))) float Bs[2][BK][BN + PB];
    // |a| max bits, |b| max bits, specials, |S| max bits of the guarded
    // pieces, in two slots used by alternate pieces
    __shared__ uint32_t s_track[2][4];
    // FP16 operands on the guarded path: per k of a staged slab, the smallest
    // nonzero |a| over the tile's rows and |b| over its columns (bit pattern
    // minus one, ~0 for none), in three slots used by successive slabs
    __shared__ uint32_t s_kmin[P16 ? 3 : 1][2][P16 ? BK : 1];

    const int tid = threadIdx.x;
    const int ly = tid / LN, lx = tid % LN;

    // a thread word: 4 FP8 codes (4 bytes) or 4 FP16 codes (8 bytes)
    typedef typename std::conditional<P16, uint2, uint32_t>::type Word;
    Word ra[WA], rb[WB];
    float P[TM][TN], S[TM][TN];
    int gslot = 0;
    if (tid < 6) (&s_track[0][0])[tid] = 0;    // ordered by the first slab's barrier
    // Slabs staged on the guarded path so far; slab c fills slot c % 3 and
    // clears slot (c + 1) % 3, whose last reader (slab c - 2) finished before
    // the barrier that precedes the staging of slab c.
    int sc = 0;
    if (P16) {
        for (int q = tid; q < 3 * 2 * BK; q += NT) (&s_kmin[0][0][0])[q] = ~0u;
        __syncthreads();
    }

    auto load_a = [&](int m0, int k0, int kend) __attribute__((always_inline)) {
        if constexpr (P16)
            slab_load16<KCA, BM, BK, NT, WA>(reinterpret_cast<const uint16_t*>(g.A), g.lda,
                                             g.a_vec, m0, g.M, k0, kend, tid, ra);
        else if constexpr (CONV)
            slab_load_conv<KCA, BM, BK, NT, WA>(g.A, g.conv, m0, g.M, k0, kend, tid, ra);
        else
            slab_load<KCA, BM, BK, NT, WA>(g.A, g.lda, g.a_vec, m0, g.M, k0, kend, tid, ra);
    };
    auto load_b = [&](int n0, int k0, int kend) __attribute__((always_inline)) {
        if constexpr (P16)
            slab_load16<KCB, BN, BK, NT, WB>(reinterpret_cast<const uint16_t*>(g.B), g.ldb,
                                             g.b_vec, n0, g.N, k0, kend, tid, rb);
        else
            slab_load<KCB, BN, BK, NT, WB>(g.B, g.ldb, g.b_vec, n0, g.N, k0, kend, tid, rb);
    };

    auto lds_read = [&](float (&a)[TM], float (&b)[TN], int buf, int kk) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < TM; ++i) a[i] = As[buf][kk][ly * TM + i];
#pragma unroll
        for (int j = 0; j < TN; ++j) b[j] = Bs[buf][kk][lx * TN + j];
    };

    // One piece: chunks [c0, c1) of tile `tile`.  lt >= 0 marks a shared tile
    // (its index among the shared tiles), whose chunk sums go to the workspace
    // when the piece does not start at chunk 0.  SAFE selects the path (see
    // the top of this file); the guarded path returns false, having written
    // nothing to C, when its check fails.
    auto piece = [&](auto safe_tag, int64_t tile, int c0, int c1, int64_t lt)
                     __attribute__((always_inline)) -> bool {
        constexpr bool SAFE = decltype(safe_tag)::value;
        // value scale of the path: 2^96 (safe, exact), 1 (guarded); the
        // fast mode's VALU variant sums plain products and scales per chunk
        constexpr int DOM = SAFE ? 96 : 0;
        constexpr int ASHIFT = FAST ? 0 : DOM;
        constexpr bool TRACK = !SAFE;

        int tr, tc;
        tile_rc(p, tile, tr, tc);
        const int m0 = tr * BM;
        const int n0 = tc * BN;
        const int kbeg = (int)((int64_t)c0 * g.CL);
        const int64_t kend64 = (int64_t)c1 * g.CL;
        const int kend = kend64 < g.K ? (int)kend64 : g.K;
        const bool to_ws = c0 > 0;
        int chunk = c0;
        float amax_a = 0.0f, amax_b = 0.0f;  // largest magnitudes decoded
        uint32_t special = 0;                // Inf/NaN codes seen
        float smax = 0.0f;                   // largest running sum at a chunk end

        auto rnd = [&](float x) __attribute__((always_inline)) -> float {
            return SAFE ? rn16s(x) : rn16v(x);
        };
        auto chunk_value = [&](float x) __attribute__((always_inline)) -> float {
            return FAST ? rn16s(x * 0x1p96f) : x;
        };
        // FP16 operands: each product is rounded to FP16 before it is added.
        // With VSPLIT (guarded path, every nonzero product of the slab at
        // least 2^-30) by Veltkamp splitting of the exact product p = a b:
        // c = a (b (2^14 + 1)) is RN(p (2^14 + 1)) -- b (2^14 + 1) is exact,
        // b having at most 10 significant bits -- and p - c = fma(a, b, -c),
        // so hi = c + fma(a, b, -c) is rn16v(p) in three instructions (a zero
        // product gives +0).  Otherwise by the clamped magic-number add.
        auto first_step = [&](auto vsplit, const float (&a)[TM], const float (&b)[TN])
                              __attribute__((always_inline)) {
            constexpr bool VSPLIT = decltype(vsplit)::value;
            float bs[TN];
#pragma unroll
            for (int j = 0; j < TN; ++j) bs[j] = VSPLIT ? b[j] * 16385.0f : 0.0f;
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    if (VSPLIT) {
                        const float c = a[i] * bs[j];
                        P[i][j] = c + __builtin_fmaf(a[i], b[j], -c);
                    } else if (P16) {
                        P[i][j] = (SAFE ? rn16_product_s(a[i] * b[j])
                                        : rn16_product(a[i] * b[j])) + 0.0f;
                    } else {
                        P[i][j] = __builtin_fmaf(a[i], b[j], 0.0f);
                    }
                }
        };
        auto fma_step = [&](auto vsplit, const float (&a)[TM], const float (&b)[TN])
                            __attribute__((always_inline)) {
            constexpr bool VSPLIT = decltype(vsplit)::value;
            float bs[TN];
#pragma unroll
            for (int j = 0; j < TN; ++j) bs[j] = VSPLIT ? b[j] * 16385.0f : 0.0f;
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    float t;
                    if (VSPLIT) {
                        const float c = a[i] * bs[j];
                        t = P[i][j] + (c + __builtin_fmaf(a[i], b[j], -c));
                    } else if (P16) {
                        t = P[i][j] + (SAFE ? rn16_product_s(a[i] * b[j])
                                            : rn16_product(a[i] * b[j]));
                    } else {
                        t = __builtin_fmaf(a[i], b[j], P[i][j]);
                    }
                    P[i][j] = FAST ? t : rnd(t);
                }
        };
        // operand slabs: HBM -> registers, registers -> LDS (decoded; on the
        // safe path FP8 A is scaled by 2^96, FP16 A and B by 2^48 and 2^16,
        // their products then by 2^64)
        auto fetch_slab = [&](int k0) __attribute__((always_inline)) {
            load_a(m0, k0, kend);
            load_b(n0, k0, kend);
        };
        auto stage_slab = [&](int buf) __attribute__((always_inline)) {
            if constexpr (P16) {
                uint32_t* km = &s_kmin[sc % 3][0][0];
                slab_store16<KCA, BM, BK, NT, WA, SAFE ? 48 : 0, TRACK>(
                    &As[buf][0][0], BM + PA, tid, ra, amax_a, special, km);
                slab_store16<KCB, BN, BK, NT, WB, SAFE ? 16 : 0, TRACK>(
                    &Bs[buf][0][0], BN + PB, tid, rb, amax_b, special, km + BK);
                if (TRACK) {
                    if (tid < 2 * BK) (&s_kmin[(sc + 1) % 3][0][0])[tid] = ~0u;
                    ++sc;
                }
            } else {
                slab_store<KCA, BM, BK, NT, WA, ASHIFT, TRACK>(&As[buf][0][0], BM + PA, tid, ra,
                                                               amax_a, special);
                slab_store<KCB, BN, BK, NT, WB, 0, TRACK>(&Bs[buf][0][0], BN + PB, tid, rb,
                                                          amax_b, special);
            }
        };

#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) { P[i][j] = 0.0f; S[i][j] = 0.0f; }

        // FP16 code of a chunk sum or running sum: on the guarded path the
        // value is on the FP16 grid and, unless the piece fails its guard
        // (and is redone on the safe path), below 2^32
        auto code = [&](float x) __attribute__((always_inline)) -> uint32_t {
            if constexpr (!SAFE && !FAST) return f32g_to_fp16(x);
            else return f32d_to_fp16<DOM>(x);
        };
        auto flush = [&]() __attribute__((always_inline)) {
            if (to_ws) {
#pragma unroll
                for (int i = 0; i < TM; ++i) {
                    uint16_t* dst = g.ws + ws_index(p, BM, BN, lt, chunk, ly * TM + i, lx * TN);
                    uint32_t w[(TN + 1) / 2];
#pragma unroll
                    for (int j = 0; j < TN; j += 2) {
                        uint32_t c = code(chunk_value(P[i][j]));
                        if (j + 1 < TN)
                            c |= code(chunk_value(P[i][j + 1])) << 16;
                        w[j / 2] = c;
                    }
                    // chunk sums are read once, by the fold pass: stored
                    // non-temporally (4 codes per store where the lane has
                    // them), so they do not evict the operands' lines
                    if constexpr (TN == 4) {
                        typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
                        const u32x2_t v = {w[0], w[1]};
                        __builtin_nontemporal_store(v, reinterpret_cast<u32x2_t*>(dst));
                    } else if (TN == 1) {
                        dst[0] = (uint16_t)w[0];
                    } else {
#pragma unroll
                        for (int j = 0; j < TN / 2; ++j) reinterpret_cast<uint32_t*>(dst)[j] = w[j];
                    }
                }
            } else {
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j) S[i][j] = rnd(S[i][j] + chunk_value(P[i][j]));
                if (TRACK) {
#pragma unroll
                    for (int i = 0; i < TM; ++i)
#pragma unroll
                        for (int j = 0; j < TN; j += 2)
                            smax = max3_abs(smax, S[i][j], S[i][TN > 1 ? j + 1 : j]);
                }
            }
            ++chunk;                     // the next chunk starts with first_step
        };

        const int nk = kend - kbeg;
        const int nslabs = (nk + BK - 1) / BK;
        int crem = g.CL;                 // products left in the current chunk
        const int sc0 = sc;              // guarded FP16: counter of this piece's first slab
        // Whether every nonzero product of the staged slab in slot `slot` is
        // at least 2^-30 (then Veltkamp splitting rounds the products): lane
        // k of each wave checks k, and the wave votes.
        auto slab_vsplit = [&](int slot) __attribute__((always_inline)) -> bool {
            bool ok = true;
            const int lane = tid & 63;
            if (lane < BK) {
                const uint32_t ka = s_kmin[slot][0][lane], kb = s_kmin[slot][1][lane];
                if (ka != ~0u && kb != ~0u)
                    ok = __uint_as_float(ka + 1u) * __uint_as_float(kb + 1u) >= 0x1p-30f;
            }
            return __all(ok);
        };
        fetch_slab(kbeg);
        stage_slab(0);
        __syncthreads();
        for (int s = 0; s < nslabs; ++s) {
            const int buf = s & 1;
            const int ks = kbeg + s * BK;
            if (s + 1 < nslabs) fetch_slab(ks + BK);
            const int kmax = min(BK, kend - ks);
            auto compute = [&](auto vsplit) __attribute__((always_inline)) {
            int kk = 0;
            while (kk < kmax) {
                const int seg = min(kmax - kk, crem);
                if (seg == BK) {
                    // Every chunk begins with a product into a zero partial
                    // sum, exact and already an FP16 value (at most 6
                    // significant bits, well inside the range): one fma with 0
                    // (which also turns -0 into +0) and no rounding.
                    const bool fresh = crem == g.CL;
                    if (PF) {
                        float a0[TM], b0[TN], a1[TM], b1[TN];
                        lds_read(a0, b0, buf, 0);
#pragma unroll
                        for (int q = 0; q < BK; q += 2) {
                            lds_read(a1, b1, buf, q + 1);
                            if (q == 0 && fresh) first_step(vsplit, a0, b0);
                            else fma_step(vsplit, a0, b0);
                            if (q + 2 < BK) lds_read(a0, b0, buf, q + 2);
                            fma_step(vsplit, a1, b1);
                        }
                    } else {
#pragma unroll
                        for (int q = 0; q < BK; ++q) {
                            float a[TM], b[TN];
                            lds_read(a, b, buf, q);
                            if (q == 0 && fresh) first_step(vsplit, a, b);
                            else fma_step(vsplit, a, b);
                        }
                    }
                } else {
                    const bool fresh = crem == g.CL;
                    for (int q = kk; q < kk + seg; ++q) {
                        float a[TM], b[TN];
                        lds_read(a, b, buf, q);
                        if (q == kk && fresh) first_step(vsplit, a, b);
                        else fma_step(vsplit, a, b);
                    }
                }
                kk += seg;
                crem -= seg;
                if (crem == 0) {
                    flush();
                    crem = g.CL;
                }
            }
            };
            if constexpr (P16 && TRACK) {
                if (slab_vsplit((sc0 + s) % 3)) compute(std::true_type{});
                else compute(std::false_type{});
            } else {
                compute(std::false_type{});
            }
            if (s + 1 < nslabs) stage_slab(buf ^ 1);
            __syncthreads();
        }
        if (crem != g.CL) flush();       // the last, shorter chunk

        if (!SAFE) {
            // Largest magnitudes over the workgroup's operands and running
            // sums of this piece (reduced within each wave, then one LDS
            // atomic per wave).  A piece that leaves chunk sums in the
            // workspace computes no running sum (the fold pass adds them in
            // the scaled domain, where overflow is exact); the first piece of
            // a shared tile and whole tiles are checked on their running sums.
            // Slot `gslot` was cleared during the previous guarded piece and
            // is read after the one barrier here; the other slot, cleared
            // now, is next written after at least one more barrier (every
            // piece has a slab).
            uint32_t* st = s_track[gslot];
            uint32_t ua = __float_as_uint(amax_a), ub = __float_as_uint(amax_b), us = special;
            uint32_t uS = __float_as_uint(smax);
            // non-negative floats: bit order
            auto umax = [](uint32_t x, uint32_t y) __attribute__((always_inline)) { return max(x, y); };
            auto uor = [](uint32_t x, uint32_t y) __attribute__((always_inline)) { return x | y; };
            ua = wave_reduce(ua, umax);
            ub = wave_reduce(ub, umax);
            us = wave_reduce(us, uor);
            uS = wave_reduce(uS, umax);
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
            if (sp) return false;                                   // Inf or NaN operand
            // chunk partial sums: at most 3 CL max|a| max|b| (CL <= K here);
            // a product rounded to FP16 is at most (1 + 2^-10) |a b|, or 2^-39
            // in the subnormal range
            const double bound = P16 ? 3.01 * (double)g.CL * (double)ma * (double)mb + 1.0
                                     : 3.0 * (double)g.CL * (double)ma * (double)mb;
            if (!(bound < 2147483648.0)) return false;             // 2^31
            if (!(sm < 2147483648.0f)) return false;               // running sums
        }
        if (to_ws) return true;
        // The first piece of a shared tile leaves its running sum for the
        // fold pass: in C, or in s_ws when only the FP8 result is wanted.
        if (lt >= 0 && !g.C) {
            uint16_t* dst = g.s_ws + (lt * BM + ly * TM) * BN + lx * TN;
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) dst[i * BN + j] = (uint16_t)code(S[i][j]);
            return true;
        }
        // The running sum: a lane's TN consecutive codes of a row are stored
        // four per 8-byte store (the 16 lanes of a row then write whole
        // 128-byte lines with one instruction), else in pairs, when
        // the whole row lies inside C and is aligned; the FP8 result (whole
        // tiles only: shared tiles get it from the fold pass) four codes per
        // 4-byte store under the same conditions, else byte by byte.
        const int nl = n0 + lx * TN;
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            const int m = m0 + ly * TM + i;
            if (m >= g.M) continue;
            if (g.C) {
                uint16_t* crow = g.C + (int64_t)m * g.ldc + nl;
                if (TN % 4 == 0 && g.c_vec8 && nl + TN <= g.N) {
#pragma unroll
                    for (int j = 0; j < TN; j += 4) {
                        uint2 c;
                        c.x = code(S[i][j]) |
                              (code(S[i][j + 1]) << 16);
                        c.y = code(S[i][j + 2]) |
                              (code(S[i][j + 3]) << 16);
                        reinterpret_cast<uint2*>(crow)[j / 4] = c;
                    }
                } else if (TN > 1 && g.c_vec && nl + TN <= g.N) {
#pragma unroll
                    for (int j = 0; j < TN; j += 2) {
                        uint32_t c = code(S[i][j]) |
                                     (code(S[i][j + 1]) << 16);
                        reinterpret_cast<uint32_t*>(crow)[j / 2] = c;
                    }
                } else {
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        if (nl + j < g.N) crow[j] = (uint16_t)code(S[i][j]);
                }
            }
            if (g.C8 && lt < 0) {
                uint8_t* qrow = g.C8 + (int64_t)m * g.ldc8 + nl;
                if (TN % 4 == 0 && g.c8_vec4 && nl + TN <= g.N) {
                    // Q8(RN32(value * scale)): the 2^-DOM scaling is exact
                    const float u = __builtin_ldexpf(1.0f, -DOM);
#pragma unroll
                    for (int j = 0; j < TN; j += 4) {
                        uint32_t q = f32x2_to_fp8x2<false>((S[i][j] * u) * g.q_scale,
                                                           (S[i][j + 1] * u) * g.q_scale, 0u);
                        q = f32x2_to_fp8x2<true>((S[i][j + 2] * u) * g.q_scale,
                                                 (S[i][j + 3] * u) * g.q_scale, q);
                        reinterpret_cast<uint32_t*>(qrow)[j / 4] = q;
                    }
                } else {
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        if (nl + j < g.N)
                            qrow[j] = (uint8_t)f32d_to_fp8_scaled<DOM>(S[i][j], g.q_scale);
                }
            }
        }
        return true;
    };

    // Work items of this workgroup: whole tiles, then its range of the
    // shared tile-chunks (gemm_plan.h).  One call site per path keeps one
    // copy of each path's code.
    const int w = blockIdx.x;
    int64_t t = w;
    int64_t s = p.L > 0 ? (int64_t)w * p.L / p.G : 0;
    const int64_t e = p.L > 0 ? (int64_t)(w + 1) * p.L / p.G : 0;
    auto fetch = [&](int64_t& tile, int64_t& lt, int& c0, int& c1)
                     __attribute__((always_inline)) -> bool {
        if (t < p.t_whole) {
            tile = whole_tile(p, t);
            lt = -1;
            c0 = 0;
            c1 = p.nch;
            t += p.G;
            return true;
        }
        if (s < e) {
            lt = s / p.nch;
            c0 = (int)(s - lt * p.nch);
            const int64_t c1l = e - lt * p.nch;
            c1 = c1l < p.nch ? (int)c1l : p.nch;
            tile = p.t_whole + lt;
            s = lt * p.nch + c1;
            return true;
        }
        return false;
    };
    int64_t tile, lt;
    int c0, c1;
    while (fetch(tile, lt, c0, c1)) {
        bool done = false;
        if (HAS_GUARDED && g.guarded)
            done = piece(std::integral_constant<bool, false>{}, tile, c0, c1, lt);
        if (!done) piece(std::integral_constant<bool, true>{}, tile, c0, c1, lt);
    }
}

// Register tiles: TM x TN outputs per lane, lane grid LM x LN, K slab BK,
// LDS prefetch PF, and the waves per SIMD the register budget must allow.
template <int C> struct ValuCfg;
template <> struct ValuCfg<0> { static constexpr int TM = 8, TN = 8, LM = 16, LN = 16, BK = 16, WPE = 2; static constexpr bool PF = false; };
template <> struct ValuCfg<1> { static constexpr int TM = 8, TN = 8, LM = 16, LN = 16, BK = 16, WPE = 2; static constexpr bool PF = true; };
template <> struct ValuCfg<2> { static constexpr int TM = 8, TN = 4, LM = 16, LN = 16, BK = 16, WPE = 3; static constexpr bool PF = true; };
template <> struct ValuCfg<3> { static constexpr int TM = 4, TN = 8, LM = 16, LN = 16, BK = 16, WPE = 3; static constexpr bool PF = true; };
template <> struct ValuCfg<4> { static constexpr int TM = 4, TN = 4, LM = 16, LN = 16, BK = 32, WPE = 4; static constexpr bool PF = true; };
template <> struct ValuCfg<5> { static constexpr int TM = 2, TN = 2, LM = 16, LN = 16, BK = 32, WPE = 8; static constexpr bool PF = false; };
template <> struct ValuCfg<6> { static constexpr int TM = 1, TN = 1, LM = 16, LN = 16, BK = 64, WPE = 8; static constexpr bool PF = false; };
template <> struct ValuCfg<7> { static constexpr int TM = 4, TN = 4, LM = 32, LN = 16, BK = 32, WPE = 4; static constexpr bool PF = true; };
template <> struct ValuCfg<8> { static constexpr int TM = 4, TN = 4, LM = 16, LN = 32, BK = 32, WPE = 4; static constexpr bool PF = true; };

template <int C, bool TA, bool TB, bool FAST>
const void* kernel_of() {
    using Q = ValuCfg<C>;
    return reinterpret_cast<const void*>(
        &chunk_gemm_valu<Q::TM, Q::TN, Q::LM, Q::LN, Q::BK, Q::PF, Q::WPE, TA, TB, FAST>);
}

// Entry addresses of every configuration for one operand layout; the fast
// variants exist for the configurations from kValuFastFirst on.
template <bool TA, bool TB>
const void* kernel_table(int cfg, int fast) {
    if (fast) {
        switch (cfg) {
            case 4: return kernel_of<4, TA, TB, true>();
            case 5: return kernel_of<5, TA, TB, true>();
            case 6: return kernel_of<6, TA, TB, true>();
            default: return nullptr;
        }
    }
    switch (cfg) {
        case 0: return kernel_of<0, TA, TB, false>();
        case 1: return kernel_of<1, TA, TB, false>();
        case 2: return kernel_of<2, TA, TB, false>();
        case 3: return kernel_of<3, TA, TB, false>();
        case 4: return kernel_of<4, TA, TB, false>();
        case 5: return kernel_of<5, TA, TB, false>();
        case 6: return kernel_of<6, TA, TB, false>();
        case 7: return kernel_of<7, TA, TB, false>();
        case 8: return kernel_of<8, TA, TB, false>();
        default: return nullptr;
    }
}

// FP16-operand kernels (chunk_gemm_p16) of the configurations built for them:
// the 4 x 4 tiles (4, 7, 8) and the small ones for few outputs (5, 6).
template <int C, bool TA, bool TB>
const void* kernel_of_p16() {
    using Q = ValuCfg<C>;
    return reinterpret_cast<const void*>(&chunk_gemm_valu<Q::TM, Q::TN, Q::LM, Q::LN, Q::BK,
                                                          Q::PF, Q::WPE, TA, TB, false, false,
                                                          true>);
}

template <bool TA, bool TB>
const void* kernel_table_p16(int cfg) {
    switch (cfg) {
        case 4: return kernel_of_p16<4, TA, TB>();
        case 5: return kernel_of_p16<5, TA, TB>();
        case 6: return kernel_of_p16<6, TA, TB>();
        case 7: return kernel_of_p16<7, TA, TB>();
        case 8: return kernel_of_p16<8, TA, TB>();
        default: return nullptr;
    }
}

template <int C>
ValuShape shape_of() {
    using Q = ValuCfg<C>;
    return ValuShape{Q::TM, Q::TN, Q::TM * Q::LM, Q::TN * Q::LN, Q::LM * Q::LN};
}

}  // namespace valu_impl
}  // namespace fp8t
