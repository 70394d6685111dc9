/*
 * Oracle: the three operations of the hot path.
 * TEST INFRASTRUCTURE ONLY (see oracle.h).
 */
#include "oracle.h"
#include "oracle_internal.h"

#include <math.h>
#include <stddef.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int orc_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads used by the OpenMP loops from now on (n >= 1); for timing the
 * oracle on one core beside the all-core run. */
void orc_set_threads(int n) {
#ifdef _OPENMP
    if (n >= 1) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* ---- operand quantization ------------------------------------------------
 * Sec. 2.1: weights, activations, errors and gradients are held in FP8 for
 * all GEMMs.  The rounding into P8 is round-to-nearest-even (the paper names
 * no mode for it).  An FP32 source is rounded once; a P16 source is first
 * decoded exactly.  The value is multiplied by `scale` in FP32 first (used for
 * loss scaling, Sec. 3). */
int cpu_fp8_quantize(const void* src, int src_format, float scale,
                     uint8_t* dst, int64_t n) {
    if (n < 0) return ORC_EINVAL;
    if (n > 0 && (!src || !dst)) return ORC_EINVAL;
    if (src_format != ORC_SRC_F32 && src_format != ORC_SRC_P16) return ORC_EINVAL;
    for (int64_t i = 0; i < n; i++) {
        float x;
        if (src_format == ORC_SRC_F32)
            x = ((const float*)src)[i];
        else
            x = (float)orc_p16_value(((const uint16_t*)src)[i]);
        volatile float xs = x * scale;          /* one FP32 product */
        dst[i] = orc_q8((double)xs);
    }
    return ORC_OK;
}

/* Round FP32 values to the nearest P16 value, ties to even (Sec. 2.2 names
 * round-to-nearest for P16; used to create P16 master weights, Sec. 3). */
int cpu_fp16_quantize(const float* src, uint16_t* dst, int64_t n) {
    if (n < 0) return ORC_EINVAL;
    if (n > 0 && (!src || !dst)) return ORC_EINVAL;
    for (int64_t i = 0; i < n; i++) dst[i] = orc_rn16((double)src[i]);
    return ORC_OK;
}

/* ---- chunk-based reduced-precision dot products --------------------------
 * Sec. 2.3, "Chunk-based Accumulation", and the dot-product algorithm of
 * Fig. 3(a): the length-K dot product is cut into chunks of CL consecutive
 * terms (starting at k = 0; the last chunk may be shorter).  Inside a chunk
 * the products are added one by one, in ascending k, into one extra variable
 * (the intra-chunk sum), rounding to P16 after every addition; after each
 * chunk that partial sum is added, again with P16 rounding, into the running
 * sum (inter-chunk accumulation).  Both sums start at +0.
 *
 * The fast mode (not in the paper) forms each chunk's partial sum exactly and
 * rounds it to P16 once, then accumulates chunks exactly as above. */

static inline uint8_t op_a(int trans_a, const uint8_t* A, int64_t lda,
                           int64_t i, int64_t k) {
    return trans_a ? A[k * lda + i] : A[i * lda + k];
}

static inline uint8_t op_b(int trans_b, const uint8_t* B, int64_t ldb,
                           int64_t k, int64_t j) {
    return trans_b ? B[j * ldb + k] : B[k * ldb + j];
}

static uint16_t chunk_dot(int trans_a, int trans_b, int64_t K, int64_t CL,
                          const uint8_t* A, int64_t lda, const uint8_t* B,
                          int64_t ldb, int mode, int64_t i, int64_t j) {
    xnum S = xn_zero(0);
    for (int64_t c0 = 0; c0 < K; c0 += CL) {
        int64_t c1 = (K - c0 < CL) ? K : c0 + CL;
        xnum P = xn_zero(0);
        if (mode == ORC_EXACT) {
            for (int64_t k = c0; k < c1; k++) {
                xnum p = xn_mul_p8(op_a(trans_a, A, lda, i, k),
                                   op_b(trans_b, B, ldb, k, j));
                P = xn_from_p16(xn_round_p16(xn_add(P, p)));
            }
        } else {
            xnum sum = xn_zero(0);
            for (int64_t k = c0; k < c1; k++) {
                xnum p = xn_mul_p8(op_a(trans_a, A, lda, i, k),
                                   op_b(trans_b, B, ldb, k, j));
                sum = xn_add(sum, p);
            }
            P = xn_from_p16(xn_round_p16(xn_add(P, sum)));
        }
        S = xn_from_p16(xn_round_p16(xn_add(S, P)));
    }
    return xn_round_p16(S);
}

static int gemm_args_ok(int trans_a, int trans_b, int64_t M, int64_t N,
                        int64_t K, int64_t CL, const uint8_t* A, int64_t lda,
                        const uint8_t* B, int64_t ldb, int mode) {
    if (M < 0 || N < 0 || K < 0 || CL < 1) return 0;
    if ((trans_a != 0 && trans_a != 1) || (trans_b != 0 && trans_b != 1)) return 0;
    if (mode != ORC_EXACT && mode != ORC_FAST) return 0;
    if (M > 0 && N > 0 && K > 0) {
        if (!A || !B) return 0;
        if (lda < (trans_a ? M : K)) return 0;
        if (ldb < (trans_b ? K : N)) return 0;
    }
    return 1;
}

int cpu_chunk_gemm(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K,
                   int64_t CL, const uint8_t* A, int64_t lda,
                   const uint8_t* B, int64_t ldb, uint16_t* C, int64_t ldc,
                   int mode) {
    if (!gemm_args_ok(trans_a, trans_b, M, N, K, CL, A, lda, B, ldb, mode))
        return ORC_EINVAL;
    if (M > 0 && N > 0 && (!C || ldc < N)) return ORC_EINVAL;
    #pragma omp parallel for schedule(dynamic, 1)
    for (int64_t i = 0; i < M; i++)
        for (int64_t j = 0; j < N; j++)
            C[i * ldc + j] = chunk_dot(trans_a, trans_b, K, CL, A, lda, B, ldb,
                                       mode, i, j);
    return ORC_OK;
}

int cpu_chunk_gemm_points(int trans_a, int trans_b, int64_t M, int64_t N,
                          int64_t K, int64_t CL, const uint8_t* A, int64_t lda,
                          const uint8_t* B, int64_t ldb, int mode,
                          const int64_t* rows, const int64_t* cols,
                          int64_t npts, uint16_t* out) {
    if (!gemm_args_ok(trans_a, trans_b, M, N, K, CL, A, lda, B, ldb, mode))
        return ORC_EINVAL;
    if (npts < 0 || (npts > 0 && (!rows || !cols || !out))) return ORC_EINVAL;
    for (int64_t p = 0; p < npts; p++)
        if (rows[p] < 0 || rows[p] >= M || cols[p] < 0 || cols[p] >= N)
            return ORC_EINVAL;
    #pragma omp parallel for schedule(dynamic, 1)
    for (int64_t p = 0; p < npts; p++)
        out[p] = chunk_dot(trans_a, trans_b, K, CL, A, lda, B, ldb, mode,
                           rows[p], cols[p]);
    return ORC_OK;
}

/* ---- the results the fast mode may give -----------------------------------
 * The fast mode (a build variant; the paper defines only the exact chunked
 * accumulation of Sec. 2.3) forms each chunk's sum without rounding to P16
 * after every addition, rounds it to P16 once, and accumulates the chunk sums
 * in order exactly as Fig. 3(a).  It has no single bit-exact result, so the
 * oracle gives bounds: a centre T_c and a half-width e_c per chunk such that
 * the chunk's sum lies in [T_c - e_c, T_c + e_c].  Rounding to P16 and P16
 * addition are monotone, so the result lies between the two chains
 *     S_lo = RN16(S_lo + RN16(T_c - e_c)),  S_hi = RN16(S_hi + RN16(T_c + e_c))
 * over the chunks in order (both from +0).  A chunk whose exact sum is Inf or
 * NaN gives the same value on both chains.
 *
 * Chunk sums in FP32 on the vector ALUs (matrix_core = 0): the products are
 * exact in FP32 and any FP32 sum of n terms, each addition rounded (to
 * nearest, or towards zero), is within n u / (1 - n u) sum|p| of the exact
 * sum s with u = 2^-22 (Higham's recursive-summation bound with one bit of
 * slack): T_c = s, e_c = that bound.
 *
 * Chunk sums on the FP8 matrix cores (matrix_core = 1): their FP8 dot
 * product is not an FP32 sum.  Measured on gfx950 (both the 32x32x16 /
 * 16x16x32 bf8 instructions and the 32x32x64 f8f6f4 one): the products of
 * each aligned group of 8 consecutive k are added in fixed point aligned to
 * the group's largest exponent E = max(e_a + e_b) over its non-zero products
 * (e the unbiased exponent of an FP8 operand, -14 for subnormals), each
 * product truncated towards zero to a multiple of 2^(E - 13); the group sums
 * are then combined, and added into the FP32 accumulator, with errors
 * measured below 2^-17 sum|p|.  Here T_c = the sum of the truncated products
 * (exact) and e_c = (2^-16 + n 2^-26) sum|p|: twice the measured
 * combination error plus one FP32 rounding of the accumulator per 16 products
 * with fourfold slack.  e_c is rounded up to the 2^-39 grid. */
static int p8_exponent(uint8_t c) {
    const int e = (c >> 2) & 31;
    return e == 0 ? -14 : e - 15;
}

static void chunk_dot_fast_bounds(int trans_a, int trans_b, int64_t K, int64_t CL,
                                  const uint8_t* A, int64_t lda, const uint8_t* B,
                                  int64_t ldb, int matrix_core, int64_t i, int64_t j,
                                  uint16_t* lo, uint16_t* hi) {
    xnum Slo = xn_zero(0), Shi = xn_zero(0);
    for (int64_t c0 = 0; c0 < K; c0 += CL) {
        int64_t c1 = (K - c0 < CL) ? K : c0 + CL;
        xnum sum = xn_zero(0), centre = xn_zero(0);
        u128 absum = 0;
        for (int64_t g0 = c0; g0 < c1; g0 += 8) {
            const int64_t g1 = (c1 - g0 < 8) ? c1 : g0 + 8;
            int E = -1000;                       /* largest exponent sum in the group */
            for (int64_t k = g0; k < g1; k++) {
                const uint8_t a = op_a(trans_a, A, lda, i, k), b = op_b(trans_b, B, ldb, k, j);
                xnum p = xn_mul_p8(a, b);
                sum = xn_add(sum, p);
                if (p.cls == XN_FIN && p.mag != 0) {
                    absum += p.mag;
                    const int e = p8_exponent(a) + p8_exponent(b);
                    if (e > E) E = e;
                }
            }
            for (int64_t k = g0; k < g1; k++) {
                xnum p = xn_mul_p8(op_a(trans_a, A, lda, i, k), op_b(trans_b, B, ldb, k, j));
                if (matrix_core && p.cls == XN_FIN) {
                    const int sh = E - 13 + 39;  /* grid 2^(E-13) in units of 2^-39 */
                    if (sh > 0) p.mag = (p.mag >> sh) << sh;
                }
                centre = xn_add(centre, p);
            }
        }
        xnum Plo = sum, Phi = sum;
        if (sum.cls == XN_FIN) {
            const u128 n = (u128)(c1 - c0);
            u128 e;
            if (matrix_core) {
                e = (absum * (((u128)1 << 10) + n) + ((u128)1 << 26) - 1) >> 26;
            } else {
                const u128 den = ((u128)1 << 22) - n;          /* 2^22 (1 - n u) */
                e = (absum * n + den - 1) / den;
            }
            xnum d = {XN_FIN, 1, e};
            Plo = xn_add(centre, d);
            d.sign = 0;
            Phi = xn_add(centre, d);
        }
        Slo = xn_from_p16(xn_round_p16(xn_add(Slo, xn_from_p16(xn_round_p16(Plo)))));
        Shi = xn_from_p16(xn_round_p16(xn_add(Shi, xn_from_p16(xn_round_p16(Phi)))));
    }
    *lo = xn_round_p16(Slo);
    *hi = xn_round_p16(Shi);
}

int cpu_chunk_gemm_fast_bounds_points(int trans_a, int trans_b, int64_t M, int64_t N,
                                      int64_t K, int64_t CL, const uint8_t* A,
                                      int64_t lda, const uint8_t* B, int64_t ldb,
                                      int matrix_core, const int64_t* rows,
                                      const int64_t* cols, int64_t npts, uint16_t* lo,
                                      uint16_t* hi) {
    if (!gemm_args_ok(trans_a, trans_b, M, N, K, CL, A, lda, B, ldb, ORC_FAST))
        return ORC_EINVAL;
    if (CL > ((int64_t)1 << 21) && K > ((int64_t)1 << 21))
        return ORC_EINVAL;                             /* keeps n u' <= 1/2 */
    if (npts < 0 || (npts > 0 && (!rows || !cols || !lo || !hi))) return ORC_EINVAL;
    for (int64_t p = 0; p < npts; p++)
        if (rows[p] < 0 || rows[p] >= M || cols[p] < 0 || cols[p] >= N)
            return ORC_EINVAL;
    #pragma omp parallel for schedule(dynamic, 1)
    for (int64_t p = 0; p < npts; p++)
        chunk_dot_fast_bounds(trans_a, trans_b, K, CL, A, lda, B, ldb, matrix_core != 0,
                              rows[p], cols[p], &lo[p], &hi[p]);
    return ORC_OK;
}

/* ---- chunk-based accumulation with stochastic rounding -------------------
 * Sec. 2.3 names two rounding modes after P16 additions -- nearest and
 * stochastic -- and Fig. 3(b) compares them on long accumulations.  This is
 * the chunk-based dot product of Fig. 3(a) with every P16 addition rounded
 * stochastically instead of to nearest: the sum of the running value and the
 * next term is first formed in FP32 (the intermediate sum held with k' = 23
 * mantissa bits) and then rounded into P16 by Eq. (1) (orc_sr16):
 *     P = SR16(fl32(P + a(i,k) b(k,j)))   for k in the chunk, ascending
 *     S = SR16(fl32(S + P))                after each chunk
 * (products of two P8 values are exact in FP32, so fl32 is one rounding of
 * the exact sum).  CL >= K is plain sequential accumulation with stochastic
 * rounding, the SR curve of Fig. 3(b).
 * Random bits (the paper names no source): Philox4x32-10 with key = seed and
 * eight 16-bit uniforms per block (the halves of its four words, low half
 * first).  One block serves four adjacent outputs of a row for two
 * consecutive products: the addition of product k into output (i, j) uses
 * uniform 4 (k mod 2) + (j mod 4) of the block with counter
 * (i, j / 4, k / 2, 2 * offset).  The addition of chunk c into the running sum
 * of output (i, j) uses uniform j mod 8 of the block with counter
 * (i, j / 8, c, 2 * offset + 1). */
static uint32_t sr_uniform(uint32_t i, uint32_t j, uint32_t q, uint32_t w3,
                           int idx, const uint32_t key[2]) {
    const uint32_t ctr[4] = {i, j, q, w3};
    uint32_t words[4];
    orc_philox4x32_10(ctr, key, words);
    const uint32_t word = words[idx / 2];
    return (idx % 2) ? (word >> 16) : (word & 0xFFFFu);
}

static uint16_t chunk_dot_sr(int trans_a, int trans_b, int64_t K, int64_t CL,
                             const uint8_t* A, int64_t lda, const uint8_t* B,
                             int64_t ldb, uint64_t seed, uint32_t offset,
                             int64_t i, int64_t j) {
    const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint16_t S = 0;                                   /* +0 */
    int64_t c = 0;
    for (int64_t c0 = 0; c0 < K; c0 += CL, c++) {
        int64_t c1 = (K - c0 < CL) ? K : c0 + CL;
        uint16_t P = 0;
        for (int64_t k = c0; k < c1; k++) {
            float p = (float)orc_p16_value(orc_mul8(op_a(trans_a, A, lda, i, k),
                                                    op_b(trans_b, B, ldb, k, j)));
            volatile float x = (float)orc_p16_value(P) + p;      /* fl32 */
            P = orc_sr16(x, sr_uniform((uint32_t)i, (uint32_t)(j / 4), (uint32_t)(k / 2),
                                       2u * offset, (int)(4 * (k % 2) + j % 4), key));
        }
        volatile float x = (float)orc_p16_value(S) + (float)orc_p16_value(P);
        S = orc_sr16(x, sr_uniform((uint32_t)i, (uint32_t)(j / 8), (uint32_t)c,
                                   2u * offset + 1u, (int)(j % 8), key));
    }
    return S;
}

static int sr_args_ok(int64_t M, int64_t N, int64_t K, uint32_t offset) {
    return M <= ((int64_t)1 << 32) && N <= ((int64_t)1 << 32) &&
           K / 2 < ((int64_t)1 << 32) && offset < 0x80000000u;
}

int cpu_chunk_gemm_sr(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K,
                      int64_t CL, const uint8_t* A, int64_t lda,
                      const uint8_t* B, int64_t ldb, uint16_t* C, int64_t ldc,
                      uint64_t seed, uint32_t offset) {
    if (!gemm_args_ok(trans_a, trans_b, M, N, K, CL, A, lda, B, ldb, ORC_EXACT))
        return ORC_EINVAL;
    if (!sr_args_ok(M, N, K, offset)) return ORC_EINVAL;
    if (M > 0 && N > 0 && (!C || ldc < N)) return ORC_EINVAL;
    #pragma omp parallel for schedule(dynamic, 1)
    for (int64_t i = 0; i < M; i++)
        for (int64_t j = 0; j < N; j++)
            C[i * ldc + j] = chunk_dot_sr(trans_a, trans_b, K, CL, A, lda, B, ldb,
                                          seed, offset, i, j);
    return ORC_OK;
}

int cpu_chunk_gemm_sr_points(int trans_a, int trans_b, int64_t M, int64_t N,
                             int64_t K, int64_t CL, const uint8_t* A, int64_t lda,
                             const uint8_t* B, int64_t ldb, uint64_t seed,
                             uint32_t offset, const int64_t* rows,
                             const int64_t* cols, int64_t npts, uint16_t* out) {
    if (!gemm_args_ok(trans_a, trans_b, M, N, K, CL, A, lda, B, ldb, ORC_EXACT))
        return ORC_EINVAL;
    if (!sr_args_ok(M, N, K, offset)) return ORC_EINVAL;
    if (npts < 0 || (npts > 0 && (!rows || !cols || !out))) return ORC_EINVAL;
    for (int64_t p = 0; p < npts; p++)
        if (rows[p] < 0 || rows[p] >= M || cols[p] < 0 || cols[p] >= N)
            return ORC_EINVAL;
    #pragma omp parallel for schedule(dynamic, 1)
    for (int64_t p = 0; p < npts; p++)
        out[p] = chunk_dot_sr(trans_a, trans_b, K, CL, A, lda, B, ldb, seed, offset,
                              rows[p], cols[p]);
    return ORC_OK;
}

/* ---- chunk-based GEMM with P16 operands ------------------------------------
 * Sec. 3 keeps the last layer's GEMMs in FP16.  Read as Fig. 3(a) with
 * FP_mult = FP_acc = P16: each product of two P16 operands is rounded to P16
 * (nearest even; the multiplication happens in FP_mult), then the products are
 * accumulated exactly as in chunk_gemm's exact mode:
 *     P = RN16(P + RN16(a(i,k) b(k,j)))   within a chunk, ascending k
 *     S = RN16(S + P)                      after each chunk
 * The product of two P16 values (at most 20 significant bits, magnitude
 * 2^-78 .. 2^64) is exact in double precision. */
static inline uint16_t op16(int trans, const uint16_t* X, int64_t ld, int64_t r, int64_t c) {
    return trans ? X[c * ld + r] : X[r * ld + c];
}

static uint16_t chunk_dot_p16(int trans_a, int trans_b, int64_t K, int64_t CL,
                              const uint16_t* A, int64_t lda, const uint16_t* B,
                              int64_t ldb, int64_t i, int64_t j) {
    uint16_t S = 0;
    for (int64_t c0 = 0; c0 < K; c0 += CL) {
        int64_t c1 = (K - c0 < CL) ? K : c0 + CL;
        uint16_t P = 0;
        for (int64_t k = c0; k < c1; k++) {
            const double a = orc_p16_value(op16(trans_a, A, lda, i, k));
            const double b = orc_p16_value(op16(trans_b, B, ldb, k, j));
            P = orc_add16(P, orc_rn16(a * b));
        }
        S = orc_add16(S, P);
    }
    return S;
}

static int p16_args_ok(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K,
                       int64_t CL, const uint16_t* A, int64_t lda, const uint16_t* B,
                       int64_t ldb) {
    if (M < 0 || N < 0 || K < 0 || CL < 1) return 0;
    if ((trans_a != 0 && trans_a != 1) || (trans_b != 0 && trans_b != 1)) return 0;
    if (M > 0 && N > 0 && K > 0) {
        if (!A || !B) return 0;
        if (lda < (trans_a ? M : K)) return 0;
        if (ldb < (trans_b ? K : N)) return 0;
    }
    return 1;
}

int cpu_chunk_gemm_p16(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K,
                       int64_t CL, const uint16_t* A, int64_t lda,
                       const uint16_t* B, int64_t ldb, uint16_t* C, int64_t ldc) {
    if (!p16_args_ok(trans_a, trans_b, M, N, K, CL, A, lda, B, ldb)) return ORC_EINVAL;
    if (M > 0 && N > 0 && (!C || ldc < N)) return ORC_EINVAL;
    #pragma omp parallel for schedule(dynamic, 1)
    for (int64_t i = 0; i < M; i++)
        for (int64_t j = 0; j < N; j++)
            C[i * ldc + j] = chunk_dot_p16(trans_a, trans_b, K, CL, A, lda, B, ldb, i, j);
    return ORC_OK;
}

int cpu_chunk_gemm_p16_points(int trans_a, int trans_b, int64_t M, int64_t N,
                              int64_t K, int64_t CL, const uint16_t* A, int64_t lda,
                              const uint16_t* B, int64_t ldb, const int64_t* rows,
                              const int64_t* cols, int64_t npts, uint16_t* out) {
    if (!p16_args_ok(trans_a, trans_b, M, N, K, CL, A, lda, B, ldb)) return ORC_EINVAL;
    if (npts < 0 || (npts > 0 && (!rows || !cols || !out))) return ORC_EINVAL;
    for (int64_t p = 0; p < npts; p++)
        if (rows[p] < 0 || rows[p] >= M || cols[p] < 0 || cols[p] >= N)
            return ORC_EINVAL;
    #pragma omp parallel for schedule(dynamic, 1)
    for (int64_t p = 0; p < npts; p++)
        out[p] = chunk_dot_p16(trans_a, trans_b, K, CL, A, lda, B, ldb, rows[p], cols[p]);
    return ORC_OK;
}

/* ---- SGD weight update in P16 with stochastic rounding -------------------
 * Sec. 2.2 (Fig. 2(b)) and Sec. 4.3: the three AXPYs of an SGD step --
 * L2 regularisation, momentum accumulation and the weight update -- all run
 * in P16 with floating-point stochastic rounding (Eq. (1)); Sec. 3 keeps a
 * P16 master copy and an FP8 copy of the weights.  Each AXPY is one FP32
 * fused multiply-add followed by one stochastic rounding into P16:
 *     g' = SR16(wd * w + g)
 *     v' = SR16(momentum * v + g')       (skipped when v is absent)
 *     w' = SR16(-lr * v' + w)            (-lr * g' + w when v is absent)
 *     w8 = Q8(w')
 * Random bits: one Philox4x32-10 block per element pair, key = seed,
 * counter = (pair index, offset), each 32-bit word split into two 16-bit
 * uniforms (low half first); element i takes uniforms 3*(i mod 2) + 0, 1, 2
 * for the three roundings in the order above. */
int cpu_sr_weight_update(uint16_t* w, const uint16_t* g, uint16_t* v,
                         uint8_t* w8, int64_t n, float lr, float momentum,
                         float weight_decay, uint64_t seed, uint64_t offset) {
    if (n < 0) return ORC_EINVAL;
    if (n > 0 && (!w || !g)) return ORC_EINVAL;
    if (momentum != 0.0f && !v) return ORC_EINVAL;
    const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; i++) {
        uint64_t pair = (uint64_t)i >> 1;
        const uint32_t ctr[4] = {(uint32_t)pair, (uint32_t)(pair >> 32),
                                 (uint32_t)offset, (uint32_t)(offset >> 32)};
        uint32_t words[4];
        orc_philox4x32_10(ctr, key, words);
        uint32_t u[8];
        for (int q = 0; q < 4; q++) {
            u[2 * q] = words[q] & 0xFFFFu;
            u[2 * q + 1] = words[q] >> 16;
        }
        const uint32_t* h = u + 3 * (i & 1);

        float wf = (float)orc_p16_value(w[i]);
        float gf = (float)orc_p16_value(g[i]);
        uint16_t g1 = orc_sr16(fmaf(weight_decay, wf, gf), h[0]);
        float step = (float)orc_p16_value(g1);
        if (v) {
            float vf = (float)orc_p16_value(v[i]);
            uint16_t v1 = orc_sr16(fmaf(momentum, vf, step), h[1]);
            v[i] = v1;
            step = (float)orc_p16_value(v1);
        }
        uint16_t w1 = orc_sr16(fmaf(-lr, step, wf), h[2]);
        w[i] = w1;
        if (w8) w8[i] = orc_q8(orc_p16_value(w1));
    }
    return ORC_OK;
}

/* ---- ADAM weight update in P16 with stochastic rounding -------------------
 * Sec. 3 also trains with the ADAM optimizer (Kingma & Ba) using FP8 GEMMs
 * and FP16 weight updates.  Read here as the SGD update above with ADAM's
 * moment estimates: every AXPY is formed in FP32 and stochastically rounded
 * into P16 (Eq. (1)), the moments are P16 buffers like the momentum buffer.
 * For element i (all FP32 operations IEEE round-to-nearest; sqrtf and the
 * division correctly rounded):
 *     g' = SR16(fmaf(wd, w, g))
 *     m' = SR16(fmaf(beta1, m, (1 - beta1) * g'))
 *     v' = SR16(fmaf(beta2, v, (1 - beta2) * (g' * g')))
 *     w' = SR16(fmaf(-alpha_t, m' / (sqrtf(v') + eps), w))
 *     w8 = Q8(w')
 * with 1 - beta1 and 1 - beta2 single FP32 subtractions, and the
 * bias-corrected step size of Kingma & Ba's efficient form,
 *     alpha_t = lr * sqrt(1 - beta2^t) / (1 - beta1^t),
 * evaluated in double precision (beta^t by binary exponentiation of the
 * double value of beta, t >= 1) and rounded once to FP32.
 * Random bits: one Philox4x32-10 block per element pair (key = seed,
 * counter = (pair index, offset)), eight 16-bit uniforms (low half first);
 * element i takes uniforms 4 (i mod 2) + 0, 1, 2, 3 for g', m', v', w'. */
static double pow_binary(double b, uint64_t t) {
    double r = 1.0;
    while (t) {
        if (t & 1) r *= b;
        b *= b;
        t >>= 1;
    }
    return r;
}

float orc_adam_step_size(float lr, float beta1, float beta2, uint64_t t) {
    const double b1t = pow_binary((double)beta1, t), b2t = pow_binary((double)beta2, t);
    return (float)((double)lr * sqrt(1.0 - b2t) / (1.0 - b1t));
}

int cpu_adam_update(uint16_t* w, const uint16_t* g, uint16_t* m, uint16_t* v,
                    uint8_t* w8, int64_t n, float lr, float beta1, float beta2,
                    float eps, float weight_decay, uint64_t t, uint64_t seed,
                    uint64_t offset) {
    if (n < 0 || t < 1) return ORC_EINVAL;
    if (n > 0 && (!w || !g || !m || !v)) return ORC_EINVAL;
    const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    const float alpha = orc_adam_step_size(lr, beta1, beta2, t);
    const float c1 = 1.0f - beta1, c2 = 1.0f - beta2;
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; i++) {
        uint64_t pair = (uint64_t)i >> 1;
        const uint32_t ctr[4] = {(uint32_t)pair, (uint32_t)(pair >> 32),
                                 (uint32_t)offset, (uint32_t)(offset >> 32)};
        uint32_t words[4];
        orc_philox4x32_10(ctr, key, words);
        uint32_t u[8];
        for (int q = 0; q < 4; q++) {
            u[2 * q] = words[q] & 0xFFFFu;
            u[2 * q + 1] = words[q] >> 16;
        }
        const uint32_t* h = u + 4 * (i & 1);

        volatile float wf = (float)orc_p16_value(w[i]);
        volatile float gf = (float)orc_p16_value(g[i]);
        volatile float mf = (float)orc_p16_value(m[i]);
        volatile float vf = (float)orc_p16_value(v[i]);
        uint16_t g1 = orc_sr16(fmaf(weight_decay, wf, gf), h[0]);
        volatile float g1f = (float)orc_p16_value(g1);
        volatile float mg = c1 * g1f;
        uint16_t m1 = orc_sr16(fmaf(beta1, mf, mg), h[1]);
        volatile float sq = g1f * g1f;
        volatile float vg = c2 * sq;
        uint16_t v1 = orc_sr16(fmaf(beta2, vf, vg), h[2]);
        volatile float m1f = (float)orc_p16_value(m1);
        volatile float v1f = (float)orc_p16_value(v1);
        volatile float den = sqrtf(v1f) + eps;
        volatile float q = m1f / den;
        uint16_t w1 = orc_sr16(fmaf(-alpha, q, wf), h[3]);
        w[i] = w1;
        m[i] = m1;
        v[i] = v1;
        if (w8) w8[i] = orc_q8(orc_p16_value(w1));
    }
    return ORC_OK;
}

/* ---- col2im: the adjoint of the convolution lowering ----------------------
 * Sec. 2.2 computes a convolution by lowering its input and a GEMM; the
 * Backward GEMM then gives the error of the lowered matrix, and col2im adds
 * each input position's entries back together.  For the NHWC input
 * X[n, ih, iw, c] the lowered matrix has rows (n, oh, ow) and columns
 * (kh, kw, c), entry X[n, oh*stride - pad + kh, ow*stride - pad + kw, c].
 * Read here: dX[n, ih, iw, c] = the P16 sum, starting at +0, in ascending
 * (kh, kw) order with rounding to nearest after every addition, of the
 * entries that map to (n, ih, iw, c). */
int cpu_col2im(const uint16_t* cols, int64_t N, int64_t H, int64_t W, int64_t C,
               int64_t KH, int64_t KW, int64_t pad, int64_t stride, uint16_t* dX) {
    if (N < 0 || H < 1 || W < 1 || C < 1 || KH < 1 || KW < 1 || pad < 0 || stride < 1)
        return ORC_EINVAL;
    if (H + 2 * pad < KH || W + 2 * pad < KW) return ORC_EINVAL;
    const int64_t OH = (H + 2 * pad - KH) / stride + 1, OW = (W + 2 * pad - KW) / stride + 1;
    const int64_t K = KH * KW * C;
    if (N * H * W * C > 0 && (!cols || !dX)) return ORC_EINVAL;
    #pragma omp parallel for schedule(static)
    for (int64_t n = 0; n < N; n++)
        for (int64_t ih = 0; ih < H; ih++)
            for (int64_t iw = 0; iw < W; iw++)
                for (int64_t c = 0; c < C; c++) {
                    uint16_t S = 0;
                    for (int64_t kh = 0; kh < KH; kh++)
                        for (int64_t kw = 0; kw < KW; kw++) {
                            const int64_t yh = ih + pad - kh, yw = iw + pad - kw;
                            if (yh < 0 || yw < 0 || yh % stride || yw % stride) continue;
                            const int64_t oh = yh / stride, ow = yw / stride;
                            if (oh >= OH || ow >= OW) continue;
                            S = orc_add16(S, cols[((n * OH + oh) * OW + ow) * K +
                                                  (kh * KW + kw) * C + c]);
                        }
                    dX[((n * H + ih) * W + iw) * C + c] = S;
                }
    return ORC_OK;
}
