/*
 * CPU oracle for the FP8-training hot path of Wang et al., "Training Deep
 * Neural Networks with 8-bit Floating Point Numbers" (NeurIPS 2018).
 *
 * TEST INFRASTRUCTURE ONLY.  This library defines what the GPU path must
 * compute; it is plain, slow and written to be checked against the paper by
 * eye.  Only the tests, the smoke check and the benchmark's CPU-baseline leg
 * load it.  It shares no source, header, table or constant generator with the
 * HIP library, and the HIP library never calls it.
 *
 * Number formats (Sec. 2.2):
 *   P8  = the paper's FP8, (sign, exponent, mantissa) = (1, 5, 2)
 *   P16 = the paper's FP16, (1, 6, 9) -- not IEEE binary16
 * Readings where the paper is silent (bias, subnormals, specials, tie-break,
 * random source) are listed in the design doc and repeated at each function.
 *
 * All arithmetic that decides a result is exact: values are held as integers
 * in units of 2^-39 (the smallest P16 step) in 128-bit integers, and every
 * rounding is applied to the exact value.
 */
#ifndef FP8T_ORACLE_H
#define FP8T_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { ORC_OK = 0, ORC_EINVAL = -1 };
enum { ORC_SRC_F32 = 0, ORC_SRC_P16 = 1 };
enum { ORC_EXACT = 0, ORC_FAST = 1 };

/* ---- formats (Sec. 2.2) ------------------------------------------------ */
double   orc_p8_value(uint8_t code);     /* exact value of a P8 code        */
double   orc_p16_value(uint16_t code);   /* exact value of a P16 code       */
uint8_t  orc_q8(double x);               /* round-to-nearest-even into P8    */
uint16_t orc_rn16(double x);             /* round-to-nearest-even into P16   */

/* ---- arithmetic primitives (Sec. 2.3) ---------------------------------- */
uint16_t orc_add16(uint16_t x, uint16_t y);     /* RN16(x + y), exact sum    */
uint16_t orc_mul8(uint8_t a, uint8_t b);        /* exact P8 x P8 product     */
uint16_t orc_sr16(float x, uint32_t u16);       /* Eq. (1), k = 9, k' = 23   */

/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11). */
void orc_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2],
                       uint32_t out[4]);

/* ---- the three entry points of the hot path ---------------------------- */
int cpu_fp8_quantize(const void* src, int src_format, float scale,
                     uint8_t* dst, int64_t n);

/* FP32 -> P16, round to nearest even (creates P16 master copies). */
int cpu_fp16_quantize(const float* src, uint16_t* dst, int64_t n);

int cpu_chunk_gemm(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K,
                   int64_t CL, const uint8_t* A, int64_t lda,
                   const uint8_t* B, int64_t ldb, uint16_t* C, int64_t ldc,
                   int mode);

/* Same as cpu_chunk_gemm, but only for the npts outputs (rows[p], cols[p]);
 * out[p] receives C(rows[p], cols[p]). */
int cpu_chunk_gemm_points(int trans_a, int trans_b, int64_t M, int64_t N,
                          int64_t K, int64_t CL, const uint8_t* A, int64_t lda,
                          const uint8_t* B, int64_t ldb, int mode,
                          const int64_t* rows, const int64_t* cols,
                          int64_t npts, uint16_t* out);

/* Bounds on what the fast mode may give at the outputs (rows[p], cols[p]),
 * defined in ops.c: chunk sums in FP32 on the vector ALUs (matrix_core = 0)
 * or on the FP8 matrix cores with their measured group truncation
 * (matrix_core = 1); lo[p] and hi[p] are the two monotone FP16 chains.
 * Requires min(CL, K) <= 2^21. */
int cpu_chunk_gemm_fast_bounds_points(int trans_a, int trans_b, int64_t M, int64_t N,
                                      int64_t K, int64_t CL, const uint8_t* A,
                                      int64_t lda, const uint8_t* B, int64_t ldb,
                                      int matrix_core, const int64_t* rows,
                                      const int64_t* cols, int64_t npts, uint16_t* lo,
                                      uint16_t* hi);

/* chunk_gemm with stochastic instead of nearest rounding after every P16
 * addition (Sec. 2.3, Fig. 3(b)); random bits keyed by (seed, i, j, k) as
 * described in ops.c.  Requires M, N <= 2^32, K / 2 < 2^32, offset < 2^31. */
int cpu_chunk_gemm_sr(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K,
                      int64_t CL, const uint8_t* A, int64_t lda,
                      const uint8_t* B, int64_t ldb, uint16_t* C, int64_t ldc,
                      uint64_t seed, uint32_t offset);
int cpu_chunk_gemm_sr_points(int trans_a, int trans_b, int64_t M, int64_t N,
                             int64_t K, int64_t CL, const uint8_t* A, int64_t lda,
                             const uint8_t* B, int64_t ldb, uint64_t seed,
                             uint32_t offset, const int64_t* rows,
                             const int64_t* cols, int64_t npts, uint16_t* out);

/* chunk_gemm with P16 operands (the last layer's GEMMs, Sec. 3): products
 * rounded to P16, then exact-mode chunked accumulation (ops.c). */
int cpu_chunk_gemm_p16(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K,
                       int64_t CL, const uint16_t* A, int64_t lda,
                       const uint16_t* B, int64_t ldb, uint16_t* C, int64_t ldc);
int cpu_chunk_gemm_p16_points(int trans_a, int trans_b, int64_t M, int64_t N,
                              int64_t K, int64_t CL, const uint16_t* A, int64_t lda,
                              const uint16_t* B, int64_t ldb, const int64_t* rows,
                              const int64_t* cols, int64_t npts, uint16_t* out);

int cpu_sr_weight_update(uint16_t* w, const uint16_t* g, uint16_t* v,
                         uint8_t* w8, int64_t n, float lr, float momentum,
                         float weight_decay, uint64_t seed, uint64_t offset);

/* ADAM step in P16 with stochastic rounding (Sec. 3, Kingma & Ba), defined
 * in ops.c; m and v are the P16 moment buffers, updated in place; t >= 1 is
 * the step number.  orc_adam_step_size is its bias-corrected step size. */
int cpu_adam_update(uint16_t* w, const uint16_t* g, uint16_t* m, uint16_t* v,
                    uint8_t* w8, int64_t n, float lr, float beta1, float beta2,
                    float eps, float weight_decay, uint64_t t, uint64_t seed,
                    uint64_t offset);
float orc_adam_step_size(float lr, float beta1, float beta2, uint64_t t);

/* col2im of P16 codes (ops.c): the adjoint of the lowering of an NHWC
 * convolution input, summed in P16 in ascending (kh, kw) order. */
int cpu_col2im(const uint16_t* cols, int64_t N, int64_t H, int64_t W, int64_t C,
               int64_t KH, int64_t KW, int64_t pad, int64_t stride, uint16_t* dX);

/* Number of OpenMP threads the oracle's parallel loops use. */
int orc_num_threads(void);
void orc_set_threads(int n);

#ifdef __cplusplus
}
#endif
#endif
