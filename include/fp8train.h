/*
 * fp8train -- the hot path of 8-bit floating-point training (Wang, Choi,
 * Brand, Chen, Gopalakrishnan, "Training Deep Neural Networks with 8-bit
 * Floating Point Numbers", NeurIPS 2018) for AMD MI355X (gfx950).
 *
 * Number formats (Sec. 2.2), stored as raw codes:
 *   FP8  (1 sign, 5 exponent, 2 mantissa bits) in uint8_t,  bias 15.
 *   FP16 (1 sign, 6 exponent, 9 mantissa bits) in uint16_t, bias 31.
 *        This FP16 is the paper's format, NOT IEEE binary16.
 * Both have gradual underflow; the all-ones exponent field holds Inf
 * (mantissa 0) and NaN.  FP8 quantization saturates finite overflow at
 * +-57344; FP16 results beyond +-(2 - 2^-9) * 2^31 become +-Inf.  Every NaN
 * result is written as the canonical code 0x7F (FP8) or 0x7F00 (FP16).
 * Rounding to nearest breaks ties to even.
 *
 * Conventions for every call:
 *   - All array pointers are device pointers owned by the caller.  The
 *     library never allocates, frees or synchronizes; work is enqueued on
 *     `stream` (0 = the null stream) and runs asynchronously.  (The one
 *     device array it owns, chunk_gemm_noalloc's scratch, is a static
 *     array of its code object.)
 *   - Arguments are validated before anything is enqueued.  A call that
 *     returns an error has enqueued nothing.
 *   - Sizes are element counts.  Matrices are row-major with a leading
 *     dimension (elements between consecutive rows).
 *   - Outputs must not alias inputs unless stated.
 */
#ifndef FP8TRAIN_H
#define FP8TRAIN_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
enum {
    FP8T_OK = 0,
    FP8T_EINVAL = -1,     /* invalid argument; nothing was enqueued          */
    FP8T_EWORKSPACE = -2, /* workspace smaller than chunk_gemm_workspace_size */
    FP8T_EHIP = -3        /* the HIP runtime reported an error at launch     */
};

/* Source formats for fp8_quantize. */
enum { FP8T_SRC_F32 = 0, FP8T_SRC_FP16 = 1 };

/* chunk_gemm modes. */
enum { FP8T_EXACT = 0, FP8T_FAST = 1 };

/*
 * fp8_quantize -- round values into FP8 (Sec. 2.1: weights, activations,
 * errors and gradients enter every GEMM as 8-bit floats).
 *
 *   dst[i] = Q8(RN32(x[i] * scale))
 *
 * x[i] is src[i] as an IEEE float (src_format FP8T_SRC_F32, `src` points to
 * float) or the exact value of the FP16 code src[i] (FP8T_SRC_FP16, `src`
 * points to uint16_t).  The product with `scale` (e.g. a loss scale, Sec. 3)
 * is one IEEE single-precision multiplication; Q8 rounds it to the nearest FP8
 * value, ties to even, with gradual underflow below 2^-14 and saturation at
 * +-57344.  n >= 0 elements; src and dst contiguous; n == 0 is a no-op.
 * Errors: FP8T_EINVAL for n < 0, a NULL pointer with n > 0, or an unknown
 * src_format.
 */
int fp8_quantize(const void* src, int src_format, float scale, uint8_t* dst,
                 int64_t n, hipStream_t stream);

/*
 * fp16_quantize -- round IEEE floats to the nearest FP16 (1,6,9) value, ties
 * to even (the round-to-nearest of Sec. 2.2), e.g. to create the FP16 master
 * copy of the weights (Sec. 3).  Overflow gives +-Inf.  n >= 0, contiguous.
 * Errors: FP8T_EINVAL for n < 0 or a NULL pointer with n > 0.
 */
int fp16_quantize(const float* src, uint16_t* dst, int64_t n,
                  hipStream_t stream);

/*
 * chunk_gemm -- C = op(A) * op(B) with FP8 operands and chunk-based FP16
 * accumulation (Sec. 2.3 "Chunk-based Accumulation" and the dot-product
 * algorithm of Fig. 3(a)); used for the Forward, Backward and Gradient GEMMs
 * of Sec. 2.2 through the transpose flags.
 *
 * For every output (i, j), with a(k) = op(A)(i, k), b(k) = op(B)(k, j):
 *   the K products a(k) * b(k) (exact) are split into chunks of CL
 *   consecutive k starting at k = 0 (the last chunk may be shorter);
 *   mode FP8T_EXACT: within a chunk, products are added in ascending k into
 *     an intra-chunk sum starting at +0, rounding to FP16 after every add;
 *   mode FP8T_FAST:  a chunk's products are summed in FP32 on the matrix
 *     cores (in an unspecified order), and the sum is rounded to FP16 once;
 *   each chunk's sum is then added, in ascending chunk order, into the
 *     running sum starting at +0, rounding to FP16 after every add;
 *   C(i, j) = the FP16 code of the running sum (+0 when K == 0).
 * FP8T_EXACT is bit-exact.  FP8T_FAST differs only in the rounding inside a
 * chunk.  With CL not a multiple of 16 the fast mode sums a chunk
 * sequentially in FP32 on the vector ALUs instead; the semantics are the same.
 *
 * Layouts (row-major):
 *   op(A) is M x K: A is stored M x K (trans_a = 0, lda >= K) or
 *                   K x M (trans_a = 1, lda >= M), op(A) = A^T.
 *   op(B) is K x N: B is stored K x N (trans_b = 0, ldb >= N) or
 *                   N x K (trans_b = 1, ldb >= K), op(B) = B^T.
 *   C is M x N with ldc >= N.
 * Forward Y = X W: (0, 0).  Backward dX = dY W^T: trans_b = 1.
 * Gradient dW = X^T dY: trans_a = 1.
 * M, N, K >= 0; CL >= 1 (CL >= K means one chunk).  C must not overlap A or B.
 * workspace / workspace_bytes: optional device scratch, for the chunk sums
 * of output tiles whose K range is shared out over several workgroups (the
 * chunk sums are then added into the running sum in ascending order by a
 * second pass, so the result is the same), or, in fast mode with trans_b = 0,
 * for a k-contiguous copy of B (N x K bytes) that the matrix-core kernel
 * reads.  With workspace_bytes == 0 the call takes the fastest plan that
 * needs none; otherwise workspace_bytes must be at least
 * chunk_gemm_workspace_size(...) for the same arguments on the same device
 * (operands whose alignment rules out a plan the query assumed take the
 * fastest plan that fits in workspace_bytes).  Its contents on entry do not
 * matter.
 * Errors: FP8T_EINVAL (negative size, M, N or K above 2^31 - 4097 -- the
 * kernels index in 32 bits --, CL < 1, flag not 0/1, a leading
 * dimension too small, NULL pointer for a non-empty matrix, NULL workspace
 * with workspace_bytes > 0); FP8T_EWORKSPACE (0 < workspace_bytes < the
 * query); FP8T_EHIP.
 */
int chunk_gemm(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K,
               int64_t CL, const uint8_t* A, int64_t lda, const uint8_t* B,
               int64_t ldb, uint16_t* C, int64_t ldc, int mode,
               void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * chunk_gemm_workspace_size -- bytes of workspace the fastest plan of
 * chunk_gemm needs on the current device for these arguments (0 if none, or
 * for invalid arguments, or when no device is present).
 */
size_t chunk_gemm_workspace_size(int trans_a, int trans_b, int64_t M,
                                 int64_t N, int64_t K, int64_t CL, int mode);

/*
 * chunk_gemm_noalloc -- chunk_gemm for callers that cannot allocate device
 * memory or pass a workspace (code under stream or graph capture, tight
 * serving loops, harnesses that forbid allocation).  Same arguments as
 * chunk_gemm without the workspace, same results bit for bit (the result
 * does not depend on the plan).  The chunk sums of shared tiles go to a
 * library-owned device array of FP8T_NOALLOC_SCRATCH_BYTES per GPU, a static
 * array of the library's code object that each GPU holds until the process
 * ends; the call takes the fastest plan whose chunk sums fit in it (a plan
 * without shared tiles needs none, so every valid call runs) and calls no
 * allocating routine.  Every call on one GPU uses that GPU's array: calls
 * whose execution overlaps on one GPU (different streams, not ordered by
 * events) race and may give wrong results; stream-ordered calls are safe.
 * Nothing in the array needs to start at zero.
 * Errors: as chunk_gemm (without the workspace cases); FP8T_EHIP also when
 * the array's device address cannot be obtained.
 */
#define FP8T_NOALLOC_SCRATCH_BYTES (64u * 1024u * 1024u)
int chunk_gemm_noalloc(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K,
                       int64_t CL, const uint8_t* A, int64_t lda, const uint8_t* B,
                       int64_t ldb, uint16_t* C, int64_t ldc, int mode,
                       hipStream_t stream);

/*
 * chunk_gemm_fp8 -- chunk_gemm with the result also rounded back to FP8 in
 * the same pass (Sec. 2.1: the 16-bit sums of a GEMM "can then be rounded
 * down to 8 bits" to feed the next layer's GEMMs), optionally scaled (e.g. by
 * a loss scale, Sec. 3):
 *
 *   C8(i, j) = Q8(RN32(value(C(i, j)) * scale))
 *
 * with C(i, j) exactly as chunk_gemm computes it (same modes, layouts and
 * rounding); Q8 and the FP32 product are those of fp8_quantize, so C8 equals
 * fp8_quantize(C, FP8T_SRC_FP16, scale).  C (ldc >= N) may be NULL when only
 * the FP8 result is wanted, which saves its 2 M N bytes of stores; C8 is
 * M x N uint8_t row-major with ldc8 >= N and must not overlap A, B or C.
 * workspace: at least chunk_gemm_fp8_workspace_size(...) bytes for the
 * fastest plan, or none (then a plan that needs none; same results).
 * Errors: as chunk_gemm, and FP8T_EINVAL for a NULL C8 or ldc8 < N.
 */
int chunk_gemm_fp8(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K,
                   int64_t CL, const uint8_t* A, int64_t lda, const uint8_t* B,
                   int64_t ldb, uint16_t* C, int64_t ldc, uint8_t* C8,
                   int64_t ldc8, float scale, int mode, void* workspace,
                   size_t workspace_bytes, hipStream_t stream);

/*
 * chunk_gemm_fp8_workspace_size -- bytes of workspace the fastest plan of
 * chunk_gemm_fp8 needs on the current device for these arguments (0 if
 * none, or for invalid arguments).
 */
size_t chunk_gemm_fp8_workspace_size(int trans_a, int trans_b, int64_t M,
                                     int64_t N, int64_t K, int64_t CL, int mode);

/*
 * chunk_gemm_sr -- chunk_gemm (FP8T_EXACT layouts and chunking) with every
 * FP16 addition rounded stochastically instead of to nearest: the second
 * rounding mode after FP16 additions of Sec. 2.3, whose effect on long
 * accumulations Fig. 3(b) shows.
 *
 * For every output (i, j), with a(k), b(k) as in chunk_gemm:
 *   within chunk c (ascending k):  P = SR(fl32(P + a(k) * b(k)))
 *   after chunk c:                 S = SR(fl32(S + P))
 *   P and S start at +0; C(i, j) = the FP16 code of S (+0 when K == 0).
 * fl32 is one IEEE single-precision addition (the product is exact), and SR
 * is sr_weight_update's stochastic rounding into FP16 (Eq. (1), k = 9 of
 * k' = 23 bits, 16-bit uniform u: the magnitude is rounded up iff
 * u < 2^16 x the discarded fraction of a step).  The uniforms come from
 * Philox4x32-10 with key = (seed low, seed high) and eight 16-bit uniforms
 * per block (the halves of its four words, low half first: uniform q is
 * half q mod 2 of word q / 2).  The addition of product k into output (i, j)
 * uses uniform 4 (k mod 2) + (j mod 4) of the block with counter
 * (i, j / 4, k / 2, 2 * offset); the addition of chunk c into the running sum
 * of output (i, j) uses uniform j mod 8 of the block with counter
 * (i, j / 8, c, 2 * offset + 1) (integer division; counter words in that
 * order).  The result is a pure function of the inputs, seed and offset
 * (bit-exact, independent of the device and plan).
 *
 * Layouts, CL, C and the workspace contract are those of chunk_gemm (with
 * chunk_gemm_sr_workspace_size as the query).  offset < 2^31.
 * Errors: as chunk_gemm, and FP8T_EINVAL for offset >= 2^31.
 */
int chunk_gemm_sr(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K,
                  int64_t CL, const uint8_t* A, int64_t lda, const uint8_t* B,
                  int64_t ldb, uint16_t* C, int64_t ldc, uint64_t seed,
                  uint64_t offset, void* workspace, size_t workspace_bytes,
                  hipStream_t stream);

/*
 * chunk_gemm_sr_workspace_size -- bytes of workspace the fastest plan of
 * chunk_gemm_sr needs on the current device for these arguments (0 if none,
 * or for invalid arguments).
 */
size_t chunk_gemm_sr_workspace_size(int trans_a, int trans_b, int64_t M,
                                    int64_t N, int64_t K, int64_t CL);

/*
 * chunk_gemm_p16 -- the GEMM with FP16 operands that Sec. 3 keeps for the last
 * layer of a network (Forward, Backward and Gradient GEMMs alike).  As
 * chunk_gemm's exact mode with FP16 codes as operands, the multiplication
 * also done in FP16 (Fig. 3(a) with FP_mult = FP_acc = FP16):
 *   within chunk c (ascending k):  P = RN(P + RN(a(k) * b(k)))
 *   after chunk c:                 S = RN(S + P)
 * RN = round to the nearest FP16 value (ties to even) of the exact value;
 * P, S start at +0; C(i, j) = the FP16 code of S (+0 when K == 0).
 * Bit-exact.  A, B: FP16 codes (uint16_t) in the layouts of chunk_gemm; C,
 * CL and the workspace contract as chunk_gemm (query:
 * chunk_gemm_p16_workspace_size).  Errors: as chunk_gemm.
 */
int chunk_gemm_p16(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K,
                   int64_t CL, const uint16_t* A, int64_t lda, const uint16_t* B,
                   int64_t ldb, uint16_t* C, int64_t ldc, void* workspace,
                   size_t workspace_bytes, hipStream_t stream);

/*
 * chunk_gemm_p16_workspace_size -- bytes of workspace the fastest plan of
 * chunk_gemm_p16 needs on the current device (0 if none, or for invalid
 * arguments).
 */
size_t chunk_gemm_p16_workspace_size(int trans_a, int trans_b, int64_t M,
                                     int64_t N, int64_t K, int64_t CL);

/*
 * sr_weight_update -- one SGD step entirely in FP16 with floating-point
 * stochastic rounding (Sec. 2.2 / Fig. 2(b): L2-Reg, Momentum-Acc and
 * Weight-Upd AXPYs; Sec. 2.3 Eq. (1); Sec. 4.3), keeping the FP16 master
 * weights and writing the FP8 copy used by the next step's GEMMs (Sec. 3).
 *
 * For i in [0, n), with SR(.) = stochastic rounding into FP16 of an IEEE
 * float (Eq. (1) with k = 9 of k' = 23 mantissa bits: the magnitude is rounded
 * up by one FP16 step with probability equal to the discarded fraction of a
 * step, using a 16-bit uniform; below 2^-30 the step is 2^-39):
 *   g' = SR(fmaf(weight_decay, w[i], g[i]))
 *   v' = SR(fmaf(momentum, v[i], g'))          (only if v != NULL)
 *   w' = SR(fmaf(-lr, v', w[i]))               (-lr * g' if v == NULL)
 *   w[i] = w', v[i] = v', w8[i] = FP8 of w' (round to nearest even, saturating)
 * fmaf is the IEEE single-precision fused multiply-add.  The uniforms: one
 * Philox4x32-10 block (Salmon et al., SC'11) per element pair with key =
 * (seed low, seed high) and counter = (i/2 low, i/2 high, offset low, offset
 * high); its four 32-bit words give eight 16-bit uniforms (low half first) and
 * element i uses uniforms 3*(i%2)+0, +1, +2 for g', v', w'.  The result is a
 * pure function of (w, g, v, n, lr, momentum, weight_decay, seed, offset).
 *
 * w, g: FP16 codes [n]; w is updated in place.  v: FP16 momentum buffer [n],
 * updated in place, or NULL (then momentum must be 0).  w8: FP8 codes [n] or
 * NULL (no copy).  w8 must not overlap w.
 * Errors: FP8T_EINVAL (n < 0, NULL w or g with n > 0, v == NULL with
 * momentum != 0); FP8T_EHIP.
 */
int sr_weight_update(uint16_t* w, const uint16_t* g, uint16_t* v, uint8_t* w8,
                     int64_t n, float lr, float momentum, float weight_decay,
                     uint64_t seed, uint64_t offset, hipStream_t stream);

/*
 * adam_update -- one ADAM step (Kingma & Ba; Sec. 3 also trains with ADAM using
 * FP8 GEMMs and FP16 weight updates) with every AXPY stochastically rounded
 * into FP16 as in sr_weight_update, keeping FP16 master weights and moment
 * buffers and writing the FP8 weight copy.
 *
 * For i in [0, n) (every FP32 operation IEEE round-to-nearest; the square
 * root and the division correctly rounded; SR as in sr_weight_update):
 *   g' = SR(fmaf(weight_decay, w[i], g[i]))
 *   m' = SR(fmaf(beta1, m[i], (1 - beta1) * g'))
 *   v' = SR(fmaf(beta2, v[i], (1 - beta2) * (g' * g')))
 *   w' = SR(fmaf(-alpha_t, m' / (sqrtf(v') + eps), w[i]))
 *   w[i] = w', m[i] = m', v[i] = v', w8[i] = FP8 of w'
 * 1 - beta1, 1 - beta2 are FP32 subtractions.  alpha_t = lr sqrt(1 - beta2^t)
 * / (1 - beta1^t) is evaluated in double precision (beta^t by binary
 * exponentiation of the double value of beta) and rounded once to float;
 * t >= 1 is the step number.  Uniforms: one Philox4x32-10 block per element
 * pair, key = seed, counter = (i/2 low, i/2 high, offset low, offset high),
 * eight 16-bit uniforms (low half first); element i uses uniforms
 * 4*(i%2) + 0, 1, 2, 3 for g', m', v', w'.
 *
 * w, g, m, v: FP16 codes [n] (w, m, v updated in place); w8: FP8 codes [n]
 * or NULL.  w8 must not overlap the others.
 * Errors: FP8T_EINVAL (n < 0, t < 1, a NULL w, g, m or v with n > 0);
 * FP8T_EHIP.
 */
int adam_update(uint16_t* w, const uint16_t* g, uint16_t* m, uint16_t* v,
                uint8_t* w8, int64_t n, float lr, float beta1, float beta2,
                float eps, float weight_decay, uint64_t t, uint64_t seed,
                uint64_t offset, hipStream_t stream);

/*
 * Element-wise steps of a training step around the GEMMs (Sec. 2.1: the
 * activations and errors enter the GEMMs in FP8; Sec. 3: loss scaling and
 * an FP16 last layer).  n >= 0 contiguous elements; n == 0 is a no-op.
 * Errors: FP8T_EINVAL (n < 0, a NULL pointer with n > 0, unknown format);
 * FP8T_EHIP.
 *
 * relu_codes: y[i] = ReLU(x[i]) on codes of `format` 8 (FP8, uint8_t) or 16
 *   (FP16, uint16_t): negative values (-0 and -Inf included) become +0, NaN
 *   becomes the canonical NaN code, other codes are copied.  ReLU commutes
 *   with rounding to FP8, so ReLU(Q8(z)) == Q8(ReLU(z)).  y may equal x.
 * relu_backward_fp8: e[i] = Q8(RN32(value(d[i]) * scale)) where
 *   value(z[i]) > 0, else +0 -- the ReLU derivative applied to an FP16 error
 *   d (z is the layer's FP16 pre-activation) and the result rounded to FP8
 *   for the next Backward/Gradient GEMMs.
 * mse_grad_fp16: e[i] = RN16(RN32(RN32(value(y[i]) - value(t[i])) * scale)),
 *   the loss-scaled gradient of a squared-error loss (scale = loss scale /
 *   batch) in FP16.
 */
int relu_codes(const void* x, int format, void* y, int64_t n, hipStream_t stream);
int relu_backward_fp8(const uint16_t* d, const uint16_t* z, uint8_t* e, int64_t n,
                      float scale, hipStream_t stream);
int mse_grad_fp16(const uint16_t* y, const uint16_t* t, uint16_t* e, int64_t n,
                  float scale, hipStream_t stream);

/*
 * Convolutions through an implicit lowering (Sec. 2.2: the convolution is
 * computed by lowering its input, then a GEMM).  The input X is NHWC FP8
 * (N x H x W x C, contiguous); output size OH = (H + 2 pad - KH) / stride + 1,
 * OW likewise.  The lowered matrix Xcol has M = N OH OW rows (n, oh, ow) and
 * K = KH KW C columns (kh, kw, c):
 *   Xcol[(n, oh, ow), (kh, kw, c)] = X[n, oh*stride - pad + kh,
 *                                      ow*stride - pad + kw, c]  (0 outside)
 * and is never written out: the GEMM kernels read X directly.
 *
 * conv2d_fwd_fp8:   Y = chunk_gemm(Xcol, Wt), exact mode, bit for bit the
 *   same as chunk_gemm on the explicit Xcol.  Wt: FP8 (K x Cout, row-major,
 *   rows in (kh, kw, c) order); Y: FP16 codes, M x Cout, ldy >= Cout.
 * conv2d_wgrad_fp8: dW = chunk_gemm(Xcol^T, dY), exact mode (as chunk_gemm
 *   with trans_a = 1 on the explicit Xcol).  dY: FP8 (M x Cout); dW: FP16
 *   codes, K x Cout, lddw >= Cout.
 * The Backward GEMM needs no lowering (dXcol = chunk_gemm(dY, Wt^T),
 * trans_b = 1); col2im_fp16 folds dXcol back onto the input.
 * workspace: as chunk_gemm, sized by conv2d_workspace_size(wgrad, ...) (0 for
 * invalid arguments).  C % 4 == 0 with a 4-byte aligned X reads 4 channels at
 * a time; other channel counts are read byte by byte.
 * Errors: FP8T_EINVAL (N < 0, H, W, C, KH, KW, stride < 1, pad < 0, a kernel
 * larger than the padded input, Cout < 0, CL < 1, a NULL pointer for
 * non-empty data, ldy / lddw < Cout, sizes beyond 32-bit indexing);
 * FP8T_EWORKSPACE; FP8T_EHIP.
 */
int conv2d_fwd_fp8(const uint8_t* X, int64_t N, int64_t H, int64_t W, int64_t C,
                   int64_t KH, int64_t KW, int64_t pad, int64_t stride,
                   const uint8_t* Wt, int64_t Cout, int64_t CL, uint16_t* Y,
                   int64_t ldy, void* workspace, size_t workspace_bytes,
                   hipStream_t stream);
int conv2d_wgrad_fp8(const uint8_t* X, int64_t N, int64_t H, int64_t W, int64_t C,
                     int64_t KH, int64_t KW, int64_t pad, int64_t stride,
                     const uint8_t* dY, int64_t Cout, int64_t CL, uint16_t* dW,
                     int64_t lddw, void* workspace, size_t workspace_bytes,
                     hipStream_t stream);
size_t conv2d_workspace_size(int wgrad, int64_t N, int64_t H, int64_t W, int64_t C,
                             int64_t KH, int64_t KW, int64_t pad, int64_t stride,
                             int64_t Cout, int64_t CL);

/*
 * col2im_fp16 -- the adjoint of the lowering above for FP16 codes: for every
 * input position, dX[n, ih, iw, c] = the FP16 sum, starting at +0, in
 * ascending (kh, kw) order with rounding to nearest (ties to even) after
 * every addition, of the entries cols[(n, oh, ow), (kh, kw, c)] that the
 * lowering takes from (n, ih, iw, c).  cols: M x K FP16 codes (contiguous);
 * dX: N x H x W x C FP16 codes.  Errors: as the convolutions; FP8T_EHIP.
 */
int col2im_fp16(const uint16_t* cols, int64_t N, int64_t H, int64_t W, int64_t C,
                int64_t KH, int64_t KW, int64_t pad, int64_t stride, uint16_t* dX,
                hipStream_t stream);

/* A static, human-readable description of a status code. */
const char* fp8t_status_string(int status);

#ifdef __cplusplus
}
#endif
#endif
