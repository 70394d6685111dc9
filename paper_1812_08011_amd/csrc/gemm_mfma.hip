// chunk_gemm fast mode on the matrix cores.
//
// The fast mode (a build variant, not in the paper) sums each chunk's CL
// products in FP32 on the matrix cores, in an unspecified order, rounds that
// chunk sum to FP16 once, and then adds the chunk sums into the running sum
// in ascending order with FP16 rounding after every add -- the inter-chunk
// half of Sec. 2.3's chunk-based accumulation is exactly the paper's.
//
// FP8 bytes are the OCP E5M2 ("bf8") encoding (bias 15, gradual underflow,
// exponent 31 for Inf/NaN), so the codes feed the bf8 MFMA instructions
// directly.  A workgroup is 4 waves in a 2 x 2 grid; each wave owns FM x FN
// blocks of BW x BW outputs:
//   BW = 32: v_mfma_f32_32x32x16_bf8_bf8 (16 products per instruction);
//   BW = 16: v_mfma_f32_16x16x32_bf8_bf8 (32 products per instruction).
// A chunk is accumulated from zero on the matrix cores; at its end the VALU
// epilogue rounds it and adds it into S.  The epilogue dominates (at CL = 64
// the matrix cores finish a chunk several times faster than the VALU rounds
// it), so two epilogues exist, as in the exact mode:
//   * guarded: plain values, Veltkamp rounding (rn16v), 9 full-rate VALU ops
//     per output per chunk including a running max of |p| and |S|; a piece in
//     which any value reached 2^32 (where FP16 would overflow to Inf) is
//     recomputed with
//   * safe: values scaled by 2^96 so FP16 overflow is FP32 overflow, integer
//     rounding on the raw bits (rn16s).
// NaN chunk sums propagate identically on both paths, so the two give the
// same bits.  Operand slabs of 64 k are staged through LDS k-contiguous (a
// 4 x 4 byte transpose in registers for operands stored with the row index
// contiguous), double-buffered in LDS, with several slabs in flight from HBM
// in registers.  Work is shared out over a persistent grid by the
// plan of gemm_plan.h.
#include "fp8t_device.h"
#include "gemm_mfma.h"

namespace fp8t {
namespace {

typedef float v16f __attribute__((ext_vector_type(16)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kNT = 256;            // threads per workgroup

// The 4 bytes (r, c .. c+3) of a row-major byte matrix with `rows` x `cols`
// valid elements and leading dimension ld; bytes outside are 0.
__device__ __forceinline__ uint32_t load4(const uint8_t* __restrict__ p, int64_t ld, int r,
                                          int c, int rows, int cols, int vec) {
    if (r >= rows) return 0u;
    const uint8_t* row = p + (int64_t)r * ld;
    if (vec && c + 3 < cols) return *reinterpret_cast<const uint32_t*>(row + c);
    uint32_t v = 0;
#pragma unroll
    for (int b = 0; b < 4; ++b)
        if (c + b < cols) v |= (uint32_t)row[c + b] << (8 * b);
    return v;
}

// 4 x 4 byte transpose: out[i] byte j = in[j] byte i.
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

// One operand slab: R rows (m or n) x kBK k, written k-contiguous into LDS.
// KC: k is contiguous in memory (element (r, k) at p[r * ld + k]) -- R x 16
// words; otherwise the row index is (element at p[k * ld + r]) -- (R/4) x 16
// blocks of 4 x 4 bytes, transposed in registers.
template <bool KC, int R, int kBK>
struct Slab {
    static constexpr int kPitch = kBK + 8;     // bytes per LDS row (k-contiguous)
    static constexpr int U = KC ? R * (kBK / 4) : (R / 4) * (kBK / 4);
    static constexpr int PER = (U + kNT - 1) / kNT;
    static constexpr int NW = KC ? PER : 4 * PER;
    uint32_t r[NW];

    __device__ __forceinline__ void load(const uint8_t* __restrict__ p, int64_t ld, int row0,
                                         int k0, int rows, int kend, int vec, int tid) {
#pragma unroll
        for (int q = 0; q < PER; ++q) {
            const int u = tid + kNT * q;
            if (U % kNT != 0 && u >= U) continue;
            if (KC) {
                const int rr = u / (kBK / 4), kq = (u % (kBK / 4)) * 4;
                r[q] = load4(p, ld, row0 + rr, k0 + kq, rows, kend, vec);
            } else {
                const int rg = u % (R / 4), kg = u / (R / 4);
#pragma unroll
                for (int b = 0; b < 4; ++b)
                    r[q * 4 + b] = load4(p, ld, k0 + kg * 4 + b, row0 + rg * 4, kend, rows, vec);
            }
        }
    }

    // The same when the whole slab lies inside the matrix and 4-byte loads
    // are aligned: no bounds checks, and the addresses are one uniform base
    // (the slab's first byte) plus per-thread 32-bit offsets fixed for the
    // whole kernel, so the loads take the scalar-base form with no per-slab
    // address arithmetic.
    __device__ __forceinline__ static void offsets(int64_t ld, int tid, uint32_t (&o)[NW]) {
#pragma unroll
        for (int q = 0; q < PER; ++q) {
            const int u = min(tid + kNT * q, U - 1);
            if (KC) {
                const int rr = u / (kBK / 4), kq = (u % (kBK / 4)) * 4;
                o[q] = (uint32_t)(rr * ld + kq);
            } else {
                const int rg = u % (R / 4), kg = u / (R / 4);
#pragma unroll
                for (int b = 0; b < 4; ++b) o[q * 4 + b] = (uint32_t)((kg * 4 + b) * ld + rg * 4);
            }
        }
    }
    __device__ __forceinline__ void load_fast(const uint8_t* __restrict__ base, const uint32_t (&o)[NW],
                                              int tid) {
#pragma unroll
        for (int q = 0; q < PER; ++q) {
            const int u = tid + kNT * q;
            if (U % kNT != 0 && u >= U) continue;
#pragma unroll
            for (int b = 0; b < (KC ? 1 : 4); ++b)
                r[q * (KC ? 1 : 4) + b] = *reinterpret_cast<const uint32_t*>(base + o[q * (KC ? 1 : 4) + b]);
        }
    }

    __device__ __forceinline__ void store(uint8_t (*lds)[kPitch], int tid) {
#pragma unroll
        for (int q = 0; q < PER; ++q) {
            const int u = tid + kNT * q;
            if (U % kNT != 0 && u >= U) continue;
            if (KC) {
                const int rr = u / (kBK / 4), kq = (u % (kBK / 4)) * 4;
                *reinterpret_cast<uint32_t*>(&lds[rr][kq]) = r[q];
            } else {
                const int rg = u % (R / 4), kg = u / (R / 4);
                uint32_t d[4] = {r[q * 4 + 0], r[q * 4 + 1], r[q * 4 + 2], r[q * 4 + 3]};
                transpose4x4(d);
#pragma unroll
                for (int b = 0; b < 4; ++b)
                    *reinterpret_cast<uint32_t*>(&lds[rg * 4 + b][kg * 4]) = d[b];
            }
        }
    }
};

// Register layouts of the two instructions (per lane l of the wave):
//   32x32x16: operand bytes = row l % 32, k 8 (l / 32) .. +7 of the 16-k step;
//             result register r = row 8 (r / 4) + 4 (l / 32) + r % 4, column l % 32.
//   16x16x32: operand bytes = row l % 16, k 8 (l / 16) .. +7 of the 32-k step;
//             result register r = row 4 (l / 16) + r, column l % 16.
template <int BW> struct Mfma;
template <> struct Mfma<32> {
    static constexpr int KI = 16, NR = 16;
    typedef v16f acc_t;
    __device__ static int row(int l) { return l % 32; }
    __device__ static int koff(int l) { return 8 * (l / 32); }
    __device__ static int out_row(int l, int r) { return 8 * (r / 4) + 4 * (l / 32) + r % 4; }
    __device__ static int out_col(int l) { return l % 32; }
    __device__ static acc_t mac(long a, long b, acc_t c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf8_bf8(a, b, c, 0, 0, 0);
    }
};
template <> struct Mfma<16> {
    static constexpr int KI = 32, NR = 4;
    typedef v4f acc_t;
    __device__ static int row(int l) { return l % 16; }
    __device__ static int koff(int l) { return 8 * (l / 16); }
    __device__ static int out_row(int l, int r) { return 4 * (l / 16) + r; }
    __device__ static int out_col(int l) { return l % 16; }
    __device__ static acc_t mac(long a, long b, acc_t c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf8_bf8(a, b, c, 0, 0, 0);
    }
};

template <int BW, int FM, int FN, int kStages, int kBK, bool TA, bool TB>
__global__ __launch_bounds__(kNT) void chunk_gemm_mfma(GemmArgs g, Plan p) {
    constexpr int kPitch = kBK + 8;     // bytes per LDS row (k-contiguous)
    using I = Mfma<BW>;
    constexpr int BM = 2 * FM * BW, BN = 2 * FN * BW;
    constexpr int KI = I::KI, NR = I::NR;
    typedef typename I::acc_t acc_t;

    __shared__ __attribute__((aligned(16))) uint8_t As[2][BM][kPitch];
    __shared__ __attribute__((aligned(16))) uint8_t Bs[2][BN][kPitch];
    __shared__ uint32_t s_vote[2];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wy = wave >> 1, wx = wave & 1;
    if (tid == 0) s_vote[0] = s_vote[1] = 0u;     // ordered by the first slab's barrier
    int vslot = 0;

    Slab<!TA, BM, kBK> la[kStages];      // A is k-contiguous unless transposed
    Slab<TB, BN, kBK> lb[kStages];       // B is k-contiguous only when transposed

    acc_t acc[FM][FN];
    float S[FM][FN][NR];
    // per-thread offsets of the interior load path (see Slab::load_fast)
    typedef Slab<!TA, BM, kBK> SlabA;
    typedef Slab<TB, BN, kBK> SlabB;
    uint32_t offa[SlabA::NW], offb[SlabB::NW];
    SlabA::offsets(g.lda, tid, offa);
    SlabB::offsets(g.ldb, tid, offb);

    auto piece = [&](auto safe_tag, int64_t tile, int c0, int c1, int64_t lt)
                     __attribute__((always_inline)) -> bool {
        constexpr bool SAFE = decltype(safe_tag)::value;
        constexpr int DOM = SAFE ? 96 : 0;
        int tr, tc;
        tile_rc(p, tile, tr, tc);
        const int m0 = tr * BM;
        const int n0 = tc * BN;
        const int kbeg = (int)((int64_t)c0 * g.CL);
        const int64_t kend64 = (int64_t)c1 * g.CL;
        const int kend = kend64 < g.K ? (int)kend64 : g.K;
        const bool to_ws = c0 > 0;
        int chunk = c0;
        float vmax = 0.0f;                 // guarded: largest |S| at chunk ends
        bool nonfinite = false;            // guarded: a chunk sum for the fold was not finite

#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int r = 0; r < NR; ++r) { acc[i][j][r] = 0.0f; S[i][j][r] = 0.0f; }

        // chunk end: round each chunk sum, add it into S (or, for a piece
        // that does not start the tile, store it for the fold pass)
        auto flush_sum = [&](acc_t (&acc)[FM][FN]) __attribute__((always_inline)) {
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j) {
#pragma unroll
                    for (int r = 0; r < NR; ++r) {
                        S[i][j][r] = SAFE ? rn16s(S[i][j][r] + rn16s(acc[i][j][r] * 0x1p96f))
                                          : rn16v(S[i][j][r] + rn16v(acc[i][j][r]));
                        acc[i][j][r] = 0.0f;
                    }
                    // the guard: running sums at chunk ends (a chunk sum that
                    // overflowed shows in them; v_max3 drops NaN, which the
                    // check of the final sums catches)
                    if (!SAFE) {
#pragma unroll
                        for (int r = 0; r < NR; r += 2)
                            vmax = max3_abs(vmax, S[i][j][r], S[i][j][NR > 1 ? r + 1 : r]);
                    }
                }
        };
        auto flush_ws = [&](acc_t (&acc)[FM][FN]) __attribute__((always_inline)) {
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j) {
                    const int r0 = wy * FM * BW + i * BW;
                    const int c = wx * FN * BW + j * BW + I::out_col(lane);
#pragma unroll
                    for (int r = 0; r < NR; ++r) {
                        float pv;
                        if (SAFE) {
                            pv = rn16s(acc[i][j][r] * 0x1p96f);
                        } else {
                            // Veltkamp rounding turns an Inf sum into NaN
                            pv = rn16v(acc[i][j][r]);
                            nonfinite |= !(fabsf(pv) < 2147483648.0f);
                        }
                        g.ws[ws_index(p, BM, BN, lt, chunk, r0 + I::out_row(lane, r), c)] =
                            fp16_code<DOM>(pv);
                        acc[i][j][r] = 0.0f;
                    }
                }
        };
        auto flush = [&]() __attribute__((always_inline)) {
            if (to_ws) flush_ws(acc);
            else flush_sum(acc);
            ++chunk;
        };

        // kStages slabs are in flight from HBM at any time (in registers)
        // while a slab is consumed from LDS: a slab holds little arithmetic
        // (64 k of MFMA and one chunk's epilogue), so one slab of prefetch
        // would not cover the memory latency.
        const int nslabs = (kend - kbeg + kBK - 1) / kBK;
        int crem = g.CL;
        // interior tiles with aligned operands load without bounds checks;
        // chunk lengths that are whole slabs end chunks only at slab ends
        const bool interior = m0 + BM <= g.M && n0 + BN <= g.N && g.a_vec && g.b_vec;
        const bool slab_chunks = g.CL % kBK == 0;
        auto issue = [&](int u, int kk) __attribute__((always_inline)) {
            if (interior && kk + kBK <= kend) {
                const uint8_t* ba = TA ? g.A + (int64_t)kk * g.lda + m0 : g.A + (int64_t)m0 * g.lda + kk;
                const uint8_t* bb = TB ? g.B + (int64_t)n0 * g.ldb + kk : g.B + (int64_t)kk * g.ldb + n0;
                la[u].load_fast(ba, offa, tid);
                lb[u].load_fast(bb, offb, tid);
            } else {
                la[u].load(g.A, g.lda, m0, kk, g.M, kend, g.a_vec, tid);
                lb[u].load(g.B, g.ldb, n0, kk, g.N, kend, g.b_vec, tid);
            }
        };
#pragma unroll
        for (int u = 0; u < kStages; ++u)
            if (u < nslabs) issue(u, kbeg + u * kBK);
        for (int s0 = 0; s0 < nslabs; s0 += kStages) {
#pragma unroll
            for (int u = 0; u < kStages; ++u) {
                const int s = s0 + u;
                if (s >= nslabs) break;
                const int buf = s & 1;
                const int ks = kbeg + s * kBK;
                // buffer buf last held slab s - 2, which every wave finished
                // before the barrier of slab s - 1
                la[u].store(As[buf], tid);
                lb[u].store(Bs[buf], tid);
                if (s + kStages < nslabs) issue(u, ks + kStages * kBK);
                __syncthreads();
                auto read = [&](long (&a)[FM], long (&b)[FN], int st) __attribute__((always_inline)) {
#pragma unroll
                    for (int i = 0; i < FM; ++i)
                        a[i] = *reinterpret_cast<const long*>(
                            &As[buf][wy * FM * BW + i * BW + I::row(lane)][st * KI + I::koff(lane)]);
#pragma unroll
                    for (int j = 0; j < FN; ++j)
                        b[j] = *reinterpret_cast<const long*>(
                            &Bs[buf][wx * FN * BW + j * BW + I::row(lane)][st * KI + I::koff(lane)]);
                };
                auto mma = [&](const long (&a)[FM], const long (&b)[FN]) __attribute__((always_inline)) {
#pragma unroll
                    for (int i = 0; i < FM; ++i)
#pragma unroll
                        for (int j = 0; j < FN; ++j) acc[i][j] = I::mac(a[i], b[j], acc[i][j]);
                };
                if (slab_chunks && ks + kBK <= kend) {
                    // a full slab inside one chunk: operand reads, then the chain
                    long a[kBK / KI][FM], b[kBK / KI][FN];
#pragma unroll
                    for (int st = 0; st < kBK / KI; ++st) read(a[st], b[st], st);
#pragma unroll
                    for (int st = 0; st < kBK / KI; ++st) mma(a[st], b[st]);
                    crem -= kBK;
                    if (crem == 0) {
                        flush();
                        crem = g.CL;
                    }
                } else if (kBK % 64 == 0 && kBK > 64 && g.CL == 64 && ks + kBK <= kend) {
                    // the paper's chunk length, several chunks per full slab
                    // (slabs start on chunk boundaries)
#pragma unroll
                    for (int q = 0; q < kBK / 64; ++q) {
                        long a[64 / KI][FM], b[64 / KI][FN];
#pragma unroll
                        for (int st = 0; st < 64 / KI; ++st) read(a[st], b[st], q * (64 / KI) + st);
#pragma unroll
                        for (int st = 0; st < 64 / KI; ++st) mma(a[st], b[st]);
                        flush();
                    }
                } else {
                    const int nsteps = (min(kBK, kend - ks) + KI - 1) / KI;
                    for (int st = 0; st < nsteps; ++st) {
                        long a[FM], b[FN];
                        read(a, b, st);
                        mma(a, b);
                        crem -= KI;
                        if (crem == 0) {
                            flush();
                            crem = g.CL;
                        }
                    }
                }
            }
        }
        __syncthreads();                   // LDS is reused by the next piece
        if (crem != g.CL) flush();         // the last, shorter chunk

        // The guard: running sums below 2^31 at every chunk end, so no chunk
        // sum or sum reached FP16's overflow threshold (one that did would
        // leave a running sum at 2^31 or more); and no Inf/NaN operand, whose
        // chunk sum the guarded rounding turns into a NaN that then stays in
        // the running sum to the end (v_max3 drops NaN: the comparison of
        // the final sums catches it).
        if (!SAFE) {
            bool bad = !(vmax < 2147483648.0f) || nonfinite;
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
#pragma unroll
                    for (int r = 0; r < NR; ++r) bad |= !(fabsf(S[i][j][r]) < 2147483648.0f);
            if (block_any(bad, s_vote, vslot)) return false;
        }
        if (to_ws) return true;
        // Results leave through LDS (free after the last slab's barrier): the
        // tile's FP16 codes are staged there, then every thread writes 8
        // consecutive codes of a row -- 16-byte stores of C, 8-byte stores of
        // the FP8 result.  The first piece of a shared tile leaves its running
        // sum for the fold pass instead (in C, or in s_ws when only the FP8
        // result is wanted); whole tiles write the results.
        uint16_t* ot = reinterpret_cast<uint16_t*>(&As[0][0][0]);
        static_assert(BM * BN * 2 <= (int)sizeof(As), "staging tile exceeds LDS slab");
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int r = 0; r < NR; ++r)
                    ot[(wy * FM * BW + i * BW + I::out_row(lane, r)) * BN + wx * FN * BW +
                       j * BW + I::out_col(lane)] = fp16_code<DOM>(S[i][j][r]);
        __syncthreads();
        const bool keep = lt >= 0 && !g.C;
        for (int u = tid; u < BM * BN / 8; u += kNT) {
            const int row = u / (BN / 8), col = (u % (BN / 8)) * 8;
            const uint4 q = *reinterpret_cast<const uint4*>(&ot[row * BN + col]);
            if (keep) {
                *reinterpret_cast<uint4*>(g.s_ws + (lt * BM + row) * BN + col) = q;
                continue;
            }
            const int m = m0 + row, n = n0 + col;
            if (m >= g.M) continue;
            const uint32_t cw[4] = {q.x, q.y, q.z, q.w};
            if (g.C) {
                uint16_t* cp = g.C + (int64_t)m * g.ldc + n;
                if (g.c_vec16 && n + 8 <= g.N) {
                    *reinterpret_cast<uint4*>(cp) = q;
                } else {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (n + e < g.N) cp[e] = (uint16_t)(cw[e / 2] >> (16 * (e % 2)));
                }
            }
            if (g.C8 && lt < 0) {
                auto val = [&](int e) __attribute__((always_inline)) {
                    return fp16_to_f32((cw[e / 2] >> (16 * (e % 2))) & 0xFFFFu) * g.q_scale;
                };
                uint2 v;
                v.x = f32x2_to_fp8x2<true>(val(2), val(3), f32x2_to_fp8x2<false>(val(0), val(1), 0u));
                v.y = f32x2_to_fp8x2<true>(val(6), val(7), f32x2_to_fp8x2<false>(val(4), val(5), 0u));
                uint8_t* qp = g.C8 + (int64_t)m * g.ldc8 + n;
                if (g.c8_vec8 && n + 8 <= g.N) {
                    *reinterpret_cast<uint2*>(qp) = v;
                } else {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (n + e < g.N) qp[e] = (uint8_t)((e < 4 ? v.x : v.y) >> (8 * (e % 4)));
                }
            }
        }
        __syncthreads();                   // the staging tile is the next piece's slab
        return true;
    };

    const int w = blockIdx.x;
    int64_t t = w;
    int64_t s = p.L > 0 ? (int64_t)w * p.L / p.G : 0;
    const int64_t e = p.L > 0 ? (int64_t)(w + 1) * p.L / p.G : 0;
    for (;;) {
        int64_t tile, lt;
        int c0, c1;
        if (t < p.t_whole) {
            tile = whole_tile(p, t);
            lt = -1;
            c0 = 0;
            c1 = p.nch;
            t += p.G;
        } else if (s < e) {
            lt = s / p.nch;
            c0 = (int)(s - lt * p.nch);
            const int64_t c1l = e - lt * p.nch;
            c1 = c1l < p.nch ? (int)c1l : p.nch;
            tile = p.t_whole + lt;
            s = lt * p.nch + c1;
        } else {
            break;
        }
        bool done = false;
        if (g.guarded) done = piece(std::integral_constant<bool, false>{}, tile, c0, c1, lt);
        if (!done) piece(std::integral_constant<bool, true>{}, tile, c0, c1, lt);
    }
}

template <int BW, int FM, int FN, int ST, int BK>
const void* kernel_sel(int ta, int tb) {
    if (!ta && !tb) return reinterpret_cast<const void*>(&chunk_gemm_mfma<BW, FM, FN, ST, BK, false, false>);
    if (!ta && tb) return reinterpret_cast<const void*>(&chunk_gemm_mfma<BW, FM, FN, ST, BK, false, true>);
    if (ta && !tb) return reinterpret_cast<const void*>(&chunk_gemm_mfma<BW, FM, FN, ST, BK, true, false>);
    return reinterpret_cast<const void*>(&chunk_gemm_mfma<BW, FM, FN, ST, BK, true, true>);
}

}  // namespace

MfmaShape mfma_shape(int cfg) {
    switch (cfg) {
        case 0: return MfmaShape{32, 64, 64, kNT, 16, 64};
        case 2: return MfmaShape{32, 64, 64, kNT, 64, 64};      // CL a multiple of 64
        case 3: return MfmaShape{32, 64, 64, 1024, 64, 256};    // CL = 64, 16 waves
        case 4: return MfmaShape{16, 64, 64, 1024, 64, 256};    // CL = 64, 16 waves
        case 5: return MfmaShape{32, 32, 128, kNT, 64, 128};   // CL a multiple of 64, 4 waves
        default: return MfmaShape{16, 32, 32, kNT, 32, 128};
    }
}

const void* mfma_kernel(int cfg, int ta, int tb) {
    switch (cfg) {
        case 0: return kernel_sel<32, 1, 1, 2, 64>(ta, tb);
        case 1: return kernel_sel<16, 1, 1, 2, 128>(ta, tb);
        case 2: return mfma_stream_kernel(ta, tb);
        case 3: return mfma_kx_kernel(ta, tb);
        case 4: return mfma_kx16_kernel(ta, tb);
        case 5: return (void)tb, mfma_wave_kernel(ta);
        default: return nullptr;
    }
}

}  // namespace fp8t
