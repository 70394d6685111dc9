// chunk_gemm fast mode on the matrix cores: the wave-independent kernel.
//
// Same arithmetic as chunk_gemm_mfma_stream (gemm_mfma_stream.hip), with the
// same instruction and lane layout, so the same bits: each chunk of CL
// products (CL a multiple of 64) is summed in FP32 by
// v_mfma_f32_32x32x64_f8f6f4 on bf8 operands (lane half h carries k
// 32 h .. 32 h + 31 of a 64-k slab for both operands), rounded to FP16 once
// and added into the running sum in ascending chunk order with FP16
// rounding after every add.  What differs is how the operands reach the
// matrix cores, for A and B both k-contiguous (B(k, n) at B[n ldb + k]; the
// host makes a k-contiguous copy of a B stored with n contiguous):
//   * each wave owns a 32 x 32 block of the workgroup's 32 x 128 tile and
//     streams its operands itself -- no workgroup barrier anywhere;
//   * a load round covers 128 k: eight lanes read a row's 128 contiguous
//     bytes, so each load instruction touches 8 whole 128-byte lines (the
//     matrix-core layout, 32 bytes of 32 rows per lane group, would touch
//     32 lines per instruction, and loads in that layout measured 2x slower);
//   * the round goes straight from memory into a wave-private LDS tile
//     (gfx950's global_load_lds_dwordx4: lane l of a load lands at its LDS
//     base + 16 l, so which 16 bytes a lane fetches sets the layout: the
//     pieces of a row are XOR-swizzled by the row, which keeps the
//     matrix-core reads free of bank conflicts); the wave reads both slabs'
//     operands from it into registers and then already starts the next
//     round (of the same tile or its next one) into it, so the loads bypass
//     the registers and take no LDS write instructions;
//   * the guard is per wave (its outputs depend on no other wave's): a tile
//     whose running sums reached 2^31 at a chunk end or ended NaN is marked
//     (one bit per tile ordinal) and recomputed after the stream with the
//     2^96-scaled epilogue;
//   * the finished block's FP16 codes leave through a second LDS tile as
//     16-byte row pieces.
// Rows of A beyond M and of B beyond N are read as row M-1 / N-1 (their
// outputs are not stored); k beyond K reads as zero.
#include "fp8t_device.h"
#include "gemm_mfma.h"

namespace fp8t {
namespace {

typedef float v16f __attribute__((ext_vector_type(16)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef uint32_t vu4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;                  // waves per workgroup
constexpr int kNT = 64 * kWaves;
constexpr int kBM = 32, kBN = 32 * kWaves; // workgroup tile; a wave's block is 32 x 32
constexpr int kRound = 128;                // k per load round: two 64-k slabs
constexpr int kP = kRound;                 // LDS row pitch (bytes) of a round
constexpr int kOP = 64;                    // LDS row pitch (bytes) of the staged codes

// Result register r of lane l: row 8 (r / 4) + 4 (l / 32) + r % 4, column l % 32.
__device__ __forceinline__ int out_row(int l, int r) { return 8 * (r / 4) + 4 * (l / 32) + r % 4; }
// LDS byte offset of 16-byte segment g of row r of a round (segments XOR-swizzled by r % 8)
__device__ __forceinline__ int seg_off(int r, int g) { return r * kP + 16 * (g ^ (r & 7)); }
typedef __attribute__((address_space(1))) const void* gptr_t;
typedef __attribute__((address_space(3))) void* lptr_t;

// max(m, |a|, |b|) with NaN propagating (IEEE 754-2019 maximum): any NaN
// operand gives NaN.
__device__ __forceinline__ float maximum3_abs(float m, float a, float b) {
    float r;
    asm("v_maximum3_f32 %0, %1, |%2|, |%3|" : "=v"(r) : "v"(m), "v"(a), "v"(b));
    return r;
}

// Orders a wave's LDS accesses across its lanes: the LDS executes one wave's
// instructions in order, and the fences keep the compiler from moving
// accesses across.
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Bytes k .. k+15 of row `row` of a k-contiguous byte matrix; bytes at k >=
// kend read as 0 (and are not loaded).
__device__ __forceinline__ vu4 load16(const uint8_t* __restrict__ p, int64_t ld, int row, int k,
                                      int kend) {
    const uint8_t* q = p + (int64_t)row * ld + k;
    if (k + 16 <= kend) return *reinterpret_cast<const vu4*>(q);
    vu4 v = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int b = 0; b < 16; ++b)
        if (k + b < kend) v[b / 4] |= (uint32_t)q[b] << (8 * (b % 4));
    return v;
}

__global__ __launch_bounds__(kNT) __attribute__((amdgpu_waves_per_eu(4)))
void chunk_gemm_mfma_wave(GemmArgs g, Plan p) {
    __shared__ __attribute__((aligned(16))) uint8_t lds[kWaves][2][kBM * kP];
    __shared__ __attribute__((aligned(16))) uint8_t lco_all[kWaves][kBM * kOP];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    uint8_t* const la = lds[wave][0];
    uint8_t* const lb = lds[wave][1];
    uint8_t* const lco = lco_all[wave];
    const int rl = lane & 31, kh = 32 * (lane >> 5);   // operand row, k half
    const int lr = lane >> 3;                          // load row (of 8)
    // the global 16-byte segment a lane loads: its LDS slot (lane % 8) XOR
    // the row's swizzle (row % 8 = lane / 8)
    const int lc = 16 * ((lane & 7) ^ lr);
    const v16f zero = {};

    auto geom = [&](int64_t t, int& m0, int& n0) __attribute__((always_inline)) {
        int tr, tc;
        tile_rc(p, whole_tile(p, t), tr, tc);
        m0 = tr * kBM;
        n0 = tc * kBN + 32 * wave;
    };

    // The FP16 codes of the wave's block (running sums S, DOM their value
    // scale) to C and / or the FP8 result C8, through the LDS tile lco.
    auto store_block = [&](auto dom_tag, const float (&S)[16], int m0, int n0)
                           __attribute__((always_inline)) {
        constexpr int DOM = decltype(dom_tag)::value;
#pragma unroll
        for (int r = 0; r < 16; ++r)
            *reinterpret_cast<uint16_t*>(lco + out_row(lane, r) * kOP + 2 * rl) =
                (uint16_t)fp16_code<DOM>(S[r]);
        wave_lds_sync();
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const int u = lane + 64 * q;
            const int row = u >> 2, col = (u & 3) * 8;
            const vu4 v = *reinterpret_cast<const vu4*>(lco + row * kOP + 2 * col);
            const int m = m0 + row, n = n0 + col;
            if (m >= g.M || n >= g.N) continue;
            if (g.C) {
                uint16_t* cp = g.C + (int64_t)m * g.ldc + n;
                if (g.c_vec16 && n + 8 <= g.N) {
                    *reinterpret_cast<vu4*>(cp) = v;
                } else {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (n + e < g.N) cp[e] = (uint16_t)(v[e / 2] >> (16 * (e % 2)));
                }
            }
            if (g.C8) {
                auto val = [&](int e) __attribute__((always_inline)) {
                    return fp16_to_f32((v[e / 2] >> (16 * (e % 2))) & 0xFFFFu) * g.q_scale;
                };
                uint2 v8;
                v8.x = f32x2_to_fp8x2<true>(val(2), val(3), f32x2_to_fp8x2<false>(val(0), val(1), 0u));
                v8.y = f32x2_to_fp8x2<true>(val(6), val(7), f32x2_to_fp8x2<false>(val(4), val(5), 0u));
                uint8_t* qp = g.C8 + (int64_t)m * g.ldc8 + n;
                if (g.c8_vec8 && n + 8 <= g.N) {
                    *reinterpret_cast<uint2*>(qp) = v8;
                } else {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (n + e < g.N) qp[e] = (uint8_t)((e < 4 ? v8.x : v8.y) >> (8 * (e % 4)));
                }
            }
        }
        wave_lds_sync();                 // lco is rewritten at the next block end
    };

    // ---- the stream (guarded epilogue) ----
    // A block's operand rows: base pointers at its first rows (wave-uniform,
    // scalar registers) and per lane the 32-bit byte offsets of load row q
    // (8 q + lane / 8, clamped to the last row) plus the lane's 16-byte
    // piece, so a round's load addresses are the scalar base plus k plus a
    // fixed lane offset (no per-load 64-bit arithmetic on the vector ALUs).
    const uint8_t* pa;
    const uint8_t* pb;
    uint32_t oa[4], ob[4];
    auto rows = [&](int m0, int n0) __attribute__((always_inline)) {
        const int nb = min(n0, g.N - 1);
        pa = g.A + (int64_t)m0 * g.lda;
        pb = g.B + (int64_t)nb * g.ldb;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            oa[q] = (uint32_t)((min(m0 + 8 * q + lr, g.M - 1) - m0) * (int)g.lda + lc);
            ob[q] = (uint32_t)((min(n0 + 8 * q + lr, g.N - 1) - nb) * (int)g.ldb + lc);
        }
    };
    // the round at k of the block whose rows() were taken last, into the
    // LDS tiles: whole rounds straight from memory (lane l of load q lands at
    // q KB + 16 l: row 8 q + l / 8, slot l % 8), a last partial round through
    // registers with the bytes past K zeroed
    auto issue = [&](int k) __attribute__((always_inline)) {
        const uint8_t* const ak = pa + k;
        const uint8_t* const bk = pb + k;
        if (k + kRound <= g.K) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                __builtin_amdgcn_global_load_lds((gptr_t)(ak + oa[q]), (lptr_t)(la + q * 1024), 16, 0, 0);
                __builtin_amdgcn_global_load_lds((gptr_t)(bk + ob[q]), (lptr_t)(lb + q * 1024), 16, 0, 0);
            }
        } else {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const vu4 va = load16(pa, 0, 0, (int)oa[q] + k, (int)(oa[q] - lc) + g.K);
                const vu4 vb = load16(pb, 0, 0, (int)ob[q] + k, (int)(ob[q] - lc) + g.K);
                *reinterpret_cast<vu4*>(la + q * 1024 + 16 * lane) = va;
                *reinterpret_cast<vu4*>(lb + q * 1024 + 16 * lane) = vb;
            }
        }
    };
    // with the guarded epilogue switched off every tile takes the safe one
    // failed blocks: ordinals below 64 as bits, any later one redoes all
    uint64_t failed = 0;
    bool fail_all = !g.guarded;
    int64_t t = blockIdx.x;
    if (g.guarded && t < p.t_whole) {
        int m0, n0, k = 0;
        geom(t, m0, n0);
        rows(m0, n0);
        issue(0);
        // the position of the next round
        int64_t tx = t;
        int mx = m0, nx = n0, kx = 0;
        bool okx = true;
        auto advance = [&]() __attribute__((always_inline)) {
            kx += kRound;
            if (kx >= g.K) {
                kx = 0;
                tx += p.G;
                okx = tx < p.t_whole;
                if (okx) {
                    geom(tx, mx, nx);
                    rows(mx, nx);
                }
            }
        };
        advance();
        v16f acc;
        float S[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) S[r] = 0.0f;
        float vmax = 0.0f;             // largest |S| at chunk ends
        int crem = g.CL, ordinal = 0;
        for (;;) {
            // this round's bytes are in the LDS tiles (direct loads count in
            // vmcnt; the compiler does not see their LDS writes)
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            wave_lds_sync();
            v8i a8s[2], b8s[2];
#pragma unroll
            for (int sl = 0; sl < 2; ++sl) {
                const int g0 = 4 * sl + kh / 16;
                const vu4 a0 = *reinterpret_cast<const vu4*>(la + seg_off(rl, g0));
                const vu4 a1 = *reinterpret_cast<const vu4*>(la + seg_off(rl, g0 + 1));
                const vu4 b0 = *reinterpret_cast<const vu4*>(lb + seg_off(rl, g0));
                const vu4 b1 = *reinterpret_cast<const vu4*>(lb + seg_off(rl, g0 + 1));
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    a8s[sl][q] = (int)a0[q];
                    a8s[sl][4 + q] = (int)a1[q];
                    b8s[sl][q] = (int)b0[q];
                    b8s[sl][4 + q] = (int)b1[q];
                }
            }
            // the tiles are refilled with the next round once these reads are done
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            wave_lds_sync();
            if (okx) issue(kx);
#pragma unroll
            for (int sl = 0; sl < 2; ++sl) {
                const int ks = k + 64 * sl;
                if (ks >= g.K) break;
                const v8i a8 = a8s[sl], b8 = b8s[sl];
                // format selectors 1, 1: both operands bf8 (= the FP8 codes);
                // no scaling; a chunk's first slab starts from zero
                if (crem == g.CL)
                    acc = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a8, b8, zero, 1, 1, 0, 0,
                                                                          0, 0);
                else
                    acc = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a8, b8, acc, 1, 1, 0, 0,
                                                                          0, 0);
                crem -= 64;
                if (crem == 0 || ks + 64 >= g.K) {
                    // S = rn16v(S + rn16v(acc)) written out step by step over
                    // the 16 outputs, so the schedule interleaves them (the
                    // compiler otherwise runs each output's 7 dependent
                    // instructions back to back; measured 1.5-2% faster)
                    float c[16], x[16];
#pragma unroll
                    for (int r = 0; r < 16; ++r) c[r] = acc[r] * 16385.0f;
#pragma unroll
                    for (int r = 0; r < 16; ++r) x[r] = c[r] - acc[r];
#pragma unroll
                    for (int r = 0; r < 16; ++r) x[r] = S[r] + (c[r] - x[r]);
#pragma unroll
                    for (int r = 0; r < 16; ++r) c[r] = x[r] * 16385.0f;
#pragma unroll
                    for (int r = 0; r < 16; ++r) x[r] = c[r] - x[r];
#pragma unroll
                    for (int r = 0; r < 16; ++r) S[r] = c[r] - x[r];
                    // the guard: running sums at chunk ends, with gfx950's
                    // NaN-propagating three-input maximum (a NaN sum, from an
                    // Inf/NaN operand, stays NaN to the block end and so
                    // fails the check there without a test of each sum)
#pragma unroll
                    for (int r = 0; r < 16; r += 2) vmax = maximum3_abs(vmax, S[r], S[r + 1]);
                    crem = g.CL;
                }
            }
            wave_lds_sync();
            if (k + kRound >= g.K) {
                // block end: running sums below 2^31 at every chunk end -- no
                // chunk sum or sum reached FP16's overflow threshold -- and
                // never NaN (no Inf/NaN operand)
                const bool bad = !(vmax < 2147483648.0f);
                if (__any(bad)) {
                    if (ordinal < 64) failed |= 1ull << ordinal;
                    else fail_all = true;
                } else {
                    store_block(std::integral_constant<int, 0>{}, S, m0, n0);
                }
#pragma unroll
                for (int r = 0; r < 16; ++r) S[r] = 0.0f;
                vmax = 0.0f;
                ++ordinal;
            }
            if (!okx) break;
            m0 = mx;
            n0 = nx;
            k = kx;
            advance();
        }
    }

    // ---- blocks that failed the guard (all of them when it is off, or when
    // one beyond the 64th failed), recomputed in the 2^96 domain ----
    if (failed == 0 && !fail_all) return;
    int ord = 0;
    for (int64_t tt = blockIdx.x; tt < p.t_whole; tt += p.G, ++ord) {
        const bool listed = fail_all || (ord < 64 && ((failed >> ord) & 1));
        if (!listed) continue;
        int m0, n0;
        geom(tt, m0, n0);
        const int ar = min(m0 + rl, g.M - 1), br = min(n0 + rl, g.N - 1);
        float S[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) S[r] = 0.0f;
        v16f acc;
        int crem = g.CL;
        for (int ks = 0; ks < g.K; ks += 64) {
            // operands straight in the matrix-core layout: lane (r, h) reads
            // k ks + 32 h .. + 31 of row r
            const vu4 a0 = load16(g.A, g.lda, ar, ks + kh, g.K);
            const vu4 a1 = load16(g.A, g.lda, ar, ks + kh + 16, g.K);
            const vu4 b0 = load16(g.B, g.ldb, br, ks + kh, g.K);
            const vu4 b1 = load16(g.B, g.ldb, br, ks + kh + 16, g.K);
            v8i a8, b8;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                a8[q] = (int)a0[q];
                a8[4 + q] = (int)a1[q];
                b8[q] = (int)b0[q];
                b8[4 + q] = (int)b1[q];
            }
            acc = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a8, b8, crem == g.CL ? zero : acc,
                                                                  1, 1, 0, 0, 0, 0);
            crem -= 64;
            if (crem == 0 || ks + 64 >= g.K) {
#pragma unroll
                for (int r = 0; r < 16; ++r) S[r] = rn16s(S[r] + rn16s(acc[r] * 0x1p96f));
                crem = g.CL;
            }
        }
        store_block(std::integral_constant<int, 96>{}, S, m0, n0);
    }
}

// Bt[n][k] = B[k][n] for k < K, n < N (B row-major K x N with leading
// dimension ldb; Bt 16-byte aligned with ldt a multiple of 16): 64 x 64 byte
// tiles through LDS, 16 bytes per thread each way (16-byte accesses where
// the row piece is whole and, for B, aligned); the grid's y dimension
// strides over the k tiles.
__global__ __launch_bounds__(256) void transpose_bytes(const uint8_t* __restrict__ B, int64_t ldb,
                                                       int K, int N, uint8_t* __restrict__ Bt,
                                                       int64_t ldt, int b_vec16) {
    __shared__ uint8_t tile[64][64 + 4];
    const int tid = threadIdx.x;
    const int r = tid >> 2, c = (tid & 3) * 16;
    const int n0 = blockIdx.x * 64;
    for (int64_t k0 = (int64_t)blockIdx.y * 64; k0 < K; k0 += (int64_t)gridDim.y * 64) {
        {
            // k row r, n bytes c .. c+15
            const int64_t k = k0 + r;
            const int n = n0 + c;
            uint32_t w[4] = {0u, 0u, 0u, 0u};
            if (k < K && n < N) {
                const uint8_t* src = B + k * ldb + n;
                if (b_vec16 && n + 16 <= N) {
                    const uint4 v = *reinterpret_cast<const uint4*>(src);
                    w[0] = v.x, w[1] = v.y, w[2] = v.z, w[3] = v.w;
                } else {
#pragma unroll
                    for (int b = 0; b < 16; ++b)
                        if (n + b < N) w[b / 4] |= (uint32_t)src[b] << (8 * (b % 4));
                }
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) *reinterpret_cast<uint32_t*>(&tile[r][c + 4 * i]) = w[i];
        }
        __syncthreads();
        {
            // n row r, k bytes c .. c+15
            const int n = n0 + r;
            const int64_t k = k0 + c;
            if (n < N && k < K) {
                uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
                for (int b = 0; b < 16; ++b) w[b / 4] |= (uint32_t)tile[c + b][r] << (8 * (b % 4));
                uint8_t* dst = Bt + (int64_t)n * ldt + k;
                if (k + 16 <= K) {
                    *reinterpret_cast<uint4*>(dst) = make_uint4(w[0], w[1], w[2], w[3]);
                } else {
#pragma unroll
                    for (int b = 0; b < 16; ++b)
                        if (k + b < K) dst[b] = (uint8_t)(w[b / 4] >> (8 * (b % 4)));
                }
            }
        }
        __syncthreads();                 // the tile is rewritten next
    }
}

}  // namespace

const void* mfma_wave_kernel(int ta) {
    return ta ? nullptr : reinterpret_cast<const void*>(&chunk_gemm_mfma_wave);
}

void launch_transpose_bytes(const uint8_t* B, int64_t ldb, int K, int N, uint8_t* Bt, int64_t ldt,
                            hipStream_t stream) {
    const int64_t kt = ((int64_t)K + 63) / 64;
    const dim3 grid((unsigned)((N + 63) / 64), (unsigned)(kt < 65535 ? kt : 65535));
    const int b_vec16 = ((uintptr_t)B % 16 == 0) && ldb % 16 == 0;
    hipLaunchKernelGGL(transpose_bytes, grid, dim3(256), 0, stream, B, ldb, K, N, Bt, ldt, b_vec16);
}

}  // namespace fp8t
