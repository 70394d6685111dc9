// chunk_gemm fast mode on the matrix cores for GEMMs with few outputs and a
// long K (the weight-gradient shape): chunks spread over a workgroup's waves.
//
// Same arithmetic as the other fast-mode kernels, for CL = 64: each chunk of
// 64 products is summed in FP32 by one v_mfma_f32_32x32x64_f8f6f4 with both
// operands bf8 (the FP8 codes are OCP E5M2 = bf8), rounded to FP16 once, and
// added into the running sum in ascending chunk order with FP16 rounding after
// every add.  The work is cut differently:
//   * a workgroup of 16 waves owns a 64 x 64 output tile; wave w computes
//     quadrant w / 4 (32 x 32 outputs) of chunk 4 s + w % 4 at step s, so the
//     four chunks of a step run side by side and one workgroup keeps all four
//     SIMDs of a CU at four waves even when the GEMM has few tiles (2304 x 256
//     outputs make 144 tiles; a K of 50176 makes 196 steps per tile);
//   * each wave rounds its chunk sums and leaves them in LDS; after a barrier
//     every thread adds the four chunk sums of its 4 outputs into their
//     running sums, in chunk order (the additions of a whole-tile pass, in
//     the same order, so the bits do not depend on the kernel);
//   * a step's operands (64 rows of A and 64 columns of B by 256 k) go
//     through one LDS buffer k-contiguous, operands stored with the row index
//     contiguous transposed 4 x 4 bytes in registers.  A tile 64 wide reads
//     64-byte runs of such operands (a 32-wide one read 32 of every line the
//     memory pipeline moves, and was bound by it);
//   * the bytes of the next two steps are in flight in two register sets
//     while the current one is consumed; with every step interior and 16-byte
//     aligned (AL) there is one load path, so the compiler waits for one set
//     only; the workgroup streams on across its tiles;
//   * the guarded epilogue (plain values, Veltkamp rounding, running max of
//     |p| -- taken by the wave that rounds p -- and of |S|) runs in the
//     stream; a tile in which a value reached 2^32 (FP16 overflow) is
//     remembered and recomputed after the stream with the
//     2^96-scaled epilogue (integer rounding on raw bits), which gives the
//     same bits wherever the guarded one is valid.
// Tiles are whole (no shared tiles, no workspace).
#include "fp8t_device.h"
#include "gemm_mfma.h"

namespace fp8t {
namespace {

typedef float v16f __attribute__((ext_vector_type(16)));
typedef int v8i __attribute__((ext_vector_type(8)));

constexpr int kNT = 1024;               // 16 waves: 4 chunks x 4 quadrants
constexpr int kT = 64;                  // tile rows = columns
constexpr int kCL = 64;                 // chunk length (one instruction)
constexpr int kWaves = 4;               // chunks per step
constexpr int kSK = kCL * kWaves;       // k per step
constexpr int kPitch = kSK + 8;         // LDS bytes per operand row
constexpr int kRedoMax = 64;            // failed tiles remembered per workgroup

// Bytes (r, c .. c+3) of a row-major byte matrix (rows x cols valid, leading
// dimension ld); 0 outside.
__device__ __forceinline__ uint32_t ld4(const uint8_t* __restrict__ p, int64_t ld, int r, int c,
                                        int rows, int cols, int vec) {
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
__device__ __forceinline__ void tr4(uint32_t d[4]) {
    const uint32_t lo01 = __builtin_amdgcn_perm(d[1], d[0], 0x05010400u);
    const uint32_t hi01 = __builtin_amdgcn_perm(d[1], d[0], 0x07030602u);
    const uint32_t lo23 = __builtin_amdgcn_perm(d[3], d[2], 0x05010400u);
    const uint32_t hi23 = __builtin_amdgcn_perm(d[3], d[2], 0x07030602u);
    d[0] = __builtin_amdgcn_perm(lo23, lo01, 0x05040100u);
    d[1] = __builtin_amdgcn_perm(lo23, lo01, 0x07060302u);
    d[2] = __builtin_amdgcn_perm(hi23, hi01, 0x05040100u);
    d[3] = __builtin_amdgcn_perm(hi23, hi01, 0x07060302u);
}

// LDS byte offset, within an operand row, of the 8-byte k slot q: slots are
// swizzled by bits 4-5 of the row, which spreads the 4-byte stores of the
// transposed operands (16 rows 4 apart per half-wave) over all banks and
// keeps each 32-byte half of a chunk where the matrix-core reads expect it.
__device__ __forceinline__ int slot_off(int row, int q) { return 8 * (q ^ ((row >> 4) & 3)); }

// One operand's share of a step (64 rows by 256 k): 16 bytes per thread.
//   KC (element (r, k) at p[r ld + k]): row t / 16, k bytes 16 (t % 16) .. +15;
//   otherwise (element (r, k) at p[k ld + r]): k rows 4 (t / 16) .. +3 by r
//     bytes 4 (t % 16) .. +3, a 4 x 4 block transposed on the way into LDS.
template <bool KC>
struct StepShare {
    uint32_t w[4];

    // AL: every step is interior and 16-byte aligned (one load path, so the
    // compiler can count the loads in flight and wait for one set only).
    template <bool AL>
    __device__ __forceinline__ void load(const uint8_t* __restrict__ p, int64_t ld, int r0,
                                         int rows, int k0, int kend, int vec, int vec16,
                                         int tid) {
        const bool interior = AL || (r0 + kT <= rows && k0 + kSK <= kend);
        if (KC) {
            const int r = r0 + (tid >> 4), k = k0 + (tid & 15) * 16;
            if (interior && (AL || vec16)) {
                const uint4 v = *reinterpret_cast<const uint4*>(p + (int64_t)r * ld + k);
                w[0] = v.x, w[1] = v.y, w[2] = v.z, w[3] = v.w;
            } else if (interior && vec) {
                const uint32_t* q = reinterpret_cast<const uint32_t*>(p + (int64_t)r * ld + k);
#pragma unroll
                for (int i = 0; i < 4; ++i) w[i] = q[i];
            } else {
#pragma unroll
                for (int i = 0; i < 4; ++i) w[i] = ld4(p, ld, r, k + 4 * i, rows, kend, vec);
            }
        } else {
            const int k = k0 + (tid >> 4) * 4, r = r0 + (tid & 15) * 4;
            if (interior && (AL || vec)) {
#pragma unroll
                for (int b = 0; b < 4; ++b)
                    w[b] = *reinterpret_cast<const uint32_t*>(p + (int64_t)(k + b) * ld + r);
            } else {
#pragma unroll
                for (int b = 0; b < 4; ++b) w[b] = ld4(p, ld, k + b, r, kend, rows, vec);
            }
        }
    }

    __device__ __forceinline__ void store(uint8_t (*lds)[kPitch], int tid) {
        if (KC) {
            const int r = tid >> 4, q = (tid & 15) * 2;
            *reinterpret_cast<uint2*>(&lds[r][slot_off(r, q)]) = make_uint2(w[0], w[1]);
            *reinterpret_cast<uint2*>(&lds[r][slot_off(r, q + 1)]) = make_uint2(w[2], w[3]);
        } else {
            uint32_t d[4] = {w[0], w[1], w[2], w[3]};
            tr4(d);
            const int kg = (tid >> 4) * 4, rg = (tid & 15) * 4;
#pragma unroll
            for (int i = 0; i < 4; ++i)
                *reinterpret_cast<uint32_t*>(&lds[rg + i][slot_off(rg + i, kg >> 3) + (kg & 4)]) = d[i];
        }
    }
};

// The block-per-wave kernel's share of a step (64 rows by 256 k, 16 bytes per
// thread) and its LDS layout:
//   KC: as StepShare (rows of k bytes, 8-byte k slots swizzled);
//   otherwise (row index contiguous in memory): k row t / 4, row bytes
//     16 (t % 4) .. +15, stored as they are -- LDS holds the step k-major
//     (kTrPitch bytes per k) and the matrix-core operands are read with
//     gfx950's transposing LDS read (ds_read_b64_tr_b8), so staging needs no
//     byte transposes in registers.
constexpr int kTrPitch = kT + 16;          // LDS bytes per k of a k-major step
template <bool KC>
struct StepShare16 {
    static constexpr int kRows = KC ? kT : kSK;
    static constexpr int kRowBytes = KC ? kPitch : kTrPitch;
    uint32_t w[4];

    template <bool AL>
    __device__ __forceinline__ void load(const uint8_t* __restrict__ p, int64_t ld, int r0,
                                         int rows, int k0, int kend, int vec, int vec16,
                                         int tid) {
        if (KC) {
            const bool interior = AL || (r0 + kT <= rows && k0 + kSK <= kend);
            const int r = r0 + (tid >> 4), k = k0 + (tid & 15) * 16;
            if (interior && (AL || vec16)) {
                const uint4 v = *reinterpret_cast<const uint4*>(p + (int64_t)r * ld + k);
                w[0] = v.x, w[1] = v.y, w[2] = v.z, w[3] = v.w;
            } else if (interior && vec) {
                const uint32_t* q = reinterpret_cast<const uint32_t*>(p + (int64_t)r * ld + k);
#pragma unroll
                for (int i = 0; i < 4; ++i) w[i] = q[i];
            } else {
#pragma unroll
                for (int i = 0; i < 4; ++i) w[i] = ld4(p, ld, r, k + 4 * i, rows, kend, vec);
            }
        } else {
            const int k = k0 + (tid >> 2), r = r0 + (tid & 3) * 16;
            const bool interior = AL || (r0 + kT <= rows && k0 + kSK <= kend);
            if (interior && (AL || vec16)) {
                const uint4 v = *reinterpret_cast<const uint4*>(p + (int64_t)k * ld + r);
                w[0] = v.x, w[1] = v.y, w[2] = v.z, w[3] = v.w;
            } else if (interior && vec) {
                const uint32_t* q = reinterpret_cast<const uint32_t*>(p + (int64_t)k * ld + r);
#pragma unroll
                for (int i = 0; i < 4; ++i) w[i] = q[i];
            } else {
#pragma unroll
                for (int i = 0; i < 4; ++i) w[i] = ld4(p, ld, k, r + 4 * i, kend, rows, vec);
            }
        }
    }

    __device__ __forceinline__ void store(uint8_t* lds, int tid) {
        if (KC) {
            const int r = tid >> 4, q = (tid & 15) * 2;
            uint8_t* row = lds + r * kRowBytes;
            *reinterpret_cast<uint2*>(row + slot_off(r, q)) = make_uint2(w[0], w[1]);
            *reinterpret_cast<uint2*>(row + slot_off(r, q + 1)) = make_uint2(w[2], w[3]);
        } else {
            *reinterpret_cast<uint4*>(lds + (tid >> 2) * kRowBytes + (tid & 3) * 16) =
                make_uint4(w[0], w[1], w[2], w[3]);
        }
    }

    // The 8 operand bytes of lane l for the 16x16x32 instruction over k kb ..
    // kb + 31: row r0 + l % 16, k kb + 8 (l / 16) .. +7.  k-major: the
    // transposing read gives lane i of each 16-lane group, as its byte b,
    // byte i % 8 of the 8-byte piece that lane 2 b + i / 8 of the group
    // addresses (b = 0 .. 7; measured on gfx950), so lane l of group
    // g = l / 16 addresses k kb + 8 g + (l % 16) / 2 at row bytes
    // r0 + 8 (l % 2) .. +7.
    __device__ __forceinline__ long operand(const uint8_t* lds, int r0, int kb, int lane) const {
        if (KC) {
            const int r = r0 + (lane & 15);
            const int q = kb / 8 + (lane >> 4);
            return *reinterpret_cast<const long*>(lds + r * kRowBytes + slot_off(r, q));
        } else {
            typedef int v2i __attribute__((ext_vector_type(2)));
            const int s = lane & 15;
            const uint8_t* a = lds + (kb + 8 * (lane >> 4) + (s >> 1)) * kRowBytes + r0 + 8 * (s & 1);
            const v2i v = __builtin_amdgcn_ds_read_tr8_b64_v2i32(
                (__attribute__((address_space(3))) v2i*)(a));
            return (long)(uint32_t)v.x | ((long)(uint32_t)v.y << 32);
        }
    }
};

// Result register r of lane l (32 x 32 block): row 8 (r / 4) + 4 (l / 32) + r % 4,
// column l % 32; operand bytes of lane l: row (or column) l % 32.
__device__ __forceinline__ int res_row(int l, int r) { return 8 * (r / 4) + 4 * (l / 32) + r % 4; }

template <bool TA, bool TB, bool AL>
__global__ __launch_bounds__(kNT) __attribute__((amdgpu_waves_per_eu(4)))
void chunk_gemm_mfma_kx(GemmArgs g, Plan p) {
    __shared__ __attribute__((aligned(16))) uint8_t As[kT][kPitch];
    __shared__ __attribute__((aligned(16))) uint8_t Bs[kT][kPitch];
    // chunk sums of a step: wave w's result register r of lane l at [w][64 r + l]
    __shared__ __attribute__((aligned(16))) float Ps[kNT / 64][16 * 64];
    __shared__ __attribute__((aligned(16))) uint16_t Os[kT * kT];
    __shared__ int redo[kRedoMax];
    __shared__ int n_redo;
    __shared__ uint32_t s_vote[2];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    // wave: chunk wc of the step, quadrant wq (rows 32 (wq / 2), columns 32 (wq % 2))
    const int wc = wave & 3, wq = wave >> 2;
    const int arow = 32 * (wq >> 1) + (lane & 31), bcol = 32 * (wq & 1) + (lane & 31);
    const int kq = kCL * wc + 32 * (lane >> 5);
    // the 4 outputs a thread adds up: quadrant cq, slots 4 u .. 4 u + 3 of its
    // waves' Ps (u = tid % 256), i.e. result register u / 16 of lanes 4 (u % 16) + i
    const int cq = tid >> 8, u = tid & 255;
    const int sr = u >> 4, sl = 4 * (u & 15);
    const int orow0 = 32 * (cq >> 1), ocol0 = 32 * (cq & 1);
    if (tid == 0) {
        n_redo = g.guarded ? 0 : kRedoMax + 1;
        s_vote[0] = s_vote[1] = 0u;
    }
    int vslot = 0;

    StepShare<!TA> sa[2];          // A is k-contiguous unless transposed
    StepShare<TB> sb[2];           // B is k-contiguous only when transposed
    float S[4];
    float vmax = 0.0f;
    const v16f zero = {};
    const int nch = p.nch;
    const int nsteps = (nch + kWaves - 1) / kWaves;

    auto tile_origin = [&](int64_t t, int& m0, int& n0) __attribute__((always_inline)) {
        int tr, tc;
        tile_rc(p, whole_tile(p, t), tr, tc);
        m0 = tr * kT;
        n0 = tc * kT;
    };
    auto load = [&](StepShare<!TA>& ra, StepShare<TB>& rb, int m0, int n0, int k0)
                    __attribute__((always_inline)) {
        ra.template load<AL>(g.A, g.lda, m0, g.M, k0, g.K, g.a_vec, g.a_vec16, tid);
        rb.template load<AL>(g.B, g.ldb, n0, g.N, k0, g.K, g.b_vec, g.b_vec16, tid);
    };
    auto store = [&](StepShare<!TA>& ra, StepShare<TB>& rb) __attribute__((always_inline)) {
        ra.store(As, tid);
        rb.store(Bs, tid);
    };

    // Wave w's chunk of step s: one instruction over its 64 k (zeros past K),
    // the sum rounded to FP16 and left in Ps.  Lane half h carries k
    // 32 h .. 32 h + 31 of both operands: the instruction sums over all 64 k,
    // so only the pairing of A and B bytes matters.
    auto chunk_sum = [&](auto safe_tag, int s) __attribute__((always_inline)) {
        constexpr bool SAFE = decltype(safe_tag)::value;
        if (!AL && s * kWaves + wc >= nch) return;
        v8i a8, b8;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const long av = *reinterpret_cast<const long*>(&As[arow][slot_off(arow, kq / 8 + j)]);
            const long bv = *reinterpret_cast<const long*>(&Bs[bcol][slot_off(bcol, kq / 8 + j)]);
            a8[2 * j] = (int)av;
            a8[2 * j + 1] = (int)(av >> 32);
            b8[2 * j] = (int)bv;
            b8[2 * j + 1] = (int)(bv >> 32);
        }
        // format selectors 1, 1: both operands bf8 (= the FP8 codes); no scaling
        const v16f acc = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a8, b8, zero, 1, 1, 0, 0,
                                                                        0, 0);
        float* dst = &Ps[wave][lane];
        float pr[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            pr[r] = SAFE ? rn16s(acc[r] * 0x1p96f) : rn16v(acc[r]);
            dst[64 * r] = pr[r];
        }
    };

    // The running sums of the thread's 4 outputs over the step's chunks, in
    // chunk order.
    auto chain = [&](auto safe_tag, int s) __attribute__((always_inline)) {
        constexpr bool SAFE = decltype(safe_tag)::value;
        const int nv = AL ? kWaves : min(kWaves, nch - s * kWaves);
        float4 pvs[kWaves];
        if (AL) {
#pragma unroll
            for (int c = 0; c < kWaves; ++c)
                pvs[c] = *reinterpret_cast<const float4*>(&Ps[4 * cq + c][64 * sr + sl]);
        }
#pragma unroll
        for (int c = 0; c < kWaves; ++c) {
            if (c >= nv) break;
            const float4 pv =
                AL ? pvs[c] : *reinterpret_cast<const float4*>(&Ps[4 * cq + c][64 * sr + sl]);
            const float pp[4] = {pv.x, pv.y, pv.z, pv.w};
#pragma unroll
            for (int i = 0; i < 4; ++i) S[i] = SAFE ? rn16s(S[i] + pp[i]) : rn16v(S[i] + pp[i]);
            if (!SAFE) {
                vmax = max3_abs(vmax, S[0], S[1]);
                vmax = max3_abs(vmax, S[2], S[3]);
            }
        }
    };

    // The finished tile: FP16 codes through Os, 16-byte rows to C (and the
    // FP8 result to C8).  Os is free: its previous readers finished before
    // the barrier that ended at least one step since.
    auto write_tile = [&](auto safe_tag, int m0, int n0) __attribute__((always_inline)) {
        constexpr int DOM = decltype(safe_tag)::value ? 96 : 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int l = sl + i;
            Os[(orow0 + res_row(l, sr)) * kT + ocol0 + (l & 31)] = fp16_code<DOM>(S[i]);
        }
        __syncthreads();
        if (tid < kT * kT / 8) {
            const int row = tid >> 3, col = (tid & 7) * 8;
            const int m = m0 + row, n = n0 + col;
            if (m < g.M) {
                const uint4 v = *reinterpret_cast<const uint4*>(&Os[row * kT + col]);
                const uint32_t cw[4] = {v.x, v.y, v.z, v.w};
                if (g.C) {
                    uint16_t* cp = g.C + (int64_t)m * g.ldc + n;
                    if (g.c_vec16 && n + 8 <= g.N) {
                        *reinterpret_cast<uint4*>(cp) = v;
                    } else {
#pragma unroll
                        for (int e = 0; e < 8; ++e)
                            if (n + e < g.N) cp[e] = (uint16_t)(cw[e / 2] >> (16 * (e % 2)));
                    }
                }
                if (g.C8) {
                    auto val = [&](int e) __attribute__((always_inline)) {
                        return fp16_to_f32((cw[e / 2] >> (16 * (e % 2))) & 0xFFFFu) * g.q_scale;
                    };
                    uint2 v8;
                    v8.x = f32x2_to_fp8x2<true>(val(2), val(3),
                                               f32x2_to_fp8x2<false>(val(0), val(1), 0u));
                    v8.y = f32x2_to_fp8x2<true>(val(6), val(7),
                                               f32x2_to_fp8x2<false>(val(4), val(5), 0u));
                    uint8_t* qp = g.C8 + (int64_t)m * g.ldc8 + n;
                    if (g.c8_vec8 && n + 8 <= g.N) {
                        *reinterpret_cast<uint2*>(qp) = v8;
                    } else {
#pragma unroll
                        for (int e = 0; e < 8; ++e)
                            if (n + e < g.N)
                                qp[e] = (uint8_t)((e < 4 ? v8.x : v8.y) >> (8 * (e % 4)));
                    }
                }
            }
        }
    };

    // ---- the stream (guarded epilogue): steps of the workgroup's tiles in
    // order.  The current step is consumed from LDS while the next one waits
    // in one register set and the one after it is loaded into the other, so
    // a load has two steps to arrive ----
    const int64_t T = p.t_whole;
    struct Pos {
        int64_t t;                   // work item (tile t of the workgroup's sequence)
        int s, m0, n0;               // step within the tile, tile origin
    };
    auto step_next = [&](Pos& q) __attribute__((always_inline)) {
        if (++q.s >= nsteps) {
            q.t += p.G;
            q.s = 0;
            if (q.t < T) tile_origin(q.t, q.m0, q.n0);
        }
    };
    if (g.guarded && (int64_t)blockIdx.x < T && nsteps > 0) {
        Pos cur;
        cur.t = blockIdx.x;
        cur.s = 0;
        tile_origin(cur.t, cur.m0, cur.n0);
        load(sa[0], sb[0], cur.m0, cur.n0, 0);
        store(sa[0], sb[0]);
        __syncthreads();
        Pos p1 = cur, p2;
        step_next(p1);
        if (p1.t < T) load(sa[0], sb[0], p1.m0, p1.n0, p1.s * kSK);
        p2 = p1;
        if (p2.t < T) step_next(p2);
        int ordinal = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) S[i] = 0.0f;
        // One step; register set Q holds step p1.
        auto body = [&](auto q_tag) __attribute__((always_inline)) -> bool {
            constexpr int Q = decltype(q_tag)::value;
            if (AL) {
                // past the last step, reload the current one (never stored)
                const Pos& lp = p2.t < T ? p2 : cur;
                load(sa[Q ^ 1], sb[Q ^ 1], lp.m0, lp.n0, lp.s * kSK);
            } else if (p2.t < T) {
                load(sa[Q ^ 1], sb[Q ^ 1], p2.m0, p2.n0, p2.s * kSK);
            }
            chunk_sum(std::integral_constant<bool, false>{}, cur.s);
            __syncthreads();                     // Ps written, As / Bs consumed
            chain(std::integral_constant<bool, false>{}, cur.s);
            if (cur.s + 1 == nsteps) {
                // tile end: the guard over the whole workgroup
                // running sums below 2^31 at every chunk end (see chain), and
                // no Inf/NaN operand: the guarded rounding turns an Inf chunk
                // sum into NaN, which stays in the running sum to the end and
                // which v_max3 drops, so the final sums are compared
                bool bad_l = !(vmax < 2147483648.0f);
#pragma unroll
                for (int i = 0; i < 4; ++i) bad_l |= !(fabsf(S[i]) < 2147483648.0f);
                const bool bad = block_any(bad_l, s_vote, vslot);
                if (bad) {
                    if (tid == 0) {
                        if (n_redo < kRedoMax) redo[n_redo] = ordinal;
                        ++n_redo;
                    }
                } else {
                    write_tile(std::integral_constant<bool, false>{}, cur.m0, cur.n0);
                }
                vmax = 0.0f;
#pragma unroll
                for (int i = 0; i < 4; ++i) S[i] = 0.0f;
                ++ordinal;
            }
            if (p1.t >= T) return false;
            store(sa[Q], sb[Q]);
            __syncthreads();                     // As / Bs written, Ps read
            cur = p1;
            p1 = p2;
            if (p2.t < T) step_next(p2);
            return true;
        };
        for (;;) {
            if (!body(std::integral_constant<int, 0>{})) break;
            if (!body(std::integral_constant<int, 1>{})) break;
        }
    }

    // ---- tiles that failed the guard (all of them when it is off, or when
    // more failed than the list holds), recomputed in the 2^96 domain ----
    __syncthreads();
    const int nr = n_redo;
    if (nr == 0 || nsteps == 0) return;
    int ord = 0, next_listed = 0;
    for (int64_t u = blockIdx.x; u < T; u += p.G, ++ord) {
        const bool listed = nr > kRedoMax || (next_listed < nr && redo[next_listed] == ord);
        if (!listed) continue;
        if (nr <= kRedoMax) ++next_listed;
        int m0, n0;
        tile_origin(u, m0, n0);
#pragma unroll
        for (int i = 0; i < 4; ++i) S[i] = 0.0f;
        for (int s = 0; s < nsteps; ++s) {
            load(sa[0], sb[0], m0, n0, s * kSK);
            __syncthreads();                     // As / Bs consumed, Ps read
            store(sa[0], sb[0]);
            __syncthreads();
            chunk_sum(std::integral_constant<bool, true>{}, s);
            __syncthreads();
            chain(std::integral_constant<bool, true>{}, s);
        }
        __syncthreads();                         // Os readers of the previous tile are done
        write_tile(std::integral_constant<bool, true>{}, m0, n0);
    }
}

// ---------------------------------------------------------------------------
// The same work cut per wave instead of per chunk: wave w of the workgroup
// owns the 16 x 16 block (w / 4, w % 4) of the 64 x 64 tile over the whole
// K, so each output's running sum stays in the registers of the lane that
// forms it and no chunk sum crosses LDS.  A chunk of 64 products is two
// v_mfma_f32_16x16x32_bf8_bf8 (k 0..31, then 32..63, accumulated from zero),
// the instruction sequence of the 16 x 16 block kernel (gemm_mfma.hip), so
// the bits are that kernel's.  A step's operands (64 rows of A and 64
// columns of B by 256 k) are staged as above into one of two LDS buffers: the
// next step's bytes are stored into the other buffer while this step's chunk
// sums are formed, and one barrier per step orders the two.
// ---------------------------------------------------------------------------
typedef float v4f __attribute__((ext_vector_type(4)));

template <bool TA, bool TB, bool AL>
__global__ __launch_bounds__(kNT) __attribute__((amdgpu_waves_per_eu(4)))
void chunk_gemm_mfma_kx16(GemmArgs g, Plan p) {
    typedef StepShare16<!TA> ShareA;  // A is k-contiguous unless transposed
    typedef StepShare16<TB> ShareB;   // B is k-contiguous only when transposed
    __shared__ __attribute__((aligned(16))) uint8_t As[2][ShareA::kRows * ShareA::kRowBytes];
    __shared__ __attribute__((aligned(16))) uint8_t Bs[2][ShareB::kRows * ShareB::kRowBytes];
    __shared__ __attribute__((aligned(16))) uint16_t Os[kT * kT];
    __shared__ int redo[kRedoMax];
    __shared__ int n_redo;
    __shared__ uint32_t s_vote[2];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    // the wave's block: rows 16 bi .., columns 16 bj ..; lane l holds operand
    // row (column) l % 16, k bytes 8 (l / 16) .. +7 of each 32-k instruction,
    // and results at rows 4 (l / 16) + r, column l % 16 of the block
    const int bi = wave >> 2, bj = wave & 3;
    const int kg = lane >> 4;
    const int orow = 16 * bi + 4 * kg, ocol = 16 * bj + (lane & 15);
    if (tid == 0) {
        n_redo = g.guarded ? 0 : kRedoMax + 1;
        s_vote[0] = s_vote[1] = 0u;
    }
    int vslot = 0;

    ShareA sa;
    ShareB sb;
    float S[4];
    float vmax = 0.0f;
    const v4f zero = {};
    const int nch = p.nch;
    const int nsteps = (nch + kWaves - 1) / kWaves;

    auto tile_origin = [&](int64_t t, int& m0, int& n0) __attribute__((always_inline)) {
        int tr, tc;
        tile_rc(p, whole_tile(p, t), tr, tc);
        m0 = tr * kT;
        n0 = tc * kT;
    };
    auto load = [&](int m0, int n0, int k0) __attribute__((always_inline)) {
        sa.template load<AL>(g.A, g.lda, m0, g.M, k0, g.K, g.a_vec, g.a_vec16, tid);
        sb.template load<AL>(g.B, g.ldb, n0, g.N, k0, g.K, g.b_vec, g.b_vec16, tid);
    };
    auto store = [&](int buf) __attribute__((always_inline)) {
        sa.store(As[buf], tid);
        sb.store(Bs[buf], tid);
    };

    // The step's chunk sums of the wave's block (chunks past K are not formed).
    auto chunk_sums = [&](int buf, int s, v4f (&acc)[kWaves]) __attribute__((always_inline)) {
#pragma unroll
        for (int c = 0; c < kWaves; ++c) {
            acc[c] = zero;
            if (!AL && s * kWaves + c >= nch) continue;
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int kb = kCL * c + 32 * h;
                const long av = sa.operand(As[buf], 16 * bi, kb, lane);
                const long bv = sb.operand(Bs[buf], 16 * bj, kb, lane);
                acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf8_bf8(av, bv, acc[c], 0, 0, 0);
            }
        }
    };
    // Each chunk sum rounded to FP16 and added into the running sums, in
    // chunk order; the guarded path keeps the largest |S| at chunk ends.
    auto chain = [&](auto safe_tag, int s, const v4f (&acc)[kWaves]) __attribute__((always_inline)) {
        constexpr bool SAFE = decltype(safe_tag)::value;
        const int nv = AL ? kWaves : min(kWaves, nch - s * kWaves);
#pragma unroll
        for (int c = 0; c < kWaves; ++c) {
            if (c >= nv) break;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float pr = SAFE ? rn16s(acc[c][r] * 0x1p96f) : rn16v(acc[c][r]);
                S[r] = SAFE ? rn16s(S[r] + pr) : rn16v(S[r] + pr);
            }
            if (!SAFE) {
                vmax = max3_abs(vmax, S[0], S[1]);
                vmax = max3_abs(vmax, S[2], S[3]);
            }
        }
    };

    // The finished tile: FP16 codes through Os, 16-byte rows to C (and the
    // FP8 result to C8).  Os is free: its previous readers finished before
    // the barrier that ended at least one step since.
    // (staging the codes and storing them from Os are split so that the
    // guarded stream's tile-end vote barrier orders the two)
    auto stage_tile = [&](auto safe_tag) __attribute__((always_inline)) {
        constexpr int DOM = decltype(safe_tag)::value ? 96 : 0;
#pragma unroll
        for (int r = 0; r < 4; ++r) Os[(orow + r) * kT + ocol] = fp16_code<DOM>(S[r]);
    };
    auto store_tile = [&](int m0, int n0) __attribute__((always_inline)) {
        if (tid < kT * kT / 8) {
            const int row = tid >> 3, col = (tid & 7) * 8;
            const int m = m0 + row, n = n0 + col;
            if (m < g.M) {
                const uint4 v = *reinterpret_cast<const uint4*>(&Os[row * kT + col]);
                const uint32_t cw[4] = {v.x, v.y, v.z, v.w};
                if (g.C) {
                    uint16_t* cp = g.C + (int64_t)m * g.ldc + n;
                    if (g.c_vec16 && n + 8 <= g.N) {
                        *reinterpret_cast<uint4*>(cp) = v;
                    } else {
#pragma unroll
                        for (int e = 0; e < 8; ++e)
                            if (n + e < g.N) cp[e] = (uint16_t)(cw[e / 2] >> (16 * (e % 2)));
                    }
                }
                if (g.C8) {
                    auto val = [&](int e) __attribute__((always_inline)) {
                        return fp16_to_f32((cw[e / 2] >> (16 * (e % 2))) & 0xFFFFu) * g.q_scale;
                    };
                    uint2 v8;
                    v8.x = f32x2_to_fp8x2<true>(val(2), val(3),
                                               f32x2_to_fp8x2<false>(val(0), val(1), 0u));
                    v8.y = f32x2_to_fp8x2<true>(val(6), val(7),
                                               f32x2_to_fp8x2<false>(val(4), val(5), 0u));
                    uint8_t* qp = g.C8 + (int64_t)m * g.ldc8 + n;
                    if (g.c8_vec8 && n + 8 <= g.N) {
                        *reinterpret_cast<uint2*>(qp) = v8;
                    } else {
#pragma unroll
                        for (int e = 0; e < 8; ++e)
                            if (n + e < g.N)
                                qp[e] = (uint8_t)((e < 4 ? v8.x : v8.y) >> (8 * (e % 4)));
                    }
                }
            }
        }
    };
    auto write_tile = [&](auto safe_tag, int m0, int n0) __attribute__((always_inline)) {
        stage_tile(safe_tag);
        __syncthreads();
        store_tile(m0, n0);
    };

    // ---- the stream (guarded epilogue): steps of the workgroup's tiles in
    // order.  Step cur is consumed from LDS buffer buf while step p1, held in
    // the registers, is stored into the other buffer and step p2 is loaded
    // into the registers ----
    const int64_t T = p.t_whole;
    struct Pos {
        int64_t t;                   // work item (tile t of the workgroup's sequence)
        int s, m0, n0;               // step within the tile, tile origin
    };
    auto step_next = [&](Pos& q) __attribute__((always_inline)) {
        if (++q.s >= nsteps) {
            q.t += p.G;
            q.s = 0;
            if (q.t < T) tile_origin(q.t, q.m0, q.n0);
        }
    };
    if (g.guarded && (int64_t)blockIdx.x < T && nsteps > 0) {
        Pos cur;
        cur.t = blockIdx.x;
        cur.s = 0;
        tile_origin(cur.t, cur.m0, cur.n0);
        load(cur.m0, cur.n0, 0);
        store(0);
        Pos p1 = cur;
        step_next(p1);
        if (p1.t < T) load(p1.m0, p1.n0, p1.s * kSK);
        __syncthreads();
        int buf = 0, ordinal = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) S[i] = 0.0f;
        for (;;) {
            v4f acc[kWaves];
            chunk_sums(buf, cur.s, acc);
            // buffer buf ^ 1 was last read by the previous step, before the
            // barrier that ended it
            Pos p2 = p1;
            if (p1.t < T) {
                store(buf ^ 1);
                step_next(p2);
                if (p2.t < T) load(p2.m0, p2.n0, p2.s * kSK);
            }
            chain(std::integral_constant<bool, false>{}, cur.s, acc);
            if (cur.s + 1 == nsteps) {
                // tile end: the guard over the whole workgroup (running sums
                // below 2^31 at every chunk end; NaN from an Inf operand stays
                // in the running sum and fails the final comparison)
                bool bad_l = !(vmax < 2147483648.0f);
#pragma unroll
                for (int i = 0; i < 4; ++i) bad_l |= !(fabsf(S[i]) < 2147483648.0f);
                // the codes go to Os before the vote (a failed tile's are
                // never stored), whose barrier then orders them for the stores
                stage_tile(std::integral_constant<bool, false>{});
                const bool bad = block_any(bad_l, s_vote, vslot);
                if (bad) {
                    if (tid == 0) {
                        if (n_redo < kRedoMax) redo[n_redo] = ordinal;
                        ++n_redo;
                    }
                } else {
                    store_tile(cur.m0, cur.n0);
                }
                vmax = 0.0f;
#pragma unroll
                for (int i = 0; i < 4; ++i) S[i] = 0.0f;
                ++ordinal;
            }
            if (p1.t >= T) break;
            __syncthreads();                     // buf read, buf ^ 1 written
            buf ^= 1;
            cur = p1;
            p1 = p2;
        }
    }

    // ---- tiles that failed the guard (all of them when it is off, or when
    // more failed than the list holds), recomputed in the 2^96 domain ----
    __syncthreads();
    const int nr = n_redo;
    if (nr == 0 || nsteps == 0) return;
    int ord = 0, next_listed = 0;
    for (int64_t u = blockIdx.x; u < T; u += p.G, ++ord) {
        const bool listed = nr > kRedoMax || (next_listed < nr && redo[next_listed] == ord);
        if (!listed) continue;
        if (nr <= kRedoMax) ++next_listed;
        int m0, n0;
        tile_origin(u, m0, n0);
#pragma unroll
        for (int i = 0; i < 4; ++i) S[i] = 0.0f;
        for (int s = 0; s < nsteps; ++s) {
            load(m0, n0, s * kSK);
            __syncthreads();                     // buffer 0 read by the previous step
            store(0);
            __syncthreads();
            v4f acc[kWaves];
            chunk_sums(0, s, acc);
            chain(std::integral_constant<bool, true>{}, s, acc);
        }
        __syncthreads();                         // Os readers of the previous tile are done
        write_tile(std::integral_constant<bool, true>{}, m0, n0);
    }
}

template <bool AL>
const void* kx16_sel(int ta, int tb) {
    if (!ta && !tb) return reinterpret_cast<const void*>(&chunk_gemm_mfma_kx16<false, false, AL>);
    if (!ta && tb) return reinterpret_cast<const void*>(&chunk_gemm_mfma_kx16<false, true, AL>);
    if (ta && !tb) return reinterpret_cast<const void*>(&chunk_gemm_mfma_kx16<true, false, AL>);
    return reinterpret_cast<const void*>(&chunk_gemm_mfma_kx16<true, true, AL>);
}

template <bool AL>
const void* kx_sel(int ta, int tb) {
    if (!ta && !tb) return reinterpret_cast<const void*>(&chunk_gemm_mfma_kx<false, false, AL>);
    if (!ta && tb) return reinterpret_cast<const void*>(&chunk_gemm_mfma_kx<false, true, AL>);
    if (ta && !tb) return reinterpret_cast<const void*>(&chunk_gemm_mfma_kx<true, false, AL>);
    return reinterpret_cast<const void*>(&chunk_gemm_mfma_kx<true, true, AL>);
}

}  // namespace

const void* mfma_kx_kernel(int ta, int tb) { return kx_sel<false>(ta, tb); }

bool mfma_kx_aligned(const GemmArgs& g) {
    return g.M % kT == 0 && g.N % kT == 0 && g.K % kSK == 0 && g.a_vec16 && g.b_vec16;
}

const void* mfma_kx_kernel_aligned(int ta, int tb) { return kx_sel<true>(ta, tb); }

const void* mfma_kx16_kernel(int ta, int tb) { return kx16_sel<false>(ta, tb); }

const void* mfma_kx16_kernel_aligned(int ta, int tb) { return kx16_sel<true>(ta, tb); }

}  // namespace fp8t
