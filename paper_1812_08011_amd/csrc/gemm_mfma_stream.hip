// chunk_gemm fast mode on the matrix cores: the streamed 64 x 64 kernel.
//
// Same arithmetic as chunk_gemm_mfma (gemm_mfma.hip), for CL a multiple of
// 64: each chunk of CL products is summed in FP32 by v_mfma_f32_32x32x64_f8f6f4 with both
// operands bf8 (the FP8 codes are OCP E5M2 = bf8), rounded to FP16 once, and added into the running sum
// in ascending chunk order with FP16 rounding after every add.  The design
// differs in how the work reaches the matrix cores and the VALU:
//   * the register budget allows 4 waves per SIMD (the VALU epilogue, 8
//     full-rate instructions per output per chunk, is the bound; the matrix
//     cores and the memory pipeline need other waves to hide behind);
//   * the workgroup's work items (whole tiles, then its share of the split
//     tiles' chunks, from the plan of gemm_plan.h) form one stream of 64-k
//     slabs: the next slab -- of the same piece or the next one -- is loaded
//     from memory while the current one is consumed, so short pieces (K of a
//     few chunks) do not pay the memory latency once per tile;
//   * only the guarded epilogue (plain values, Veltkamp rounding, running
//     max of |S| at chunk ends) runs in the stream.  A piece in which a
//     running sum reached 2^31 (so a chunk sum or sum may have overflowed
//     FP16) or ended NaN (Inf operands: Veltkamp rounding of Inf gives NaN,
//     which stays) is remembered and recomputed after the stream with the
//     2^96-scaled epilogue (integer rounding on raw bits), which gives the
//     same bits wherever the guarded one is valid.
// Slabs are staged in LDS k-contiguous (operands stored with the row index
// contiguous are transposed 4 x 4 bytes in registers), double-buffered with
// one barrier per slab.  The finished tile's FP16 codes leave through an LDS
// staging tile as 16-byte rows.
#include "fp8t_device.h"
#include "gemm_mfma.h"

namespace fp8t {
namespace {

typedef float v16f __attribute__((ext_vector_type(16)));
typedef int v8i __attribute__((ext_vector_type(8)));

constexpr int kNT = 256;               // 4 waves, 2 x 2 blocks of 32 x 32
constexpr int kB = 64;                 // tile rows = columns = slab k
constexpr int kPitch = kB + 8;         // LDS bytes per operand row
constexpr int kRedoMax = 64;           // failed pieces remembered per workgroup

// Bytes (r, c .. c+3) of a row-major byte matrix (rows x cols valid, leading
// dimension ld); 0 outside.
__device__ __forceinline__ uint32_t load4s(const uint8_t* __restrict__ p, int64_t ld, int r, int c,
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
__device__ __forceinline__ void transpose4(uint32_t d[4]) {
    const uint32_t lo01 = __builtin_amdgcn_perm(d[1], d[0], 0x05010400u);
    const uint32_t hi01 = __builtin_amdgcn_perm(d[1], d[0], 0x07030602u);
    const uint32_t lo23 = __builtin_amdgcn_perm(d[3], d[2], 0x05010400u);
    const uint32_t hi23 = __builtin_amdgcn_perm(d[3], d[2], 0x07030602u);
    d[0] = __builtin_amdgcn_perm(lo23, lo01, 0x05040100u);
    d[1] = __builtin_amdgcn_perm(lo23, lo01, 0x07060302u);
    d[2] = __builtin_amdgcn_perm(hi23, hi01, 0x05040100u);
    d[3] = __builtin_amdgcn_perm(hi23, hi01, 0x07060302u);
}

// One operand's share of a 64 x 64 slab: 16 bytes per thread.
//   KC (k contiguous in memory, element (r, k) at p[r ld + k]): row t / 4,
//     k bytes 16 (t % 4) .. +15 -- one 16-byte or four 4-byte loads;
//   otherwise (element (r, k) at p[k ld + r]): the 4 x 4 block of k rows
//     4 (t / 16) .. +3 and r bytes 4 (t % 16) .. +3, transposed on the way
//     into LDS.
template <bool KC>
struct Share {
    uint32_t w[4];

    __device__ __forceinline__ void load(const uint8_t* __restrict__ p, int64_t ld, int r0,
                                         int rows, int k0, int kend, int vec, int vec16,
                                         bool interior, int tid) {
        if (KC) {
            const int r = r0 + (tid >> 2), k = k0 + (tid & 3) * 16;
            if (interior && vec16) {
                const uint4 v = *reinterpret_cast<const uint4*>(p + (int64_t)r * ld + k);
                w[0] = v.x, w[1] = v.y, w[2] = v.z, w[3] = v.w;
            } else if (interior && vec) {
                const uint32_t* q = reinterpret_cast<const uint32_t*>(p + (int64_t)r * ld + k);
#pragma unroll
                for (int i = 0; i < 4; ++i) w[i] = q[i];
            } else {
#pragma unroll
                for (int i = 0; i < 4; ++i) w[i] = load4s(p, ld, r, k + 4 * i, rows, kend, vec);
            }
        } else {
            const int k = k0 + (tid >> 4) * 4, r = r0 + (tid & 15) * 4;
            if (interior && vec) {
#pragma unroll
                for (int b = 0; b < 4; ++b)
                    w[b] = *reinterpret_cast<const uint32_t*>(p + (int64_t)(k + b) * ld + r);
            } else {
#pragma unroll
                for (int b = 0; b < 4; ++b) w[b] = load4s(p, ld, k + b, r, kend, rows, vec);
            }
        }
    }

    __device__ __forceinline__ void store(uint8_t (*lds)[kPitch], int tid) {
        if (KC) {
            uint8_t* d = &lds[tid >> 2][(tid & 3) * 16];
            *reinterpret_cast<uint2*>(d) = make_uint2(w[0], w[1]);
            *reinterpret_cast<uint2*>(d + 8) = make_uint2(w[2], w[3]);
        } else {
            uint32_t d[4] = {w[0], w[1], w[2], w[3]};
            transpose4(d);
            const int rg = (tid & 15) * 4, kg = (tid >> 4) * 4;
#pragma unroll
            for (int b = 0; b < 4; ++b) *reinterpret_cast<uint32_t*>(&lds[rg + b][kg]) = d[b];
        }
    }
};

// A work item: chunks [c0, c1) of tile `tile`; lt >= 0 marks a split tile.
// Its geometry (first row m0 and column n0, k range [kbeg, kend)) is worked
// out once, when the item is fetched.
struct Item {
    int64_t tile, lt;
    int c0, c1;
    int m0, n0, kbeg, kend;
};

// The workgroup's items in order: whole tiles, then its range of the split
// tiles' chunks (the same decomposition as the other kernels).
struct Work {
    int64_t t, s, e;
    __device__ __forceinline__ void start(const Plan& p, int w) {
        t = w;
        s = p.L > 0 ? (int64_t)w * p.L / p.G : 0;
        e = p.L > 0 ? (int64_t)(w + 1) * p.L / p.G : 0;
    }
    __device__ __forceinline__ bool next(const Plan& p, const GemmArgs& g, Item& it) {
        if (t < p.t_whole) {
            it.tile = whole_tile(p, t);
            it.lt = -1;
            it.c0 = 0;
            it.c1 = p.nch;
            t += p.G;
        } else if (s < e) {
            it.lt = s / p.nch;
            it.c0 = (int)(s - it.lt * p.nch);
            const int64_t c1l = e - it.lt * p.nch;
            it.c1 = c1l < p.nch ? (int)c1l : p.nch;
            it.tile = p.t_whole + it.lt;
            s = it.lt * p.nch + it.c1;
        } else {
            return false;
        }
        int tr, tc;
        tile_rc(p, it.tile, tr, tc);
        it.m0 = tr * kB;
        it.n0 = tc * kB;
        it.kbeg = (int)((int64_t)it.c0 * g.CL);
        const int64_t ke = (int64_t)it.c1 * g.CL;
        it.kend = ke < g.K ? (int)ke : g.K;
        return true;
    }
};

// Result register r of lane l (32 x 32 blocks): row 8 (r / 4) + 4 (l / 32) + r % 4,
// column l % 32; operand bytes of lane l: row (or column) l % 32.
__device__ __forceinline__ int out_row(int l, int r) { return 8 * (r / 4) + 4 * (l / 32) + r % 4; }

template <bool TA, bool TB>
__global__ __launch_bounds__(kNT) __attribute__((amdgpu_waves_per_eu(4)))
void chunk_gemm_mfma_stream(GemmArgs g, Plan p) {
    __shared__ __attribute__((aligned(16))) uint8_t As[2][kB][kPitch];
    __shared__ __attribute__((aligned(16))) uint8_t Bs[2][kB][kPitch];
    __shared__ __attribute__((aligned(16))) uint16_t Os[kB * kB];
    __shared__ int redo[kRedoMax];
    __shared__ int n_redo;
    __shared__ uint32_t s_vote[2];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wy = wave >> 1, wx = wave & 1;
    const int arow = wy * 32 + (lane & 31), bcol = wx * 32 + (lane & 31);
    const int kq = 32 * (lane >> 5);
    // with the guarded epilogue switched off every piece takes the safe one
    if (tid == 0) {
        n_redo = g.guarded ? 0 : kRedoMax + 1;
        s_vote[0] = s_vote[1] = 0u;
    }
    int vslot = 0;

    Share<!TA> sa;                 // A is k-contiguous unless transposed
    Share<TB> sb;                  // B is k-contiguous only when transposed
    v16f acc;
    float S[16];
    float vmax = 0.0f;             // guarded: largest |S| at chunk ends
    bool nonfinite = false;        // guarded: a chunk sum for the fold was not finite
    const v16f zero = {};

    auto geom = [&](const Item& it, int& m0, int& n0, int& kbeg, int& kend)
                    __attribute__((always_inline)) {
        m0 = it.m0;
        n0 = it.n0;
        kbeg = it.kbeg;
        kend = it.kend;
    };
    auto load = [&](const Item& it, int k0) __attribute__((always_inline)) {
        const bool kin = k0 + kB <= it.kend;
        sa.load(g.A, g.lda, it.m0, g.M, k0, it.kend, g.a_vec, g.a_vec16,
                kin && it.m0 + kB <= g.M, tid);
        sb.load(g.B, g.ldb, it.n0, g.N, k0, it.kend, g.b_vec, g.b_vec16,
                kin && it.n0 + kB <= g.N, tid);
    };

    // Chunk end: round the chunk sum and add it into S (or, for a piece that
    // does not start its tile, store it for the fold pass).
    auto chunk_end = [&](auto safe_tag, const Item& it, int m0, int n0, int chunk)
                         __attribute__((always_inline)) {
        constexpr bool SAFE = decltype(safe_tag)::value;
        constexpr int DOM = SAFE ? 96 : 0;
        if (it.c0 > 0) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                float pv;
                if (SAFE) {
                    pv = rn16s(acc[r] * 0x1p96f);
                } else {
                    // Veltkamp rounding turns an Inf sum into NaN
                    pv = rn16v(acc[r]);
                    nonfinite |= !(fabsf(pv) < 2147483648.0f);
                }
                g.ws[ws_index(p, kB, kB, it.lt, chunk, wy * 32 + out_row(lane, r), bcol)] =
                    fp16_code<DOM>(pv);
            }
        } else {
#pragma unroll
            for (int r = 0; r < 16; ++r)
                S[r] = SAFE ? rn16s(S[r] + rn16s(acc[r] * 0x1p96f)) : rn16v(S[r] + rn16v(acc[r]));
            // the guard: running sums at chunk ends (a chunk sum that
            // overflowed shows in them; v_max3 drops NaN, which the check of
            // the final sums catches)
            if (!SAFE) {
#pragma unroll
                for (int r = 0; r < 16; r += 2) vmax = max3_abs(vmax, S[r], S[r + 1]);
            }
        }
        (void)m0;
        (void)n0;
    };

    // The products of one slab (LDS buffer buf, k from ks) of item it.  CL is
    // a multiple of 64, so a chunk ends only at a slab end: a slab is one
    // 32 x 32 x 64 matrix-core instruction per wave (past kend the operands
    // are zero), and crem counts the k left in the current chunk.  The
    // instruction sums over all 64 k of its operands, so which lane half and
    // byte holds which k only has to agree between A and B: lane half h holds
    // k 32 h .. 32 h + 31 of both, in order.
    auto slab = [&](auto safe_tag, const Item& it, int buf, int ks, int& crem, int& chunk)
                    __attribute__((always_inline)) {
        v8i a8, b8;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const long av = *reinterpret_cast<const long*>(&As[buf][arow][kq + 8 * j]);
            const long bv = *reinterpret_cast<const long*>(&Bs[buf][bcol][kq + 8 * j]);
            a8[2 * j] = (int)av;
            a8[2 * j + 1] = (int)(av >> 32);
            b8[2 * j] = (int)bv;
            b8[2 * j + 1] = (int)(bv >> 32);
        }
        // format selectors 1, 1: both operands bf8 (= the FP8 codes); no scaling
        if (crem == g.CL)
            acc = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a8, b8, zero, 1, 1, 0, 0, 0, 0);
        else
            acc = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a8, b8, acc, 1, 1, 0, 0, 0, 0);
        crem -= kB;
        if (crem == 0 || ks + kB >= it.kend) {
            chunk_end(safe_tag, it, it.m0, it.n0, chunk);
            crem = g.CL;
            ++chunk;
        }
    };

    // Piece end: results of a piece that starts its tile (the running sums:
    // C / C8 for a whole tile, C or s_ws for the first piece of a split tile).
    // Staging the codes and storing them from Os are split so that the
    // guarded stream's piece-end vote barrier orders the two.
    auto stage_sums = [&](auto safe_tag) __attribute__((always_inline)) {
        constexpr int DOM = decltype(safe_tag)::value ? 96 : 0;
#pragma unroll
        for (int r = 0; r < 16; ++r)
            Os[(wy * 32 + out_row(lane, r)) * kB + bcol] = fp16_code<DOM>(S[r]);
    };
    auto store_sums = [&](const Item& it) __attribute__((always_inline)) {
        int m0, n0, kbeg, kend;
        geom(it, m0, n0, kbeg, kend);
        const bool keep = it.lt >= 0 && !g.C;
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const int u = tid + kNT * q;
            const int row = u >> 3, col = (u & 7) * 8;
            const uint4 v = *reinterpret_cast<const uint4*>(&Os[row * kB + col]);
            if (keep) {
                *reinterpret_cast<uint4*>(g.s_ws + (it.lt * kB + row) * kB + col) = v;
                continue;
            }
            const int m = m0 + row, n = n0 + col;
            if (m >= g.M) continue;
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
            if (g.C8 && it.lt < 0) {
                auto val = [&](int e) __attribute__((always_inline)) {
                    return fp16_to_f32((cw[e / 2] >> (16 * (e % 2))) & 0xFFFFu) * g.q_scale;
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
        // Os is next written after at least one more barrier
    };
    auto write_sums = [&](auto safe_tag, const Item& it) __attribute__((always_inline)) {
        stage_sums(safe_tag);
        __syncthreads();
        store_sums(it);
    };

    // ---- the stream (guarded epilogue) ----
    // Slab positions in stream order: cur is consumed from LDS while the next
    // slab is in flight in registers.
    Work work;
    work.start(p, blockIdx.x);
    struct Pos {
        Item it;
        int ks;
        int ok;                    // an int: a copy of Pos has no padding bytes (which
                                   // went through scratch memory with a bool here)
    };
    Pos cur;
    cur.ok = g.guarded && work.next(p, g, cur.it);
    if (cur.ok) {
        cur.ks = cur.it.kbeg;
        load(cur.it, cur.ks);
        sa.store(As[0], tid);
        sb.store(Bs[0], tid);
        __syncthreads();
        Pos nx = cur;
        auto adv = [&]() __attribute__((always_inline)) {
            if (nx.ks + kB < nx.it.kend) {
                nx.ks += kB;
            } else {
                nx.ok = work.next(p, g, nx.it);
                nx.ks = nx.it.kbeg;
            }
            if (nx.ok) load(nx.it, nx.ks);
        };
        adv();
        int buf = 0, crem = g.CL, chunk = cur.it.c0, ordinal = 0;
#pragma unroll
        for (int r = 0; r < 16; ++r) S[r] = 0.0f;
        for (;;) {
            slab(std::integral_constant<bool, false>{}, cur.it, buf, cur.ks, crem, chunk);
            if (cur.ks + kB >= cur.it.kend) {
                // piece end: the guard over the whole workgroup
                // running sums below 2^31 at every chunk end: no chunk sum
                // or sum reached FP16's overflow threshold; no Inf/NaN
                // operand (its NaN stays in the running sum to the end)
                bool bad_l = !(vmax < 2147483648.0f) || nonfinite;
#pragma unroll
                for (int r = 0; r < 16; ++r) bad_l |= !(fabsf(S[r]) < 2147483648.0f);
                // the codes go to Os before the vote (a failed piece's are
                // never stored), whose barrier then orders them for the stores
                if (cur.it.c0 == 0) stage_sums(std::integral_constant<bool, false>{});
                const bool bad = block_any(bad_l, s_vote, vslot);
                if (bad) {
                    if (tid == 0) {
                        if (n_redo < kRedoMax) redo[n_redo] = ordinal;
                        ++n_redo;
                    }
                } else if (cur.it.c0 == 0) {
                    store_sums(cur.it);
                }
                vmax = 0.0f;
                nonfinite = false;
#pragma unroll
                for (int r = 0; r < 16; ++r) S[r] = 0.0f;
                crem = g.CL;
                chunk = nx.it.c0;
                ++ordinal;
            }
            if (!nx.ok) break;
            sa.store(As[buf ^ 1], tid);
            sb.store(Bs[buf ^ 1], tid);
            __syncthreads();
            buf ^= 1;
            cur = nx;
            adv();
        }
    }

    // ---- pieces that failed the guard (all of them when it is off, or when
    // more failed than the list holds), recomputed in the 2^96 domain ----
    __syncthreads();
    const int nr = n_redo;
    if (nr == 0) return;
    Work again;
    again.start(p, blockIdx.x);
    Item it;
    int ord = 0, next_listed = 0;
    while (again.next(p, g, it)) {
        const bool listed = nr > kRedoMax || (next_listed < nr && redo[next_listed] == ord);
        ++ord;
        if (!listed) continue;
        if (nr <= kRedoMax) ++next_listed;
        int m0, n0, kbeg, kend;
        geom(it, m0, n0, kbeg, kend);
        int crem = g.CL, chunk = it.c0;
#pragma unroll
        for (int r = 0; r < 16; ++r) S[r] = 0.0f;
        for (int ks = kbeg; ks < kend; ks += kB) {
            load(it, ks);
            __syncthreads();             // every wave is done with buffer 0
            sa.store(As[0], tid);
            sb.store(Bs[0], tid);
            __syncthreads();
            slab(std::integral_constant<bool, true>{}, it, 0, ks, crem, chunk);
        }
        if (it.c0 == 0) {
            __syncthreads();             // Os readers of the previous piece are done
            write_sums(std::integral_constant<bool, true>{}, it);
        }
    }
}

}  // namespace

const void* mfma_stream_kernel(int ta, int tb) {
    if (!ta && !tb) return reinterpret_cast<const void*>(&chunk_gemm_mfma_stream<false, false>);
    if (!ta && tb) return reinterpret_cast<const void*>(&chunk_gemm_mfma_stream<false, true>);
    if (ta && !tb) return reinterpret_cast<const void*>(&chunk_gemm_mfma_stream<true, false>);
    return reinterpret_cast<const void*>(&chunk_gemm_mfma_stream<true, true>);
}

}  // namespace fp8t
