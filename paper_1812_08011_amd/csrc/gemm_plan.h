// Work decomposition shared by the chunk_gemm kernels.
//
// The output is cut into BM x BN tiles numbered row-major (t = tm * tiles_n +
// tn).  A tile's K range is cut into nch chunks of CL products starting at
// k = 0 (Sec. 2.3: chunks are independent until their sums are added, in
// order, into the running sum).  A launch has G workgroups:
//
//   * tiles [0, t_whole) are processed whole, workgroup w taking tiles
//     w, w + G, w + 2G, ...: the chunk sums go straight into the running sum
//     and the FP16 result into C;
//   * the remaining T - t_whole tiles, laid end to end as L = (T - t_whole) *
//     nch tile-chunks, are shared out as contiguous ranges
//     [w * L / G, (w + 1) * L / G), so every workgroup ends with the same
//     number of chunks.  A range piece that starts at chunk 0 of its tile
//     writes the running sum of its chunks to C; a piece that starts later
//     writes each chunk's FP16 sum to the workspace (ws_index), and
//     chunk_fold then continues the running sum from C over those chunk sums
//     in ascending order.  The additions are the same ones, in the same order, as when a
//     tile is processed whole, so the result does not depend on the plan.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fp8t {

// Implicit lowering of a convolution (Sec. 2.2: a convolution is computed by
// lowering its input and then a GEMM): the lowered matrix Xcol, M = N * OH *
// OW rows (output pixels, row-major n, oh, ow) by KH * KW * C columns (order
// kh, kw, c), is read straight from the NHWC input X:
//   Xcol(p, (kh, kw, c)) = X[n, oh * stride - pad + kh, ow * stride - pad + kw, c]
// (0 outside the image).
struct ConvGeom {
    int H, W, C;        // input height, width, channels
    int KW, KWC;        // kernel width, KW * C
    int OW, OHW;        // output width, OH * OW
    int pad, stride;
    int vec;            // C % 4 == 0 and X 4-byte aligned: 4 channels per load
};

struct GemmArgs {
    const uint8_t* A;
    const uint8_t* B;
    uint16_t* C;        // FP16 result (may be null when C8 is set)
    uint16_t* ws;       // chunk sums of the shared tiles (null when L == 0)
    uint16_t* s_ws;     // running sums of the shared tiles' first pieces when C is null
    uint8_t* C8;        // FP8 result Q8(value * q_scale), or null
    int64_t ldc8;
    float q_scale;
    int64_t lda, ldb, ldc;
    int M, N, K, CL;
    int a_vec;          // A, lda allow 4-byte loads (and lda < 2^24)
    int b_vec;          // B, ldb allow 4-byte loads (and ldb < 2^24)
    int a_vec16;        // A, lda allow 16-byte loads
    int b_vec16;        // B, ldb allow 16-byte loads
    int c_vec;          // C, ldc allow 4-byte stores of code pairs
    int c_vec8;         // C, ldc allow 8-byte stores (4 codes)
    int c_vec16;        // C, ldc allow 16-byte stores (8 codes)
    int c8_vec8;        // C8, ldc8 allow 8-byte stores
    int c8_vec4;        // C8, ldc8 allow 4-byte stores
    int guarded;        // exact mode: try the guarded path first
    ConvGeom conv;      // A is the implicit lowering of an NHWC input (conv kernels)
};

struct Plan {
    int64_t tiles_n;
    int64_t t_whole;
    int64_t L;          // tile-chunks shared out
    int nch;            // chunks per tile
    int G;              // workgroups
    int xcd_remap;      // whole tiles are grouped by XCD (see whole_tile)
};

// Tile of whole-tile work item t.  Workgroups are dealt to the 8 XCDs of the
// chip round-robin (workgroup w runs on XCD w % 8), and with G a multiple of 8
// item t runs on XCD t % 8.  With xcd_remap, XCD x gets the contiguous range
// of row-major tiles [x * t_whole / 8, (x + 1) * t_whole / 8): tiles that
// share operand rows then share that XCD's L2.
__host__ __device__ inline int64_t whole_tile(const Plan& p, int64_t t) {
    if (!p.xcd_remap) return t;
    return (t % 8) * (p.t_whole / 8) + t / 8;
}

// Row and column of tile `tile` in the row-major tile grid.  The tile index
// of any output that fits in device memory is below 2^32, where a 32-bit
// division is a fraction of the 64-bit instruction sequence (a per-tile cost
// on the scalar unit); the 64-bit form stays for the rest.
__host__ __device__ inline void tile_rc(const Plan& p, int64_t tile, int& tr, int& tc) {
    if ((uint64_t)tile < (1ull << 32) && (uint64_t)p.tiles_n < (1ull << 32)) {
        const uint32_t t = (uint32_t)tile, n = (uint32_t)p.tiles_n, q = t / n;
        tr = (int)q;
        tc = (int)(t - q * n);
    } else {
        const int64_t q = tile / p.tiles_n;
        tr = (int)q;
        tc = (int)(tile - q * p.tiles_n);
    }
}

// Workspace index of the chunk sum of chunk `chunk` of output (r, c) of
// shared tile lt (BM x BN tiles, BM a multiple of 4): the tile's rows in
// bands of 4, each band's sums of one chunk a run of 4 BN codes, the runs of
// a band in chunk order.  The fold pass, one wave per band, then reads each
// band's successive chunks from consecutive memory.
__host__ __device__ inline int64_t ws_index(const Plan& p, int BM, int BN, int64_t lt, int chunk,
                                            int r, int c) {
    return ((lt * (BM / 4) + r / 4) * p.nch + chunk) * (int64_t)(4 * BN) + (r % 4) * BN + c;
}

// First chunk of shared tile lt that the workspace holds: the end of the
// piece that starts at the tile's chunk 0 (nch if the tile is not split).
__host__ __device__ inline int first_piece_end(const Plan& p, int64_t lt) {
    const int64_t x = lt * p.nch;                       // tile start
    const int64_t w0 = ((x + 1) * p.G - 1) / p.L;       // range holding x
    const int64_t e = (w0 + 1) * p.L / p.G;             // its end
    const int64_t a = e - x;
    return a < p.nch ? (int)a : p.nch;
}

}  // namespace fp8t
