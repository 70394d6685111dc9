// Matrix-core chunk_gemm kernels of the fast mode (gemm_mfma.hip): tile
// shapes and kernel entry addresses, for the host-side planner in
// chunk_gemm.hip.
#pragma once

#include "gemm_plan.h"

namespace fp8t {

// Workgroup-wide OR of one flag per thread with a single barrier (the fast
// kernels' guard vote at a piece end; __syncthreads_or took three barriers
// and a load of the workgroup size): each wave votes, one lane of a wave
// with a set flag writes 1 into slots[s] (all writers write the same value),
// thread 0 clears the other slot for the next vote, and after the barrier
// every thread reads slots[s]; s alternates.  Both slots start at 0, and a
// caller has at least one barrier between two votes, so the readers of the
// other slot's previous vote are past it when thread 0 clears it.
__device__ __forceinline__ bool block_any(bool flag, uint32_t* slots, int& s) {
    if (__any(flag) && (threadIdx.x & 63) == 0) slots[s] = 1u;
    if (threadIdx.x == 0) slots[s ^ 1] = 0u;
    __syncthreads();
    const bool r = slots[s] != 0u;
    s ^= 1;
    return r;
}

struct MfmaShape {
    int BW;         // MFMA block (32: 32x32x16, 16: 16x16x32)
    int BM, BN;     // outputs per workgroup
    int NT;         // threads per workgroup
    int kstep;      // products per instruction: CL must be a multiple
    int BK;         // k per LDS slab
};

constexpr int kMfmaConfigs = 6;

MfmaShape mfma_shape(int cfg);

// __global__ function of configuration cfg (0 .. kMfmaConfigs-1) for the
// given operand layouts, taking (GemmArgs, Plan).
const void* mfma_kernel(int cfg, int ta, int tb);

// The streamed 64 x 64 kernel (gemm_mfma_stream.hip), configuration 2.
const void* mfma_stream_kernel(int ta, int tb);

// 64 x 64 tiles with a step's four chunks spread over the workgroup's 16 waves
// (gemm_mfma_kx.hip), configuration 3: CL = 64 only, whole tiles only.
const void* mfma_kx_kernel(int ta, int tb);
// Its variant for M and N multiples of 64, K a multiple of 256 and 16-byte
// loads of both operands (mfma_kx_aligned): one load path, deeper prefetch.
bool mfma_kx_aligned(const GemmArgs& g);
const void* mfma_kx_kernel_aligned(int ta, int tb);

// The same tiles with each of the 16 waves owning a 16 x 16 block over the
// whole K (gemm_mfma_kx.hip), configuration 4: CL = 64 only, whole tiles
// only; its aligned variant under the same conditions.
const void* mfma_kx16_kernel(int ta, int tb);
const void* mfma_kx16_kernel_aligned(int ta, int tb);

// 32 x 128 tiles, each of the 4 waves streaming its own 32 x 32 block with
// no workgroup barrier (gemm_mfma_wave.hip), configuration 5: CL a multiple
// of 64, whole tiles only, A k-contiguous (trans_a = 0) and 16-byte loads of
// A and of a k-contiguous B (B itself when trans_b = 1, else the copy
// launch_transpose_bytes makes), leading dimensions below 2^26; nullptr for
// trans_a = 1.
const void* mfma_wave_kernel(int ta);
// Bt[n * ldt + k] = B[k * ldb + n] for k < K, n < N, on `stream` (Bt 16-byte
// aligned, ldt a multiple of 16).
void launch_transpose_bytes(const uint8_t* B, int64_t ldb, int K, int N, uint8_t* Bt, int64_t ldt,
                            hipStream_t stream);

}  // namespace fp8t
