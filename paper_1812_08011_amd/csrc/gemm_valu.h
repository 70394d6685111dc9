// Vector-ALU chunk_gemm kernels (gemm_valu.hip): register-tile shapes and
// kernel entry addresses, for the host-side planner in chunk_gemm.hip.
#pragma once

#include "gemm_plan.h"

namespace fp8t {

struct ValuShape {
    int TM, TN;     // outputs per lane
    int BM, BN;     // outputs per workgroup
    int NT;         // threads per workgroup
};

// Configurations 0-8 are chunk_gemm_valu register tiles (gemm_valu_impl.h);
// configurations 9, 10, 11 are chunk_gemm_chain (gemm_chain.hip) with 2 x 2,
// 1 x 2 and 1 x 1 outputs per lane: whole tiles, CL a multiple of 4 or
// covering K.
constexpr int kValuConfigs = 12;
constexpr int kChainConfig = 9;
inline bool is_chain(int cfg) { return cfg >= kChainConfig && cfg < kChainConfig + 3; }

ValuShape valu_shape(int cfg);

// __global__ function of register-tile configuration cfg (0 .. kValuConfigs-1)
// for the given operand layouts and mode (fast: sum a chunk in FP32 and round
// once), taking (GemmArgs, Plan); null where that variant is not built (the
// fast variants exist for the small tiles only: the fast mode runs here only
// for chunk lengths the matrix cores cannot split).
const void* valu_kernel(int cfg, int ta, int tb, int fast);

// Kernel of configuration cfg with FP16 operands (chunk_gemm_p16: products
// rounded to FP16, exact mode); null where not built (configurations 4-8).
const void* valu_p16_kernel(int cfg, int ta, int tb);

// Exact-mode kernel of configuration cfg whose A operand is an implicitly
// lowered convolution input (GemmArgs::conv); trans_b = 0; null where not
// built (only configuration 4).
const void* valu_conv_kernel(int cfg, int ta);

// chunk_gemm_chain with 2 x 2 (shape 0), 1 x 2 (1) or 1 x 1 (2) outputs per
// lane for the given operand layouts and mode (fast: sum a chunk in FP32 and
// round once) (gemm_chain.hip).
const void* chain_kernel(int shape, int ta, int tb, int fast);

}  // namespace fp8t
