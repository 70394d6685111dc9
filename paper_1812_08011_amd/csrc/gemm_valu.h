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

constexpr int kValuConfigs = 9;

ValuShape valu_shape(int cfg);

// __global__ function of register-tile configuration cfg (0 .. kValuConfigs-1)
// for the given operand layouts and mode (fast: sum a chunk in FP32 and round
// once), taking (GemmArgs, Plan); null where that variant is not built (the
// fast variants exist for the small tiles only: the fast mode runs here only
// for chunk lengths the matrix cores cannot split).
const void* valu_kernel(int cfg, int ta, int tb, int fast);

// Exact-mode kernel of configuration cfg whose A operand is an implicitly
// lowered convolution input (GemmArgs::conv); trans_b = 0; null where not
// built (only configuration 4).
const void* valu_conv_kernel(int cfg, int ta);

}  // namespace fp8t
