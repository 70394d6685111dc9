// chunk_gemm_valu instances whose A operand is an implicitly lowered NHWC
// convolution input (trans_a = 0: the Forward GEMM Xcol W; trans_a = 1: the
// Gradient GEMM Xcol^T dY), exact mode, 4 x 4 register tiles.
#include "gemm_valu_impl.h"

namespace fp8t {

const void* valu_conv_kernel(int cfg, int ta) {
    using Q = valu_impl::ValuCfg<4>;
    if (cfg != 4) return nullptr;
    if (!ta)
        return reinterpret_cast<const void*>(&valu_impl::chunk_gemm_valu<
            Q::TM, Q::TN, Q::LM, Q::LN, Q::BK, Q::PF, Q::WPE, false, false, false, true>);
    return reinterpret_cast<const void*>(&valu_impl::chunk_gemm_valu<
        Q::TM, Q::TN, Q::LM, Q::LN, Q::BK, Q::PF, Q::WPE, true, false, false, true>);
}

}  // namespace fp8t
