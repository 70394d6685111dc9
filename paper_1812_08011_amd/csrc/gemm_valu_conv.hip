// chunk_gemm_valu instances whose A operand is an implicitly lowered NHWC
// convolution input (trans_a = 0: the Forward GEMM Xcol W; trans_a = 1: the
// Gradient GEMM Xcol^T dY), exact mode, 4 x 4 register tiles on 64 x 64
// (configuration 4) or 128 x 64 (configuration 7) workgroup tiles.
#include "gemm_valu_impl.h"

namespace fp8t {
namespace {

template <int C>
const void* conv_kernel_of(int ta) {
    using Q = valu_impl::ValuCfg<C>;
    if (!ta)
        return reinterpret_cast<const void*>(&valu_impl::chunk_gemm_valu<
            Q::TM, Q::TN, Q::LM, Q::LN, Q::BK, Q::PF, Q::WPE, false, false, false, true>);
    return reinterpret_cast<const void*>(&valu_impl::chunk_gemm_valu<
        Q::TM, Q::TN, Q::LM, Q::LN, Q::BK, Q::PF, Q::WPE, true, false, false, true>);
}

}  // namespace

const void* valu_conv_kernel(int cfg, int ta) {
    if (cfg == 4) return conv_kernel_of<4>(ta);
    if (cfg == 7) return conv_kernel_of<7>(ta);
    return nullptr;
}

}  // namespace fp8t
