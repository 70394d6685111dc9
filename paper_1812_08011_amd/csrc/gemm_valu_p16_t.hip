// chunk_gemm_valu instances with FP16 operands for trans_a = 1
// (kernel template in gemm_valu_impl.h).
#include "gemm_valu_impl.h"

namespace fp8t {

const void* valu_p16_kernel_t(int cfg, int tb) {
    return tb ? valu_impl::kernel_table_p16<true, true>(cfg)
              : valu_impl::kernel_table_p16<true, false>(cfg);
}

}  // namespace fp8t
