// chunk_gemm_valu instances for trans_a = 1, trans_b = 0
// (kernel template in gemm_valu_impl.h; one file per layout so the builds run
// in parallel).
#include "gemm_valu_impl.h"

namespace fp8t {

const void* valu_kernel_tn(int cfg, int fast) {
    return valu_impl::kernel_table<true, false>(cfg, fast);
}

}  // namespace fp8t
