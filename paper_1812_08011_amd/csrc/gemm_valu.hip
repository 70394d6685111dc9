// Dispatch tables of the vector-ALU chunk_gemm kernels (gemm_valu_impl.h).
#include "gemm_valu_impl.h"

namespace fp8t {

const void* valu_kernel_nn(int cfg, int fast);
const void* valu_kernel_nt(int cfg, int fast);
const void* valu_kernel_tn(int cfg, int fast);
const void* valu_kernel_tt(int cfg, int fast);
const void* valu_p16_kernel_n(int cfg, int tb);
const void* valu_p16_kernel_t(int cfg, int tb);

ValuShape valu_shape(int cfg) {
    switch (cfg) {
        case 0: return valu_impl::shape_of<0>();
        case 1: return valu_impl::shape_of<1>();
        case 2: return valu_impl::shape_of<2>();
        case 3: return valu_impl::shape_of<3>();
        case 4: return valu_impl::shape_of<4>();
        case 5: return valu_impl::shape_of<5>();
        case 7: return valu_impl::shape_of<7>();
        case 8: return valu_impl::shape_of<8>();
        case kChainConfig: return ValuShape{2, 2, 32, 32, 256};
        case kChainConfig + 1: return ValuShape{1, 2, 16, 32, 256};
        case kChainConfig + 2: return ValuShape{1, 1, 16, 16, 256};
        default: return valu_impl::shape_of<6>();
    }
}

const void* valu_kernel(int cfg, int ta, int tb, int fast) {
    if (cfg < 0 || cfg >= kValuConfigs) return nullptr;
    if (is_chain(cfg)) return chain_kernel(cfg - kChainConfig, ta, tb, fast);
    if (!ta && !tb) return valu_kernel_nn(cfg, fast);
    if (!ta && tb) return valu_kernel_nt(cfg, fast);
    if (ta && !tb) return valu_kernel_tn(cfg, fast);
    return valu_kernel_tt(cfg, fast);
}

const void* valu_p16_kernel(int cfg, int ta, int tb) {
    if (cfg < 0 || cfg >= kValuConfigs || is_chain(cfg)) return nullptr;
    return ta ? valu_p16_kernel_t(cfg, tb) : valu_p16_kernel_n(cfg, tb);
}

}  // namespace fp8t
