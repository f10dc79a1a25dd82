// k_spmm_mfma_f16.hip -- the general matrix-core product for binary16 operands.
#include "k_spmm_mfma.hpp"

nmg_status nmg_internal::spmm_general_f16(const SpmmArgs &a) {
    return launch_mfma<_Float16>(a.L, a.values, a.indices, a.X, a.ldx, a.N, a.Y, a.ldy, a.stream);
}
