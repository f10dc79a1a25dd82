// k_spmm_mfma_f32.hip -- the general matrix-core product for binary32 operands.
#include "k_spmm_mfma.hpp"

nmg_status nmg_internal::spmm_general_f32(const SpmmArgs &a) {
    return launch_mfma<float>(a.L, a.values, a.indices, a.X, a.ldx, a.N, a.Y, a.ldy, a.stream);
}

bool nmg_internal::spmm_general_supported(const nmg_layout *L, int64_t N) {
    return mfma_supported(L, N);
}
