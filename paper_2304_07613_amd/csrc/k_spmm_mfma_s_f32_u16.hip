// k_spmm_mfma_s_f32_u16.hip -- scalar-indexed matrix-core product, binary32,
// group units of 16 rows.
#include "k_spmm_mfma_s.hpp"

nmg_status nmg_internal::spmm_scalar_f32_u16(const SpmmArgs &a) {
    const int tpl = fast_tpl(a.L, a.N);
    if (tpl == 4) return launch_fast_ut<float, 16, 4>(a.L, a.values, a.indices, a.X, a.ldx, a.N, a.Y, a.ldy, a.stream);
    if (tpl == 2) return launch_fast_ut<float, 16, 2>(a.L, a.values, a.indices, a.X, a.ldx, a.N, a.Y, a.ldy, a.stream);
    return launch_fast_ut<float, 16, 1>(a.L, a.values, a.indices, a.X, a.ldx, a.N, a.Y, a.ldy, a.stream);
}
