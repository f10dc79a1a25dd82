// k_spmm_mfma_s_f16.hip -- scalar-indexed matrix-core product, binary16 operands
// (widened to binary32 on the way to LDS), every group unit.
#include "k_spmm_mfma_s.hpp"

namespace {

template <int U>
nmg_status f16_unit(const SpmmArgs &a) {
    const int tpl = fast_tpl(a.L, a.N);
    if (tpl == 4) return launch_fast_ut<_Float16, U, 4>(a.L, a.values, a.indices, a.X, a.ldx, a.N, a.Y, a.ldy, a.stream);
    if (tpl == 2) return launch_fast_ut<_Float16, U, 2>(a.L, a.values, a.indices, a.X, a.ldx, a.N, a.Y, a.ldy, a.stream);
    return launch_fast_ut<_Float16, U, 1>(a.L, a.values, a.indices, a.X, a.ldx, a.N, a.Y, a.ldy, a.stream);
}

}  // namespace

nmg_status nmg_internal::spmm_scalar_f16(const SpmmArgs &a) {
    switch (mfma_unit(a.L) >= 16 ? 16 : mfma_unit(a.L)) {
        case 16: return f16_unit<16>(a);
        case 8: return f16_unit<8>(a);
        case 4: return f16_unit<4>(a);
        default: return NMG_ERR_UNSUPPORTED;
    }
}

bool nmg_internal::spmm_scalar_supported(const nmg_layout *L, const uint8_t *indices,
                                         int64_t ldx) {
    return fast_supported(L, indices, ldx);
}

nmg_status nmg_internal::spmm_scalar(const SpmmArgs &a) {
    if (a.L->dtype == NMG_F16) return spmm_scalar_f16(a);
    switch (mfma_unit(a.L) >= 16 ? 16 : mfma_unit(a.L)) {
        case 16: return spmm_scalar_f32_u16(a);
        case 8: return spmm_scalar_f32_u8(a);
        case 4: return spmm_scalar_f32_u4(a);
        default: return NMG_ERR_UNSUPPORTED;
    }
}
