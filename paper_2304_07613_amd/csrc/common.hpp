// common.hpp -- shared by the translation units of libnmg: host-side helpers
// and the internal launcher interface (namespace nmg_internal), and device
// helpers (one private copy per translation unit).
//
// Paper: STen (arXiv 2304.07613), Section 5.  The layout, selection rule and
// product are specified in include/nmg.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <atomic>
#include <type_traits>
#include <utility>

#include "nmg.h"

namespace nmg_internal {

inline nmg_status check_layout(const nmg_layout *L) {
    if (!L) return NMG_ERR_NULL;
    if (L->dtype != NMG_F32 && L->dtype != NMG_F16) return NMG_ERR_DTYPE;
    if (L->M < 1 || L->K < 1 || L->n < 1 || L->m < L->n || L->m > 255 || L->g < 1)
        return NMG_ERR_PARAM;
    if (L->M % L->g != 0) return NMG_ERR_SHAPE;
    const int32_t C = (L->K + L->m - 1) / L->m;
    if (L->C != C) return NMG_ERR_PARAM;
    if (L->K - (C - 1) * L->m < L->n) return NMG_ERR_SHAPE;
    return NMG_OK;
}

inline size_t elem_size(nmg_dtype d) { return d == NMG_F32 ? 4 : 2; }

inline bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

// X rows start on 4-element boundaries: four tokens come in one vector load.
inline bool x_vectorisable(const nmg_layout *L, const void *X, int64_t ldx) {
    return aligned(X, 4 * elem_size(L->dtype)) && ldx % 4 == 0;
}

// A launch's status is read right after it with hipGetLastError.  Each entry
// point first clears whatever error earlier runtime calls on the thread left
// pending (prelaunch), so that such an error is not reported as the failure
// of this library's launch; the host queries the launchers make on the way
// (device_cus, kernel_occupancy) clear their own errors.
inline void prelaunch() { (void)hipGetLastError(); }
inline nmg_status launched() {
    return hipGetLastError() == hipSuccess ? NMG_OK : NMG_ERR_LAUNCH;
}

// Rows per group unit of the matrix-core kernels: the largest of 32, 16, 8,
// 4 that divides g; 0 if g % 4 != 0.
inline int mfma_unit(const nmg_layout *L) {
    for (int u = 32; u >= 4; u /= 2)
        if (L->g % u == 0) return u;
    return 0;
}

// Compute units of the current device (cached per device), and workgroups of
// `kernel` with `threads` threads that fit one of its compute units (cached
// per device, kernel and size).  Both are safe to call from any thread.
int device_cus();
int kernel_occupancy(const void *kernel, int threads);

// One product launch: arguments validated by the C ABI.
struct SpmmArgs {
    const nmg_layout *L;
    const void *values;
    const uint8_t *indices;
    const void *X;
    int64_t ldx;
    int N;
    void *Y;
    int64_t ldy;
    hipStream_t stream;
    nmg_epilogue epi = NMG_EPILOGUE_NONE;  // applied by kernels that fuse it
    const void *R = nullptr;               // residual (NMG_EPILOGUE_ADD)
    int64_t ldr = 0;
};

nmg_status launch_compress(const nmg_layout *L, const void *W, int64_t ldw, void *values,
                           uint8_t *indices, hipStream_t stream);
nmg_status launch_repack(const nmg_layout *L, const void *W, int64_t ldw, const uint8_t *indices,
                         void *values, hipStream_t stream);
// `zeros` (may be NULL): K bytes set to 0 on the way (the index bytes of the
// expanded weight's one-column chunks)
nmg_status launch_densify(const nmg_layout *L, const void *values, const uint8_t *indices,
                          void *W_out, int64_t ldw, hipStream_t stream, uint8_t *zeros = nullptr);
nmg_status launch_gelu(nmg_dtype dtype, const void *in, void *out, int64_t count,
                       hipStream_t stream);
nmg_status launch_add(nmg_dtype dtype, const void *a, const void *b, void *out, int64_t count,
                      hipStream_t stream);

nmg_status spmm_valu(const SpmmArgs &a);
bool spmm_valu_staged_supported(const nmg_layout *L, const void *X, int64_t ldx, int64_t N);
bool spmm_valu_staged_preferred(const nmg_layout *L, const void *X, int64_t ldx, int64_t N);
nmg_status spmm_valu_staged(const SpmmArgs &a);

bool spmm_general_supported(const nmg_layout *L, int64_t N);
nmg_status spmm_general_f32(const SpmmArgs &a);
nmg_status spmm_general_f16(const SpmmArgs &a);

bool spmm_scalar_supported(const nmg_layout *L, const uint8_t *indices, int64_t ldx);
nmg_status spmm_scalar(const SpmmArgs &a);
nmg_status spmm_scalar_f32_u16(const SpmmArgs &a);
nmg_status spmm_scalar_f32_u8(const SpmmArgs &a);
nmg_status spmm_scalar_f32_u4(const SpmmArgs &a);
nmg_status spmm_scalar_f16(const SpmmArgs &a);

bool spmm_direct_supported(const nmg_layout *L, int64_t ldx);
bool spmm_direct_preferred(const nmg_layout *L, int64_t N, int64_t ldx);
nmg_status spmm_direct(const SpmmArgs &a);

bool spmm_smfmac_supported(const nmg_layout *L, const void *values, const uint8_t *indices,
                           const void *X, int64_t ldx, int64_t N);
nmg_status spmm_smfmac(const SpmmArgs &a);

bool spmm_half_supported(const nmg_layout *L, const void *X, int64_t ldx, int64_t N);

// the 16 x 16 x 32 products (k_spmm_x16.hip): layout and argument checks,
// size of the prepared operands, preparation and product
bool x16_layout_supported(const nmg_layout *L);
// the layout the kernels run: n == m keeps every column, so every index row
// is 0 .. m-1 and the whole weight is one group (g = M); else L itself
const nmg_layout *effective_layout(const nmg_layout *L, nmg_layout *tmp);
// Where a product's scratch memory comes from: a function that returns
// `bytes` of device memory that is the call's alone until its work on the
// stream is done, or NULL with *st set (NMG_ERR_CAPACITY when the request is
// too large for it).
typedef void *(*scratch_source)(int64_t bytes, hipStream_t stream, nmg_status *st);
// nmg_spmm_epilogue; the families with scratch memory (the 16 x 16 x 32
// products' prepared operands, the expanded weight) take it from `scratch`,
// or from a stream-ordered allocation when scratch is NULL
nmg_status spmm_epilogue_ws(const nmg_layout *L, nmg_kernel kernel, nmg_epilogue epi,
                            const void *values, const uint8_t *indices, const void *X, int64_t ldx,
                            int64_t N, const void *R, int64_t ldr, void *Y, int64_t ldy,
                            hipStream_t stream, scratch_source scratch);
// The expanded product: W_s written out dense (zeros elsewhere) as a layout
// of one group with one-column chunks, multiplied by the binary32 /
// widened-binary16 matrix-core kernel.  Scratch bytes it needs; whether it
// takes the layout.
int64_t expand_scratch_bytes(const nmg_layout *L);
bool expand_supported(const nmg_layout *L, int64_t ldx);
bool expand_preferred(const nmg_layout *L, int64_t ldx);
// the fused residual sum of the 16 x 16 x 32 products reads R 16 bytes at a time
inline bool x16_residual_supported(const nmg_layout *L, const void *R, int64_t ldr) {
    const int64_t es = L->dtype == NMG_F32 ? 4 : 2;
    return aligned(R, 16) && ldr % (16 / es) == 0;
}
bool x16_args_supported(const nmg_layout *L, const void *X, int64_t ldx, const void *Y,
                        int64_t ldy, int64_t N);
int64_t x16_prepared_bytes(const nmg_layout *L);
nmg_status x16_prepare(const nmg_layout *L, const void *values, const uint8_t *indices,
                       void *prepared, hipStream_t stream);
// epi: NMG_EPILOGUE_NONE / _ADD (R read 16 bytes at a time) / _GELU;
// NMG_ERR_UNSUPPORTED, before any launch, for a GELU the chosen tile cannot
// fold in (binary32, or outputs that leave no room for the table)
nmg_status x16_product(const nmg_layout *L, const void *prepared, const void *X, int64_t ldx,
                       int N, void *Y, int64_t ldy, int epi, const void *R, int64_t ldr,
                       hipStream_t stream);

nmg_status check_p_layout(const nmg_p_layout *L);
int p_pattern_count(int m, int n);
nmg_status launch_p_compress(const nmg_p_layout *L, const void *W, int64_t ldw, void *values,
                             uint8_t *index, hipStream_t stream);
nmg_status launch_p_densify(const nmg_p_layout *L, const void *values, const uint8_t *index,
                            void *W_out, int64_t ldw, hipStream_t stream);
nmg_status launch_p_refine(const nmg_p_layout *L, const void *W, int64_t ldw, void *values,
                           uint8_t *index, hipStream_t stream);
nmg_status launch_p_spmm(const nmg_p_layout *L, nmg_kernel kernel, const void *values,
                         const uint8_t *index, const void *X, int64_t ldx, int N, void *Y,
                         int64_t ldy, hipStream_t stream);
nmg_status spmm_half(const SpmmArgs &a);

}  // namespace nmg_internal

namespace {

using namespace nmg_internal;

typedef float v4f __attribute__((ext_vector_type(4)));
typedef _Float16 h4 __attribute__((ext_vector_type(4)));

constexpr int kBlock = 256;  // threads per workgroup for every kernel

template <typename T> struct Bits;
template <> struct Bits<float> { using type = uint32_t; };
template <> struct Bits<_Float16> { using type = uint16_t; };

template <int... S, typename F>
__device__ __forceinline__ void static_for_impl(std::integer_sequence<int, S...>, F &&f) {
    (f(std::integral_constant<int, S>{}), ...);
}
// f(std::integral_constant<int, s>) for s = 0 .. N-1, fully unrolled.
template <int N, typename F>
__device__ __forceinline__ void static_for(F &&f) {
    static_for_impl(std::make_integer_sequence<int, N>{}, f);
}

// Four consecutive elements of row `p` (token t .. t+3) widened to binary32;
// entries at or beyond `valid` are zero.  `vec` (uniform) says p is aligned to
// four elements, so one vector load serves.
template <typename T>
__device__ __forceinline__ v4f load4(const T *p, int valid, bool vec) {
    v4f v = {0.f, 0.f, 0.f, 0.f};
    if (vec && valid >= 4) {
        if constexpr (std::is_same<T, float>::value) {
            v = *reinterpret_cast<const v4f *>(p);
        } else {
            h4 h = *reinterpret_cast<const h4 *>(p);
            v = v4f{(float)h[0], (float)h[1], (float)h[2], (float)h[3]};
        }
    } else {
        for (int j = 0; j < 4; ++j)
            if (j < valid) v[j] = (float)p[j];
    }
    return v;
}

// XCD-aware tile order.  Workgroups are dealt round-robin to the 8 XCDs
// (workgroup i runs on XCD i % 8); this maps them so that each XCD receives
// one contiguous range of logical tiles, in which the row tiles of a token
// tile are adjacent and share that token tile's X rows in the XCD's L2.
__device__ __forceinline__ int xcd_tile(int i, int total) {
    constexpr int kXcd = 8;
    const int per = total / kXcd, rem = total % kXcd;
    const int x = i % kXcd, j = i / kXcd;
    return x * per + (x < rem ? x : rem) + j;
}

// 16 bytes per lane from global memory straight into LDS: a buffer load with
// an LDS destination (buffer_load_dwordx4 ... lds) from byte offset `off` of
// the buffer `r` to lds + 16 * lane (`lds` wave-uniform).  Not the global
// form (global_load_lds_dwordx4): the compiler takes a flat-encoded LDS copy
// in flight as an access to both memory and LDS, and then makes every later
// use of a loaded register or LDS read wait for all memory operations
// (vmcnt(0) / lgkmcnt(0)); buffer copies are counted like other loads, so
// its waits stay counts.  The descriptor covers `bytes` from
// `base` (raw: stride 0, 32-bit data format, no swizzle or thread-id offset,
// the gfx9-family raw-buffer word 3); offsets must fit 32 bits.
#if defined(__HIP_DEVICE_COMPILE__)
typedef __amdgpu_buffer_rsrc_t buf_rsrc_t;
__device__ __forceinline__ buf_rsrc_t buf_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes,
                                             0x00020000);
}
__device__ __forceinline__ void lds_copy16_buf(buf_rsrc_t r, uint32_t off, void *lds) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void *)lds, 16,
                                             (int)off, 0, 0, 0);
}
#else
typedef int buf_rsrc_t;
__device__ inline buf_rsrc_t buf_rsrc(const void *, uint32_t) { return 0; }
__device__ inline void lds_copy16_buf(buf_rsrc_t, uint32_t, void *) {}
#endif

// Wait for every outstanding memory operation of this wave.
__device__ __forceinline__ void wait_all_memory() {
#if defined(__HIP_DEVICE_COMPILE__)
    __builtin_amdgcn_s_waitcnt(0);
#endif
}

constexpr int ilog2(int v) { return v <= 1 ? 0 : 1 + ilog2(v / 2); }

}  // namespace
