// abi.hip -- the C ABI of libnmg (include/nmg.h): host-side validation and
// dispatch to the kernels' launchers.  Nothing here touches the GPU except
// through those launchers and two cached runtime queries (compute units per
// device, occupancy per kernel and workgroup size).
//
// Paper: STen (arXiv 2304.07613), Section 5.
#include <mutex>

#include "common.hpp"

namespace nmg_internal {

namespace {
// Per-device figures are cached for devices 0 .. kMaxDevices-1; others are
// queried on every call.
constexpr int kMaxDevices = 64;

int current_device() {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) {
        (void)hipGetLastError();  // leave no error pending for the next launch
        return -1;
    }
    return dev;
}
}  // namespace

int device_cus() {
    static std::atomic<int> cus[kMaxDevices];  // 0 = not yet queried
    const int dev = current_device();
    if (dev >= 0 && dev < kMaxDevices) {
        const int v = cus[dev].load(std::memory_order_relaxed);
        if (v > 0) return v;
    }
    int c = 0;
    if (dev < 0 || hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) !=
                       hipSuccess || c < 1) {
        (void)hipGetLastError();
        c = 256;
    }
    // every thread computes the same value for a device, so a plain store is
    // race-free in effect
    if (dev >= 0 && dev < kMaxDevices) cus[dev].store(c, std::memory_order_relaxed);
    return c;
}

// Occupancy figures from the HIP runtime, cached per (device, kernel, threads)
// in a table guarded by one mutex: an entry is written whole before any
// thread can read it, so every caller sees either no entry or the complete
// figure, and every call on a device gets the same launch shape.
int kernel_occupancy(const void *kernel, int threads) {
    struct Entry {
        const void *kernel;
        int device, threads, occ;
    };
    constexpr int kSlots = 512;
    static std::mutex lock;
    static Entry table[kSlots];
    static int used = 0;
    const int dev = current_device();
    {
        std::lock_guard<std::mutex> guard(lock);
        for (int i = 0; i < used; ++i)
            if (table[i].kernel == kernel && table[i].threads == threads &&
                table[i].device == dev)
                return table[i].occ;
    }
    int nb = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, kernel, threads, 0) != hipSuccess ||
        nb < 1) {
        (void)hipGetLastError();
        nb = 1;
    }
    std::lock_guard<std::mutex> guard(lock);
    for (int i = 0; i < used; ++i)  // another thread may have filled it meanwhile
        if (table[i].kernel == kernel && table[i].threads == threads && table[i].device == dev)
            return table[i].occ;
    if (dev >= 0 && used < kSlots) table[used++] = Entry{kernel, dev, threads, nb};
    return nb;
}

}  // namespace nmg_internal

using namespace nmg_internal;

extern "C" {

nmg_status nmg_layout_init(nmg_layout *layout, int32_t M, int32_t K, int32_t n, int32_t m,
                           int32_t g, nmg_dtype dtype) {
    if (!layout) return NMG_ERR_NULL;
    nmg_layout L;
    L.M = M;
    L.K = K;
    L.n = n;
    L.m = m;
    L.g = g;
    L.C = (m >= 1 && K >= 1) ? (K + m - 1) / m : 0;
    L.dtype = dtype;
    const nmg_status st = check_layout(&L);
    if (st != NMG_OK) return st;
    *layout = L;
    return NMG_OK;
}

int64_t nmg_values_numel(const nmg_layout *layout) {
    if (check_layout(layout) != NMG_OK) return -1;
    return (int64_t)layout->M * layout->C * layout->n;
}

int64_t nmg_indices_numel(const nmg_layout *layout) {
    if (check_layout(layout) != NMG_OK) return -1;
    return (int64_t)(layout->M / layout->g) * layout->C * layout->n;
}

nmg_status nmg_compress(const nmg_layout *L, const void *W, int64_t ldw, void *values,
                        uint8_t *indices, hipStream_t stream) {
    nmg_status st = check_layout(L);
    if (st != NMG_OK) return st;
    if (!W || !values || !indices) return NMG_ERR_NULL;
    if (ldw < L->K) return NMG_ERR_PARAM;
    const size_t es = elem_size(L->dtype);
    if (!aligned(W, es) || !aligned(values, es)) return NMG_ERR_ALIGN;
    prelaunch();
    return launch_compress(L, W, ldw, values, indices, stream);
}

nmg_status nmg_repack(const nmg_layout *L, const void *W, int64_t ldw, const uint8_t *indices,
                      void *values, hipStream_t stream) {
    nmg_status st = check_layout(L);
    if (st != NMG_OK) return st;
    if (!W || !indices || !values) return NMG_ERR_NULL;
    if (ldw < L->K) return NMG_ERR_PARAM;
    const size_t es = elem_size(L->dtype);
    if (!aligned(W, es) || !aligned(values, es)) return NMG_ERR_ALIGN;
    prelaunch();
    return launch_repack(L, W, ldw, indices, values, stream);
}

nmg_kernel nmg_spmm_auto_kernel(const nmg_layout *L, int64_t N) {
    if (check_layout(L) != NMG_OK) return NMG_KERNEL_AUTO;
    nmg_layout dense;
    if (L->n == L->m && L->g != L->M) {  // as in nmg_spmm_epilogue
        dense = *L;
        dense.g = L->M;
        L = &dense;
    }
    if (spmm_half_supported(L, nullptr, N, N)) return NMG_KERNEL_MFMA_F16;
    if (spmm_smfmac_supported(L, nullptr, nullptr, nullptr, N, N)) return NMG_KERNEL_SMFMAC_F16;
    if (spmm_direct_preferred(L, N, N)) return NMG_KERNEL_MFMA_DIRECT;
    if (spmm_scalar_supported(L, nullptr, N)) return NMG_KERNEL_MFMA_SCALAR;
    if (spmm_general_supported(L, N)) return NMG_KERNEL_MFMA_GENERAL;
    if (expand_preferred(L, N)) return NMG_KERNEL_MFMA_EXPAND;
    return spmm_valu_staged_preferred(L, nullptr, N, N) ? NMG_KERNEL_VALU_STAGED : NMG_KERNEL_VALU;
}

nmg_status nmg_spmm_with(const nmg_layout *L, nmg_kernel kernel, const void *values,
                         const uint8_t *indices, const void *X, int64_t ldx, int64_t N, void *Y,
                         int64_t ldy, hipStream_t stream) {
    return nmg_spmm_epilogue(L, kernel, NMG_EPILOGUE_NONE, values, indices, X, ldx, N, nullptr, 0,
                             Y, ldy, stream);
}

nmg_status nmg_spmm_epilogue(const nmg_layout *L, nmg_kernel kernel, nmg_epilogue epi,
                             const void *values, const uint8_t *indices, const void *X,
                             int64_t ldx, int64_t N, const void *R, int64_t ldr, void *Y,
                             int64_t ldy, hipStream_t stream) {
    return spmm_epilogue_ws(L, kernel, epi, values, indices, X, ldx, N, R, ldr, Y, ldy, stream,
                            nullptr);
}

}  // extern "C"

namespace {

// The expanded weight as a layout: one group, chunks of one column, every
// column kept (its index bytes are all 0)
nmg_layout expanded_layout(const nmg_layout *L) {
    nmg_layout D = *L;
    D.n = 1;
    D.m = 1;
    D.g = L->M;
    D.C = L->K;
    return D;
}

constexpr int64_t round256(int64_t b) { return (b + 255) / 256 * 256; }

// Scratch memory from the caller's source, else in stream order
void *take_scratch(scratch_source src, int64_t bytes, hipStream_t stream, nmg_status *st) {
    if (src) return src(bytes, stream, st);
    void *p = nullptr;
    if (hipMallocAsync(&p, (size_t)bytes, stream) != hipSuccess || p == nullptr) {
        (void)hipGetLastError();
        *st = NMG_ERR_LAUNCH;
        return nullptr;
    }
    return p;
}

nmg_status give_back_scratch(scratch_source src, void *p, hipStream_t stream, nmg_status st) {
    if (!src && hipFreeAsync(p, stream) != hipSuccess) {
        (void)hipGetLastError();
        if (st == NMG_OK) st = NMG_ERR_LAUNCH;
    }
    return st;
}

// The epilogue as a second pass over Y (row by row when rows are not contiguous)
nmg_status epilogue_pass(const nmg_layout *L, nmg_epilogue epi, void *Y, int64_t ldy,
                         const void *R, int64_t ldr, int64_t N, hipStream_t stream) {
    const size_t es = elem_size(L->dtype);
    const bool flat = ldy == N && (epi != NMG_EPILOGUE_ADD || ldr == N);
    const int64_t rows = flat ? 1 : L->M, count = flat ? (int64_t)L->M * N : N;
    for (int64_t r = 0; r < rows; ++r) {
        char *y = static_cast<char *>(Y) + (size_t)(r * ldy) * es;
        const nmg_status st =
            epi == NMG_EPILOGUE_GELU
                ? launch_gelu(L->dtype, y, y, count, stream)
                : launch_add(L->dtype, y, static_cast<const char *>(R) + (size_t)(r * ldr) * es, y,
                             count, stream);
        if (st != NMG_OK) return st;
    }
    return NMG_OK;
}

// The 16 x 16 x 32 product with its epilogue folded in where the kernel
// takes it (the residual sum with 16-byte aligned R, GELU where the tile
// leaves room for the table), else as a second pass
nmg_status x16_with_epilogue(const nmg_layout *L, const void *prepared, nmg_epilogue epi,
                             const void *X, int64_t ldx, int64_t N, const void *R, int64_t ldr,
                             void *Y, int64_t ldy, hipStream_t stream) {
    if (epi == NMG_EPILOGUE_GELU ||
        (epi == NMG_EPILOGUE_ADD && x16_residual_supported(L, R, ldr))) {
        const nmg_status st = x16_product(L, prepared, X, ldx, (int)N, Y, ldy, epi, R, ldr, stream);
        if (st != NMG_ERR_UNSUPPORTED) return st;
    }
    const nmg_status st =
        x16_product(L, prepared, X, ldx, (int)N, Y, ldy, NMG_EPILOGUE_NONE, nullptr, 0, stream);
    if (st != NMG_OK || epi == NMG_EPILOGUE_NONE) return st;
    return epilogue_pass(L, epi, Y, ldy, R, ldr, N, stream);
}

}  // namespace

// AUTO's binary32 choice among the families for groups the grouped
// matrix-core kernels cannot share: the expanded product does m / n times
// the useful work at the matrix rate, the staged vector kernel the useful
// work at about a seventh of it (measured break-even near m / n = 10)
bool nmg_internal::expand_preferred(const nmg_layout *L, int64_t ldx) {
    return L->dtype == NMG_F32 && L->m <= 8 * L->n && expand_supported(L, ldx);
}

int64_t nmg_internal::expand_scratch_bytes(const nmg_layout *L) {
    return round256((int64_t)L->M * L->K * (int64_t)elem_size(L->dtype)) + round256(L->K);
}

bool nmg_internal::expand_supported(const nmg_layout *L, int64_t ldx) {
    if ((int64_t)L->M * L->K >= ((int64_t)1 << 31)) return false;
    const nmg_layout D = expanded_layout(L);
    return check_layout(&D) == NMG_OK && spmm_scalar_supported(&D, nullptr, ldx);
}

const nmg_layout *nmg_internal::effective_layout(const nmg_layout *L, nmg_layout *tmp) {
    // n == m keeps every column, so every index row is 0 .. m-1: the whole
    // weight is one group and the grouped kernels apply whatever g is
    if (L->n == L->m && L->g != L->M) {
        *tmp = *L;
        tmp->g = L->M;
        return tmp;
    }
    return L;
}

nmg_status nmg_internal::spmm_epilogue_ws(const nmg_layout *L, nmg_kernel kernel, nmg_epilogue epi,
                                          const void *values, const uint8_t *indices,
                                          const void *X, int64_t ldx, int64_t N, const void *R,
                                          int64_t ldr, void *Y, int64_t ldy, hipStream_t stream,
                                          scratch_source scratch) {
    nmg_status st = check_layout(L);
    if (st != NMG_OK) return st;
    if (!values || !indices || !X || !Y) return NMG_ERR_NULL;
    if (N < 1 || N > INT32_MAX || ldx < N || ldy < N) return NMG_ERR_PARAM;
    const size_t es = elem_size(L->dtype);
    if (!aligned(X, es) || !aligned(values, es) || !aligned(Y, es)) return NMG_ERR_ALIGN;
    if (epi != NMG_EPILOGUE_NONE && epi != NMG_EPILOGUE_GELU && epi != NMG_EPILOGUE_ADD)
        return NMG_ERR_PARAM;
    if (epi == NMG_EPILOGUE_ADD) {
        if (!R) return NMG_ERR_NULL;
        if (ldr < N) return NMG_ERR_PARAM;
        if (!aligned(R, es)) return NMG_ERR_ALIGN;
        // R must not overlap Y (the unfused families write Y before reading R)
        const uintptr_t r0 = reinterpret_cast<uintptr_t>(R), y0 = reinterpret_cast<uintptr_t>(Y);
        const uintptr_t r1 = r0 + (uintptr_t)(((int64_t)(L->M - 1) * ldr + N) * (int64_t)es);
        const uintptr_t y1 = y0 + (uintptr_t)(((int64_t)(L->M - 1) * ldy + N) * (int64_t)es);
        if (r0 < y1 && y0 < r1) return NMG_ERR_PARAM;
    }
    nmg_layout dense;
    L = effective_layout(L, &dense);
    prelaunch();
    SpmmArgs a{L, values, indices, X, ldx, (int)N, Y, ldy, stream};
    const bool half_ok = spmm_half_supported(L, X, ldx, N);
    const bool scalar_ok = spmm_scalar_supported(L, indices, ldx);
    if (kernel == NMG_KERNEL_AUTO || kernel == NMG_KERNEL_MFMA) {
        const bool direct = spmm_direct_preferred(L, N, ldx);
        kernel = half_ok     ? NMG_KERNEL_MFMA_F16
                 : spmm_smfmac_supported(L, values, indices, X, ldx, N) ? NMG_KERNEL_SMFMAC_F16
                 : direct    ? NMG_KERNEL_MFMA_DIRECT
                 : scalar_ok ? NMG_KERNEL_MFMA_SCALAR
                 : spmm_general_supported(L, N) || kernel == NMG_KERNEL_MFMA
                     ? NMG_KERNEL_MFMA_GENERAL
                 : expand_preferred(L, ldx) ? NMG_KERNEL_MFMA_EXPAND
                 : spmm_valu_staged_preferred(L, X, ldx, N) ? NMG_KERNEL_VALU_STAGED
                                                              : NMG_KERNEL_VALU;
    }
    switch (kernel) {
        case NMG_KERNEL_MFMA_F16:
            if (!half_ok) return NMG_ERR_UNSUPPORTED;
            a.epi = epi;  // applied in the product kernel
            a.R = R;
            a.ldr = ldr;
            return spmm_half(a);
        case NMG_KERNEL_SMFMAC_F16:
            if (!spmm_smfmac_supported(L, values, indices, X, ldx, N)) return NMG_ERR_UNSUPPORTED;
            a.epi = epi;  // applied in the product kernel
            a.R = R;
            a.ldr = ldr;
            return spmm_smfmac(a);
        case NMG_KERNEL_MFMA_DIRECT:
            if (!spmm_direct_supported(L, ldx)) return NMG_ERR_UNSUPPORTED;
            st = spmm_direct(a);
            break;
        case NMG_KERNEL_MFMA_SCALAR:
            if (!scalar_ok) return NMG_ERR_UNSUPPORTED;
            st = spmm_scalar(a);
            break;
        case NMG_KERNEL_MFMA_GENERAL:
            if (!spmm_general_supported(L, N)) return NMG_ERR_UNSUPPORTED;
            st = L->dtype == NMG_F32 ? spmm_general_f32(a) : spmm_general_f16(a);
            break;
        case NMG_KERNEL_VALU:
            st = spmm_valu(a);
            break;
        case NMG_KERNEL_VALU_STAGED:
            if (!spmm_valu_staged_supported(L, X, ldx, N)) return NMG_ERR_UNSUPPORTED;
            st = spmm_valu_staged(a);
            break;
        case NMG_KERNEL_MFMA_WIDE:
        case NMG_KERNEL_MFMA_SPLIT: {
            if ((kernel == NMG_KERNEL_MFMA_SPLIT) != (L->dtype == NMG_F32) ||
                !x16_args_supported(L, X, ldx, Y, ldy, N))
                return NMG_ERR_UNSUPPORTED;
            // the prepared operands live for this call only
            void *prepared = take_scratch(scratch, x16_prepared_bytes(L), stream, &st);
            if (!prepared) return st;
            st = x16_prepare(L, values, indices, prepared, stream);
            if (st == NMG_OK)
                st = x16_with_epilogue(L, prepared, epi, X, ldx, N, R, ldr, Y, ldy, stream);
            return give_back_scratch(scratch, prepared, stream, st);
        }
        case NMG_KERNEL_MFMA_EXPAND: {
            if (!expand_supported(L, ldx)) return NMG_ERR_UNSUPPORTED;
            // the dense weight and its index bytes live for this call only
            void *ws = take_scratch(scratch, expand_scratch_bytes(L), stream, &st);
            if (!ws) return st;
            const nmg_layout D = expanded_layout(L);
            char *wd = static_cast<char *>(ws);
            uint8_t *zi = reinterpret_cast<uint8_t *>(
                wd + round256((int64_t)L->M * L->K * (int64_t)es));
            st = launch_densify(L, values, indices, wd, L->K, stream, zi);
            if (st == NMG_OK)  // the epilogue goes with the dense product
                st = spmm_epilogue_ws(&D, NMG_KERNEL_MFMA_SCALAR, epi, wd, zi, X, ldx, N, R, ldr,
                                      Y, ldy, stream, scratch);
            return give_back_scratch(scratch, ws, stream, st);
        }
        default:
            return NMG_ERR_PARAM;
    }
    if (st != NMG_OK || epi == NMG_EPILOGUE_NONE) return st;
    return epilogue_pass(L, epi, Y, ldy, R, ldr, N, stream);
}

extern "C" {

nmg_status nmg_p_layout_init(nmg_p_layout *layout, int32_t M, int32_t K, int32_t n, int32_t m,
                             int32_t g, nmg_dtype dtype) {
    if (!layout) return NMG_ERR_NULL;
    if (dtype != NMG_F32 && dtype != NMG_F16) return NMG_ERR_DTYPE;
    if (M < 1 || K < 1 || n < 1 || m < n || m > 255 || g < 1) return NMG_ERR_PARAM;
    nmg_p_layout L;
    L.M = M;
    L.K = K;
    L.n = n;
    L.m = m;
    L.g = g;
    L.P = p_pattern_count(m, n);
    if (L.P > 256) return NMG_ERR_PARAM;
    L.S = L.P * g;
    L.B = K / m;
    L.dtype = dtype;
    const nmg_status st = check_p_layout(&L);
    if (st != NMG_OK) return st;
    *layout = L;
    return NMG_OK;
}

nmg_status nmg_p_compress(const nmg_p_layout *L, const void *W, int64_t ldw, void *values,
                          uint8_t *index, hipStream_t stream) {
    nmg_status st = check_p_layout(L);
    if (st != NMG_OK) return st;
    if (!W || !values || !index) return NMG_ERR_NULL;
    if (ldw < L->K) return NMG_ERR_PARAM;
    const size_t es = elem_size(L->dtype);
    if (!aligned(W, es) || !aligned(values, es)) return NMG_ERR_ALIGN;
    prelaunch();
    return launch_p_compress(L, W, ldw, values, index, stream);
}

nmg_status nmg_p_refine(const nmg_p_layout *L, const void *W, int64_t ldw, void *values,
                        uint8_t *index, hipStream_t stream) {
    nmg_status st = check_p_layout(L);
    if (st != NMG_OK) return st;
    if (!W || !values || !index) return NMG_ERR_NULL;
    if (ldw < L->K) return NMG_ERR_PARAM;
    const size_t es = elem_size(L->dtype);
    if (!aligned(W, es) || !aligned(values, es)) return NMG_ERR_ALIGN;
    prelaunch();
    return launch_p_refine(L, W, ldw, values, index, stream);
}

nmg_status nmg_p_spmm_with(const nmg_p_layout *L, nmg_kernel kernel, const void *values,
                           const uint8_t *index, const void *X, int64_t ldx, int64_t N, void *Y,
                           int64_t ldy, hipStream_t stream) {
    nmg_status st = check_p_layout(L);
    if (st != NMG_OK) return st;
    if (kernel != NMG_KERNEL_AUTO && kernel != NMG_KERNEL_VALU && kernel != NMG_KERNEL_MFMA)
        return NMG_ERR_UNSUPPORTED;
    if (!values || !index || !X || !Y) return NMG_ERR_NULL;
    if (N < 1 || N > INT32_MAX || ldx < N || ldy < N) return NMG_ERR_PARAM;
    const size_t es = elem_size(L->dtype);
    if (!aligned(X, es) || !aligned(values, es) || !aligned(Y, es)) return NMG_ERR_ALIGN;
    prelaunch();
    return launch_p_spmm(L, kernel, values, index, X, ldx, (int)N, Y, ldy, stream);
}

nmg_status nmg_p_spmm(const nmg_p_layout *L, const void *values, const uint8_t *index,
                      const void *X, int64_t ldx, int64_t N, void *Y, int64_t ldy,
                      hipStream_t stream) {
    return nmg_p_spmm_with(L, NMG_KERNEL_AUTO, values, index, X, ldx, N, Y, ldy, stream);
}

nmg_status nmg_p_densify(const nmg_p_layout *L, const void *values, const uint8_t *index,
                         void *W_out, int64_t ldw, hipStream_t stream) {
    nmg_status st = check_p_layout(L);
    if (st != NMG_OK) return st;
    if (!values || !index || !W_out) return NMG_ERR_NULL;
    if (ldw < L->K) return NMG_ERR_PARAM;
    const size_t es = elem_size(L->dtype);
    if (!aligned(values, es) || !aligned(W_out, es)) return NMG_ERR_ALIGN;
    prelaunch();
    return launch_p_densify(L, values, index, W_out, ldw, stream);
}

nmg_status nmg_spmm(const nmg_layout *L, const void *values, const uint8_t *indices,
                    const void *X, int64_t ldx, int64_t N, void *Y, int64_t ldy,
                    hipStream_t stream) {
    return nmg_spmm_with(L, NMG_KERNEL_AUTO, values, indices, X, ldx, N, Y, ldy, stream);
}

int64_t nmg_x16_prepared_bytes(const nmg_layout *L) {
    if (check_layout(L) != NMG_OK) return -1;
    return x16_prepared_bytes(L);
}

nmg_status nmg_x16_prepare(const nmg_layout *L, const void *values, const uint8_t *indices,
                           void *prepared, hipStream_t stream) {
    nmg_status st = check_layout(L);
    if (st != NMG_OK) return st;
    if (!values || !indices || !prepared) return NMG_ERR_NULL;
    if (!x16_layout_supported(L)) return NMG_ERR_UNSUPPORTED;
    if (!aligned(values, elem_size(L->dtype)) || !aligned(prepared, 16)) return NMG_ERR_ALIGN;
    prelaunch();
    return x16_prepare(L, values, indices, prepared, stream);
}

nmg_status nmg_spmm_x16_epilogue(const nmg_layout *L, const void *prepared, nmg_epilogue epi,
                                 const void *X, int64_t ldx, int64_t N, const void *R, int64_t ldr,
                                 void *Y, int64_t ldy, hipStream_t stream) {
    nmg_status st = check_layout(L);
    if (st != NMG_OK) return st;
    if (!prepared || !X || !Y) return NMG_ERR_NULL;
    if (N < 1 || N > INT32_MAX || ldx < N || ldy < N) return NMG_ERR_PARAM;
    if (epi != NMG_EPILOGUE_NONE && epi != NMG_EPILOGUE_GELU && epi != NMG_EPILOGUE_ADD)
        return NMG_ERR_PARAM;
    if (!aligned(prepared, 16)) return NMG_ERR_ALIGN;
    if (!x16_args_supported(L, X, ldx, Y, ldy, N)) return NMG_ERR_UNSUPPORTED;
    if (epi == NMG_EPILOGUE_ADD) {
        if (!R) return NMG_ERR_NULL;
        if (ldr < N) return NMG_ERR_PARAM;
        if (!x16_residual_supported(L, R, ldr)) return NMG_ERR_UNSUPPORTED;
        const size_t es = elem_size(L->dtype);
        const uintptr_t r0 = reinterpret_cast<uintptr_t>(R), y0 = reinterpret_cast<uintptr_t>(Y);
        const uintptr_t r1 = r0 + (uintptr_t)(((int64_t)(L->M - 1) * ldr + N) * (int64_t)es);
        const uintptr_t y1 = y0 + (uintptr_t)(((int64_t)(L->M - 1) * ldy + N) * (int64_t)es);
        if (r0 < y1 && y0 < r1) return NMG_ERR_PARAM;
    }
    prelaunch();
    return x16_with_epilogue(L, prepared, epi, X, ldx, N, R, ldr, Y, ldy, stream);
}

nmg_status nmg_spmm_x16(const nmg_layout *L, const void *prepared, const void *X, int64_t ldx,
                        int64_t N, void *Y, int64_t ldy, hipStream_t stream) {
    return nmg_spmm_x16_epilogue(L, prepared, NMG_EPILOGUE_NONE, X, ldx, N, nullptr, 0, Y, ldy,
                                 stream);
}

nmg_status nmg_densify(const nmg_layout *L, const void *values, const uint8_t *indices,
                       void *W_out, int64_t ldw, hipStream_t stream) {
    nmg_status st = check_layout(L);
    if (st != NMG_OK) return st;
    if (!values || !indices || !W_out) return NMG_ERR_NULL;
    if (ldw < L->K) return NMG_ERR_PARAM;
    const size_t es = elem_size(L->dtype);
    if (!aligned(values, es) || !aligned(W_out, es)) return NMG_ERR_ALIGN;
    prelaunch();
    return launch_densify(L, values, indices, W_out, ldw, stream);
}

nmg_status nmg_gelu(nmg_dtype dtype, const void *in, void *out, int64_t count,
                    hipStream_t stream) {
    if (dtype != NMG_F32 && dtype != NMG_F16) return NMG_ERR_DTYPE;
    if (!in || !out) return NMG_ERR_NULL;
    if (count < 0) return NMG_ERR_PARAM;
    if (count == 0) return NMG_OK;
    const size_t es = elem_size(dtype);
    if (!aligned(in, es) || !aligned(out, es)) return NMG_ERR_ALIGN;
    prelaunch();
    return launch_gelu(dtype, in, out, count, stream);
}

nmg_status nmg_add(nmg_dtype dtype, const void *a, const void *b, void *out, int64_t count,
                   hipStream_t stream) {
    if (dtype != NMG_F32 && dtype != NMG_F16) return NMG_ERR_DTYPE;
    if (!a || !b || !out) return NMG_ERR_NULL;
    if (count < 0) return NMG_ERR_PARAM;
    if (count == 0) return NMG_OK;
    const size_t es = elem_size(dtype);
    if (!aligned(a, es) || !aligned(b, es) || !aligned(out, es)) return NMG_ERR_ALIGN;
    prelaunch();
    return launch_add(dtype, a, b, out, count, stream);
}

const char *nmg_status_str(nmg_status s) {
    switch (s) {
        case NMG_OK: return "ok";
        case NMG_ERR_NULL: return "null pointer";
        case NMG_ERR_PARAM: return "invalid parameter";
        case NMG_ERR_SHAPE: return "invalid shape";
        case NMG_ERR_DTYPE: return "unknown dtype";
        case NMG_ERR_ALIGN: return "misaligned pointer or leading dimension";
        case NMG_ERR_LAUNCH: return "kernel launch failed";
        case NMG_ERR_UNSUPPORTED: return "kernel does not support this layout";
        case NMG_ERR_CAPACITY: return "layout exceeds a fixed-size working buffer";
    }
    return "unknown status";
}

const char *nmg_version(void) { return "nmg 0.2.0 gfx950"; }

}  // extern "C"
