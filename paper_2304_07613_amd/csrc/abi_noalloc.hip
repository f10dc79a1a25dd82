// nmg_spmm_epilogue_noalloc: nmg_spmm_epilogue for callers that cannot
// allocate device memory (code under HIP graph capture, serving loops,
// harnesses that forbid allocation).
//
// The only scratch memory of the library's products is the prepared operands
// that the 16 x 16 x 32 families (NMG_KERNEL_MFMA_WIDE / _SPLIT) make from
// the packed weight on every nmg_spmm_epilogue call, there in a stream-ordered
// allocation.  Here they go to one fixed array in device memory instead, a
// copy of it on every GPU the library runs on, held until the process ends.
// The preparation writes every byte of the region it uses before the product
// reads it, so nothing has to be cleared between calls; calls that overlap on
// one GPU (several host threads, or several streams) share the array and race.
// The other families use no scratch memory and run as nmg_spmm_epilogue runs
// them.
#include <hip/hip_runtime.h>

#include <atomic>
#include <mutex>

#include "common.hpp"

using namespace nmg_internal;

namespace {

constexpr int64_t kScratchBytes = (int64_t)16 << 20;  // 16 MiB per GPU
constexpr int kMaxDevices = 64;

// Device-side storage; host code never passes this name to a kernel or a
// copy (on the host it only names the symbol): the address of each GPU's
// copy comes from hipGetSymbolAddress with that GPU current.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex scratch_lock;
std::atomic<void *> scratch_ptr[kMaxDevices];

// The current device's copy of the array (looked up once per device), or
// nullptr when the runtime cannot name it.
void *scratch_address(int device) {
    void *p = scratch_ptr[device].load(std::memory_order_acquire);
    if (p) return p;
    std::lock_guard<std::mutex> guard(scratch_lock);
    p = scratch_ptr[device].load(std::memory_order_relaxed);
    if (p) return p;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) {
        (void)hipGetLastError();
        return nullptr;
    }
    scratch_ptr[device].store(p, std::memory_order_release);
    return p;
}

}  // namespace

nmg_status nmg_spmm_epilogue_noalloc(const nmg_layout *L, nmg_kernel kernel, nmg_epilogue epi,
                                     const void *values, const uint8_t *indices, const void *X,
                                     int64_t ldx, int64_t N, const void *R, int64_t ldr, void *Y,
                                     int64_t ldy, hipStream_t stream) {
    if (kernel != NMG_KERNEL_MFMA_WIDE && kernel != NMG_KERNEL_MFMA_SPLIT)
        return nmg_spmm_epilogue(L, kernel, epi, values, indices, X, ldx, N, R, ldr, Y, ldy,
                                 stream);
    nmg_status st = check_layout(L);
    if (st != NMG_OK) return st;
    if (!values || !indices || !X || !Y) return NMG_ERR_NULL;
    // the size check comes before any runtime call
    nmg_layout tmp;
    const int64_t bytes = x16_prepared_bytes(effective_layout(L, &tmp));
    if (bytes < 0) return NMG_ERR_UNSUPPORTED;
    if (bytes > kScratchBytes) return NMG_ERR_CAPACITY;
    // the array of the GPU the work runs on, which must be the current one
    int device = -1, stream_device = -1;
    if (hipGetDevice(&device) != hipSuccess || device < 0 || device >= kMaxDevices) {
        (void)hipGetLastError();
        return NMG_ERR_LAUNCH;
    }
    if (stream != nullptr) {
        if (hipStreamGetDevice(stream, &stream_device) != hipSuccess) {
            (void)hipGetLastError();
            return NMG_ERR_LAUNCH;
        }
        if (stream_device != device) return NMG_ERR_PARAM;
    }
    void *ws = scratch_address(device);
    if (!ws) return NMG_ERR_LAUNCH;
    return spmm_epilogue_ws(L, kernel, epi, values, indices, X, ldx, N, R, ldr, Y, ldy, stream, ws,
                            kScratchBytes);
}
