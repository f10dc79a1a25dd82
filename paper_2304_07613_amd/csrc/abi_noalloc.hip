// nmg_spmm_epilogue_noalloc: nmg_spmm_epilogue for callers that cannot
// allocate device memory (code under HIP graph capture, serving loops,
// harnesses that forbid allocation).
//
// The library's products have scratch memory in two families: the prepared
// operands that the 16 x 16 x 32 products (NMG_KERNEL_MFMA_WIDE / _SPLIT) make
// from the packed weight, and the dense weight of the expanded product
// (NMG_KERNEL_MFMA_EXPAND, also an NMG_KERNEL_AUTO choice), made on every
// nmg_spmm_epilogue call in a stream-ordered allocation.  Here they go to one
// fixed array in device memory instead, a copy of it on every GPU the library
// runs on, held until the process ends.  Each family writes every byte of the
// region it uses before reading it (the preparation, and the densify pass
// that also zeroes the index bytes), so nothing has to be cleared between
// calls; calls that overlap on one GPU (several host threads, or several
// streams) share the array and race.  The other families use no scratch
// memory and run as nmg_spmm_epilogue runs them.
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


// The scratch source of this entry point: the current device's array
// (after checking that the work's stream is on that device), or
// NMG_ERR_CAPACITY before any runtime call when the request exceeds it.
void *fixed_scratch(int64_t bytes, hipStream_t stream, nmg_status *st) {
    if (bytes > kScratchBytes) {
        *st = NMG_ERR_CAPACITY;
        return nullptr;
    }
    int device = -1, stream_device = -1;
    if (hipGetDevice(&device) != hipSuccess || device < 0 || device >= kMaxDevices) {
        (void)hipGetLastError();
        *st = NMG_ERR_LAUNCH;
        return nullptr;
    }
    if (stream != nullptr) {
        if (hipStreamGetDevice(stream, &stream_device) != hipSuccess) {
            (void)hipGetLastError();
            *st = NMG_ERR_LAUNCH;
            return nullptr;
        }
        if (stream_device != device) {
            *st = NMG_ERR_PARAM;
            return nullptr;
        }
    }
    void *p = scratch_address(device);
    if (!p) *st = NMG_ERR_LAUNCH;
    return p;
}

}  // namespace

nmg_status nmg_spmm_epilogue_noalloc(const nmg_layout *L, nmg_kernel kernel, nmg_epilogue epi,
                                     const void *values, const uint8_t *indices, const void *X,
                                     int64_t ldx, int64_t N, const void *R, int64_t ldr, void *Y,
                                     int64_t ldy, hipStream_t stream) {
    return spmm_epilogue_ws(L, kernel, epi, values, indices, X, ldx, N, R, ldr, Y, ldy, stream,
                            fixed_scratch);
}
