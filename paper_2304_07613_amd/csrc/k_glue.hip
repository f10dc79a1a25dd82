// k_glue.hip -- the elementwise glue between the linears of a BERT encoder
// block (not part of the paper's format): GELU and the residual sum.
//
//   k_gelu_f16  binary16: a 65536-entry table of the correctly rounded GELU of
//               every binary16 input (generated at build time), copied to LDS
//               by each workgroup; 16-byte vectors in and out.  HBM-bound.
//   k_gelu_f32  binary32: 0.5 x erfc(-x / sqrt 2) evaluated in binary32.
//   k_add       a + b in binary32, rounded once to the element type; 16-byte
//               vectors when every operand allows.
#include "common.hpp"

namespace {

// GELU(x) for every binary16 x, indexed by the bits of x
__device__ __attribute__((aligned(16))) const uint16_t g_gelu_f16[65536] = {
#include "gelu_f16_table.inc"
};

constexpr int kGlueThreads = 1024;

__global__ __launch_bounds__(kGlueThreads) void k_gelu_f16(const uint16_t *in, uint16_t *out,
                                                           int64_t count, bool vec) {
    __shared__ uint4 tab4[65536 * 2 / 16];
    const uint4 *src = reinterpret_cast<const uint4 *>(g_gelu_f16);
    for (int i = threadIdx.x; i < 65536 * 2 / 16; i += blockDim.x) tab4[i] = src[i];
    __syncthreads();
    const uint16_t *tab = reinterpret_cast<const uint16_t *>(tab4);
    auto look2 = [&](uint32_t w) { return (uint32_t)tab[w & 0xffffu] | ((uint32_t)tab[w >> 16] << 16); };

    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t done = 0;
    if (vec) {  // in and out on 16-byte boundaries: 8 elements per access
        const int64_t nv = count / 8;
        for (int64_t v = tid; v < nv; v += stride) {
            const uint4 x = reinterpret_cast<const uint4 *>(in)[v];
            reinterpret_cast<uint4 *>(out)[v] = uint4{look2(x.x), look2(x.y), look2(x.z), look2(x.w)};
        }
        done = nv * 8;
    }
    for (int64_t i = done + tid; i < count; i += stride) out[i] = tab[in[i]];
}

__global__ __launch_bounds__(kBlock) void k_gelu_f32(const float *in, float *out, int64_t count) {
    const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (i >= count) return;
    const float x = in[i];
    // 1 + erf(z) written as erfc(-z): no cancellation for negative x
    out[i] = 0.5f * x * erfcf(-x * 0.70710678118654752f);
}

template <typename T>
__global__ __launch_bounds__(kGlueThreads) void k_add(const T *a, const T *b, T *out,
                                                      int64_t count, bool vec) {
    constexpr int V = 16 / sizeof(T);  // elements per 16-byte access
    typedef T TV __attribute__((ext_vector_type(V)));
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t done = 0;
    if (vec) {
        const int64_t nv = count / V;
        for (int64_t v = tid; v < nv; v += stride) {
            const TV x = reinterpret_cast<const TV *>(a)[v], y = reinterpret_cast<const TV *>(b)[v];
            TV s;
#pragma unroll
            for (int e = 0; e < V; ++e) s[e] = (T)((float)x[e] + (float)y[e]);
            reinterpret_cast<TV *>(out)[v] = s;
        }
        done = nv * V;
    }
    for (int64_t i = done + tid; i < count; i += stride) out[i] = (T)((float)a[i] + (float)b[i]);
}

// Grid of a streaming kernel: enough workgroups for `count` elements at
// `per_block` each, at most `cap`.
unsigned glue_grid(int64_t count, int64_t per_block, int cap) {
    const int64_t want = (count + per_block - 1) / per_block;
    return (unsigned)std::max<int64_t>(1, std::min<int64_t>(want, cap));
}

}  // namespace

namespace nmg_internal {

nmg_status launch_gelu(nmg_dtype dtype, const void *in, void *out, int64_t count,
                       hipStream_t stream) {
    if (dtype == NMG_F32) {
        const int64_t blocks = (count + kBlock - 1) / kBlock;
        if (blocks > INT32_MAX) return NMG_ERR_PARAM;
        hipLaunchKernelGGL(k_gelu_f32, dim3((unsigned)blocks), dim3(kBlock), 0, stream,
                           (const float *)in, (float *)out, count);
        return launched();
    }
    // one workgroup per CU holds the 128 KB table; each one streams a share
    const bool vec = aligned(in, 16) && aligned(out, 16);
    const unsigned grid = glue_grid(count, (int64_t)kGlueThreads * 8, device_cus());
    hipLaunchKernelGGL(k_gelu_f16, dim3(grid), dim3(kGlueThreads), 0, stream,
                       (const uint16_t *)in, (uint16_t *)out, count, vec);
    return launched();
}

nmg_status launch_add(nmg_dtype dtype, const void *a, const void *b, void *out, int64_t count,
                      hipStream_t stream) {
    const bool vec = aligned(a, 16) && aligned(b, 16) && aligned(out, 16);
    const unsigned grid = glue_grid(count, (int64_t)kGlueThreads * 8, 8 * device_cus());
    if (dtype == NMG_F32)
        hipLaunchKernelGGL((k_add<float>), dim3(grid), dim3(kGlueThreads), 0, stream,
                           (const float *)a, (const float *)b, (float *)out, count, vec);
    else
        hipLaunchKernelGGL((k_add<_Float16>), dim3(grid), dim3(kGlueThreads), 0, stream,
                           (const _Float16 *)a, (const _Float16 *)b, (_Float16 *)out, count, vec);
    return launched();
}

}  // namespace nmg_internal
