// k_spmm_valu.hip -- Y = W_s X with vector FMAs; any g, n, m (Section 5.1).
// Weights are wave-uniform (scalar loads), X rows are gathered per group from
// global memory.  The fallback for layouts the matrix-core kernels decline.
#include "common.hpp"

namespace {

constexpr int kValuRowsWave = 8;
constexpr int kValuRowsWg = 4 * kValuRowsWave;   // 32 rows
constexpr int kValuTokens = 256;                 // 4 per lane

template <typename T>
__global__ __launch_bounds__(kBlock) void k_spmm_valu(
    const T *__restrict__ values, const uint8_t *__restrict__ indices,
    const T *__restrict__ X, int64_t ldx, T *__restrict__ Y, int64_t ldy,
    int M, int K, int N, int n, int m, int g, int C, int row_tiles, int tiles, bool xvec) {
    const int tile = xcd_tile(blockIdx.x, tiles);
    const int rt = tile % row_tiles, tt = tile / row_tiles;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int r0 = rt * kValuRowsWg + wave * kValuRowsWave;
    const int tok = tt * kValuTokens + 4 * lane;
    const int valid = N - tok;
    const int64_t ldv = (int64_t)C * n;

    int grp[kValuRowsWave];
    bool fresh[kValuRowsWave], live[kValuRowsWave];
#pragma unroll
    for (int r = 0; r < kValuRowsWave; ++r) {
        const int row = r0 + r;
        live[r] = row < M;
        grp[r] = live[r] ? row / g : 0;
        fresh[r] = r == 0 || grp[r] != grp[r - 1];
    }

    float acc[kValuRowsWave][4];
#pragma unroll
    for (int r = 0; r < kValuRowsWave; ++r)
        for (int j = 0; j < 4; ++j) acc[r][j] = 0.f;

    int c = 0, s = 0;  // chunk and slot of k-slot ks
    for (int64_t ks = 0; ks < ldv; ++ks) {
        v4f x = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int r = 0; r < kValuRowsWave; ++r) {
            if (!live[r]) continue;
            if (fresh[r]) {
                // clamped so that invalid indices never leave X's K rows
                const int k = min(c * m + (int)indices[(int64_t)grp[r] * ldv + ks], K - 1);
                x = load4<T>(X + (int64_t)k * ldx + tok, valid, xvec);
            }
            const float w = (float)values[(int64_t)(r0 + r) * ldv + ks];
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[r][j] = fmaf(w, x[j], acc[r][j]);
        }
        if (++s == n) { s = 0; ++c; }
    }

#pragma unroll
    for (int r = 0; r < kValuRowsWave; ++r) {
        if (!live[r]) continue;
        T *y = Y + (int64_t)(r0 + r) * ldy + tok;
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (j < valid) y[j] = (T)acc[r][j];
    }
}

template <typename T>
nmg_status launch_valu(const nmg_layout *L, const void *values, const uint8_t *indices,
                       const void *X, int64_t ldx, int N, void *Y, int64_t ldy,
                       hipStream_t stream) {
    const int row_tiles = (L->M + kValuRowsWg - 1) / kValuRowsWg;
    const int tok_tiles = (N + kValuTokens - 1) / kValuTokens;
    const int tiles = row_tiles * tok_tiles;
    const bool xvec = x_vectorisable(L, X, ldx);
    hipLaunchKernelGGL((k_spmm_valu<T>), dim3(tiles), dim3(kBlock), 0, stream,
                       (const T *)values, indices, (const T *)X, ldx, (T *)Y, ldy, L->M, L->K,
                       N, L->n, L->m, L->g, L->C, row_tiles, tiles, xvec);
    return launched();
}

}  // namespace

nmg_status nmg_internal::spmm_valu(const SpmmArgs &a) {
    return a.L->dtype == NMG_F32
               ? launch_valu<float>(a.L, a.values, a.indices, a.X, a.ldx, a.N, a.Y, a.ldy, a.stream)
               : launch_valu<_Float16>(a.L, a.values, a.indices, a.X, a.ldx, a.N, a.Y, a.ldy,
                                       a.stream);
}
