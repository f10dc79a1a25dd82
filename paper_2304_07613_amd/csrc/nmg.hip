// nmg.hip -- HIP kernels and C ABI of the n:m:g library, written for gfx950.
//
// Paper: STen (arXiv 2304.07613), Section 5.  The layout, selection rule and
// product are specified in include/nmg.h; this file states only how the GPU
// computes them.
//
// Kernels
//   k_compress      dense -> (values, indices).  One thread per column of a
//                   chunk-block: binary32 group score down the g rows
//                   (coalesced across lanes), rank by counting inside the
//                   chunk through LDS, then a coalesced copy of the kept
//                   weights.  HBM-bound.
//   k_spmm_mfma     Y = W_s X on binary32 matrix cores.  v_mfma_f32_4x4x1f32
//                   runs 16 independent 4x4 outer products; with the A-operand
//                   broadcast (CBSZ/ABID) all 16 blocks multiply the same 4
//                   weights (4 rows of one group, one k-slot) by 64 different
//                   tokens of the X row that the group selected.  One A
//                   register therefore carries the weights of 4 rows for up to
//                   16 k-slots, and the gathered X row is a plain coalesced
//                   64-lane LDS read.  A workgroup stages whole chunk windows
//                   of X (all m rows of each chunk, all its tokens) in LDS once
//                   and every group of its 256 rows gathers from there.
//   k_spmm_valu     Y = W_s X with vector FMAs; any g, n, m.  Weights are
//                   wave-uniform (scalar loads), X rows are gathered per group
//                   from global memory.
//   k_densify       (values, indices) -> dense.
//   k_gelu, k_add   elementwise glue of the linear stack.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

#include "nmg.h"

namespace {

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

// ------------------------------------------------------------------ compress

template <typename T>
__global__ __launch_bounds__(kBlock) void k_compress(
    const T *__restrict__ W, int64_t ldw, T *__restrict__ values,
    uint8_t *__restrict__ indices, int K, int n, int m, int g, int C, int cpb) {
    using B = typename Bits<T>::type;
    __shared__ uint32_t key[kBlock];
    __shared__ uint8_t keep[kBlock];
    __shared__ uint8_t sel[kBlock];

    const int G = blockIdx.x;                 // group
    const int c_first = blockIdx.y * cpb;     // first chunk of this block
    const int t = threadIdx.x;
    const int lc = t / m, o = t - lc * m;     // local chunk, in-chunk offset
    const int c = c_first + lc;
    const bool in_block = lc < cpb && c < C;
    const int w = in_block ? min(m, K - c * m) : 0;
    const bool active = in_block && o < w;
    const int64_t ldv = (int64_t)C * n;
    const int64_t row0 = (int64_t)G * g;

    // group score, binary32, rows in ascending order
    uint32_t kk = 0;
    if (active) {
        const T *p = W + row0 * ldw + (int64_t)c * m + o;
        float s = 0.0f;
        for (int i = 0; i < g; ++i) s = s + fabsf((float)p[(int64_t)i * ldw]);
        // scores are >= +0 or NaN: as unsigned integers the bit patterns of
        // non-negative floats sort like the floats; NaNs become one value
        // above +inf
        kk = __builtin_isnan(s) ? 0x7fc00000u : __float_as_uint(s);
    }
    key[t] = kk;
    __syncthreads();

    // keep iff fewer than n columns of the chunk rank above this one
    bool kp = false;
    if (active) {
        const int base = lc * m;
        int rank = 0;
        for (int i = 0; i < w; ++i) {
            const uint32_t ki = key[base + i];
            rank += (ki > kk) || (i < o && ki == kk);
        }
        kp = rank < n;
    }
    keep[t] = kp;
    __syncthreads();

    if (kp) {
        const int base = lc * m;
        int slot = 0;
        for (int i = 0; i < o; ++i) slot += keep[base + i];
        indices[(int64_t)G * ldv + (int64_t)c * n + slot] = (uint8_t)o;
        sel[lc * n + slot] = (uint8_t)o;
    }
    __syncthreads();

    // copy the kept weights of the g rows, bit for bit, coalesced on output
    const int nout = min(cpb, C - c_first) * n;
    for (int i = 0; i < g; ++i) {
        const B *src = reinterpret_cast<const B *>(W + (row0 + i) * ldw);
        B *dst = reinterpret_cast<B *>(values + (row0 + i) * ldv) + (int64_t)c_first * n;
        for (int p = t; p < nout; p += kBlock) {
            const int cc = c_first + p / n;
            dst[p] = src[(int64_t)cc * m + sel[p]];
        }
    }
}

// --------------------------------------------------------------- spmm, MFMA

constexpr int kMfmaQuads = 16;                    // row quads per wave
constexpr int kMfmaRowsWave = 4 * kMfmaQuads;     // 64 rows per wave
constexpr int kMfmaRowsWg = 4 * kMfmaRowsWave;    // 256 rows per workgroup
constexpr int kMfmaTokens = 64;                   // tokens per workgroup
constexpr int kMfmaMaxWindowRows = 128;           // X rows staged per window

constexpr int ilog2(int v) { return v <= 1 ? 0 : 1 + ilog2(v / 2); }

// U: rows per group unit (U divides g, U % 4 == 0); KSW: k-slots per window
// (a power of two <= 16 that n divides).  A window is KSW/n whole chunks.
template <typename T, int U, int KSW>
__global__ __launch_bounds__(kBlock, 2) void k_spmm_mfma(
    const T *__restrict__ values, const uint8_t *__restrict__ indices,
    const T *__restrict__ X, int64_t ldx, T *__restrict__ Y, int64_t ldy,
    int M, int K, int N, int n, int m, int g, int C, int row_tiles, int tiles, bool xvec) {
    constexpr int UNITS = kMfmaRowsWave / U;      // group units per wave
    constexpr int QPU = U / 4;                    // quads per unit
    constexpr int CBSZ = ilog2(KSW);
    constexpr int PAIRS = UNITS * KSW;            // (unit, slot) pairs per window
    constexpr int PREGS = (PAIRS + 63) / 64;
    constexpr int TN = kMfmaTokens;
    __shared__ float xs[kMfmaMaxWindowRows * TN];

    const int tile = xcd_tile(blockIdx.x, tiles);
    const int rt = tile % row_tiles, tt = tile / row_tiles;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int r0 = rt * kMfmaRowsWg + wave * kMfmaRowsWave;
    const int t0 = tt * TN;
    const int64_t ldv = (int64_t)C * n;
    const int cpw = KSW / n;                      // chunks per window
    const int rpw = cpw * m;                      // X rows per window
    const int nwin = (C + cpw - 1) / cpw;

    // Per-lane constants for the (unit, slot) pairs this lane resolves:
    // pair p = u * KSW + s lives in register p / 64, lane p % 64.
    int pair_group[PREGS], pair_slot[PREGS], pair_chunk_row[PREGS];
    bool pair_live[PREGS];
#pragma unroll
    for (int r = 0; r < PREGS; ++r) {
        const int p = r * 64 + lane;
        const int u = p / KSW, s = p % KSW;
        const int row = r0 + u * U;
        pair_live[r] = p < PAIRS && row < M;
        pair_group[r] = row / g;
        pair_slot[r] = s;
        pair_chunk_row[r] = (s / n) * m;          // first window row of s's chunk
    }

    v4f acc[kMfmaQuads];
#pragma unroll
    for (int q = 0; q < kMfmaQuads; ++q) acc[q] = v4f{0.f, 0.f, 0.f, 0.f};

    for (int win = 0; win < nwin; ++win) {
        const int ks0 = win * KSW;                // first k-slot of the window
        const int xr0 = win * rpw;                // first X row of the window

        // stage X[xr0 .. xr0+rpw) x [t0, t0+64) as binary32
        __syncthreads();
        for (int e = threadIdx.x; e < rpw * (TN / 4); e += kBlock) {
            const int rr = e / (TN / 4), c4 = e % (TN / 4);
            const int k = xr0 + rr, tok = t0 + 4 * c4;
            v4f v = {0.f, 0.f, 0.f, 0.f};
            if (k < K) v = load4<T>(X + (int64_t)k * ldx + tok, N - tok, xvec);
            *reinterpret_cast<v4f *>(&xs[rr * TN + 4 * c4]) = v;
        }

        // A operands: lane 4b+i holds row (r0 + 4q + i), k-slot ks0 + b % KSW
        float a[kMfmaQuads];
        {
            const int i = lane & 3, s = (lane >> 2) & (KSW - 1);
            const int64_t ks = ks0 + s;
#pragma unroll
            for (int q = 0; q < kMfmaQuads; ++q) {
                const int row = r0 + 4 * q + i;
                a[q] = (row < M && ks < ldv) ? (float)values[(int64_t)row * ldv + ks] : 0.f;
            }
        }

        // LDS offset (floats) of the X row each (unit, slot) pair selects
        int pair_off[PREGS];
#pragma unroll
        for (int r = 0; r < PREGS; ++r) {
            const int64_t ks = ks0 + pair_slot[r];
            int off = 0;
            if (pair_live[r] && ks < ldv) {
                // clamped so that invalid indices still address the window
                const int o = min((int)indices[(int64_t)pair_group[r] * ldv + ks], m - 1);
                off = (pair_chunk_row[r] + o) * TN;
            }
            pair_off[r] = off;
        }
        __syncthreads();

        static_for<KSW>([&](auto sc) {
            constexpr int s = decltype(sc)::value;
            static_for<UNITS>([&](auto uc) {
                constexpr int u = decltype(uc)::value;
                constexpr int p = u * KSW + s;
                const int off = __builtin_amdgcn_readlane(pair_off[p / 64], p % 64);
                const float b = xs[off + lane];
                static_for<QPU>([&](auto qc) {
                    constexpr int q = u * QPU + decltype(qc)::value;
                    acc[q] = __builtin_amdgcn_mfma_f32_4x4x1f32(a[q], b, acc[q], CBSZ, s, 0);
                });
            });
        });
    }

    // output register i of quad q at lane l is Y[r0 + 4q + i][t0 + l]
    const int tok = t0 + lane;
    if (tok < N) {
#pragma unroll
        for (int q = 0; q < kMfmaQuads; ++q)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int row = r0 + 4 * q + i;
                if (row < M) Y[(int64_t)row * ldy + tok] = (T)acc[q][i];
            }
    }
}

// --------------------------------------------------------------- spmm, VALU

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

// ------------------------------------------------------------------ densify

template <typename T>
__global__ __launch_bounds__(kBlock) void k_densify(
    const T *__restrict__ values, const uint8_t *__restrict__ indices,
    T *__restrict__ out, int64_t ldw, int K, int n, int m, int g, int C) {
    using B = typename Bits<T>::type;
    const int64_t r = blockIdx.x;
    const int k = blockIdx.y * kBlock + threadIdx.x;
    if (k >= K) return;
    const int c = k / m, o = k - c * m;
    const int64_t ldv = (int64_t)C * n;
    const uint8_t *idx = indices + (r / g) * ldv + (int64_t)c * n;
    B v = 0;
    for (int s = 0; s < n; ++s)
        if (idx[s] == o) v = reinterpret_cast<const B *>(values)[r * ldv + (int64_t)c * n + s];
    reinterpret_cast<B *>(out)[r * ldw + k] = v;
}

// ------------------------------------------------------------- elementwise

template <typename T>
__global__ __launch_bounds__(kBlock) void k_gelu(const T *in, T *out, int64_t count) {
    const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (i >= count) return;
    const float x = (float)in[i];
    // 1 + erf(z) written as erfc(-z): no cancellation for negative x
    out[i] = (T)(0.5f * x * erfcf(-x * 0.70710678118654752f));
}

template <typename T>
__global__ __launch_bounds__(kBlock) void k_add(const T *a, const T *b, T *out, int64_t count) {
    const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (i >= count) return;
    out[i] = (T)((float)a[i] + (float)b[i]);
}

// ------------------------------------------------------------ host helpers

nmg_status check_layout(const nmg_layout *L) {
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

size_t elem_size(nmg_dtype d) { return d == NMG_F32 ? 4 : 2; }

bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

// X rows start on 4-element boundaries: four tokens come in one vector load.
bool x_vectorisable(const nmg_layout *L, const void *X, int64_t ldx) {
    return aligned(X, 4 * elem_size(L->dtype)) && ldx % 4 == 0;
}

nmg_status launched() {
    return hipGetLastError() == hipSuccess ? NMG_OK : NMG_ERR_LAUNCH;
}

// Largest power-of-two window (<= 16 k-slots) that n divides and whose
// chunks fit the staged-row budget; 0 if none.
int mfma_window(const nmg_layout *L) {
    for (int ksw = 16; ksw >= 1; ksw /= 2)
        if (ksw % L->n == 0 && (ksw / L->n) * L->m <= kMfmaMaxWindowRows) return ksw;
    return 0;
}

// Rows per group unit for the MFMA kernel: the largest of 32, 16, 8, 4 that
// divides g; 0 if g % 4 != 0.
int mfma_unit(const nmg_layout *L) {
    for (int u = 32; u >= 4; u /= 2)
        if (L->g % u == 0) return u;
    return 0;
}

template <typename T, int U>
nmg_status launch_mfma_u(const nmg_layout *L, int ksw, const void *values,
                         const uint8_t *indices, const void *X, int64_t ldx,
                         int N, void *Y, int64_t ldy, hipStream_t stream) {
    const bool xvec = x_vectorisable(L, X, ldx);
    const int row_tiles = (L->M + kMfmaRowsWg - 1) / kMfmaRowsWg;
    const int tok_tiles = (N + kMfmaTokens - 1) / kMfmaTokens;
    const int tiles = row_tiles * tok_tiles;
#define NMG_LAUNCH_MFMA(KSW)                                                            \
    hipLaunchKernelGGL((k_spmm_mfma<T, U, KSW>), dim3(tiles), dim3(kBlock), 0, stream,    \
                       (const T *)values, indices, (const T *)X, ldx, (T *)Y, ldy, L->M,  \
                       L->K, N, L->n, L->m, L->g, L->C, row_tiles, tiles, xvec)
    switch (ksw) {
        case 16: NMG_LAUNCH_MFMA(16); break;
        case 8: NMG_LAUNCH_MFMA(8); break;
        case 4: NMG_LAUNCH_MFMA(4); break;
        case 2: NMG_LAUNCH_MFMA(2); break;
        case 1: NMG_LAUNCH_MFMA(1); break;
        default: return NMG_ERR_UNSUPPORTED;
    }
#undef NMG_LAUNCH_MFMA
    return launched();
}

template <typename T>
nmg_status launch_mfma(const nmg_layout *L, const void *values, const uint8_t *indices,
                       const void *X, int64_t ldx, int N, void *Y, int64_t ldy,
                       hipStream_t stream) {
    const int ksw = mfma_window(L);
    switch (mfma_unit(L)) {
        case 32: return launch_mfma_u<T, 32>(L, ksw, values, indices, X, ldx, N, Y, ldy, stream);
        case 16: return launch_mfma_u<T, 16>(L, ksw, values, indices, X, ldx, N, Y, ldy, stream);
        case 8: return launch_mfma_u<T, 8>(L, ksw, values, indices, X, ldx, N, Y, ldy, stream);
        case 4: return launch_mfma_u<T, 4>(L, ksw, values, indices, X, ldx, N, Y, ldy, stream);
        default: return NMG_ERR_UNSUPPORTED;
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

bool mfma_supported(const nmg_layout *L) { return mfma_unit(L) != 0 && mfma_window(L) != 0; }

}  // namespace

// ===================================================================== C ABI

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
    const int cpb = kBlock / L->m;  // chunks per block, >= 1 since m <= 255
    dim3 grid(L->M / L->g, (L->C + cpb - 1) / cpb);
    if (L->dtype == NMG_F32)
        hipLaunchKernelGGL((k_compress<float>), grid, dim3(kBlock), 0, stream, (const float *)W, ldw,
                           (float *)values, indices, L->K, L->n, L->m, L->g, L->C, cpb);
    else
        hipLaunchKernelGGL((k_compress<_Float16>), grid, dim3(kBlock), 0, stream,
                           (const _Float16 *)W, ldw, (_Float16 *)values, indices, L->K, L->n, L->m,
                           L->g, L->C, cpb);
    return launched();
}

nmg_kernel nmg_spmm_auto_kernel(const nmg_layout *L, int64_t N) {
    (void)N;
    if (check_layout(L) != NMG_OK) return NMG_KERNEL_AUTO;
    return mfma_supported(L) ? NMG_KERNEL_MFMA : NMG_KERNEL_VALU;
}

nmg_status nmg_spmm_with(const nmg_layout *L, nmg_kernel kernel, const void *values,
                         const uint8_t *indices, const void *X, int64_t ldx, int64_t N, void *Y,
                         int64_t ldy, hipStream_t stream) {
    nmg_status st = check_layout(L);
    if (st != NMG_OK) return st;
    if (!values || !indices || !X || !Y) return NMG_ERR_NULL;
    if (N < 1 || N > INT32_MAX || ldx < N || ldy < N) return NMG_ERR_PARAM;
    const size_t es = elem_size(L->dtype);
    if (!aligned(X, es) || !aligned(values, es) || !aligned(Y, es)) return NMG_ERR_ALIGN;
    if (kernel == NMG_KERNEL_AUTO) kernel = nmg_spmm_auto_kernel(L, N);
    const int n32 = (int)N;
    if (kernel == NMG_KERNEL_MFMA) {
        if (!mfma_supported(L)) return NMG_ERR_UNSUPPORTED;
        return L->dtype == NMG_F32
                   ? launch_mfma<float>(L, values, indices, X, ldx, n32, Y, ldy, stream)
                   : launch_mfma<_Float16>(L, values, indices, X, ldx, n32, Y, ldy, stream);
    }
    if (kernel == NMG_KERNEL_VALU)
        return L->dtype == NMG_F32
                   ? launch_valu<float>(L, values, indices, X, ldx, n32, Y, ldy, stream)
                   : launch_valu<_Float16>(L, values, indices, X, ldx, n32, Y, ldy, stream);
    return NMG_ERR_PARAM;
}

nmg_status nmg_spmm(const nmg_layout *L, const void *values, const uint8_t *indices,
                    const void *X, int64_t ldx, int64_t N, void *Y, int64_t ldy,
                    hipStream_t stream) {
    return nmg_spmm_with(L, NMG_KERNEL_AUTO, values, indices, X, ldx, N, Y, ldy, stream);
}

nmg_status nmg_densify(const nmg_layout *L, const void *values, const uint8_t *indices,
                       void *W_out, int64_t ldw, hipStream_t stream) {
    nmg_status st = check_layout(L);
    if (st != NMG_OK) return st;
    if (!values || !indices || !W_out) return NMG_ERR_NULL;
    if (ldw < L->K) return NMG_ERR_PARAM;
    const size_t es = elem_size(L->dtype);
    if (!aligned(values, es) || !aligned(W_out, es)) return NMG_ERR_ALIGN;
    dim3 grid(L->M, (L->K + kBlock - 1) / kBlock);
    if (L->dtype == NMG_F32)
        hipLaunchKernelGGL((k_densify<float>), grid, dim3(kBlock), 0, stream, (const float *)values,
                           indices, (float *)W_out, ldw, L->K, L->n, L->m, L->g, L->C);
    else
        hipLaunchKernelGGL((k_densify<_Float16>), grid, dim3(kBlock), 0, stream,
                           (const _Float16 *)values, indices, (_Float16 *)W_out, ldw, L->K, L->n,
                           L->m, L->g, L->C);
    return launched();
}

nmg_status nmg_gelu(nmg_dtype dtype, const void *in, void *out, int64_t count,
                    hipStream_t stream) {
    if (dtype != NMG_F32 && dtype != NMG_F16) return NMG_ERR_DTYPE;
    if (!in || !out) return NMG_ERR_NULL;
    if (count < 0) return NMG_ERR_PARAM;
    if (count == 0) return NMG_OK;
    const size_t es = elem_size(dtype);
    if (!aligned(in, es) || !aligned(out, es)) return NMG_ERR_ALIGN;
    const int64_t blocks = (count + kBlock - 1) / kBlock;
    if (blocks > INT32_MAX) return NMG_ERR_PARAM;
    if (dtype == NMG_F32)
        hipLaunchKernelGGL((k_gelu<float>), dim3((unsigned)blocks), dim3(kBlock), 0, stream,
                           (const float *)in, (float *)out, count);
    else
        hipLaunchKernelGGL((k_gelu<_Float16>), dim3((unsigned)blocks), dim3(kBlock), 0, stream,
                           (const _Float16 *)in, (_Float16 *)out, count);
    return launched();
}

nmg_status nmg_add(nmg_dtype dtype, const void *a, const void *b, void *out, int64_t count,
                   hipStream_t stream) {
    if (dtype != NMG_F32 && dtype != NMG_F16) return NMG_ERR_DTYPE;
    if (!a || !b || !out) return NMG_ERR_NULL;
    if (count < 0) return NMG_ERR_PARAM;
    if (count == 0) return NMG_OK;
    const size_t es = elem_size(dtype);
    if (!aligned(a, es) || !aligned(b, es) || !aligned(out, es)) return NMG_ERR_ALIGN;
    const int64_t blocks = (count + kBlock - 1) / kBlock;
    if (blocks > INT32_MAX) return NMG_ERR_PARAM;
    if (dtype == NMG_F32)
        hipLaunchKernelGGL((k_add<float>), dim3((unsigned)blocks), dim3(kBlock), 0, stream,
                           (const float *)a, (const float *)b, (float *)out, count);
    else
        hipLaunchKernelGGL((k_add<_Float16>), dim3((unsigned)blocks), dim3(kBlock), 0, stream,
                           (const _Float16 *)a, (const _Float16 *)b, (_Float16 *)out, count);
    return launched();
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
    }
    return "unknown status";
}

const char *nmg_version(void) { return "nmg 0.1.0 gfx950"; }

}  // extern "C"
