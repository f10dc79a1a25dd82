// k_spmm_mfma.hpp -- the general matrix-core product (Section 5.1 on gfx950),
// included by one translation unit per element type.
//
// v_mfma_f32_4x4x1f32 runs 16 independent 4x4 outer products; with the
// A-operand broadcast (CBSZ/ABID) all 16 blocks multiply the same 4 weights
// (4 rows of one group, one k-slot) by 64 different tokens of the X row that
// the group selected.  One A register therefore carries the weights of 4 rows
// for up to 16 k-slots, and the gathered X row is one coalesced 64-lane LDS
// read.  A workgroup stages whole chunk windows of X (all m rows of each chunk,
// all its tokens) in LDS once and every group of its rows gathers from there.
// The gathered-row offsets of a window are computed lane-parallel and moved to
// scalar registers one by one, which any index layout allows.
#pragma once
#include "common.hpp"

namespace {

constexpr int kMfmaRowsWave = 32;                  // rows per wave (8 quads)
constexpr int kMfmaRowsWg = 4 * kMfmaRowsWave;     // 128 rows per workgroup
constexpr int kMfmaStageFloats = 4096;             // 16 KB per staging buffer, two buffers

// Staged X rows per window for a token tile of 64 * TPL.
__host__ __device__ constexpr int mfma_window_rows(int tpl) { return kMfmaStageFloats / (64 * tpl); }

template <int TPL> struct TokVec;
template <> struct TokVec<1> { typedef float type; };
template <> struct TokVec<2> { typedef float type __attribute__((ext_vector_type(2))); };

template <int TPL>
__device__ __forceinline__ float tok_part(const typename TokVec<TPL>::type &v, int p) {
    if constexpr (TPL == 1) { (void)p; return v; } else { return v[p]; }
}

// U: rows per group unit (U divides g, U % 4 == 0, U <= 32); KSW: k-slots per
// window (a power of two <= 16 that n divides; a window is KSW/n whole chunks);
// TPL: tokens per lane (workgroup token tile = 64 * TPL); DIRECT: X windows go
// from global memory straight to LDS (buffer loads with an LDS destination),
// which needs binary32 X, 16-byte aligned rows, whole token tiles and byte
// offsets of X within 32 bits; otherwise X passes
// through registers (and binary16 is widened on the way).
//
// Two LDS buffers, one barrier per window: window w is computed from one
// buffer while window w+1 (X rows, weights, indices) is in flight to the
// other.  Inside a window the gathered X rows of k-slot s+1 are read from LDS
// before the matrix instructions of k-slot s.
template <typename T, int U, int KSW, int TPL, bool DIRECT>
__global__ __launch_bounds__(kBlock, 2) void k_spmm_mfma(
    const T *__restrict__ values, const uint8_t *__restrict__ indices,
    const T *__restrict__ X, int64_t ldx, T *__restrict__ Y, int64_t ldy,
    int M, int K, int N, int n, int m, int g, int C, int row_tiles, int tiles, bool xvec,
    bool yvec) {
    static_assert(!DIRECT || std::is_same<T, float>::value, "direct staging copies binary32");
    constexpr int QW = kMfmaRowsWave / 4;         // quads per wave
    constexpr int UNITS = kMfmaRowsWave / U;      // group units per wave
    constexpr int QPU = U / 4;                    // quads per unit
    constexpr int TN = 64 * TPL;                  // tokens per workgroup
    constexpr int C4 = TN / 4;                    // 4-token vectors per staged row
    constexpr int MAXR = mfma_window_rows(TPL);   // staged rows per window, max
    constexpr int XV = MAXR * C4 / kBlock;        // register-staged vectors per thread
    constexpr int RPI = 1024 / (4 * TN);          // rows per direct load instruction
    constexpr int CBSZ = ilog2(KSW);
    constexpr int PAIRS = UNITS * KSW;            // (unit, slot) pairs per window
    constexpr int PREGS = (PAIRS + 63) / 64;
    typedef typename TokVec<TPL>::type BV;
    __shared__ float xs0[kMfmaStageFloats];
    __shared__ float xs1[kMfmaStageFloats];

    const int tile = xcd_tile(blockIdx.x, tiles);
    const int rt = tile % row_tiles, tt = tile / row_tiles;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int r0 = rt * kMfmaRowsWg + wave * kMfmaRowsWave;
    const int t0 = tt * TN;
    const int64_t ldv = (int64_t)C * n;
    const int cpw = KSW / n;                      // chunks per window
    const int rpw = cpw * m;                      // X rows per window (<= MAXR)
    const int nwin = (C + cpw - 1) / cpw;

    // (unit, slot) pair p = u * KSW + s is resolved by register p / 64, lane p % 64
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
        pair_chunk_row[r] = (s / n) * m;
    }

    // ---- staging of the X rows of a window (direct: buffer loads,
    // lds_copy16_buf; host: the byte offsets of X fit 32 bits)
    const buf_rsrc_t xrs = buf_rsrc(X, DIRECT ? (uint32_t)((int64_t)K * ldx * 4) : 0u);
    auto issue_direct = [&](int win, float *buf) {
        if constexpr (DIRECT) {
            // one instruction moves RPI rows (1 KB); lane l writes 16 bytes at
            // buf + 16 l, i.e. row l / C4, tokens 4 (l % C4) .. + 3
            const int xr0 = win * rpw;
            const int ninst = (rpw + RPI - 1) / RPI;
            const int sub = lane / C4, c4 = lane % C4;
            for (int j = wave; j < ninst; j += 4) {
                // rows past K are loaded from row K-1: never selected
                const int k = min(xr0 + j * RPI + sub, K - 1);
                lds_copy16_buf(xrs, ((uint32_t)k * (uint32_t)ldx + (uint32_t)(t0 + 4 * c4)) * 4u,
                               buf + j * RPI * TN);
            }
        } else {
            (void)win;
            (void)buf;
        }
    };
    auto load_x = [&](int win, v4f (&xr)[XV]) {
        const int xr0 = win * rpw;
#pragma unroll
        for (int p = 0; p < XV; ++p) {
            const int e = threadIdx.x + p * kBlock;
            const int rr = e / C4, c4 = e % C4;
            const int k = xr0 + rr, tok = t0 + 4 * c4;
            xr[p] = v4f{0.f, 0.f, 0.f, 0.f};
            if (rr < rpw && k < K) xr[p] = load4<T>(X + (int64_t)k * ldx + tok, N - tok, xvec);
        }
    };
    auto store_x = [&](const v4f (&xr)[XV], float *buf) {
#pragma unroll
        for (int p = 0; p < XV; ++p) {
            const int e = threadIdx.x + p * kBlock;
            const int rr = e / C4, c4 = e % C4;
            if (rr < rpw) *reinterpret_cast<v4f *>(&buf[rr * TN + 4 * c4]) = xr[p];
        }
    };
    // A operands: lane 4b+i holds row (r0 + 4q + i) at k-slot ks0 + b % KSW
    auto load_a = [&](int win, float (&a)[QW]) {
        const int i = lane & 3, s = (lane >> 2) & (KSW - 1);
        const int64_t ks = (int64_t)win * KSW + s;
#pragma unroll
        for (int q = 0; q < QW; ++q) {
            const int row = r0 + 4 * q + i;
            a[q] = (row < M && ks < ldv) ? (float)values[(int64_t)row * ldv + ks] : 0.f;
        }
    };
    auto load_idx = [&](int win, int (&raw)[PREGS]) {
#pragma unroll
        for (int r = 0; r < PREGS; ++r) {
            const int64_t ks = (int64_t)win * KSW + pair_slot[r];
            raw[r] = (pair_live[r] && ks < ldv) ? (int)indices[(int64_t)pair_group[r] * ldv + ks]
                                                : 0;
        }
    };

    v4f acc[QW][TPL];
#pragma unroll
    for (int q = 0; q < QW; ++q)
#pragma unroll
        for (int p = 0; p < TPL; ++p) acc[q][p] = v4f{0.f, 0.f, 0.f, 0.f};

    v4f xr[DIRECT ? 1 : XV];
    float a_nx[QW];
    int raw_nx[PREGS];
    if constexpr (DIRECT) {
        issue_direct(0, xs0);
    } else {
        load_x(0, xr);
        store_x(xr, xs0);
    }
    load_a(0, a_nx);
    load_idx(0, raw_nx);

    auto step = [&](int win, float *cur, float *nxt) {
        if constexpr (DIRECT) wait_all_memory();  // this wave's copies into cur have landed
        __syncthreads();  // cur is complete; every wave is done with nxt
        float a[QW];
#pragma unroll
        for (int q = 0; q < QW; ++q) a[q] = a_nx[q];
        int pair_off[PREGS];  // LDS offset (floats) of each pair's row, clamped into the window
#pragma unroll
        for (int r = 0; r < PREGS; ++r) pair_off[r] = (pair_chunk_row[r] + min(raw_nx[r], m - 1)) * TN;
        const bool more = win + 1 < nwin;
        if (more) {
            if constexpr (DIRECT) issue_direct(win + 1, nxt);
            else load_x(win + 1, xr);
            load_a(win + 1, a_nx);
            load_idx(win + 1, raw_nx);
        }

        BV b[2][UNITS];
        auto read_b = [&](auto sc, BV (&dst)[UNITS]) {
            constexpr int s = decltype(sc)::value;
            static_for<UNITS>([&](auto uc) {
                constexpr int u = decltype(uc)::value;
                constexpr int p = u * KSW + s;
                // offsets are multiples of TN floats: index LDS in whole vectors
                const int off = __builtin_amdgcn_readlane(pair_off[p / 64], p % 64);
                dst[u] = reinterpret_cast<const BV *>(cur)[off / TPL + lane];
            });
        };
        read_b(std::integral_constant<int, 0>{}, b[0]);
        static_for<KSW>([&](auto sc) {
            constexpr int s = decltype(sc)::value;
            if constexpr (s + 1 < KSW) read_b(std::integral_constant<int, s + 1>{}, b[(s + 1) & 1]);
            static_for<UNITS>([&](auto uc) {
                constexpr int u = decltype(uc)::value;
                static_for<QPU>([&](auto qc) {
                    constexpr int q = u * QPU + decltype(qc)::value;
                    static_for<TPL>([&](auto pc) {
                        constexpr int p = decltype(pc)::value;
                        acc[q][p] = __builtin_amdgcn_mfma_f32_4x4x1f32(
                            a[q], tok_part<TPL>(b[s & 1][u], p), acc[q][p], CBSZ, s, 0);
                    });
                });
            });
        });
        if constexpr (!DIRECT)
            if (more) store_x(xr, nxt);
    };
    for (int win = 0; win < nwin; win += 2) {
        step(win, xs0, xs1);
        if (win + 1 < nwin) step(win + 1, xs1, xs0);
    }

    // output register i of (quad q, part p) at lane l is Y[r0 + 4q + i][t0 + TPL*l + p]
    const int tok = t0 + TPL * lane;
#pragma unroll
    for (int q = 0; q < QW; ++q)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int row = r0 + 4 * q + i;
            if (row >= M) continue;
            T *y = Y + (int64_t)row * ldy + tok;
            if constexpr (TPL == 2) {
                if (yvec && tok + 1 < N) {
                    typedef T T2 __attribute__((ext_vector_type(2)));
                    *reinterpret_cast<T2 *>(y) = T2{(T)acc[q][0][i], (T)acc[q][1][i]};
                    continue;
                }
            }
#pragma unroll
            for (int p = 0; p < TPL; ++p)
                if (tok + p < N) y[p] = (T)acc[q][p][i];
        }
}

// Tokens per lane of the MFMA kernel: the 128-token tile when it still gives
// at least two workgroups per CU, else the 64-token tile.
int mfma_tpl(const nmg_layout *L, int64_t N) {
    const int64_t row_tiles = (L->M + kMfmaRowsWg - 1) / kMfmaRowsWg;
    return row_tiles * ((N + 127) / 128) >= 512 ? 2 : 1;
}

// Largest power-of-two window (2 .. 16 k-slots) that n divides and whose
// chunks fit the staged-row budget; 0 if none.
int mfma_window(const nmg_layout *L, int tpl) {
    for (int ksw = 16; ksw >= 2; ksw /= 2)
        if (ksw % L->n == 0 && (ksw / L->n) * L->m <= mfma_window_rows(tpl)) return ksw;
    return 0;
}

template <typename T, int U, int TPL, bool DIRECT>
nmg_status launch_mfma_utd(const nmg_layout *L, int ksw, const void *values,
                           const uint8_t *indices, const void *X, int64_t ldx, int N, void *Y,
                           int64_t ldy, bool xvec, bool yvec, hipStream_t stream) {
    const int row_tiles = (L->M + kMfmaRowsWg - 1) / kMfmaRowsWg;
    const int tok_tiles = (N + 64 * TPL - 1) / (64 * TPL);
    const int tiles = row_tiles * tok_tiles;
#define NMG_LAUNCH_MFMA(KSW)                                                                   \
    hipLaunchKernelGGL((k_spmm_mfma<T, U, KSW, TPL, DIRECT>), dim3(tiles), dim3(kBlock), 0,      \
                       stream, (const T *)values, indices, (const T *)X, ldx, (T *)Y, ldy, L->M, \
                       L->K, N, L->n, L->m, L->g, L->C, row_tiles, tiles, xvec, yvec)
    switch (ksw) {
        case 16: NMG_LAUNCH_MFMA(16); break;
        case 8: NMG_LAUNCH_MFMA(8); break;
        case 4: NMG_LAUNCH_MFMA(4); break;
        case 2: NMG_LAUNCH_MFMA(2); break;
        default: return NMG_ERR_UNSUPPORTED;
    }
#undef NMG_LAUNCH_MFMA
    return launched();
}

template <typename T, int U, int TPL>
nmg_status launch_mfma_ut(const nmg_layout *L, int ksw, const void *values,
                          const uint8_t *indices, const void *X, int64_t ldx, int N, void *Y,
                          int64_t ldy, hipStream_t stream) {
    const bool xvec = x_vectorisable(L, X, ldx);
    const bool yvec = aligned(Y, 2 * elem_size(L->dtype)) && ldy % 2 == 0;
    if constexpr (std::is_same<T, float>::value) {
        // direct global -> LDS staging: 16-byte rows, whole token tiles and
        // byte offsets of X within 32 bits
        if (xvec && N % (64 * TPL) == 0 && (int64_t)L->K * ldx * 4 <= (int64_t)0xffffffff)
            return launch_mfma_utd<T, U, TPL, true>(L, ksw, values, indices, X, ldx, N, Y, ldy,
                                                    xvec, yvec, stream);
    }
    return launch_mfma_utd<T, U, TPL, false>(L, ksw, values, indices, X, ldx, N, Y, ldy, xvec,
                                             yvec, stream);
}

template <typename T, int U>
nmg_status launch_mfma_u(const nmg_layout *L, const void *values, const uint8_t *indices,
                         const void *X, int64_t ldx, int N, void *Y, int64_t ldy,
                         hipStream_t stream) {
    const int tpl = mfma_tpl(L, N);
    const int ksw = mfma_window(L, tpl);
    if (tpl == 2)
        return launch_mfma_ut<T, U, 2>(L, ksw, values, indices, X, ldx, N, Y, ldy, stream);
    return launch_mfma_ut<T, U, 1>(L, ksw, values, indices, X, ldx, N, Y, ldy, stream);
}

template <typename T>
nmg_status launch_mfma(const nmg_layout *L, const void *values, const uint8_t *indices,
                       const void *X, int64_t ldx, int N, void *Y, int64_t ldy,
                       hipStream_t stream) {
    switch (mfma_unit(L)) {
        case 32: return launch_mfma_u<T, 32>(L, values, indices, X, ldx, N, Y, ldy, stream);
        case 16: return launch_mfma_u<T, 16>(L, values, indices, X, ldx, N, Y, ldy, stream);
        case 8: return launch_mfma_u<T, 8>(L, values, indices, X, ldx, N, Y, ldy, stream);
        case 4: return launch_mfma_u<T, 4>(L, values, indices, X, ldx, N, Y, ldy, stream);
        default: return NMG_ERR_UNSUPPORTED;
    }
}

[[maybe_unused]] bool mfma_supported(const nmg_layout *L, int64_t N) {
    return mfma_unit(L) != 0 && mfma_window(L, mfma_tpl(L, N)) != 0;
}

}  // namespace
