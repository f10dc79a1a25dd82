// k_spmm_mfma_s.hpp -- the matrix-core product with scalar-loaded indices,
// included by one translation unit per (element type, group unit).
#pragma once
#include "common.hpp"

namespace {

// The fast matrix-core kernel, for layouts with n a power of two and windows
// of 4, 8 or 16 k-slots.  Differences from k_spmm_mfma: a wave owns 16 rows
// (4 quads) and 64*TPL tokens; the workgroup has a runtime number of waves so
// that the tile count fits the GPU in whole rounds; the index words of a
// window are loaded by distinct lanes and moved to scalar registers once per
// window, so every gathered-row offset is computed on the scalar unit; one LDS
// read of TPL tokens per lane feeds TPL*U/4 matrix instructions.
constexpr int kFastRowsWave = 16;                  // 4 quads
constexpr int kFastMaxWaves = 16;
// Staging buffers: 64 KB each when X is copied straight to LDS in its own
// element type, 32 KB when it passes through registers (as binary32).
__host__ __device__ constexpr int fast_stage_bytes(bool direct) { return direct ? 65536 : 32768; }
// Staged X rows per window for a token tile of 64 * TPL elements of `es` bytes.
__host__ __device__ constexpr int fast_window_rows(int tpl, bool direct, int es) {
    return fast_stage_bytes(direct) / (64 * tpl * es);
}

// TPL consecutive staged elements (the tokens one lane multiplies).
template <typename SE, int TPL> struct TokVec4 {
    typedef SE type __attribute__((ext_vector_type(TPL)));
};
template <typename SE> struct TokVec4<SE, 1> { typedef SE type; };

template <typename SE, int TPL>
__device__ __forceinline__ float tok_part4(const typename TokVec4<SE, TPL>::type &v, int p) {
    if constexpr (TPL == 1) { (void)p; return (float)v; } else { return (float)v[p]; }
}

template <typename T, int U, int KSW, int TPL, bool DIRECT>
__global__ __launch_bounds__(DIRECT ? 64 * kFastMaxWaves : 64 * kFastMaxWaves / 2) void k_spmm_mfma_s(
    const T *__restrict__ values, const uint8_t *__restrict__ indices,
    const T *__restrict__ X, int64_t ldx, T *__restrict__ Y, int64_t ldy,
    int M, int K, int N, int log2n, int m, int g, int C, int row_tiles, int tiles, bool xvec,
    bool yvec) {
    static_assert(KSW % 4 == 0 && U <= kFastRowsWave, "window of whole index words");
    // staged element: X's own type when copied directly, binary32 otherwise
    typedef typename std::conditional<DIRECT, T, float>::type SE;
    constexpr int SES = (int)sizeof(SE);
    constexpr int QW = kFastRowsWave / 4;         // quads per wave
    constexpr int UNITS = kFastRowsWave / U;      // group units per wave
    constexpr int QPU = U / 4;                    // quads per unit
    constexpr int TN = 64 * TPL;                  // tokens per workgroup
    constexpr int C4 = TN / 4;                    // 4-token vectors per staged row
    constexpr int MAXR = fast_window_rows(TPL, DIRECT, SES);  // staged rows per window, max
    constexpr int EPL = 16 / SES;                 // elements per lane of a direct copy
    constexpr int LPR = TN / EPL;                 // lanes per staged row (direct copy)
    constexpr int RPI = 64 / LPR;                 // rows per direct copy instruction (1 KB)
    constexpr int CBSZ = ilog2(KSW);
    constexpr int IW = KSW / 4;                   // index words per unit and window
    constexpr int XVMAX = (MAXR * C4 + 4 * 64 - 1) / (4 * 64);  // register staging, >= 4 waves
    typedef typename TokVec4<SE, TPL>::type BV;
    __shared__ SE xs0[fast_stage_bytes(DIRECT) / SES];
    __shared__ SE xs1[fast_stage_bytes(DIRECT) / SES];

    const int nthreads = blockDim.x;
    const int nwaves = nthreads >> 6;
    const int tile = xcd_tile(blockIdx.x, tiles);
    const int rt = tile % row_tiles, tt = tile / row_tiles;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int r0 = rt * (kFastRowsWave * nwaves) + wave * kFastRowsWave;
    const int t0 = tt * TN;
    const int n = 1 << log2n;                     // n is a power of two here
    const int ldv = C * n;                        // host checked: M * ldv < 2^31
    const int cpw = KSW >> log2n;                 // chunks per window
    const int rpw = cpw * m;                      // X rows per window (<= MAXR)
    const int nwin = (C + cpw - 1) / cpw;
    const bool ragged = nwin * KSW > ldv;         // the last window runs past the k-slots

    // index row of each unit (rows past M read the last group; never stored)
    const uint8_t *irow[UNITS];
#pragma unroll
    for (int u = 0; u < UNITS; ++u) {
        const int G = min(r0 + u * U, M - 1) / g;
        irow[u] = indices + (int64_t)G * ldv;
    }
    // per-lane offsets of the A operands: lane 4b+i holds row r0+4q+i, slot b % KSW
    int aoff[QW];
#pragma unroll
    for (int q = 0; q < QW; ++q)
        aoff[q] = min(r0 + 4 * q + (lane & 3), M - 1) * ldv + ((lane >> 2) & (KSW - 1));

    auto load_a = [&](int win, float (&a)[QW], bool guarded) {
        const T *vb = values + win * KSW;
#pragma unroll
        for (int q = 0; q < QW; ++q) {
            if (!guarded) {
                a[q] = (float)vb[aoff[q]];
            } else {
                const int s = (lane >> 2) & (KSW - 1);
                a[q] = win * KSW + s < ldv ? (float)vb[aoff[q]] : 0.f;
            }
        }
    };
    // index words of the window: lane u*IW + j loads word j of unit u with a
    // vector load (lane-distinct addresses), so that LDS waits never wait for
    // them; they reach scalar registers by readlane when the window starts
    static_assert(UNITS * IW <= 64, "one index word per lane");
    const int iw_u = min(lane / IW, UNITS - 1), iw_j = lane % IW;
    const uint8_t *iw_row = irow[0];
#pragma unroll
    for (int u = 1; u < UNITS; ++u)
        if (iw_u == u) iw_row = irow[u];
    auto load_idx = [&](int win, uint32_t &wv, bool guarded) {
        const uint8_t *p = iw_row + win * KSW + 4 * iw_j;
        if (!guarded && (reinterpret_cast<uintptr_t>(p) & 3) == 0) {
            wv = *reinterpret_cast<const uint32_t *>(p);
        } else {  // the last window, or an index row not on a 4-byte boundary
            uint32_t x = 0;
#pragma unroll
            for (int b = 0; b < 4; ++b)
                if (win * KSW + 4 * iw_j + b < ldv) x |= (uint32_t)p[b] << (8 * b);
            wv = x;
        }
    };
    // X rows of a window into LDS, by buffer loads (lds_copy16_buf; host: the
    // byte offsets of X fit 32 bits on this path)
    const buf_rsrc_t xrs = buf_rsrc(X, DIRECT ? (uint32_t)((int64_t)K * ldx * (int64_t)sizeof(T)) : 0u);
    auto issue_direct = [&](int win, SE *buf) {
        if constexpr (DIRECT) {
            // lane l copies 16 bytes: row l / LPR, elements EPL * (l % LPR) ..
            const int xr0 = win * rpw;
            const int ninst = (rpw + RPI - 1) / RPI;
            const int sub = lane / LPR, ce = EPL * (lane % LPR);
            const int lane_x = sub * (int)ldx + t0 + ce;  // host checked: K * ldx < 2^31
            for (int j = wave; j < ninst; j += nwaves) {
                const int kb = xr0 + j * RPI;  // first row of this instruction (uniform)
                // rows past K (the last window): the last row, never selected
                const uint32_t el = kb + RPI <= K
                                        ? (uint32_t)kb * (uint32_t)ldx + (uint32_t)lane_x
                                        : (uint32_t)min(kb + sub, K - 1) * (uint32_t)ldx + (uint32_t)(t0 + ce);
                lds_copy16_buf(xrs, el * (uint32_t)sizeof(T), buf + j * RPI * TN);
            }
        } else {
            (void)win;
            (void)buf;
        }
    };
    auto load_x = [&](int win, v4f (&xr)[XVMAX]) {
        const int xr0 = win * rpw;
#pragma unroll
        for (int p = 0; p < XVMAX; ++p) {
            const int e = threadIdx.x + p * nthreads;
            const int rr = e / C4, c4 = e % C4;
            const int k = xr0 + rr, tok = t0 + 4 * c4;
            xr[p] = v4f{0.f, 0.f, 0.f, 0.f};
            if (rr < rpw && k < K) xr[p] = load4<T>(X + (int64_t)k * ldx + tok, N - tok, xvec);
        }
    };
    auto store_x = [&](const v4f (&xr)[XVMAX], SE *buf) {
#pragma unroll
        for (int p = 0; p < XVMAX; ++p) {
            const int e = threadIdx.x + p * nthreads;
            const int rr = e / C4, c4 = e % C4;
            if constexpr (!DIRECT)
                if (rr < rpw) *reinterpret_cast<v4f *>(&buf[rr * TN + 4 * c4]) = xr[p];
        }
    };

    v4f acc[QW][TPL];
#pragma unroll
    for (int q = 0; q < QW; ++q)
#pragma unroll
        for (int p = 0; p < TPL; ++p) acc[q][p] = v4f{0.f, 0.f, 0.f, 0.f};

    v4f xr[DIRECT ? 1 : XVMAX];
    float a0[QW], a1[QW];       // weights of even / odd windows
    uint32_t w0 = 0, w1 = 0;    // index words of even / odd windows (one per lane)
    if constexpr (DIRECT) {
        issue_direct(0, xs0);
    } else {
        load_x(0, xr);
        store_x(xr, xs0);
    }
    load_a(0, a0, ragged && nwin == 1);
    load_idx(0, w0, ragged && nwin == 1);

    // window `win` from LDS buffer `cur` with weights `a` and index words `wv`;
    // window win+1 goes to `nxt`, `a_nxt`, `wv_nxt` meanwhile
    auto step = [&](int win, SE *cur, SE *nxt, const float (&a)[QW], uint32_t wv,
                    float (&a_nxt)[QW], uint32_t &wv_nxt) {
        if constexpr (DIRECT) wait_all_memory();  // this wave's loads for `win` have landed
        __syncthreads();  // cur is complete; every wave is done with nxt
        uint32_t w[UNITS][IW];
#pragma unroll
        for (int u = 0; u < UNITS; ++u)
#pragma unroll
            for (int j = 0; j < IW; ++j) w[u][j] = __builtin_amdgcn_readlane(wv, u * IW + j);
        const bool more = win + 1 < nwin;
        if (more) {
            const bool last_guarded = ragged && win + 2 == nwin;
            if constexpr (DIRECT) issue_direct(win + 1, nxt);
            else load_x(win + 1, xr);
            load_a(win + 1, a_nxt, last_guarded);
            load_idx(win + 1, wv_nxt, last_guarded);
        }

        const BV *cv = reinterpret_cast<const BV *>(cur);
        BV b[2][UNITS];
        auto read_b = [&](auto sc, BV (&dst)[UNITS]) {
            constexpr int s = decltype(sc)::value;
            static_for<UNITS>([&](auto uc) {
                constexpr int u = decltype(uc)::value;
                // scalar: byte s of the unit's index words, clamped into the chunk
                const uint32_t o = min((w[u][s / 4] >> (8 * (s % 4))) & 0xffu, (uint32_t)(m - 1));
                const uint32_t row = (uint32_t)((s >> log2n) * m) + o;
                const BV *rp = cv + row * 64;  // uniform row address
                dst[u] = rp[lane];
            });
        };
        read_b(std::integral_constant<int, 0>{}, b[0]);
        static_for<KSW>([&](auto sc) {
            constexpr int s = decltype(sc)::value;
            if constexpr (s + 1 < KSW) read_b(std::integral_constant<int, s + 1>{}, b[(s + 1) & 1]);
            // keep the reads of slot s+1 ahead of the matrix instructions of
            // slot s, so that their latency hides behind them
            __builtin_amdgcn_sched_barrier(0);
            static_for<UNITS>([&](auto uc) {
                constexpr int u = decltype(uc)::value;
                static_for<QPU>([&](auto qc) {
                    constexpr int q = u * QPU + decltype(qc)::value;
                    static_for<TPL>([&](auto pc) {
                        constexpr int p = decltype(pc)::value;
                        acc[q][p] = __builtin_amdgcn_mfma_f32_4x4x1f32(
                            a[q], tok_part4<SE, TPL>(b[s & 1][u], p), acc[q][p], CBSZ, s, 0);
                    });
                });
            });
        });
        if constexpr (!DIRECT)
            if (more) store_x(xr, nxt);
    };
    for (int win = 0; win < nwin; win += 2) {
        step(win, xs0, xs1, a0, w0, a1, w1);
        if (win + 1 < nwin) step(win + 1, xs1, xs0, a1, w1, a0, w0);
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
            // Y is written once and not read here again: non-temporal stores
            // keep it from evicting the X rows other workgroups still gather
            if constexpr (TPL > 1) {
                if (yvec && tok + TPL - 1 < N) {
                    typedef T TV __attribute__((ext_vector_type(TPL)));
                    TV v;
#pragma unroll
                    for (int p = 0; p < TPL; ++p) v[p] = (T)acc[q][p][i];
                    __builtin_nontemporal_store(v, reinterpret_cast<TV *>(y));
                    continue;
                }
            }
#pragma unroll
            for (int p = 0; p < TPL; ++p)
                if (tok + p < N) __builtin_nontemporal_store((T)acc[q][p][i], y + p);
        }
}

// ---------------------------------------------------- fast kernel selection

// Largest window of 16, 8 or 4 k-slots that n divides and whose chunks fit
// the staged rows of the variant; 0 if none.  (The register-staged variant's
// smaller budget decides whether the layout is taken at all.)
int fast_window(const nmg_layout *L, int tpl, bool direct = false) {
    const int es = direct ? (int)elem_size(L->dtype) : 4;
    for (int ksw = 16; ksw >= 4; ksw /= 2)
        if (ksw % L->n == 0 && (ksw / L->n) * L->m <= fast_window_rows(tpl, direct, es)) return ksw;
    return 0;
}

// `indices` may be NULL to ask about the layout alone.
[[maybe_unused]] bool fast_supported(const nmg_layout *L, const uint8_t *indices, int64_t ldx) {
    const int64_t ldv = (int64_t)L->C * L->n;
    (void)indices;
    return mfma_unit(L) != 0 && (L->n & (L->n - 1)) == 0 &&
           (int64_t)L->M * ldv < ((int64_t)1 << 31) &&
           (int64_t)L->K * ldx < ((int64_t)1 << 31) && fast_window(L, 1) != 0;
}

template <typename T, int U, int KSW, int TPL, bool DIRECT>
const void *fast_kernel() {
    return reinterpret_cast<const void *>(&k_spmm_mfma_s<T, U, KSW, TPL, DIRECT>);
}

template <typename T, int U, int KSW, int TPL, bool DIRECT>
nmg_status launch_fast_v(const nmg_layout *L, const void *values, const uint8_t *indices,
                         const void *X, int64_t ldx, int N, void *Y, int64_t ldy, bool xvec,
                         hipStream_t stream) {
    const void *kern = fast_kernel<T, U, KSW, TPL, DIRECT>();
    // waves per workgroup: the count whose tiles fill whole rounds of the GPU best
    const int cus = device_cus();
    const int tok_tiles = (N + 64 * TPL - 1) / (64 * TPL);
    int best_w = 4;
    double best_eff = -1.0;
    // register-staged variants keep more registers: at most half the waves
    for (int w = 4; w <= (DIRECT ? kFastMaxWaves : kFastMaxWaves / 2); ++w) {
        const int64_t tiles = (int64_t)((L->M + kFastRowsWave * w - 1) / (kFastRowsWave * w)) * tok_tiles;
        const int64_t slots = (int64_t)cus * kernel_occupancy(kern, 64 * w) * w;  // waves resident at once
        const int64_t rounds = (tiles * w + slots - 1) / slots;
        const double eff = (double)(tiles * w) / (double)(rounds * slots);
        // best fill of whole rounds; on a tie the larger workgroup (its staged
        // X windows feed more rows) -- unless the grid leaves CUs idle, where
        // more, smaller workgroups spread the work wider
        const bool tie = eff > best_eff - 1e-9 && eff < best_eff + 1e-9;
        if (eff > best_eff + 1e-9 || (tie && tiles >= cus)) {
            best_eff = std::max(eff, best_eff);
            best_w = w;
        }
    }
    const int row_tiles = (L->M + kFastRowsWave * best_w - 1) / (kFastRowsWave * best_w);
    const int tiles = row_tiles * tok_tiles;
    const bool yvec = aligned(Y, TPL * elem_size(L->dtype)) && ldy % TPL == 0;
    int log2n = 0;
    while ((1 << log2n) < L->n) ++log2n;
    hipLaunchKernelGGL((k_spmm_mfma_s<T, U, KSW, TPL, DIRECT>), dim3(tiles), dim3(64 * best_w), 0,
                       stream, (const T *)values, indices, (const T *)X, ldx, (T *)Y, ldy, L->M,
                       L->K, N, log2n, L->m, L->g, L->C, row_tiles, tiles, xvec, yvec);
    return launched();
}

template <typename T, int U, int TPL>
nmg_status launch_fast_ut(const nmg_layout *L, const void *values, const uint8_t *indices,
                          const void *X, int64_t ldx, int N, void *Y, int64_t ldy,
                          hipStream_t stream) {
    const bool xvec = x_vectorisable(L, X, ldx);
    // direct copies move 16 bytes per lane: 16-byte rows and whole token
    // tiles; their buffer offsets must fit 32 bits
    const bool direct = aligned(X, 16) && (ldx * (int64_t)sizeof(T)) % 16 == 0 &&
                        N % (64 * TPL) == 0 &&
                        (int64_t)L->K * ldx * (int64_t)sizeof(T) <= (int64_t)0xffffffff;
#define NMG_FAST(KSW)                                                                           \
    return direct ? launch_fast_v<T, U, KSW, TPL, true>(L, values, indices, X, ldx, N, Y, ldy,   \
                                                        xvec, stream)                           \
                  : launch_fast_v<T, U, KSW, TPL, false>(L, values, indices, X, ldx, N, Y, ldy, \
                                                         xvec, stream)
    switch (fast_window(L, TPL, direct)) {
        case 16: NMG_FAST(16);
        case 8: NMG_FAST(8);
        case 4: NMG_FAST(4);
        default: return NMG_ERR_UNSUPPORTED;
    }
#undef NMG_FAST
}

// Tokens per lane of the fast kernel: 4 when a window of at least 4 k-slots
// fits 32 staged rows and the 256-token tiles still cover every CU, else 2,
// else 1.
int fast_tpl(const nmg_layout *L, int64_t N) {
    const int cus = device_cus();
    const int64_t row_tiles = (L->M + kFastRowsWave * 8 - 1) / (kFastRowsWave * 8);
    if (fast_window(L, 4) && row_tiles * ((N + 255) / 256) >= cus) return 4;
    if (fast_window(L, 2) && row_tiles * ((N + 127) / 128) >= cus) return 2;
    return fast_window(L, 2) && N >= 128 ? 2 : 1;
}

}  // namespace
