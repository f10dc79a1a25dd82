// k_spmm_valu_s.hip -- Y = W_s X (Section 5.1) with vector FMAs on X windows
// staged in LDS: the product for layouts whose groups are not whole quads of
// rows (g % 4 != 0, g = 1 above all), where every row gathers its own X rows
// and the matrix-core kernels decline.
//
// The vector kernel (k_spmm_valu) gathers each row's X rows from global
// memory, one load per 4 multiply-adds.  Here a workgroup of 64 (or 256) rows
// x 256 tokens copies a window of whole chunks of X (global -> LDS, 16 bytes per
// lane) once, and every row reads the rows it selects from LDS: one 16-byte
// LDS read per lane feeds 4 FMAs, and each staged row serves every row of the
// workgroup that selects it.  Weights and index bytes of 16 rows x 4 slots
// come with one vector load per lane and reach scalar registers by readlane;
// the gathered row's LDS address is computed on the scalar unit.
#include "common.hpp"

namespace {

constexpr int kVsRowsWave = 16;
constexpr int kVsTok = 256;                         // 4 tokens per lane
constexpr int kVsGroups = 4;                        // groups of 4 k-slots per window, max
// Two shapes: workgroups of 4 waves (64 rows) with 32 KB staging buffers, and,
// where such a window holds a single k-slot (m > 16 at n = 1), 16 waves (256
// rows, each staged row serving 4 times as many) with 64 KB buffers, so that a
// window holds several chunks: on 3072 x 768 x 4096 at 1:20:1 220 -> 97 us
// (the gathering vector kernel: 139); at m <= 10 the small shape is faster
// (1:10:1 156 against 171 us).
constexpr int kVsSmallWaves = 4, kVsSmallStage = 32768;
constexpr int kVsWideWaves = 16, kVsWideStage = 65536;

template <typename T, int SB> constexpr int vs_rows_max() { return SB / (kVsTok * (int)sizeof(T)); }

// 4 staged tokens of row `row` at this lane
template <typename T>
__device__ __forceinline__ v4f vs_read(const T *buf, uint32_t row, int lane) {
    static_assert(sizeof(T) == 4, "binary32 staging");
    return *reinterpret_cast<const v4f *>(buf + row * kVsTok + 4 * lane);
}

template <typename T, int WAVES, int SB>
__global__ __launch_bounds__(64 * WAVES) void k_spmm_valu_s(
    const T *__restrict__ values, const uint8_t *__restrict__ indices,
    const T *__restrict__ X, int64_t ldx, T *__restrict__ Y, int64_t ldy, int M, int K, int N,
    int n, int m, int g, int C, int cpw, int row_tiles, int tiles) {
    constexpr int ES = (int)sizeof(T);
    constexpr int EPL = 16 / ES;                 // elements per 16-byte copy
    constexpr int LPR = kVsTok / EPL;            // copy lanes per staged row
    constexpr int RPI = 64 / LPR;                // staged rows per copy instruction
    __shared__ T xs0[SB / ES];
    __shared__ T xs1[SB / ES];

    const int tile = xcd_tile(blockIdx.x, tiles);
    const int rt = tile % row_tiles, tt = tile / row_tiles;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int r0 = rt * (kVsRowsWave * WAVES) + wave * kVsRowsWave;
    const int t0 = tt * kVsTok;
    const int ldv = C * n;                       // host checked: M * ldv < 2^31
    const int rpw = cpw * m;                     // staged rows per window (<= vs_rows_max)
    const int spw = cpw * n;                     // k-slots per window
    const int nwin = (C + cpw - 1) / cpw;
    const int ngrp = (spw + 3) / 4;              // groups of 4 k-slots per window (<= kVsGroups)
    // slot / n for slot < 256 by a multiply (exact: n <= 255)
    const uint32_t inv_n = ((1u << 20) + (uint32_t)n - 1) / (uint32_t)n;

    // weights and index bytes of a group: lane 4r + j holds row r0 + r, slot j
    const int wrow = min(r0 + (lane >> 2), M - 1);
    const T *wv = values + (int64_t)wrow * ldv;
    const uint8_t *wi = indices + (int64_t)(wrow / g) * ldv;
    // every group of a window at once (loaded a window ahead, before that
    // window's copies, so that waiting for them never waits for the copies)
    auto load_w = [&](int win, float (&w)[kVsGroups], uint32_t (&ix)[kVsGroups]) {
        const int wc = min(win, nwin - 1);
#pragma unroll
        for (int q = 0; q < kVsGroups; ++q) {
            const int slot = q * 4 + (lane & 3);            // within the window
            const int gs = wc * spw + slot;                 // within the row
            const bool live = slot < spw && gs < ldv;
            const int gc = live ? gs : 0;
            w[q] = live ? (float)wv[gc] : 0.f;
            ix[q] = wi[gc];
        }
    };

    // X rows of a window into LDS (rows past K: the last row, never selected;
    // tokens past N: the row's last 16 bytes, never stored)
    const int copy_sub = lane / LPR;
    const int copy_tok = min(t0 + EPL * (lane % LPR), N - EPL);   // host checked: N % EPL == 0
    // (buffer loads, lds_copy16_buf; host: the byte offsets of X fit 32 bits)
    const buf_rsrc_t xrs = buf_rsrc(X, (uint32_t)((int64_t)K * ldx * (int64_t)sizeof(T)));
    auto issue_copies = [&](int win, T *buf) {
        const int ninst = (rpw + RPI - 1) / RPI;
        for (int j = wave; j < ninst; j += WAVES) {
            const int k = min(win * rpw + j * RPI + copy_sub, K - 1);
            lds_copy16_buf(xrs, ((uint32_t)k * (uint32_t)ldx + (uint32_t)copy_tok) * (uint32_t)sizeof(T),
                           buf + j * RPI * kVsTok);
        }
    };

    v4f acc[kVsRowsWave];
#pragma unroll
    for (int r = 0; r < kVsRowsWave; ++r) acc[r] = v4f{0.f, 0.f, 0.f, 0.f};

    float w0[kVsGroups], w1[kVsGroups];
    uint32_t i0[kVsGroups], i1[kVsGroups];
    load_w(0, w0, i0);
    issue_copies(0, xs0);
    auto step = [&](int win, const T *cur, T *nxt, const float (&w)[kVsGroups],
                    const uint32_t (&ix)[kVsGroups], float (&w_nxt)[kVsGroups],
                    uint32_t (&ix_nxt)[kVsGroups]) {
        wait_all_memory();  // this wave's copies and weights for `win` have landed
        __syncthreads();    // cur is complete; every wave is done with nxt
        load_w(win + 1, w_nxt, ix_nxt);
        if (win + 1 < nwin) issue_copies(win + 1, nxt);
        static_for<kVsGroups>([&](auto qc) {
            constexpr int q = decltype(qc)::value;
            if (q >= ngrp) return;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                // the staged row of slot 4q + j (scalar), clamped into the window
                const uint32_t slot = (uint32_t)(4 * q + j);
                const uint32_t c = (slot * inv_n) >> 20;
#pragma unroll
                for (int r = 0; r < kVsRowsWave; ++r) {
                    const uint32_t o = min(__builtin_amdgcn_readlane(ix[q], 4 * r + j), (uint32_t)(m - 1));
                    const uint32_t row = min(c * (uint32_t)m + o, (uint32_t)(rpw - 1));
                    const float wr = __builtin_bit_cast(
                        float, __builtin_amdgcn_readlane(__builtin_bit_cast(uint32_t, w[q]), 4 * r + j));
                    const v4f x = vs_read<T>(cur, row, lane);
#pragma unroll
                    for (int e = 0; e < 4; ++e) acc[r][e] = fmaf(wr, x[e], acc[r][e]);
                }
            }
        });
    };
    for (int win = 0; win < nwin; win += 2) {
        step(win, xs0, xs1, w0, i0, w1, i1);
        if (win + 1 < nwin) step(win + 1, xs1, xs0, w1, i1, w0, i0);
    }

    const int tok = t0 + 4 * lane;
#pragma unroll
    for (int r = 0; r < kVsRowsWave; ++r) {
        const int row = r0 + r;
        if (row >= M) continue;
        T *y = Y + (int64_t)row * ldy + tok;
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (tok + e < N) y[e] = (T)acc[r][e];
    }
}

// chunks per window of a staging buffer of SB bytes
template <typename T, int SB>
int vs_cpw(const nmg_layout *L) {
    return std::max(1, std::min(vs_rows_max<T, SB>() / L->m, 4 * kVsGroups / L->n));
}
// the wide shape where a small window would hold a single k-slot
template <typename T>
bool vs_wide(const nmg_layout *L) { return vs_cpw<T, kVsSmallStage>(L) * L->n < 2; }

template <typename T, int WAVES, int SB>
nmg_status launch_valu_s_shape(const SpmmArgs &a) {
    const nmg_layout *L = a.L;
    const int cpw = vs_cpw<T, SB>(L);
    const int row_tiles = (L->M + kVsRowsWave * WAVES - 1) / (kVsRowsWave * WAVES);
    const int tiles = row_tiles * ((a.N + kVsTok - 1) / kVsTok);
    hipLaunchKernelGGL((k_spmm_valu_s<T, WAVES, SB>), dim3(tiles), dim3(64 * WAVES), 0, a.stream,
                       (const T *)a.values, a.indices, (const T *)a.X, a.ldx, (T *)a.Y, a.ldy,
                       L->M, L->K, a.N, L->n, L->m, L->g, L->C, cpw, row_tiles, tiles);
    return launched();
}

template <typename T>
nmg_status launch_valu_s(const SpmmArgs &a) {
    return vs_wide<T>(a.L) ? launch_valu_s_shape<T, kVsWideWaves, kVsWideStage>(a)
                           : launch_valu_s_shape<T, kVsSmallWaves, kVsSmallStage>(a);
}

}  // namespace

// The staged vector kernel takes binary32 layouts whose chunks fit the
// staging buffer (m <= 32 rows of 256 tokens) with n <= 16 (a window of at
// least one chunk keeps 16 k-slots at most), and X that can be copied 16
// bytes at a time (X and ldx on 16-byte boundaries, N % 4 == 0); value
// offsets within 31 bits, byte offsets of X within 32 bits.  (Binary16 layouts of g % 4 != 0 go to the sparse matrix
// instruction, or the vector kernel.)
bool nmg_internal::spmm_valu_staged_supported(const nmg_layout *L, const void *X, int64_t ldx,
                                              int64_t N) {
    return L->dtype == NMG_F32 && L->m <= vs_rows_max<float, kVsSmallStage>() && L->n <= 4 * kVsGroups &&
           (X == nullptr || aligned(X, 16)) && ldx % 4 == 0 && N % 4 == 0 &&
           (int64_t)L->M * L->C * L->n < ((int64_t)1 << 31) &&
           (int64_t)L->K * ldx * 4 <= (int64_t)0xffffffff;
}

nmg_status nmg_internal::spmm_valu_staged(const SpmmArgs &a) { return launch_valu_s<float>(a); }

// AUTO's choice between this kernel and the gathering vector kernel: staging
// pays when a window holds at least 2 k-slots (with one, every slot costs a
// copy and a barrier for a single FMA per row and token); the wide shape's
// windows hold 2 or more chunks for every supported m.
bool nmg_internal::spmm_valu_staged_preferred(const nmg_layout *L, const void *X, int64_t ldx,
                                              int64_t N) {
    return spmm_valu_staged_supported(L, X, ldx, N) &&
           (vs_wide<float>(L) ? vs_cpw<float, kVsWideStage>(L) : vs_cpw<float, kVsSmallStage>(L)) * L->n >= 2;
}
