// k_spmm_mfma_d.hip -- Y = W_s X (Section 5.1) for binary32 layouts, with
// each group's selected X rows gathered straight from global memory.
//
// The staged kernels copy every X row of a window into LDS, so a workgroup
// reads K rows of its token tile however few of them its groups select; at
// m/n = 10 most of that copy is unused.  This kernel reads only the selected
// rows: per (group unit, k-slot) one coalesced load of the unit's gathered row
// (TPL tokens per lane), which feeds the unit's quads directly as the MFMA B
// operand (the same 4x4x1 instruction with the weight block broadcast).  The
// index words come by scalar loads two windows ahead, the rows and weights of
// window w+1 by vector loads issued before the matrix instructions of window
// w.
// The k-slots can also be split over the waves of a workgroup, whose partial
// sums are added through LDS in split order at the end: a layer with few rows
// or few tokens (768 x 768 x 128) still gives every CU waves to run.  Layers
// that fill the GPU anyway take 4 tokens per lane (the wide shape, DConf).
#include "common.hpp"

namespace {

constexpr int kDRowsWave = 16;   // 4 quads

// The window, tokens per lane and largest workgroup of each group unit, in two
// shapes.  Two windows of gathered rows are in registers at once.
//   WIDE, for layers whose 256-token tiles alone cover the CUs: 4 tokens a
//   lane and 4-slot windows in workgroups of at most 8 waves (up to about 250
//   registers; units of 4 rows spill 4, which costs less than one wave a
//   SIMD: 1:20:4 29.5 us against 34.8 in 4-wave workgroups).  Against the
//   narrow shape on 3072 x 768 x 4096: 1:20:4 51.6 -> 29.8 us, 1:10:4 90.9 ->
//   51.6, 1:20:8 32.4 -> 23.7, 1:10:8 53.3 -> 38.6, and on 768 x 3072 x 4096
//   at 1:10:16 40.7 -> 33.1.
//   Narrow, for layers that need the k-split to fill the GPU (768 x 768 x 128
//   at 2:4:4 takes 13.4 us so, 21.2 wide): 16-wave workgroups, 2 tokens a
//   lane (1 for units of 4).
__host__ __device__ constexpr int d_waves(int tpl) { return tpl == 4 ? 8 : 16; }
template <int U, bool WIDE> struct DConf;
template <int U> struct DConf<U, true> { static constexpr int ksw = 4, tpl = 4, waves = d_waves(4); };
template <> struct DConf<16, false> { static constexpr int ksw = 8, tpl = 2, waves = d_waves(2); };
template <> struct DConf<8, false> { static constexpr int ksw = 4, tpl = 2, waves = d_waves(2); };
template <> struct DConf<4, false> { static constexpr int ksw = 4, tpl = 1, waves = d_waves(1); };

template <int TPL> struct DTok { typedef float type __attribute__((ext_vector_type(TPL))); };
template <> struct DTok<1> { typedef float type; };
template <int TPL>
__device__ __forceinline__ float d_part(const typename DTok<TPL>::type &v, int p) {
    if constexpr (TPL == 1) { (void)p; return v; } else { return v[p]; }
}

template <int U, int KSW, int TPL, bool VEC>
__global__ __launch_bounds__(64 * d_waves(TPL)) void k_spmm_mfma_d(
    const float *__restrict__ values, const uint8_t *__restrict__ indices,
    const float *__restrict__ X, int64_t ldx, float *__restrict__ Y, int64_t ldy, int M, int K,
    int N, int log2n, int m, int g, int C, int row_tiles, int tiles, int split, bool yvec) {
    static_assert(KSW % 4 == 0 && KSW <= 16 && U % 4 == 0 && U <= kDRowsWave, "window of index words");
    constexpr int QW = kDRowsWave / 4;   // quads per wave
    constexpr int UNITS = kDRowsWave / U;
    constexpr int QPU = U / 4;           // quads per unit
    constexpr int IW = KSW / 4;          // index words per unit and window
    constexpr int CBSZ = ilog2(KSW);
    constexpr int TN = 64 * TPL;
    typedef typename DTok<TPL>::type BV;
    extern __shared__ v4f red[];         // partial sums of every wave (k-splits only)

    const int nwaves = blockDim.x >> 6;
    const int nrw = nwaves / split;      // row-waves (host: nwaves % split == 0)
    const int tile = xcd_tile(blockIdx.x, tiles);
    const int rt = tile % row_tiles, tt = tile / row_tiles;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int rw = wave % nrw, sp = wave / nrw;
    const int r0 = rt * (kDRowsWave * nrw) + rw * kDRowsWave;
    const int tok = tt * TN + TPL * lane;
    const int valid = N - tok;
    const int n = 1 << log2n;            // n is a power of two here
    const int ldv = C * n;               // host checked: M * ldv < 2^31
    const int nwin = (ldv + KSW - 1) / KSW;
    // this wave's k-split: a contiguous range of windows
    const int wbeg = (int)((int64_t)nwin * sp / split), wend = (int)((int64_t)nwin * (sp + 1) / split);

    // Every load of the main loop is unconditional, with its address clamped
    // into its buffer, so that the compiler counts the loads in flight
    // exactly and waits for one window's loads only when they are used.
    // Lanes past N load a clamped token and are never stored; the k-slots past
    // the last chunk are zeroed in the last window, after their loads.
    //
    // A operands: lane 4b+i holds row r0+4q+i, slot b % KSW of the window
    const int a_slot = (lane >> 2) & (KSW - 1);
    const int vmax = M * ldv - 1;
    int aoff[QW];
#pragma unroll
    for (int q = 0; q < QW; ++q) aoff[q] = min(r0 + 4 * q + (lane & 3), M - 1) * ldv + a_slot;
    auto load_a = [&](int win, float (&a)[QW]) {
#pragma unroll
        for (int q = 0; q < QW; ++q) a[q] = values[min(win * KSW + aoff[q], vmax)];
    };
    // index bytes of a window: per unit, the IW + 1 aligned words that cover
    // its KSW bytes, by scalar loads (the unit's index row is the same for
    // the whole wave).  Addresses are clamped to the last word of the index
    // array, so every word read holds at least one byte of the array (and
    // lies on its pages); the bytes outside a unit's window are shifted out
    // or clamped away.  KSW % 4 == 0, so a unit's bytes start at the same
    // offset within a word in every window.
    struct IdxWords {
        uint32_t lo[UNITS][IW], hi[UNITS][IW];   // words j and j+1 of each unit
    };
    // the index array as aligned words: word w holds bytes 4w - mis .. of it
    const int mis = (int)(reinterpret_cast<uintptr_t>(indices) & 3);
    // (read through the constant address space: nothing writes the indices
    // while the kernel runs, and uniform loads from it become scalar loads)
    typedef const __attribute__((address_space(4))) uint32_t *ConstWords;
    const ConstWords iwords = (ConstWords)(indices - mis);
    const int wlast = (mis + (M / g) * ldv - 1) >> 2;   // host checked: M * ldv < 2^31
    int ibyte[UNITS], ishift[UNITS];
#pragma unroll
    for (int u = 0; u < UNITS; ++u) {
        ibyte[u] = mis + (min(r0 + u * U, M - 1) / g) * ldv;  // unit's row, from the first word
        ishift[u] = 8 * (ibyte[u] & 3);
    }
    auto load_idx = [&](int win, IdxWords &d) {
#pragma unroll
        for (int u = 0; u < UNITS; ++u) {
            const int w0 = (ibyte[u] + win * KSW) >> 2;
#pragma unroll
            for (int j = 0; j < IW; ++j) {
                d.lo[u][j] = iwords[min(w0 + j, wlast)];
                d.hi[u][j] = iwords[min(w0 + j + 1, wlast)];
            }
        }
    };
    // X row offsets (elements) of a window's gathered rows, one per (k-slot,
    // unit), computed on the scalar unit from the index bytes
    auto gather_rows = [&](int win, const IdxWords &d, uint32_t (&ro)[KSW][UNITS]) {
#pragma unroll
        for (int u = 0; u < UNITS; ++u)
#pragma unroll
            for (int j = 0; j < IW; ++j) {
                const uint32_t w =
                    (uint32_t)((((uint64_t)d.hi[u][j] << 32) | d.lo[u][j]) >> ishift[u]);
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    const int s = 4 * j + b;
                    const int o = min((int)((w >> (8 * b)) & 0xffu), m - 1);
                    ro[s][u] = (uint32_t)min(((win * KSW + s) >> log2n) * m + o, K - 1) * (uint32_t)ldx;
                }
            }
    };
    // the gathered rows, TPL tokens per lane: one vector load when X rows are
    // vector-aligned and N % TPL == 0 (a lane's tokens are then all valid or
    // all past N), else TPL loads with each token clamped below N
    const int tok_c = VEC ? min(tok, N - TPL) : tok;
    auto load_x = [&](const uint32_t (&ro)[KSW][UNITS], BV (&bx)[KSW][UNITS]) {
#pragma unroll
        for (int s = 0; s < KSW; ++s)
#pragma unroll
            for (int u = 0; u < UNITS; ++u) {
                const float *row = X + ro[s][u];
                if constexpr (VEC) {
                    bx[s][u] = *reinterpret_cast<const BV *>(row + tok_c);
                } else if constexpr (TPL == 1) {
                    bx[s][u] = row[min(tok, N - 1)];
                } else {
#pragma unroll
                    for (int e = 0; e < TPL; ++e) bx[s][u][e] = row[min(tok + e, N - 1)];
                }
            }
    };

    v4f acc[QW][TPL];
#pragma unroll
    for (int q = 0; q < QW; ++q)
#pragma unroll
        for (int p = 0; p < TPL; ++p) acc[q][p] = v4f{0.f, 0.f, 0.f, 0.f};

    auto mfma_window = [&](const float (&a)[QW], const BV (&bx)[KSW][UNITS]) {
        static_for<KSW>([&](auto sc) {
            constexpr int s = decltype(sc)::value;
            static_for<UNITS>([&](auto uc) {
                constexpr int u = decltype(uc)::value;
                static_for<QPU>([&](auto qc) {
                    constexpr int q = u * QPU + decltype(qc)::value;
                    static_for<TPL>([&](auto pc) {
                        constexpr int p = decltype(pc)::value;
                        acc[q][p] = __builtin_amdgcn_mfma_f32_4x4x1f32(
                            a[q], d_part<TPL>(bx[s][u], p), acc[q][p], CBSZ, s, 0);
                    });
                });
            });
        });
    };
    // the last window of this wave: k-slots past the last chunk contribute 0
    auto last_window = [&](int win, float (&a)[QW], BV (&bx)[KSW][UNITS]) {
        if ((win + 1) * KSW > ldv) {
            const bool a_ok = win * KSW + a_slot < ldv;
#pragma unroll
            for (int q = 0; q < QW; ++q) a[q] = a_ok ? a[q] : 0.f;
#pragma unroll
            for (int s = 0; s < KSW; ++s)
#pragma unroll
                for (int u = 0; u < UNITS; ++u)
                    if (win * KSW + s >= ldv) bx[s][u] = BV{};
        }
        mfma_window(a, bx);
    };

    if (wbeg < wend) {
        float a0[QW], a1[QW];
        IdxWords i0, i1;         // index words of even / odd windows
        BV b0[KSW][UNITS], b1[KSW][UNITS];
        uint32_t ro[KSW][UNITS];
        load_idx(wbeg, i0);
        load_idx(min(wbeg + 1, wend - 1), i1);
        gather_rows(wbeg, i0, ro);
        load_x(ro, b0);
        load_a(wbeg, a0);
        // window `win` from (a, bx) while the index words of win+2 go to
        // i_nn and window win+1's rows (its words i_nxt came a window
        // earlier) to bx_nxt
        auto step = [&](int win, const float (&a)[QW], const BV (&bx)[KSW][UNITS],
                        const IdxWords &i_nxt, float (&a_nxt)[QW], BV (&bx_nxt)[KSW][UNITS],
                        IdxWords &i_nn) {
            gather_rows(win + 1, i_nxt, ro);
            load_idx(min(win + 2, wend - 1), i_nn);
            load_x(ro, bx_nxt);
            load_a(win + 1, a_nxt);
            // keep the loads of win+1 ahead of win's matrix instructions
            __builtin_amdgcn_sched_barrier(0);
            mfma_window(a, bx);
            __builtin_amdgcn_sched_barrier(0);
        };
        int win = wbeg;
        for (; win + 2 < wend; win += 2) {
            step(win, a0, b0, i1, a1, b1, i0);
            step(win + 1, a1, b1, i0, a0, b0, i1);
        }
        if (win + 2 == wend) {
            step(win, a0, b0, i1, a1, b1, i0);
            last_window(win + 1, a1, b1);
        } else {
            last_window(win, a0, b0);
        }
    }

    // output register i of (quad q, part p) at lane l is Y[r0 + 4q + i][tok + p]
    auto store_quad = [&](int q, const v4f (&s)[TPL]) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int row = r0 + 4 * q + i;
            if (row >= M) continue;
            float *y = Y + (int64_t)row * ldy + tok;
            if constexpr (TPL > 1) {
                if (yvec && valid >= TPL) {
                    BV v;
#pragma unroll
                    for (int p = 0; p < TPL; ++p) v[p] = s[p][i];
                    __builtin_nontemporal_store(v, reinterpret_cast<BV *>(y));
                    continue;
                }
            }
#pragma unroll
            for (int p = 0; p < TPL; ++p)
                if (p < valid) __builtin_nontemporal_store(s[p][i], y + p);
        }
    };
    if (split == 1) {
#pragma unroll
        for (int q = 0; q < QW; ++q) store_quad(q, acc[q]);
        return;
    }
    // k-splits: every wave's partial sums go to LDS; then the wave of split
    // sp adds quads sp, sp + split, .. of its row-wave over the splits in
    // split order (a fixed order for a given launch shape) and stores them
    v4f *part = red + (size_t)(sp * nrw + rw) * (QW * TPL * 64);
#pragma unroll
    for (int q = 0; q < QW; ++q)
#pragma unroll
        for (int p = 0; p < TPL; ++p) part[(q * TPL + p) * 64 + lane] = acc[q][p];
    __syncthreads();
    for (int q = sp; q < QW; q += split) {
        v4f s[TPL];
        const v4f *src = red + (size_t)rw * (QW * TPL * 64) + q * TPL * 64 + lane;
#pragma unroll
        for (int p = 0; p < TPL; ++p) s[p] = src[p * 64];
        for (int t = 1; t < split; ++t) {
            const v4f *st = src + (size_t)t * nrw * (QW * TPL * 64);
#pragma unroll
            for (int p = 0; p < TPL; ++p) s[p] += st[p * 64];
        }
        store_quad(q, s);
    }
}

// Row-waves x k-splits per workgroup.  Each shape is priced as rounds of the
// GPU times the windows one wave runs, plus one window's worth per extra
// split for the reduction; the cheapest wins, and on a tie the one with fewer
// splits, then more row-waves.  A round is as many workgroups per CU as are
// resident at once (the runtime's occupancy and the LDS of the reduction);
// a last, partial round counts for the share of it that each CU runs, since
// the CUs' load paths, not the waves, bound the gathers (1:20:16 on 384
// workgroups of 16 waves, one and a half rounds: 32.8 us; on 768 of 8, two
// resident a CU: 24.9).
struct DShape {
    int nrw, split;
    size_t lds;
};
template <int U, bool WIDE>
DShape d_shape(const nmg_layout *L, int N) {
    constexpr int KSW = DConf<U, WIDE>::ksw, TPL = DConf<U, WIDE>::tpl, WAVES = DConf<U, WIDE>::waves;
    const void *kern = reinterpret_cast<const void *>(&k_spmm_mfma_d<U, KSW, TPL, true>);
    const int cus = device_cus();
    const int rws = (L->M + kDRowsWave - 1) / kDRowsWave;
    const int64_t tt = (N + 64 * TPL - 1) / (64 * TPL);
    const int nwin = ((int)L->C * L->n + KSW - 1) / KSW;
    constexpr size_t kWaveLds = (size_t)4 * TPL * 64 * sizeof(v4f);  // one wave's partial sums
    DShape best{1, 1, 0};
    double best_cost = 0.0;
    for (int split = 1; split <= WAVES && split <= nwin; split *= 2) {
        for (int nrw = 1; nrw * split <= WAVES && nrw <= rws; ++nrw) {
            const int wg = nrw * split;
            const size_t lds = split > 1 ? (size_t)wg * kWaveLds : 0;
            if (lds > 65536) continue;
            int per_cu = kernel_occupancy(kern, 64 * wg);
            if (lds > 0) per_cu = std::min<int>(per_cu, (int)(163840 / lds));
            per_cu = std::max(per_cu, 1);
            const int64_t tiles = (int64_t)((rws + nrw - 1) / nrw) * tt;
            const double rounds = std::max((double)((tiles + cus - 1) / cus) / per_cu, 1.0);
            const double cost = rounds * ((nwin + split - 1) / split + (split > 1 ? 1 : 0));
            if (best_cost == 0.0 || cost < best_cost - 1e-9 ||
                (cost < best_cost + 1e-9 && split == best.split && nrw > best.nrw)) {
                best = DShape{nrw, split, lds};
                best_cost = cost;
            }
        }
    }
    return best;
}

template <int U, bool WIDE>
nmg_status launch_d(const SpmmArgs &a) {
    constexpr int KSW = DConf<U, WIDE>::ksw, TPL = DConf<U, WIDE>::tpl;
    const nmg_layout *L = a.L;
    const DShape sh = d_shape<U, WIDE>(L, a.N);
    const int rws = (L->M + kDRowsWave - 1) / kDRowsWave;
    const int row_tiles = (rws + sh.nrw - 1) / sh.nrw;
    const int tiles = row_tiles * ((a.N + 64 * TPL - 1) / (64 * TPL));
    // whole-vector loads: X rows aligned to TPL elements and N % TPL == 0
    const bool vec = aligned(a.X, 4 * TPL) && a.ldx % TPL == 0 && a.N % TPL == 0;
    const bool yvec = aligned(a.Y, 4 * TPL) && a.ldy % TPL == 0;
    int log2n = 0;
    while ((1 << log2n) < L->n) ++log2n;
    auto kern = vec ? k_spmm_mfma_d<U, KSW, TPL, true> : k_spmm_mfma_d<U, KSW, TPL, false>;
    hipLaunchKernelGGL(kern, dim3(tiles), dim3(64 * sh.nrw * sh.split), sh.lds, a.stream,
                       (const float *)a.values, a.indices, (const float *)a.X, a.ldx,
                       (float *)a.Y, a.ldy, L->M, L->K, a.N, log2n, L->m, L->g, L->C, row_tiles,
                       tiles, sh.split, yvec);
    return launched();
}

// The wide shape when its 256-token tiles of 16 rows cover the CUs.
bool d_wide(const nmg_layout *L, int64_t N) {
    const int64_t rws = (L->M + kDRowsWave - 1) / kDRowsWave;
    return rws * ((N + 255) / 256) >= device_cus();
}

}  // namespace

// The gathering kernel takes binary32 layouts with g % 4 == 0 and n a power of
// two, with value and X offsets within 31 bits.
bool nmg_internal::spmm_direct_supported(const nmg_layout *L, int64_t ldx) {
    return L->dtype == NMG_F32 && mfma_unit(L) != 0 && (L->n & (L->n - 1)) == 0 &&
           (int64_t)L->M * L->C * L->n < ((int64_t)1 << 31) &&
           (int64_t)L->K * ldx < ((int64_t)1 << 31);
}

nmg_status nmg_internal::spmm_direct(const SpmmArgs &a) {
    const bool wide = d_wide(a.L, a.N);
    switch (std::min(mfma_unit(a.L), 16)) {
        case 16: return wide ? launch_d<16, true>(a) : launch_d<16, false>(a);
        case 8: return wide ? launch_d<8, true>(a) : launch_d<8, false>(a);
        case 4: return wide ? launch_d<4, true>(a) : launch_d<4, false>(a);
        default: return NMG_ERR_UNSUPPORTED;
    }
}

// AUTO's choice between this kernel and the staged one.  A staged workgroup of
// about 8 waves (128 rows) reads all K rows of its token tile; a gathering
// unit of U rows reads its C * n selected rows.  In the wide shape, units of
// 8 or more rows win up to 1.75 times the staged kernel's rows (measured on
// 3072 x 768 x 4096: 1:10:8, 1.6 times, 38.6 against 53.5 us; 1:4:16, 2 times,
// 64.2 against 54.6), units of 4 up to 3.5 times (1:10:4, 3.2 times, 51.6
// against 58.2; 1:4:4, 8 times, 116 against 65); in the narrow one up to the
// same rows.  Gathering also wins whenever the staged kernel would leave most
// CUs idle (it has no k-split).
bool nmg_internal::spmm_direct_preferred(const nmg_layout *L, int64_t N, int64_t ldx) {
    if (!spmm_direct_supported(L, ldx)) return false;
    const int64_t U = std::min(mfma_unit(L), 16);
    const int64_t ldv = (int64_t)L->C * L->n;
    const int64_t lim = !d_wide(L, N) ? 4 : U >= 8 ? 7 : 14;   // 4 x the ratio of rows read
    if (4 * 128 * ldv <= lim * U * L->K) return true;
    const int64_t staged_waves = (int64_t)((L->M + 15) / 16) * ((N + 127) / 128);
    return staged_waves < 2 * device_cus();
}
