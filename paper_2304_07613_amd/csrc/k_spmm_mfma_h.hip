// k_spmm_mfma_h.hip -- the product Y = W_s X for binary16 layouts on the
// binary16 matrix cores (v_mfma_f32_4x4x4_16b_f16, binary32 accumulation).
//
// Paper: STen (arXiv 2304.07613), Section 5.1 (the sparse x dense product of
// the grouped n:m layout); the kernel itself is this library's design.
//
// The binary32 kernels multiply one gathered X row (one k-slot) per matrix
// instruction.  The binary16 instruction contracts over 4 k-slots at once, so
// each lane needs, for its token, the 4 gathered X values of 4 consecutive
// k-slots side by side.  X is staged in LDS row-major as in the other
// kernels, and one transposing LDS read (ds_read_b64_tr_b16) delivers exactly
// that: within each 16-lane group, lane i receives element i % 4 of the 8-byte
// loads of lanes i/4, i/4 + 4, i/4 + 8 and i/4 + 12.  So the lanes 4k .. 4k+3
// of a group load 16 consecutive tokens of the gathered row of slot k, and
// every lane gets its own token's 4 slots, with no shuffles.  The A operand
// (4 rows x 4 k-slots of weights) is broadcast from one block to all 16
// blocks of the instruction, so one instruction covers 4 rows x 64 tokens x 4
// k-slots.  A wave covers 64 * TPL tokens: lane l owns tokens l + 64p.
//
// With 4 tokens per lane (256-token rows, 512 bytes) the staged rows of odd
// chunks have the two 64-token halves of each 128 tokens swapped: a
// transposing read touches 4 rows of 128 bytes, and with n = 1 or 2 they come
// from chunks of both parities, so two land in each half of the banks.
//
// Epilogues (fused, so that Y is written once): GELU looks the rounded
// product up in the binary16 GELU table, copied into the staging buffers once
// the last window is done; ADD reads the residual beside the store.  Both
// give exactly what the product followed by nmg_gelu or nmg_add gives.
#include "common.hpp"

namespace {

typedef _Float16 h4 __attribute__((ext_vector_type(4)));

// GELU(x) for every binary16 x, indexed by the bits of x (the table nmg_gelu
// uses, generated at build time)
__device__ __attribute__((aligned(16))) const uint16_t g_gelu_f16[65536] = {
#include "gelu_f16_table.inc"
};

constexpr int kHalfRowsWave = 16;        // 4 quads of 4 rows
constexpr int kHalfMaxWaves = 12;        // 128 KB of LDS: one workgroup per CU
constexpr int kHalfStageBytes = 65536;   // per staging buffer
// staged X rows per window for 64 * TPL tokens per row
__host__ __device__ constexpr int half_window_rows(int tpl) { return kHalfStageBytes / (128 * tpl); }

typedef short s4 __attribute__((ext_vector_type(4)));

// The transposing LDS read of 8 bytes at `p` (an address in LDS).
__device__ __forceinline__ h4 lds_read_tr(const _Float16 *p) {
#if defined(__HIP_DEVICE_COMPILE__)
    return __builtin_bit_cast(
        h4, __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s4 *)p));
#else
    (void)p;
    return h4{};
#endif
}

// AVEC: values rows start on 8-byte and index rows on 4-byte boundaries
// (ldv % 4 == 0, aligned bases), so a lane loads its 4 weights and an index
// word with one load each.
template <int U, int KSW, int TPL, bool AVEC>
__global__ __launch_bounds__(64 * kHalfMaxWaves) void k_spmm_mfma_h(
    const _Float16 *__restrict__ values, const uint8_t *__restrict__ indices,
    const _Float16 *__restrict__ X, int64_t ldx, _Float16 *__restrict__ Y, int64_t ldy,
    const _Float16 *__restrict__ R, int64_t ldr, int M, int K, int N, int log2n, int m, int g,
    int C, int row_tiles, int tiles, int epi) {
    static_assert(KSW % 4 == 0 && KSW <= 64 && U % 4 == 0 && U <= kHalfRowsWave, "k-groups of 4 slots");
    constexpr int QW = kHalfRowsWave / 4;   // quads per wave
    constexpr int UNITS = kHalfRowsWave / U;
    constexpr int QPU = U / 4;              // quads per unit
    constexpr int KG = KSW / 4;             // k-groups per window
    constexpr int CBSZ = ilog2(KG);         // broadcast group of KG blocks
    constexpr int IW = KSW / 4;             // index words per unit and window
    constexpr int TN = 64 * TPL;            // tokens per wave and workgroup
    constexpr int LPR = TN / 8;             // lanes per staged row (16 bytes each)
    constexpr int RPI = 64 / LPR;           // rows per copy instruction
    static_assert(UNITS * IW <= 64, "one index word per lane");
    __shared__ _Float16 xs0[kHalfStageBytes / 2];
    __shared__ _Float16 xs1[kHalfStageBytes / 2];

    const int nwaves = blockDim.x >> 6;
    const int tile = xcd_tile(blockIdx.x, tiles);
    const int rt = tile % row_tiles, tt = tile / row_tiles;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int r0 = rt * (kHalfRowsWave * nwaves) + wave * kHalfRowsWave;
    const int t0 = tt * TN;
    const int n = 1 << log2n;
    const int ldv = C * n;                  // host checked: M * ldv < 2^31
    const int cpw = KSW >> log2n;           // chunks per window
    const int rpw = cpw * m;                // X rows per window (<= half_window_rows(TPL))
    const int nwin = (C + cpw - 1) / cpw;

    // index row of each unit (rows past M read the last group; never stored)
    const uint8_t *irow[UNITS];
#pragma unroll
    for (int u = 0; u < UNITS; ++u) irow[u] = indices + (int64_t)(min(r0 + u * U, M - 1) / g) * ldv;

    // A operands: lane 4b+i holds row r0+4q+i, k-slots 4(b % KG) .. 4(b % KG)+3
    // of the window (blocks beyond KG repeat the first KG, as the broadcast
    // groups of CBSZ expect)
    const int a_slot = 4 * ((lane >> 2) & (KG - 1));
    int aoff[QW];
#pragma unroll
    for (int q = 0; q < QW; ++q) aoff[q] = min(r0 + 4 * q + (lane & 3), M - 1) * ldv + a_slot;
    // Every load is unconditional, its slot clamped into the row, and what
    // is loaded is used only in the window that needs it (slots past the row
    // get weight 0 there): a branch around a load, or an operation on its
    // result right after it, would make the compiler wait for every load in
    // flight -- the next window's copies included -- at that point.  (Not
    // so for unaligned rows, AVEC false: their elements are combined as they
    // arrive, which keeps the registers within the budget.)
    auto load_a = [&](int win, h4 (&a)[QW]) {
        const int s0 = win * KSW + a_slot;      // first of this lane's 4 slots
#pragma unroll
        for (int q = 0; q < QW; ++q) {
            const _Float16 *vr = values + (aoff[q] - a_slot);   // the row
            if constexpr (AVEC) {
                a[q] = *reinterpret_cast<const h4 *>(vr + min(s0, ldv - 4));
            } else {
#pragma unroll
                for (int k = 0; k < 4; ++k) a[q][k] = vr[min(s0 + k, ldv - 1)];
            }
        }
    };
    auto use_a = [&](int win, h4 v) {
        const int s0 = win * KSW + a_slot;
#pragma unroll
        for (int k = 0; k < 4; ++k) v[k] = s0 + k < ldv ? v[k] : (_Float16)0.f;
        return v;
    };
    // index words of the window: lane u*IW + j loads word j of unit u
    const int iw_u = min(lane / IW, UNITS - 1), iw_j = lane % IW;
    const uint8_t *iw_row = irow[0];
#pragma unroll
    for (int u = 1; u < UNITS; ++u)
        if (iw_u == u) iw_row = irow[u];
    // (slots past the row read a clamped byte: their weight is 0 and every
    // offset is clamped into its chunk where it is used)
    auto load_idx = [&](int win, uint32_t &wv) {
        const int s0 = win * KSW + 4 * iw_j;
        if constexpr (AVEC) {
            wv = *reinterpret_cast<const uint32_t *>(iw_row + min(s0, ldv - 4));
        } else {
            uint32_t x = 0;
#pragma unroll
            for (int b = 0; b < 4; ++b) x |= (uint32_t)iw_row[min(s0 + b, ldv - 1)] << (8 * b);
            wv = x;
        }
    };
    // X rows of a window into LDS: lane l copies 16 bytes (8 tokens) of row
    // l / LPR; tokens past N (a ragged last token tile) re-read the row's last
    // 8 tokens (host checked: N % 8 == 0), rows past K the last row -- both
    // are staged but never used for a stored output.
    // Staged rows of odd chunks (counted within the window) swap the 64-token
    // halves of each 128 tokens when TPL == 4, so that a transposing read of
    // 4 slots from two chunks (n = 1, 2) puts 2 rows in each half of the LDS
    // banks.  The copies are addressed on the scalar unit where they can be:
    // a uniform row base plus a per-lane offset fixed for the whole kernel,
    // one per swap parity; a row's chunk parity comes from a multiply.
    const int copy_sub = lane / LPR;
    const int copy_tk = 8 * (lane % LPR);
    // element offsets of this lane from its instruction's first row (K * ldx < 2^31)
    const int sub_off = copy_sub * (int)ldx;
    const int lane_x0 = sub_off + min(t0 + copy_tk, N - 8);
    const int lane_x1 = sub_off + min(t0 + (copy_tk ^ 64), N - 8);
    // r / m by a multiply, exact for r < 2^16 / m (rows of a window: r <= 128)
    const uint32_t inv_m = (65536u + (uint32_t)m - 1) / (uint32_t)m;
    // the copies are buffer loads (lds_copy16_buf; K ldx < 2^31 elements, so
    // every byte offset fits 32 bits)
    const buf_rsrc_t xrs = buf_rsrc(X, (uint32_t)((int64_t)K * ldx * 2));
    auto issue_copies = [&](int win, _Float16 *buf) {
        const int ninst = (rpw + RPI - 1) / RPI;
        for (int j = wave; j < ninst; j += nwaves) {
            const int rb = __builtin_amdgcn_readfirstlane(j * RPI);   // first row in the window
            const int kb = __builtin_amdgcn_readfirstlane(win * rpw + rb);   // and in X
            int lx = lane_x0;
            if constexpr (TPL == 4) {
                // RPI == 2: the chunk parities of rows rb and rb + 1
                const int p0 = __builtin_amdgcn_readfirstlane((int)(((uint32_t)rb * inv_m) >> 16) & 1);
                const int p1 = __builtin_amdgcn_readfirstlane((int)(((uint32_t)(rb + 1) * inv_m) >> 16) & 1);
                lx = (copy_sub ? p1 : p0) ? lane_x1 : lane_x0;
            }
            // rows past K (the last window) read the last row, never selected
            const int lim = K - kb;
            const int clamp = __builtin_amdgcn_readfirstlane((lim - 1) * (int)ldx);
            lx = copy_sub < lim ? lx : lx - sub_off + clamp;
            lds_copy16_buf(xrs, ((uint32_t)kb * (uint32_t)ldx + (uint32_t)lx) * 2u, buf + rb * TN);
        }
    };

    // transposing reads: lane l loads slot k_l = (l >> 2) & 3 of a k-group,
    // 4 tokens at tr_tok = 16 (l >> 4) + 4 (l & 3) of each 64-token block
    const int k_l = (lane >> 2) & 3;
    const uint32_t tr_shift = 8 * k_l;                    // its byte of an index word
    const uint32_t tr_chunk = (uint32_t)((k_l >> log2n) * m);  // its slot's chunk within the k-group
    const uint32_t tr_tok = 16 * (lane >> 4) + 4 * (lane & 3);
    const uint32_t tr_par = (uint32_t)((k_l >> log2n) & 1);

    v4f acc[QW][TPL];
#pragma unroll
    for (int q = 0; q < QW; ++q)
#pragma unroll
        for (int p = 0; p < TPL; ++p) acc[q][p] = v4f{0.f, 0.f, 0.f, 0.f};

    h4 a0[QW], a1[QW];          // weights of even / odd windows, as loaded
    uint32_t w0 = 0, w1 = 0;    // index words of even / odd windows (one per lane)
    issue_copies(0, xs0);
    load_a(0, a0);
    load_idx(0, w0);

    auto step = [&](int win, _Float16 *cur, _Float16 *nxt, const h4 (&a_raw)[QW], uint32_t wv,
                    h4 (&a_nxt)[QW], uint32_t &wv_nxt) {
        wait_all_memory();  // this wave's copies and loads for `win` have landed
        __syncthreads();    // cur is complete; every wave is done with nxt
        h4 a[QW];
#pragma unroll
        for (int q = 0; q < QW; ++q) a[q] = use_a(win, a_raw[q]);
        uint32_t w[UNITS][IW];
#pragma unroll
        for (int u = 0; u < UNITS; ++u)
#pragma unroll
            for (int j = 0; j < IW; ++j) w[u][j] = __builtin_amdgcn_readlane(wv, u * IW + j);
        if (win + 1 < nwin) {
            issue_copies(win + 1, nxt);
            load_a(win + 1, a_nxt);
            load_idx(win + 1, wv_nxt);
        }

        // steps t = kg * UNITS + u: the B operands of k-group kg of unit u
        // (one transposing read per 64-token block), read one step ahead
        h4 r[2][TPL];
        auto read_step = [&](auto tc, h4 (&dst)[TPL]) {
            constexpr int kg = decltype(tc)::value / UNITS, u = decltype(tc)::value % UNITS;
            // this lane's slot 4 kg + k_l: chunk base, then its offset (clamped into the chunk)
            const uint32_t base = (uint32_t)(((4 * kg) >> log2n) * m) + tr_chunk;
            const uint32_t o = min((w[u][kg] >> tr_shift) & 0xffu, (uint32_t)(m - 1));
            const _Float16 *rp = cur + (base + o) * TN + tr_tok;
            if constexpr (TPL == 4) {
                const uint32_t sw = 64u * ((((4 * kg) >> log2n) & 1) ^ tr_par);
                static_for<TPL>([&](auto pc) {
                    constexpr int p = decltype(pc)::value;
                    dst[p] = lds_read_tr(cur + (base + o) * TN + tr_tok + ((64u * p) ^ sw));
                });
            } else {
                static_for<TPL>([&](auto pc) {
                    constexpr int p = decltype(pc)::value;
                    dst[p] = lds_read_tr(rp + 64 * p);
                });
            }
        };
        read_step(std::integral_constant<int, 0>{}, r[0]);
        static_for<KG * UNITS>([&](auto tc) {
            constexpr int t = decltype(tc)::value;
            constexpr int kg = t / UNITS, u = t % UNITS;
            if constexpr (t + 1 < KG * UNITS) read_step(std::integral_constant<int, t + 1>{}, r[(t + 1) & 1]);
            // keep the reads of step t+1 ahead of the work of step t
            __builtin_amdgcn_sched_barrier(0);
            static_for<TPL>([&](auto pc) {
                constexpr int p = decltype(pc)::value;
                static_for<QPU>([&](auto qc) {
                    constexpr int q = u * QPU + decltype(qc)::value;
                    acc[q][p] = __builtin_amdgcn_mfma_f32_4x4x4f16(a[q], r[t & 1][p], acc[q][p], CBSZ, kg, 0);
                });
            });
        });
    };
    for (int win = 0; win < nwin; win += 2) {
        step(win, xs0, xs1, a0, w0, a1, w1);
        if (win + 1 < nwin) step(win + 1, xs1, xs0, a1, w1, a0, w0);
    }

    if (epi == NMG_EPILOGUE_GELU) {
        // the GELU table into the staging buffers: entries of non-negative
        // inputs (sign bit clear) in xs0, of negative ones in xs1
        __syncthreads();  // every wave is done with the last window
        const uint4 *src = reinterpret_cast<const uint4 *>(g_gelu_f16);
        constexpr int HALF4 = kHalfStageBytes / 16;
        for (int i = threadIdx.x; i < 2 * HALF4; i += blockDim.x)
            reinterpret_cast<uint4 *>(i < HALF4 ? xs0 : xs1)[i % HALF4] = src[i];
        __syncthreads();
    }
    // output register i of (quad q, block p) at lane l is Y[r0 + 4q + i][t0 + 64p + l];
    // each store instruction writes 64 consecutive tokens
    auto store_all = [&](auto ec) {
        constexpr int E = decltype(ec)::value;
#pragma unroll
        for (int q = 0; q < QW; ++q)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int row = r0 + 4 * q + i;
                if (row >= M) continue;
#pragma unroll
                for (int p = 0; p < TPL; ++p) {
                    const int tok = t0 + 64 * p + lane;
                    if (tok >= N) continue;
                    const _Float16 h = (_Float16)acc[q][p][i];  // nearest even, as nmg_spmm stores it
                    _Float16 out = h;
                    if constexpr (E == NMG_EPILOGUE_GELU) {
                        const uint16_t b = __builtin_bit_cast(uint16_t, h);
                        const uint16_t *tab = reinterpret_cast<const uint16_t *>((b & 0x8000u) ? xs1 : xs0);
                        out = __builtin_bit_cast(_Float16, tab[b & 0x7fffu]);
                    } else if constexpr (E == NMG_EPILOGUE_ADD) {
                        out = (_Float16)((float)h + (float)R[(int64_t)row * ldr + tok]);
                    }
                    __builtin_nontemporal_store(out, Y + (int64_t)row * ldy + tok);
                }
            }
    };
    if (epi == NMG_EPILOGUE_GELU) store_all(std::integral_constant<int, NMG_EPILOGUE_GELU>{});
    else if (epi == NMG_EPILOGUE_ADD) store_all(std::integral_constant<int, NMG_EPILOGUE_ADD>{});
    else store_all(std::integral_constant<int, NMG_EPILOGUE_NONE>{});
}

// Largest window of 4 .. 32 k-slots (64 with one token per lane: one A
// register covers 64) that n divides and whose chunks fit the staging buffer;
// 0 if none.
int half_window(const nmg_layout *L, int tpl) {
    for (int ksw = tpl == 1 ? 64 : 32; ksw >= 4; ksw /= 2)
        if (ksw % L->n == 0 && (ksw / L->n) * L->m <= half_window_rows(tpl)) return ksw;
    return 0;
}

// Tokens per lane: 4 (256-token tiles, fewer LDS reads per matrix instruction)
// when the layer gives every SIMD two such waves; else 1 (64-token tiles: the
// same waves then cover 4x the rows, so each staged X row feeds 4x the work)
int half_tpl(const nmg_layout *L, int64_t N) {
    const int64_t waves4 = (int64_t)((L->M + kHalfRowsWave - 1) / kHalfRowsWave) * ((N + 255) / 256);
    return waves4 >= 8 * (int64_t)device_cus() && half_window(L, 4) ? 4 : 1;
}

template <int U, int KSW, int TPL, bool AVEC>
nmg_status launch_half(const SpmmArgs &a) {
    const nmg_layout *L = a.L;
    const void *kern = reinterpret_cast<const void *>(&k_spmm_mfma_h<U, KSW, TPL, AVEC>);
    // waves per workgroup: the count whose tiles fill whole rounds of the GPU best
    const int cus = device_cus();
    const int tok_tiles = (a.N + 64 * TPL - 1) / (64 * TPL);
    int best_w = 4;
    double best_eff = -1.0;
    for (int w = 4; w <= kHalfMaxWaves; ++w) {
        const int64_t tiles = (int64_t)((L->M + kHalfRowsWave * w - 1) / (kHalfRowsWave * w)) * tok_tiles;
        const int64_t slots = (int64_t)cus * kernel_occupancy(kern, 64 * w) * w;
        const int64_t rounds = (tiles * w + slots - 1) / slots;
        const double eff = (double)(tiles * w) / (double)(rounds * slots);
        const bool tie = eff > best_eff - 1e-9 && eff < best_eff + 1e-9;
        if (eff > best_eff + 1e-9 || (tie && tiles >= cus)) {
            best_eff = std::max(eff, best_eff);
            best_w = w;
        }
    }
    const int row_tiles = (L->M + kHalfRowsWave * best_w - 1) / (kHalfRowsWave * best_w);
    const int tiles = row_tiles * tok_tiles;
    int log2n = 0;
    while ((1 << log2n) < L->n) ++log2n;
    hipLaunchKernelGGL((k_spmm_mfma_h<U, KSW, TPL, AVEC>), dim3(tiles), dim3(64 * best_w), 0, a.stream,
                       (const _Float16 *)a.values, a.indices, (const _Float16 *)a.X, a.ldx,
                       (_Float16 *)a.Y, a.ldy, (const _Float16 *)a.R, a.ldr, L->M, L->K, a.N,
                       log2n, L->m, L->g, L->C, row_tiles, tiles, (int)a.epi);
    return launched();
}

template <int U, int KSW, int TPL>
nmg_status launch_half_v(const SpmmArgs &a) {
    const int64_t ldv = (int64_t)a.L->C * a.L->n;
    const bool avec = aligned(a.values, 8) && aligned(a.indices, 4) && ldv % 4 == 0;
    return avec ? launch_half<U, KSW, TPL, true>(a) : launch_half<U, KSW, TPL, false>(a);
}

template <int U>
nmg_status launch_half_u(const SpmmArgs &a) {
    if (half_tpl(a.L, a.N) == 4) {
        switch (half_window(a.L, 4)) {
            case 32: return launch_half_v<U, 32, 4>(a);
            case 16: return launch_half_v<U, 16, 4>(a);
            case 8: return launch_half_v<U, 8, 4>(a);
            case 4: return launch_half_v<U, 4, 4>(a);
            default: return NMG_ERR_UNSUPPORTED;
        }
    }
    switch (half_window(a.L, 1)) {
        case 64: return launch_half_v<U, 64, 1>(a);
        case 32: return launch_half_v<U, 32, 1>(a);
        case 16: return launch_half_v<U, 16, 1>(a);
        case 8: return launch_half_v<U, 8, 1>(a);
        case 4: return launch_half_v<U, 4, 1>(a);
        default: return NMG_ERR_UNSUPPORTED;
    }
}

}  // namespace

// The binary16 matrix-core kernel takes binary16 layouts whose groups are
// whole quads (g % 4 == 0) with n a power of two and a window that fits its
// staging buffer, and X that can be copied to LDS 16 bytes at a time: rows on
// 16-byte boundaries (X and ldx) and N a multiple of 8.  Index and values
// offsets must fit 31 bits.  `X` may be NULL to ask about the layout alone.
bool nmg_internal::spmm_half_supported(const nmg_layout *L, const void *X, int64_t ldx, int64_t N) {
    const int64_t ldv = (int64_t)L->C * L->n;
    return L->dtype == NMG_F16 && mfma_unit(L) != 0 && (L->n & (L->n - 1)) == 0 &&
           half_window(L, 1) != 0 && (X == nullptr || aligned(X, 16)) && ldx % 8 == 0 && N % 8 == 0 &&
           (int64_t)L->M * ldv < ((int64_t)1 << 31) && (int64_t)L->K * ldx < ((int64_t)1 << 31);
}

nmg_status nmg_internal::spmm_half(const SpmmArgs &a) {
    switch (mfma_unit(a.L) >= 16 ? 16 : mfma_unit(a.L)) {
        case 16: return launch_half_u<16>(a);
        case 8: return launch_half_u<8>(a);
        case 4: return launch_half_u<4>(a);
        default: return NMG_ERR_UNSUPPORTED;
    }
}
