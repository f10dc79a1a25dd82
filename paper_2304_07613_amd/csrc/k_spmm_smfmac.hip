// k_spmm_smfmac.hip -- Y = W_s X (Section 5.1) for binary16 layouts whose
// kept columns fit the matrix cores' own 2-of-4 sparsity: n <= 2 kept of every
// m in {4, 8, 16} columns, so no aligned group of 4 columns holds more than 2.
//
// gfx950's sparse matrix instruction v_smfmac_f32_16x16x64_f16 multiplies a
// 16 x 64 weight block, stored as 2 values (and their 2-bit positions) per
// aligned group of 4 columns, by a dense 64 x 16 block of X.  The layout's
// kept columns become those stored values directly -- padded with zeros where
// a group of 4 holds fewer than 2 -- so X is read as contiguous rows, the
// same 64 rows for every weight row of a workgroup, as in a dense product:
// no gathered rows, no per-group staging, and every staged X value feeds all
// the workgroup's rows.  The selection of columns is done by the hardware from
// the positions, which this kernel builds from the layout's indices while it
// runs (the weights stay in the layout nmg_compress writes).
//
// Lane layouts (checked on the GPU with in-bounds probes): the weight operand
// of lane l holds row l % 16 and stored values e = 0..7 at logical k =
// 16 (l / 16) + 4 (e / 2) + pos_e, pos_e in bits 2e, 2e+1 of the index word
// (duplicate or descending positions add up); the X operand of lane l holds
// token l % 16 and logical k = 8 (l / 16) + e for e < 8, 32 + 8 (l / 16) +
// e - 8 for e >= 8; the result register r of lane l is row 4 (l / 16) + r,
// token l % 16.  The X operand comes from the staged rows by four transposing
// LDS reads (ds_read_b64_tr_b16: lanes 4k'..4k'+3 of a 16-lane group read 4
// tokens of row k', and lane i receives token i of the 4 rows).
//
// Staged X rows are XOR-swizzled by 32-byte segments (segment s of row r is
// stored at s ^ f(r)), so that the 16 rows one transposing read touches fall
// on distinct bank groups.
#include "common.hpp"

namespace {

typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef _Float16 h4 __attribute__((ext_vector_type(4)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef _Float16 h16 __attribute__((ext_vector_type(16)));
typedef short s4 __attribute__((ext_vector_type(4)));

// GELU(x) for every binary16 x, indexed by the bits of x (the table nmg_gelu
// uses, generated at build time)
__device__ __attribute__((aligned(16))) const uint16_t g_gelu_f16_s[65536] = {
#include "gelu_f16_table.inc"
};

constexpr int kSmMaxWaves = 16;
constexpr int kSmKStep = 64;   // X rows per step (one sparse instruction's k)

// The transposing LDS read of 8 bytes at `p` (an address in LDS).
__device__ __forceinline__ h4 sm_read_tr(const _Float16 *p) {
#if defined(__HIP_DEVICE_COMPILE__)
    return __builtin_bit_cast(
        h4, __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s4 *)p));
#else
    (void)p;
    return h4{};
#endif
}

// The 32-byte segment swizzle of staged row r: rows 8a + 4b + c (c < 4) of a
// transposing read differ in (c, a & 1), which this maps to 8 distinct values.
__device__ __forceinline__ int sm_swz(int r) { return (r & 3) | ((r >> 1) & 4); }

// SPW kept slots per 16-column window: raw values and index bytes as loaded.
template <int SPW> struct SmRaw;
template <> struct SmRaw<1> { _Float16 v; uint8_t o; };
template <> struct SmRaw<2> { h2 v; uint16_t o; };
template <> struct SmRaw<4> { h4 v; uint32_t o; };
template <> struct SmRaw<8> { h8 v; uint64_t o; };

// the bits of kept value j, and of the pair of values 2k, 2k+1 (a word)
template <int SPW>
__device__ __forceinline__ uint32_t raw_half(const SmRaw<SPW> &r, int j) {
    if constexpr (SPW == 1) { (void)j; return __builtin_bit_cast(uint16_t, r.v); }
    else { return __builtin_bit_cast(uint16_t, (_Float16)r.v[j]); }
}
template <int SPW>
__device__ __forceinline__ uint32_t raw_word(const SmRaw<SPW> &r, int k) {
    if constexpr (SPW == 2) { (void)k; return __builtin_bit_cast(uint32_t, r.v); }
    else {
        typedef uint32_t uw __attribute__((ext_vector_type(SPW / 2)));
        return __builtin_bit_cast(uw, r.v)[k];
    }
}
template <int SPW>
__device__ __forceinline__ uint32_t raw_index(const SmRaw<SPW> &r, int j) {
    return (uint32_t)((uint64_t)r.o >> (8 * j)) & 0xffu;
}

// LM4 = log2(m / 4), NN = n; R x T blocks of 16 rows x 16 tokens per wave;
// WR x WT waves per workgroup; EPI = the epilogue.
template <int LM4, int NN, int R, int T, int WR, int WT, int EPI>
__global__ __launch_bounds__(64 * WR * WT) void k_spmm_smfmac(
    const _Float16 *__restrict__ values, const uint8_t *__restrict__ indices,
    const _Float16 *__restrict__ X, int64_t ldx, _Float16 *__restrict__ Y, int64_t ldy,
    const _Float16 *__restrict__ Rs, int64_t ldr, int M, int K, int N, int g, int C,
    int row_tiles, int tiles) {
    constexpr int MM = 4 << LM4;                  // m
    constexpr int SPW = 16 * NN / MM;             // kept slots per 16 columns
    constexpr int BM = WR * R * 16, BN = WT * T * 16;
    constexpr int PITCH = BN;                     // staged row, in halves
    constexpr int STAGE = kSmKStep * PITCH;       // halves per staging buffer
    // two staging buffers; X reaches them through registers, loaded two
    // steps ahead (three register sets), so every wait is on a register and
    // the compiler counts it exactly.  The GELU table (32K halves for each
    // sign) takes the buffers' place at the end.
    constexpr int BUF = EPI == NMG_EPILOGUE_GELU && STAGE < 32768 ? 32768 : STAGE;
    constexpr int LPR = BN / 8;                   // lanes per staged row (16 bytes each)
    constexpr int RPI = 64 / LPR;                 // staged rows per 1 KB wave store
    constexpr int NCOPY = kSmKStep / RPI;         // 1 KB pieces per step
    constexpr int NCW = NCOPY / (WR * WT);        // ... loaded and stored by each wave
    static_assert(NCOPY % (WR * WT) == 0, "every wave moves the same pieces");
    static_assert(BN >= 128 && WR * WT <= kSmMaxWaves, "tile shape");
    __shared__ _Float16 xs0[BUF];
    __shared__ _Float16 xs1[BUF];

    const int nwaves = WR * WT;
    const int tile = xcd_tile(blockIdx.x, tiles);
    const int rt = tile % row_tiles, tt = tile / row_tiles;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wr = wave % WR, wt = wave / WR;
    const int r0 = rt * BM + wr * R * 16;         // this wave's first row
    const int t0 = tt * BN;                       // the workgroup's first token
    const int ldv = C * NN;                       // host checked: ldv % 8 == 0, M * ldv < 2^31
    const int nsteps = (K + kSmKStep - 1) / kSmKStep;
    const int grp = lane >> 4, li = lane & 15;

    // ---- weights: per row block, the lane's row and its 16 columns of a step
    const _Float16 *vrow[R];
    const uint8_t *irow[R];
#pragma unroll
    for (int b = 0; b < R; ++b) {
        const int row = min(r0 + 16 * b + li, M - 1);   // rows past M: never stored
        vrow[b] = values + (int64_t)row * ldv;
        irow[b] = indices + (int64_t)(row / g) * ldv;
    }
    // slot of the first kept column of this lane's 16 columns in step s
    auto slot0 = [&](int s) { return (s * kSmKStep + 16 * grp) / MM * NN; };
    auto load_raw = [&](int s, SmRaw<SPW> (&raw)[R]) {
        const int sl = slot0(min(s, nsteps - 1));
        const int slc = sl < ldv ? sl : 0;             // a window past the last chunk: zeros below
#pragma unroll
        for (int b = 0; b < R; ++b) {
            raw[b].v = *reinterpret_cast<const decltype(raw[b].v) *>(vrow[b] + slc);
            raw[b].o = *reinterpret_cast<const decltype(raw[b].o) *>(irow[b] + slc);
        }
    };
    // the stored values and index word of one row block: element (q, t) of
    // the 4-column group q takes kept slot j = (q >> LM4) * NN + t when that
    // slot's column lies in group q (else 0); its position is the column's
    // offset within the group.  Built a pair of elements (a word) at a time.
    auto build_a = [&](int s, const SmRaw<SPW> &raw, h8 &a, uint32_t &idx) {
        const uint32_t live = slot0(s) < ldv ? 0xffffffffu : 0u;
        typedef uint32_t u4w __attribute__((ext_vector_type(4)));
        u4w w;
        if constexpr (LM4 == 1 && NN == 2) {
            // 2 of 8: slots 0, 1 in the first chunk, 2, 3 in the second; bit 2
            // of an offset says which group of 4 of its chunk it lies in
            const uint32_t O = raw.o;
            const uint32_t B = (O >> 2) & 0x01010101u;
            const uint32_t m01 = ((B & 1u) | ((B & 0x100u) << 8)) * 0xffffu;           // slots 0, 1 in group 1
            const uint32_t m23 = (((B >> 16) & 1u) | ((B >> 8) & 0x10000u)) * 0xffffu;  // slots 2, 3 in group 3
            const uint32_t v01 = raw_word<SPW>(raw, 0) & live, v23 = raw_word<SPW>(raw, 1) & live;
            w = u4w{v01 & ~m01, v01 & m01, v23 & ~m23, v23 & m23};
            const uint32_t Q = O & 0x03030303u;
            const uint32_t z = Q | (Q >> 6);   // positions of slots 0,1 in bits 0-3, of 2,3 in 16-19
            idx = ((z & 0xfu) | ((z >> 8) & 0xf00u)) * 0x11u;
        } else {
            constexpr uint32_t GM = (1u << LM4) - 1;   // groups of 4 per chunk, minus 1
            idx = 0;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint32_t h = (uint32_t)q & GM;
                if constexpr (NN == 2) {
                    const int j0 = 2 * (q >> LM4);
                    const uint32_t o0 = raw_index<SPW>(raw, j0), o1 = raw_index<SPW>(raw, j0 + 1);
                    uint32_t m = 0xffffffffu;
                    if constexpr (LM4 > 0)
                        m = (((o0 >> 2) & GM) == h ? 0xffffu : 0u) | (((o1 >> 2) & GM) == h ? 0xffff0000u : 0u);
                    w[q] = raw_word<SPW>(raw, j0 / 2) & m & live;
                    idx |= ((o0 & 3u) << (4 * q)) | ((o1 & 3u) << (4 * q + 2));
                } else {
                    const int j = q >> LM4;
                    const uint32_t o = raw_index<SPW>(raw, j);
                    const bool here = LM4 == 0 || ((o >> 2) & GM) == h;
                    w[q] = here ? raw_half<SPW>(raw, j) & live : 0u;
                    idx |= (o & 3u) << (4 * q);
                }
            }
        }
        a = __builtin_bit_cast(h8, w);
    };

    // ---- X: 64 rows x BN tokens per step into LDS, swizzled
    const int copy_row = lane / LPR, copy_pc = lane % LPR;
    typedef uint32_t u4 __attribute__((ext_vector_type(4)));
    // piece j of step s: staged row r = j * RPI + copy_row, 16 bytes at the
    // lane's swizzled place (steps past the last load clamped rows)
    int xrow[NCW];
    uint32_t xtok[NCW];
#pragma unroll
    for (int c = 0; c < NCW; ++c) {
        const int r = (wave + c * nwaves) * RPI + copy_row;  // staged row
        const int seg = (copy_pc >> 1) ^ sm_swz(r);           // logical 32-byte segment
        xrow[c] = r;
        xtok[c] = (uint32_t)min(t0 + 16 * seg + 8 * (copy_pc & 1), N - 8);  // host checked: N % 8 == 0
    }
    auto load_x = [&](int s, u4 (&xr)[NCW]) {
        const int k0 = min(s, nsteps - 1) * kSmKStep;
#pragma unroll
        for (int c = 0; c < NCW; ++c) {
            const uint32_t k = (uint32_t)min(k0 + xrow[c], K - 1);  // rows past K: zero weights
            xr[c] = *reinterpret_cast<const u4 *>(X + (k * (uint32_t)ldx + xtok[c]));  // K * ldx < 2^31
        }
    };
    auto store_x = [&](const u4 (&xr)[NCW], _Float16 *buf) {
#pragma unroll
        for (int c = 0; c < NCW; ++c) {
            const int j = wave + c * nwaves;
            *reinterpret_cast<u4 *>(buf + j * RPI * PITCH + 8 * lane) = xr[c];
        }
    };
    // transposing read q of token block tb: rows (q >> 1) * 32 + 8 grp + 4 (q & 1) + k'
    const int tr_k = (lane & 15) >> 2, tr_t = 4 * (lane & 3);
    auto read_b = [&](const _Float16 *__restrict__ buf, int tb, h16 &bv) {
        const int seg = wt * T + tb;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int r = (q >> 1) * 32 + 8 * grp + 4 * (q & 1) + tr_k;
            const h4 v = sm_read_tr(buf + r * PITCH + 16 * (seg ^ sm_swz(r)) + tr_t);
#pragma unroll
            for (int i = 0; i < 4; ++i) bv[4 * q + i] = v[i];
        }
    };

    v4f acc[R][T];
#pragma unroll
    for (int b = 0; b < R; ++b)
#pragma unroll
        for (int t = 0; t < T; ++t) acc[b][t] = v4f{0.f, 0.f, 0.f, 0.f};

    SmRaw<SPW> raw0[R], raw1[R];
    u4 xr0[NCW], xr1[NCW], xr2[NCW];
    // step s reads buffer s % 2 (stored during step s-1), stores X of step
    // s+1 into the other one from register set (s+1) % 3 (loaded two steps
    // earlier), and loads X of step s+3 into set s % 3 and the weights of
    // step s+1.  No load is conditional (steps past the last load clamped
    // data nobody uses), so the compiler's waits stay exact.
    load_x(0, xr0);
    load_x(1, xr1);
    load_raw(0, raw0);
    load_x(2, xr2);
    store_x(xr0, xs0);

    auto step = [&](int s, const _Float16 *cur, _Float16 *nxt, const SmRaw<SPW> (&raw)[R],
                    SmRaw<SPW> (&raw_nxt)[R], const u4 (&x_nxt)[NCW], u4 (&x_new)[NCW]) {
        // this wave's LDS stores are done; after the barrier every wave's are,
        // and every wave is done reading nxt (step s-1)
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
        store_x(x_nxt, nxt);
        load_raw(s + 1, raw_nxt);
        load_x(s + 3, x_new);
        h8 a[R];
        uint32_t ix[R];
#pragma unroll
        for (int b = 0; b < R; ++b) build_a(s, raw[b], a[b], ix[b]);
        h16 bv[2];
        read_b(cur, 0, bv[0]);
#pragma unroll
        for (int tb = 0; tb < T; ++tb) {
            if (tb + 1 < T) read_b(cur, tb + 1, bv[(tb + 1) & 1]);
            // keep the reads of block tb+1 ahead of block tb's instructions
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int b = 0; b < R; ++b)
                acc[b][tb] = __builtin_amdgcn_smfmac_f32_16x16x64_f16(a[b], bv[tb & 1], acc[b][tb],
                                                                      (int)ix[b], 0, 0);
        }
    };
    // six steps per iteration (buffers period 2, weights 2, register sets 3),
    // no branch inside; the last steps after the loop
    int s = 0;
    for (; s + 6 <= nsteps; s += 6) {
        step(s, xs0, xs1, raw0, raw1, xr1, xr0);
        step(s + 1, xs1, xs0, raw1, raw0, xr2, xr1);
        step(s + 2, xs0, xs1, raw0, raw1, xr0, xr2);
        step(s + 3, xs1, xs0, raw1, raw0, xr1, xr0);
        step(s + 4, xs0, xs1, raw0, raw1, xr2, xr1);
        step(s + 5, xs1, xs0, raw1, raw0, xr0, xr2);
    }
    if (s < nsteps) step(s, xs0, xs1, raw0, raw1, xr1, xr0);
    if (s + 1 < nsteps) step(s + 1, xs1, xs0, raw1, raw0, xr2, xr1);
    if (s + 2 < nsteps) step(s + 2, xs0, xs1, raw0, raw1, xr0, xr2);
    if (s + 3 < nsteps) step(s + 3, xs1, xs0, raw1, raw0, xr1, xr0);
    if (s + 4 < nsteps) step(s + 4, xs0, xs1, raw0, raw1, xr2, xr1);

    if constexpr (EPI == NMG_EPILOGUE_GELU) {
        // the GELU table into the first two staging buffers: entries of
        // non-negative inputs (sign bit clear) in xs0, of negative ones in xs1
        __syncthreads();  // every wave is done with the last step (and its stores)
        const uint4 *src = reinterpret_cast<const uint4 *>(g_gelu_f16_s);
        for (int i = threadIdx.x; i < 8192; i += blockDim.x)
            reinterpret_cast<uint4 *>(i < 4096 ? xs0 : xs1)[i % 4096] = src[i];
        __syncthreads();
    }
    // result register r of (row block b, token block tb) at lane l is
    // Y[r0 + 16 b + 4 (l / 16) + r][t0 + 16 (wt T + tb) + l % 16]
#pragma unroll
    for (int b = 0; b < R; ++b)
#pragma unroll
        for (int tb = 0; tb < T; ++tb)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = r0 + 16 * b + 4 * grp + r;
                const int tok = t0 + 16 * (wt * T + tb) + li;
                if (row >= M || tok >= N) continue;
                const _Float16 h = (_Float16)acc[b][tb][r];  // nearest even, as nmg_spmm stores it
                _Float16 out = h;
                if constexpr (EPI == NMG_EPILOGUE_GELU) {
                    const uint16_t bits = __builtin_bit_cast(uint16_t, h);
                    out = ((bits & 0x8000u) ? xs1 : xs0)[bits & 0x7fffu];
                } else if constexpr (EPI == NMG_EPILOGUE_ADD) {
                    out = (_Float16)((float)h + (float)Rs[(int64_t)row * ldr + tok]);
                }
                __builtin_nontemporal_store(out, Y + (int64_t)row * ldy + tok);
            }
}

template <int LM4, int NN, int R, int T, int WR, int WT, int EPI>
nmg_status launch_sm_cfg(const SpmmArgs &a) {
    const nmg_layout *L = a.L;
    constexpr int BM = WR * R * 16, BN = WT * T * 16;
    const int row_tiles = (L->M + BM - 1) / BM;
    const int tiles = row_tiles * ((a.N + BN - 1) / BN);
    hipLaunchKernelGGL((k_spmm_smfmac<LM4, NN, R, T, WR, WT, EPI>), dim3(tiles), dim3(64 * WR * WT), 0,
                       a.stream, (const _Float16 *)a.values, a.indices, (const _Float16 *)a.X, a.ldx,
                       (_Float16 *)a.Y, a.ldy, (const _Float16 *)a.R, a.ldr, L->M, L->K, a.N, L->g,
                       L->C, row_tiles, tiles);
    return launched();
}

// Workgroup tile: 64 rows x 128 tokens (4 waves of 32 x 64) for layers of
// 1536 rows or more, else 128 x 128 (8 waves of 32 x 64).  Measured on the
// BERT layers (4096 tokens) against 128 x 256 and other shapes.
template <int LM4, int NN, int EPI>
nmg_status launch_sm_epi(const SpmmArgs &a) {
    if (a.L->M >= 1536) return launch_sm_cfg<LM4, NN, 2, 4, 2, 2, EPI>(a);
    return launch_sm_cfg<LM4, NN, 2, 4, 4, 2, EPI>(a);
}

template <int LM4, int NN>
nmg_status launch_sm(const SpmmArgs &a) {
    switch (a.epi) {
        case NMG_EPILOGUE_GELU: return launch_sm_epi<LM4, NN, NMG_EPILOGUE_GELU>(a);
        case NMG_EPILOGUE_ADD: return launch_sm_epi<LM4, NN, NMG_EPILOGUE_ADD>(a);
        default: return launch_sm_epi<LM4, NN, NMG_EPILOGUE_NONE>(a);
    }
}

}  // namespace

// The sparse-matrix-core kernel takes binary16 layouts with n in {1, 2} and m
// in {4, 8, 16} (every aligned group of 4 columns then keeps at most 2), any
// g, value and index rows on 16-byte boundaries (C * n % 8 == 0, values and
// indices 16-byte aligned), and X that can be copied to LDS 16 bytes at a time
// (X and ldx on 16-byte boundaries, N % 8 == 0); offsets within 31 bits.
// `values`, `indices` and `X` may be NULL to ask about the layout alone.
bool nmg_internal::spmm_smfmac_supported(const nmg_layout *L, const void *values,
                                         const uint8_t *indices, const void *X, int64_t ldx,
                                         int64_t N) {
    const int64_t ldv = (int64_t)L->C * L->n;
    return L->dtype == NMG_F16 && (L->n == 1 || L->n == 2) &&
           (L->m == 4 || L->m == 8 || L->m == 16) && ldv % 8 == 0 &&
           (values == nullptr || aligned(values, 16)) && (indices == nullptr || aligned(indices, 16)) &&
           (X == nullptr || aligned(X, 16)) && ldx % 8 == 0 && N % 8 == 0 &&
           (int64_t)L->M * ldv < ((int64_t)1 << 31) && (int64_t)L->K * ldx < ((int64_t)1 << 31);
}

nmg_status nmg_internal::spmm_smfmac(const SpmmArgs &a) {
    const int lm4 = a.L->m == 4 ? 0 : a.L->m == 8 ? 1 : 2;
    switch (lm4 * 2 + a.L->n - 1) {
        case 0: return launch_sm<0, 1>(a);
        case 1: return launch_sm<0, 2>(a);
        case 2: return launch_sm<1, 1>(a);
        case 3: return launch_sm<1, 2>(a);
        case 4: return launch_sm<2, 1>(a);
        case 5: return launch_sm<2, 2>(a);
        default: return NMG_ERR_UNSUPPORTED;
    }
}
