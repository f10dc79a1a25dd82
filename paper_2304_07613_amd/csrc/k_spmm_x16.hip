// k_spmm_x16.hip -- the product Y = W_s X on the 16 x 16 x 32 binary16 matrix
// instruction of gfx950 (v_mfma_f32_16x16x32_f16, binary32 accumulation), in
// two modes:
//
//   HALF   binary16 layouts (binary16 in and out);
//   SPLIT  binary32 layouts: every binary32 operand v is carried as two
//          binary16 numbers, hi = fp16(v) and lo = fp16(v - hi) (for X the
//          remainder scaled by 2^11, and the weights it meets scaled by 2^-11,
//          so that it stays a normal number), and the four products hi*hi,
//          hi*lo, lo*hi and lo*lo are all formed (exactly, in binary32) and
//          summed in binary32.  hi + lo holds 22 of v's 24 significant bits,
//          so each product is within about 2^-21 of the binary32 one; see
//          nmg.h for the range in which this holds.
//
// Paper: STen (arXiv 2304.07613), Section 5.1 (the sparse x dense product of
// the grouped n:m layout); the kernel itself is this library's design.
//
// Orientation.  One instruction computes D[t][j] += sum_k A[t][k] B[k][j] for
// 16 tokens t, 16 columns j and 32 contraction indices k.  A holds gathered X
// (a group's k-slots select the X rows, so the 32 k of one instruction are 32
// k-slots of one group), B the group's weights; a column j is a weight row
// (HALF: 16 rows of a group, or 8 with the other 8 columns zero), or in SPLIT
// mode a (row, part) pair: columns 0-7 carry the hi parts of 8 rows, 8-15 the
// lo parts, and one instruction reads the hi parts of X, a second one the lo
// parts.  Lane l holds A[l % 16][8 (l / 16) + e] and B[8 (l / 16) + e][l % 16],
// e = 0..7, and gets D[4 (l / 16) + i][l % 16], i = 0..3 (fitted to an
// in-bounds probe of the instruction): 4 consecutive tokens of one row per
// lane, a 16-byte store.
//
// Staging.  A workgroup covers R rows and a tile of 128 tokens; windows of 32
// k-slots (32 / n whole chunks, all m X rows of each) are staged in LDS, in
// rotating buffers, one barrier per window.  HALF copies X rows straight
// from global memory into LDS (buffer loads with an LDS destination), two or
// three windows ahead; SPLIT loads binary32 X into registers one window
// ahead, splits it and writes a hi plane and a lo plane.  The A operand comes from two transposing
// LDS reads (ds_read_b64_tr_b16): in each 16-lane group, lanes 4k .. 4k+3
// read 16 tokens of the row of k-slot k, and lane i receives token i of the 4
// rows side by side.
//
// LDS banks.  One transposing read touches 16 row segments of 32 bytes, and
// each half-wave's 8 segments should fall on the 8 distinct 32-byte quarters
// of the 256-byte bank window.  A row's in-chunk offset is data, so rows are
// laid out with a stride that is a multiple of 256 bytes and chunks with a
// stride of 32 bytes more: a segment's bank quarter depends only on its chunk
// (and the token tile), and the order of k-slots inside a window (kb_slot)
// puts 8 consecutive chunks in each half-wave's read.
//
// Scaling (SPLIT).  Each unit of 8 rows is multiplied by a power of two that
// brings its largest |weight| into [2^13, 2^14), so the lo parts of its
// weights are binary16 normal numbers whatever the weights' magnitude; the
// output is multiplied back (exact).
#include "common.hpp"

namespace {

typedef _Float16 h4 __attribute__((ext_vector_type(4)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef short s4 __attribute__((ext_vector_type(4)));
typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kXSlots = 32;    // k-slots per window (one instruction's contraction)
constexpr int kXTok = 128;     // tokens per tile
constexpr int kXTiles = 8;     // 16-token sub-tiles per tile

// The k-slot (0..31, within the window) that lane group q (= lane / 16) puts
// at contraction index 8 q + e.  The transposing read r = e / 4 of half-wave h
// = q / 2 reads the slots of "pass" P = 2 r + h: 8 slots from 8 consecutive
// chunks (n <= 2), at pass position ps = 4 (q % 2) + e % 4.
__host__ __device__ constexpr int kb_slot(int n, int q, int e) {
    const int P = 2 * (e >> 2) + (q >> 1);
    const int ps = 4 * (q & 1) + (e & 3);
    const int cgroups = (kXSlots / n) / 8;  // groups of 8 chunks in a window
    return (8 * (P % cgroups) + ps) * n + P / cgroups;
}

typedef __attribute__((address_space(3))) char lds_char;

// GELU(x) for every binary16 x, indexed by the bits of x (the table nmg_gelu
// uses, generated at build time), and where it is a rule instead
__device__ __attribute__((aligned(16))) const uint16_t g_x16_gelu[65536] = {
#include "gelu_f16_table.inc"
};
#include "gelu_f16_bounds.inc"
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) u32x2 lds_u2;

// The transposing LDS read of 8 bytes at `p`.
__device__ __forceinline__ h4 lds_read_tr(lds_char *p) {
#if defined(__HIP_DEVICE_COMPILE__)
    return __builtin_bit_cast(h4, __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s4 *)p));
#else
    (void)p;
    return h4{};
#endif
}

// s_waitcnt immediate: at most n vector-memory operations of this wave
// outstanding, and (lgkm0) none of its LDS operations; expcnt left at its
// maximum
[[maybe_unused]] __host__ __device__ constexpr int waitcnt_imm(int n, bool lgkm0) {
    return (n & 0xf) | ((n >> 4) << 14) | (0x7 << 4) | ((lgkm0 ? 0 : 0xf) << 8);
}

// The end of a window: this wave's copies into LDS up to `n` vector-memory
// operations ago and all its LDS writes have landed (the waits are explicit:
// a workgroup fence would also wait for the loads still in flight for later
// windows, LDS copies counting as LDS writes), then the workgroup barrier; the
// memory clobber keeps the compiler from moving LDS accesses across it.
template <int n>
__device__ __forceinline__ void window_barrier() {
#if defined(__HIP_DEVICE_COMPILE__)
    __builtin_amdgcn_s_waitcnt(waitcnt_imm(n, true));
    asm volatile("s_barrier" ::: "memory");
#endif
}

// All LDS operations of this wave done, then the workgroup barrier (memory
// operations, LDS copies included, may stay in flight)
__device__ __forceinline__ void lds_barrier() {
#if defined(__HIP_DEVICE_COMPILE__)
    __builtin_amdgcn_s_waitcnt(waitcnt_imm(63, true));
    asm volatile("s_barrier" ::: "memory");
#endif
}

// a + (the value of lane l ^ 8 of the same 16-lane row)
__device__ __forceinline__ float add_row_ror8(float a) {
#if defined(__HIP_DEVICE_COMPILE__)
    const int o = __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, a), 0x128, 0xf, 0xf, false);
    return a + __builtin_bit_cast(float, o);
#else
    return a;
#endif
}

#ifndef X16_NT_STORE
#define X16_NT_STORE 1
#endif
template <typename T>
__device__ __forceinline__ void store_y(T v, T *p) {
    if constexpr (X16_NT_STORE) __builtin_nontemporal_store(v, p);
    else *p = v;
}

__device__ __forceinline__ uint32_t pack_h2(_Float16 lo, _Float16 hi) {
    return (uint32_t)__builtin_bit_cast(uint16_t, lo) | ((uint32_t)__builtin_bit_cast(uint16_t, hi) << 16);
}

// Workgroup geometry, shared by the kernel and its launcher.
template <bool SPLIT, bool U16, int GW, int NW>
struct XGeom {
    static constexpr int rows_unit = SPLIT ? 8 : (U16 ? 16 : 8);
    static constexpr int rows_wave = GW * rows_unit;
    static constexpr int rows_wg = NW * rows_wave;
    // bytes of one staged X row: SPLIT [hi 64 tokens | lo 64 tokens] twice,
    // HALF 128 binary16 tokens
    static constexpr int row_bytes = SPLIT ? 512 : 256;
};

// Fused GELU (binary16): after the last window the staging buffers take the
// table entries that are not a rule -- non-negative inputs below
// NMG_GELU_F16_IDENTITY_FROM in buffer 0, negative ones below
// NMG_GELU_F16_NEGZERO_FROM in buffer 1 -- and the waves' output regions go
// to buffers 2 (and 3) and to what the tables leave of buffers 0 and 1.
constexpr int kGeluPosBytes = (2 * NMG_GELU_F16_IDENTITY_FROM + 255) / 256 * 256;
constexpr int kGeluNegBytes = (2 * (NMG_GELU_F16_NEGZERO_FROM - 0x8000) + 255) / 256 * 256;
__host__ __device__ constexpr int x16_out_region(bool split, int rows_wave) {
    return rows_wave * (kXTok * (split ? 4 : 2) + 32);
}
__host__ __device__ constexpr bool x16_gelu_fits(bool split, int rows_wave, int waves, int bufcap,
                                                 int nbuf) {
    return !split && nbuf >= 3 && kGeluPosBytes <= bufcap && kGeluNegBytes <= bufcap &&
           (nbuf - 2) * (bufcap / x16_out_region(split, rows_wave)) +
                   (bufcap - kGeluPosBytes) / x16_out_region(split, rows_wave) +
                   (bufcap - kGeluNegBytes) / x16_out_region(split, rows_wave) >=
               waves;
}

// LDS bytes of one staging buffer (a multiple of 256)
inline int x16_buffer_bytes(int n, int m, int row_bytes) {
    const int cs = m * row_bytes + 32;
    return ((kXSlots / n) * cs + 255) / 256 * 256;
}
// Staging buffers: binary16 DP + 1 when windows are copied DP ahead (four
// of 40 KB when a window fits, copies three windows ahead; else three of 52
// KB, two ahead), binary32 two (its X passes through registers one window
// ahead, DP = 1)
template <bool SPLIT, int DP> constexpr int x16_nbuf() { return SPLIT ? 2 : DP + 1; }
template <bool SPLIT, int DP> constexpr int x16_buf_cap() {
    return SPLIT ? 81920 : DP == 3 ? 40960 : 53248;
}

// ---------------------------------------------------------------- prepared operands
//
// The product's per-window operands, computed once per packed weight: for
// every unit of RU rows and window of 32 k-slots, each lane's B operand (8
// binary16: the weights of its column at the slots kb_slot(q, 0..7), SPLIT
// the hi or lo part of the scaled binary32 weight) and the in-chunk offsets
// of the two rows its transposing reads fetch (the index bytes of slots
// kb_slot(q, p / 4) and kb_slot(q, 4 + p / 4)); and per unit the exponent of
// its scale (SPLIT).  Layout, for U units and W windows:
//   frag   U * W * 64 entries of 16 bytes   [(unit * W + window) * 64 + lane]
//   offs   U * W * 64 entries of 2 bytes    (low byte: read 0, high: read 1)
//   scale  U bytes                          (signed exponent; 0 for binary16)
struct XPrep {
    int units, nwin;
    size_t frag, offs, scale, bytes;  // byte offsets and total
};
inline XPrep x16_prep_layout(const nmg_layout *L, int ru) {
    XPrep P;
    P.units = L->M / ru;
    P.nwin = (L->C * L->n + kXSlots - 1) / kXSlots;
    const size_t e = (size_t)P.units * P.nwin * 64;
    P.frag = 0;
    P.offs = e * 16;
    P.scale = P.offs + e * 2;
    P.bytes = (P.scale + P.units + 255) / 256 * 256;
    return P;
}

template <bool SPLIT, int NS, int RU>
__global__ __launch_bounds__(64) void k_x16_prepare(const void *__restrict__ values_,
                                                    const uint8_t *__restrict__ indices, h8 *frag,
                                                    uint16_t *offs, int8_t *scale, int M, int m,
                                                    int g, int C, int nwin) {
    const int unit = blockIdx.x;
    const int lane = threadIdx.x;
    const int q = lane >> 4, p = lane & 15;
    const int ldv = C * NS;
    const int r0 = unit * RU;
    const int grp = r0 / g;
    // column -> row of the unit (SPLIT: row p % 8, part p / 8; binary16
    // 8-row units: columns 8-15 are zero)
    const int b_row = (SPLIT || RU == 16) ? (RU == 16 ? p : (p & 7)) : (p & 7);
    const bool b_lo = SPLIT && p >= 8;
    const bool b_zero = !SPLIT && RU == 8 && p >= 8;
    int sc = 0;
    if constexpr (SPLIT) {
        // the unit's RU rows are contiguous: 8 independent loads per lane in flight
        const float *vr = reinterpret_cast<const float *>(values_) + (int64_t)r0 * ldv;
        const int nv = RU * ldv;
        float mx = 0.f;
        for (int i0 = 0; i0 < nv; i0 += 8 * 64) {
            float x[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) x[k] = vr[min(i0 + k * 64 + lane, nv - 1)];
#pragma unroll
            for (int k = 0; k < 8; ++k) mx = fmaxf(mx, fabsf(x[k]));
        }
#pragma unroll
        for (int sh = 32; sh >= 1; sh >>= 1) mx = fmaxf(mx, __shfl_xor(mx, sh, 64));
        if (mx > 0.f && mx <= 3.4e38f) {
            int e = 0;
            (void)frexpf(mx, &e);  // mx in [2^(e-1), 2^e): scaled max in [2^13, 2^14)
            sc = 14 - e;
        }
        if (lane == 0) scale[unit] = (int8_t)sc;
    } else {
        if (lane == 0) scale[unit] = 0;
    }
    const float mul = __builtin_ldexpf(1.f, sc);
    for (int win = 0; win < nwin; ++win) {
        const int slot0 = win * kXSlots;
        const size_t e0 = ((size_t)unit * nwin + win) * 64 + lane;
        // A offsets
        uint32_t oo = 0;
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const int sl = slot0 + kb_slot(NS, q, 4 * r + (p >> 2));
            const uint32_t o = sl < ldv ? min((uint32_t)indices[(int64_t)grp * ldv + sl], (uint32_t)(m - 1)) : 0u;
            oo |= o << (8 * r);
        }
        offs[e0] = (uint16_t)oo;
        // B operand
        h8 b;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int sl = slot0 + kb_slot(NS, q, e);
            _Float16 h = (_Float16)0.f;
            if (sl < ldv && !b_zero) {
                if constexpr (SPLIT) {
                    const float w = reinterpret_cast<const float *>(values_)[(int64_t)(r0 + b_row) * ldv + sl] * mul;
                    const _Float16 hi = (_Float16)w;
                    const _Float16 lo = (_Float16)(w - (float)hi);
                    h = b_lo ? lo : hi;
                } else {
                    h = reinterpret_cast<const _Float16 *>(values_)[(int64_t)(r0 + b_row) * ldv + sl];
                }
            }
            b[e] = h;
        }
        frag[e0] = b;
    }
}

// ---------------------------------------------------------------- the product

// R_ == nullptr: Y = P; else Y = P + R (the sum in binary32 of the product
// rounded to the element type and R, rounded again)
template <bool SPLIT, int NS, bool U16, int GW, int NW, int NSTG, int DP, int TPW>
__global__ __launch_bounds__(64 * NW) void k_spmm_x16(
    const h8 *__restrict__ frag, const uint16_t *__restrict__ offs, const int8_t *__restrict__ scale,
    const void *__restrict__ X_, int64_t ldx, void *__restrict__ Y_, int64_t ldy,
    const void *__restrict__ R_, int64_t ldr, int epi, int M, int K, int N, int m, int nwin,
    int row_blocks) {
    using G = XGeom<SPLIT, U16, GW, NW>;
    constexpr int RU = G::rows_unit, ROWB = G::row_bytes;
    constexpr int CPW = kXSlots / NS;  // chunks per window
    constexpr int NBUF = x16_nbuf<SPLIT, DP>();
    constexpr int BUFCAP = x16_buf_cap<SPLIT, DP>();
    static_assert(NS == 1 || NS == 2, "n of 1 or 2");
    static_assert(TPW == 1 || (TPW == 2 && !SPLIT && DP == 2), "two tiles: binary16, two windows ahead");
    // the staging buffers as distinct objects, so that the compiler can tell
    // the copies into one from the reads of another
    __shared__ __attribute__((aligned(256))) char xs0[BUFCAP];
    __shared__ __attribute__((aligned(256))) char xs1[BUFCAP];
    __shared__ __attribute__((aligned(256))) char xs2[NBUF >= 3 ? BUFCAP : 16];
    __shared__ __attribute__((aligned(256))) char xs3[NBUF >= 4 ? BUFCAP : 16];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int q = lane >> 4, p = lane & 15;
    const int cs = m * ROWB + 32;   // chunk stride in LDS
    const int rw = CPW * m;         // X rows per window
    const int units = M / RU;

    // this workgroup's tiles: row block rb, TPW tiles of 128 tokens from t0
    // (tiles of one token range are adjacent, so an XCD's workgroups share X
    // in its L2); its steps are the windows of its tiles, one after the other
    const int tile = xcd_tile(blockIdx.x, gridDim.x);
    const int rb = tile % row_blocks;
    const int t0 = (tile / row_blocks) * (TPW * kXTok);
    const int ntile = TPW == 1 ? 1 : min(TPW, (N - t0 + kXTok - 1) / kXTok);
    const int nstep = ntile * nwin;
    const int row_w = rb * G::rows_wg + wave * G::rows_wave;  // first row of this wave
    int ug[GW];                                               // this wave's units (clamped)
#pragma unroll
    for (int u = 0; u < GW; ++u) ug[u] = min((row_w + u * RU) / RU, units - 1);

    // transposing reads: lane (q, p) reads, for read r, row o_r of the chunk
    // of slot kb_slot(q, 4 r + p / 4), tokens 4 (p % 4) .. +3 of the sub-tile
    uint32_t rbase[2];
#pragma unroll
    for (int r = 0; r < 2; ++r) {
        int s = 0;
#pragma unroll
        for (int qq = 0; qq < 4; ++qq)
#pragma unroll
            for (int kk = 0; kk < 4; ++kk)
                if (qq == q && kk == (p >> 2)) s = kb_slot(NS, qq, 4 * r + kk);
        rbase[r] = (uint32_t)((s / NS) * cs + (p & 3) * 8);
    }

    // ---- staging
    const float *Xf = reinterpret_cast<const float *>(X_);
    // binary16 X as a buffer of K rows, copied into LDS by buffer loads (see
    // lds_copy16_buf; host: K ldx < 2^31 elements, so every byte offset fits
    // 32 bits)
    const buf_rsrc_t xr16 = buf_rsrc(X_, SPLIT ? 0u : (uint32_t)((int64_t)K * ldx * 2));
    // SPLIT: item i of a window = (row i / 32, tokens 4 (i % 32) .. +3); lane
    // takes items lane_g + k 64 NW (rows st_row0 + k SROWS, one token offset);
    // items past the last are clamped to the last row (a duplicate writes the
    // same bytes twice)
    constexpr int SROWS = SPLIT ? 64 * NW / (kXTok / 4) : 1;
    const int lane_g = wave * 64 + lane;
    const int st_row0 = SPLIT ? lane_g / (kXTok / 4) : 0;
    const int st_ti = lane_g % (kXTok / 4);
    const uint32_t st_sub = (uint32_t)((st_ti >> 4) * 256 + (st_ti & 15) * 8);  // within a row
    const int st_tok = min(t0 + 4 * st_ti, N - 4);   // tokens past N: never stored
    // HALF: copy instruction j = wave + k NW moves 4 rows (16 lanes of 16
    // bytes each): rows 4 j .. 4 j + 3 of the window, one chunk (m % 4 == 0),
    // 1 KB contiguous in LDS; instructions past the last repeat the last one
    // (same bytes to the same place), so every wave issues exactly NSTG copies
    const int ninst = rw / 4;
    // r / m for the rows of a window (r < 32 m, m <= 45) by a multiply
    const uint32_t inv_m = (65536u + (uint32_t)m - 1) / (uint32_t)m;
    auto div_m = [&](int r) __attribute__((always_inline)) { return (int)(((uint32_t)r * inv_m) >> 16); };
    const int cp_sub = lane >> 4;                 // row within the instruction's 4
    const int cp_tok = 8 * (lane & 15);           // token offset within the tile
    f4 stg[NSTG];
    // item k of window w's staging
    auto stage_one = [&](int w, char *buf, auto kc) __attribute__((always_inline)) {
        constexpr int k = decltype(kc)::value;
        // step w: window w % nwin of tile w / nwin
        const int tj = (TPW > 1 && w >= nwin) ? 1 : 0;
        const int k0 = (w - tj * nwin) * rw;
        if constexpr (SPLIT) {
            const int row = min(st_row0 + k * SROWS, rw - 1);
            const int xr = min(k0 + row, K - 1);           // rows past K: never selected
            stg[k] = *reinterpret_cast<const f4 *>(Xf + (int64_t)xr * ldx + st_tok);
        } else {
            const int j = min(wave + k * NW, ninst - 1);   // uniform
            const int row0 = 4 * j;                         // first row of the four, in the window
            const int c = div_m(row0), o = row0 - c * m;    // its chunk and offset (uniform)
            const int xr = min(k0 + row0 + cp_sub, K - 1);
            const int tok = min(t0 + tj * kXTok + cp_tok, N - 8);
            lds_copy16_buf(xr16, ((uint32_t)xr * (uint32_t)ldx + (uint32_t)tok) * 2u,
                           buf + c * cs + o * ROWB);
        }
    };
    auto stage_issue = [&](int w, char *buf) __attribute__((always_inline)) {
        static_for<NSTG>([&](auto kc) { stage_one(w, buf, kc); });
    };
    // SPLIT: the registers of one window, split and written to LDS
    auto stage_write_one = [&](char *buf, auto kc) __attribute__((always_inline)) {
        constexpr int k = decltype(kc)::value;
        if constexpr (SPLIT) {
            lds_char *lb = (lds_char *)buf;
            const int row = min(st_row0 + k * SROWS, rw - 1);
            const int c = div_m(row), o = row - c * m;
            const uint32_t off = (uint32_t)(c * cs + o * ROWB) + st_sub;
            _Float16 hi[4], lo[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                hi[i] = (_Float16)stg[k][i];
                // the remainder (exact in binary32) scaled by 2^11 (exact), so
                // that it stays a normal binary16 number down to |x| of about
                // 2^-14; the products with it are scaled back through the
                // weights (compute)
                lo[i] = (_Float16)((stg[k][i] - (float)hi[i]) * 2048.f);
            }
            *(lds_u2 *)(lb + off) = u32x2{pack_h2(hi[0], hi[1]), pack_h2(hi[2], hi[3])};
            *(lds_u2 *)(lb + off + 128) = u32x2{pack_h2(lo[0], lo[1]), pack_h2(lo[2], lo[3])};
        }
    };
    auto stage_write = [&](char *buf) __attribute__((always_inline)) {
        static_for<NSTG>([&](auto kc) { stage_write_one(buf, kc); });
    };

    // ---- a window's prepared operands (windows past the last: the last one)
    struct Ops {
        h8 b[GW];
        uint32_t o[GW];
    };
    // (binary16 8-row units: columns 8-15 are zero; those lanes load the
    // fragment of column p - 8, so a unit's fragments are 512 distinct bytes,
    // and zero it where it is used)
    const int flane = (!SPLIT && !U16) ? (lane & ~8) : lane;
    auto load_one = [&](int w, Ops &op, auto uc) __attribute__((always_inline)) {
        constexpr int u = decltype(uc)::value;
        const int wc = min(w, nstep - 1);
        const size_t e = ((size_t)ug[u] * nwin + ((TPW > 1 && wc >= nwin) ? wc - nwin : wc)) * 64;
        op.b[u] = frag[e + flane];
        op.o[u] = offs[e + lane];
    };
    auto load_ops = [&](int w, Ops &op) __attribute__((always_inline)) {
        static_for<GW>([&](auto uc) { load_one(w, op, uc); });
    };
    // A addresses of a window (byte offsets within its buffer)
    auto addresses = [&](const Ops &op, uint32_t (&aa)[GW][2]) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < GW; ++u) {
            aa[u][0] = rbase[0] + (op.o[u] & 0xffu) * (uint32_t)ROWB;
            aa[u][1] = rbase[1] + (op.o[u] >> 8) * (uint32_t)ROWB;
        }
    };

    f4 acc[GW][kXTiles];
#pragma unroll
    for (int u = 0; u < GW; ++u)
#pragma unroll
        for (int t = 0; t < kXTiles; ++t) acc[u][t] = f4{0.f, 0.f, 0.f, 0.f};

    // ---- the products of one window: NM instructions, each fed by two
    // transposing reads issued PD instructions ahead
    constexpr int NPL = SPLIT ? 2 : 1;
    constexpr int NM = NPL * GW * kXTiles;
    constexpr int PD = 3;
    // The loads for later windows (NJ jobs) are issued between the
    // instructions, one every JS of them, so that the load path works while
    // the matrix cores do (issued all at once, they would queue on the load
    // path while the matrix cores wait at the next barrier).
    constexpr int NJ = NSTG + GW;
    constexpr int JS = (SPLIT ? NM / 2 : NM) / NJ > 0 ? (SPLIT ? NM / 2 : NM) / NJ : 1;
    // SPLIT: the X of window w + 1, loaded by the jobs, is split and written
    // to LDS (NSTG items) between the instructions of the second half, one
    // every WS of them.
    constexpr int WS = (NM / 2) / NSTG > 0 ? (NM / 2) / NSTG : 1;
    auto compute = [&](const char *buf, const Ops &op, const uint32_t (&aa)[GW][2], auto &&job,
                       auto &&post) __attribute__((always_inline)) {
        lds_char *lb = (lds_char *)buf;
        h4 ra[PD][2];
        auto issue = [&](auto ic) __attribute__((always_inline)) {
            constexpr int i = decltype(ic)::value;
            constexpr int pl = i / (GW * kXTiles), u = (i / kXTiles) % GW, t = i % kXTiles;
            constexpr uint32_t toff = SPLIT ? (uint32_t)((t >> 2) * 256 + pl * 128 + (t & 3) * 32)
                                            : (uint32_t)(t * 32);
            ra[i % PD][0] = lds_read_tr(lb + aa[u][0] + toff);
            ra[i % PD][1] = lds_read_tr(lb + aa[u][1] + toff);
        };
        // SPLIT: the lo plane of X holds remainders scaled by 2^11; its
        // instructions take the weights scaled by 2^-11 (exact while normal)
        h8 bl[GW];
#pragma unroll
        for (int u = 0; u < GW; ++u) {
            if constexpr (SPLIT) {
                const _Float16 k = (_Float16)(1.f / 2048.f);
                bl[u] = op.b[u] * h8{k, k, k, k, k, k, k, k};
            } else if constexpr (!U16) {
                const h8 z = {};
                bl[u] = p < 8 ? op.b[u] : z;
            } else {
                bl[u] = op.b[u];
            }
        }
        static_for<PD>([&](auto ic) { issue(ic); });
        static_for<NM>([&](auto ic) {
            constexpr int i = decltype(ic)::value;
            constexpr int pl = i / (GW * kXTiles), u = (i / kXTiles) % GW, t = i % kXTiles;
            const h4 a0 = ra[i % PD][0], a1 = ra[i % PD][1];
            const h8 a = {a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], a1[2], a1[3]};
            if constexpr (i + PD < NM) issue(std::integral_constant<int, i + PD>{});
            acc[u][t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, (SPLIT && pl == 0) ? op.b[u] : bl[u],
                                                               acc[u][t], 0, 0, 0);
            if constexpr (i % JS == 0 && i / JS < NJ) job(std::integral_constant<int, i / JS>{});
            if constexpr (i >= NM / 2 && (i - NM / 2) % WS == 0 && (i - NM / 2) / WS < NSTG)
                post(std::integral_constant<int, (i - NM / 2) / WS>{});
        });
        // jobs and post jobs the instructions did not reach
        static_for<NJ>([&](auto jc) {
            constexpr int j = decltype(jc)::value;
            if constexpr (j * JS >= NM) job(jc);
        });
        static_for<NSTG>([&](auto kc) {
            constexpr int k = decltype(kc)::value;
            if constexpr (NM / 2 + k * WS >= NM) post(kc);
        });
    };

    // ---- the outputs go through LDS: each wave writes its rows x 128 tokens
    // into a region of its own (rows padded by 32 bytes, so that the 8 rows a
    // write instruction touches fall on distinct banks; by 16 where a tile's
    // outputs must fit the one buffer free in the middle of the pipeline),
    // then stores whole rows, 16 bytes per lane (a full 256- or 512-byte run
    // per row, instead of 32- or 64-byte pieces from the instruction's own
    // layout)
    constexpr int ES = SPLIT ? 4 : 2;
    constexpr int RSTRIDE = kXTok * ES + ((TPW > 1 && NW * G::rows_wave * (kXTok * ES + 32) > BUFCAP) ? 16 : 32);
    constexpr int RB = G::rows_wave * RSTRIDE;       // one wave's region
    static_assert(TPW > 1 || RB == x16_out_region(SPLIT, G::rows_wave), "one region formula");
    static_assert(TPW == 1 || NW * RB <= BUFCAP, "a tile's outputs fit one staging buffer");
    constexpr int LPR = kXTok * ES / 16;              // lanes per row
    constexpr int RPI = 64 / LPR;                     // rows per instruction
    constexpr int NST = G::rows_wave / RPI;           // store instructions per wave and tile
    bool after_out = false;                           // the steps after a tile's outputs

    // a tile's outputs: acc -> this wave's region at ob -> whole rows of Y
    // (tokens from tb), GELU or the residual sum applied on the way
    constexpr bool GELU_OK = TPW == 1 && x16_gelu_fits(SPLIT, G::rows_wave, NW, BUFCAP, NBUF);
    auto tile_out = [&](lds_char *ob, int tb, bool gelu) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < GW; ++u) {
            const float sc = SPLIT ? __builtin_ldexpf(1.f, -(int)scale[ug[u]]) : 1.f;
#pragma unroll
            for (int t = 0; t < kXTiles; ++t) {
                f4 d = acc[u][t];
                const uint32_t col = (uint32_t)((16 * t + 4 * q) * ES);
                if constexpr (SPLIT) {
#pragma unroll
                    for (int i = 0; i < 4; ++i) d[i] = add_row_ror8(d[i]) * sc;
                    if (p < 8) *(__attribute__((address_space(3))) f4 *)(ob + (u * RU + p) * RSTRIDE + col) = d;
                } else {
                    if (U16 || p < 8)
                        *(lds_u2 *)(ob + (u * RU + p) * RSTRIDE + col) =
                            u32x2{pack_h2((_Float16)d[0], (_Float16)d[1]), pack_h2((_Float16)d[2], (_Float16)d[3])};
                }
            }
        }
        const int orow = lane / LPR, ocol = lane % LPR;
        const int tok = tb + ocol * (16 / ES);
        // a wave whose rows and tokens are all inside Y stores without a guard per
        // row, so that the compiler may overlap the rows' LDS reads
        const bool whole = row_w + G::rows_wave <= M && tb + kXTok <= N;
        auto store_rows = [&](auto guarded) __attribute__((always_inline)) {
#pragma unroll
        for (int r0 = 0; r0 < G::rows_wave; r0 += RPI) {
            const int r = r0 + orow;
            f4 v = *(__attribute__((address_space(3))) f4 *)(ob + r * RSTRIDE + ocol * 16);
            const int row = row_w + r;
            if (!decltype(guarded)::value || (row < M && tok < N)) {
                if constexpr (GELU_OK) {
                    if (gelu) {
                        typedef __attribute__((address_space(3))) const uint16_t lds_u16;
                        typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
                        const u32x4 a = __builtin_bit_cast(u32x4, v);  // 8 binary16, two per word
                        u32x4 o = {0u, 0u, 0u, 0u};
                        lds_u16 *const tab0 = (lds_u16 *)(lds_char *)xs0;
                        lds_u16 *const tab1 = (lds_u16 *)(lds_char *)xs1;
                        // branch-free: one LDS read per element, at an in-bounds
                        // entry of the sign's table (all 8 issued before any is
                        // used), then the rule where the table has no entry
                        uint32_t bb[8], lim[8], tv[8];
#pragma unroll
                        for (int i = 0; i < 8; ++i) {
                            bb[i] = (a[i >> 1] >> (16 * (i & 1))) & 0xffffu;
                            lim[i] = (bb[i] >> 15) ? (uint32_t)(NMG_GELU_F16_NEGZERO_FROM - 0x8001)
                                                   : (uint32_t)(NMG_GELU_F16_IDENTITY_FROM - 1);
                            tv[i] = ((bb[i] >> 15) ? tab1 : tab0)[min(bb[i] & 0x7fffu, lim[i])];
                        }
#pragma unroll
                        for (int i = 0; i < 8; ++i) {
                            const uint32_t b = bb[i];
                            const uint32_t rule = b <= 0x7c00u ? b
                                                  : (b - 0x8000u) < 0x7c00u ? 0x8000u
                                                                           : (uint32_t)NMG_GELU_F16_NAN_OUT;
                            o[i >> 1] |= ((b & 0x7fffu) <= lim[i] ? tv[i] : rule) << (16 * (i & 1));
                        }
                        v = __builtin_bit_cast(f4, o);
                    }
                }
                if (R_ != nullptr) {
                    const f4 rv = *reinterpret_cast<const f4 *>(reinterpret_cast<const char *>(R_) +
                                                                ((int64_t)row * ldr + tok) * ES);
                    if constexpr (SPLIT) {
                        v = v + rv;
                    } else {
                        const h8 a = __builtin_bit_cast(h8, v), b = __builtin_bit_cast(h8, rv);
                        h8 o;
#pragma unroll
                        for (int i = 0; i < 8; ++i) o[i] = (_Float16)((float)a[i] + (float)b[i]);
                        v = __builtin_bit_cast(f4, o);
                    }
                }
                store_y(v, reinterpret_cast<f4 *>(reinterpret_cast<char *>(Y_) + ((int64_t)row * ldy + tok) * ES));
            }
        }
        };
        if (whole) store_rows(std::false_type{});
        else store_rows(std::true_type{});
    };

    // ---- the pipeline.  HALF: operands and X copies DP windows ahead (DP +
    // 1 buffers); at the end of window w the copies of w + 1 must have
    // landed, and after them this wave issued only the operand loads (2 GW)
    // and the copies (NSTG) of windows w + 2 .. w + DP: it waits until at
    // most that many are outstanding.  SPLIT: operands and X one window
    // ahead (X through registers, split and written after the products).
    constexpr int DIST = SPLIT ? 1 : DP;    // windows ahead
    static_assert(SPLIT ? DP == 1 : (DP == 2 || DP == 3), "pipeline depth");
    constexpr int NOPS = DIST + 1;          // operand sets in rotation
    char *const bufs[4] = {xs0, xs1, xs2, xs3};
    Ops ops[NOPS];
    uint32_t aa[2][GW][2];
    if constexpr (SPLIT) {
        load_ops(0, ops[0]);
        stage_issue(0, xs0);
        stage_write(xs0);
        wait_all_memory();
        addresses(ops[0], aa[0]);
        __syncthreads();
    } else {
        // window by window, operands then copies; window 0 starts once its
        // own copies have landed (the count at a window's end: the (DIST -
        // 1) (2 GW + NSTG) loads of windows 1 .. DIST - 1 may stay in
        // flight); step 0 makes window 1's addresses
        static_for<DIST>([&](auto dc) {
            load_ops(decltype(dc)::value, ops[decltype(dc)::value]);
            stage_issue(decltype(dc)::value, bufs[decltype(dc)::value]);
        });
        addresses(ops[0], aa[0]);
        window_barrier<(DIST - 1) * (2 * GW + NSTG)>();
    }
    // step w (W6 = w % PERIOD, so that operand sets, address sets and buffers
    // rotate statically): window w from bufs[W6 % NBUF]
    constexpr int PERIOD = NOPS == 4 ? 4 : 6;  // a multiple of NOPS, NBUF and 2
    auto step = [&](int w, auto w6c) __attribute__((always_inline)) {
        constexpr int W6 = decltype(w6c)::value;
        Ops &cur = ops[W6 % NOPS];
        Ops &nxt = ops[(W6 + 1) % NOPS];
        Ops &tgt = ops[(W6 + DIST) % NOPS];
        uint32_t (&ac)[GW][2] = aa[W6 % 2];
        uint32_t (&an)[GW][2] = aa[(W6 + 1) % 2];
        // jobs: the copies (or X loads) of window w + DIST first, then its
        // operands (so that at the window's end the copies of w + 1 are
        // followed by exactly the window's own 2 GW + NSTG loads or more)
        char *sbuf = bufs[(W6 + DIST) % NBUF];
        const int ws = min(w + DIST, nstep - 1);
        compute(
            bufs[W6 % NBUF], cur, ac,
            [&](auto jc) __attribute__((always_inline)) {
                constexpr int j = decltype(jc)::value;
                if constexpr (j < NSTG) stage_one(ws, sbuf, std::integral_constant<int, j>{});
                else load_one(w + DIST, tgt, std::integral_constant<int, j - NSTG>{});
            },
            [&](auto kc) __attribute__((always_inline)) { stage_write_one(sbuf, kc); });
        if constexpr (SPLIT) {
            addresses(nxt, an);
            window_barrier<2 * GW>();  // operand loads of w + 1 may stay in flight
        } else {
            addresses(nxt, an);
            if constexpr (TPW > 1 && W6 < DIST - 1) {
                // the first steps after a tile's outputs: its NST stores,
                // issued after the copies of window w + 1, may stay in flight
                if (after_out) window_barrier<(DIST - 1) * (2 * GW + NSTG) + NST>();
                else window_barrier<(DIST - 1) * (2 * GW + NSTG)>();
            } else {
                window_barrier<(DIST - 1) * (2 * GW + NSTG)>();
            }
        }
    };
    static_assert(PERIOD % NOPS == 0 && PERIOD % NBUF == 0 && PERIOD % 2 == 0, "static rotation");
    if constexpr (TPW > 1) {
        // nwin % PERIOD == 0 (host): every tile ends a block of PERIOD steps
        for (int w = 0; w < nstep; w += PERIOD) {
            static_for<PERIOD>([&](auto kc) { step(w + decltype(kc)::value, kc); });
            after_out = false;
            if (w + PERIOD < nstep && (w + PERIOD) % nwin == 0) {
                // a tile's outputs through the buffer of its last window (the
                // step's barrier: every wave is done with it) while the next
                // tile's first windows are in flight into the other buffers
                tile_out((lds_char *)bufs[(PERIOD - 1) % NBUF] + wave * RB,
                         t0 + ((w + PERIOD) / nwin - 1) * kXTok, false);
                lds_barrier();  // every region read back: the buffer takes copies again
#pragma unroll
                for (int u = 0; u < GW; ++u)
#pragma unroll
                    for (int t = 0; t < kXTiles; ++t) acc[u][t] = f4{0.f, 0.f, 0.f, 0.f};
                after_out = true;
            }
        }
    } else {
        int w = 0;
        for (; w + PERIOD <= nwin; w += PERIOD)
            static_for<PERIOD>([&](auto kc) { step(w + decltype(kc)::value, kc); });
        static_for<PERIOD - 1>([&](auto kc) {
            if (w + decltype(kc)::value < nwin) step(w + decltype(kc)::value, kc);
        });
    }

    // ---- the outputs of the last tile (all staging buffers free)
    constexpr int WPA = BUFCAP / RB;                 // regions per staging buffer
    static_assert(WPA >= 1 && WPA * NBUF >= NW, "output regions fit the staging buffers");
    const bool gelu = GELU_OK && epi == NMG_EPILOGUE_GELU;  // the host asks only when it fits
    // the GELU table's non-rule entries, 16 bytes a thread and step, all loads
    // in flight together before the barrier (the buffers are free after it)
    constexpr int TPB = 64 * NW;
    constexpr int NTP = kGeluPosBytes / 16, NTN = kGeluNegBytes / 16;
    constexpr int IP = GELU_OK ? (NTP + TPB - 1) / TPB : 1, IN = GELU_OK ? (NTN + TPB - 1) / TPB : 1;
    f4 tabp[IP], tabn[IN];
    if constexpr (GELU_OK) {
        if (gelu) {
            const f4 *src = reinterpret_cast<const f4 *>(g_x16_gelu);
#pragma unroll
            for (int j = 0; j < IP; ++j)
                tabp[j] = src[min((int)threadIdx.x + j * TPB, NTP - 1)];
#pragma unroll
            for (int j = 0; j < IN; ++j)
                tabn[j] = src[0x8000 * 2 / 16 + min((int)threadIdx.x + j * TPB, NTN - 1)];
        }
    }
    window_barrier<0>();  // copies for windows past the last have landed; every wave is done
    const int oreg = wave / WPA;
    lds_char *ob = (lds_char *)(oreg == 0 ? xs0 : (NBUF == 2 || oreg == 1) ? xs1 : (NBUF == 3 || oreg == 2) ? xs2 : xs3) +
                   (wave % WPA) * RB;
    if constexpr (GELU_OK) {
        if (gelu) {
            // into buffers 0 (non-negative inputs) and 1 (negative ones)
            typedef __attribute__((address_space(3))) f4 lds_f4;
#pragma unroll
            for (int j = 0; j < IP; ++j)
                if ((int)threadIdx.x + j * TPB < NTP)
                    ((lds_f4 *)(lds_char *)xs0)[threadIdx.x + j * TPB] = tabp[j];
#pragma unroll
            for (int j = 0; j < IN; ++j)
                if ((int)threadIdx.x + j * TPB < NTN)
                    ((lds_f4 *)(lds_char *)xs1)[threadIdx.x + j * TPB] = tabn[j];
            window_barrier<0>();  // every wave's table writes are done
            constexpr int W2 = BUFCAP / RB, W3 = NBUF >= 4 ? BUFCAP / RB : 0;
            constexpr int W0 = (BUFCAP - kGeluPosBytes) / RB;
            ob = wave < W2 ? (lds_char *)xs2 + wave * RB
                 : wave < W2 + W3 ? (lds_char *)xs3 + (wave - W2) * RB
                 : wave < W2 + W3 + W0 ? (lds_char *)xs0 + kGeluPosBytes + (wave - W2 - W3) * RB
                                       : (lds_char *)xs1 + kGeluNegBytes + (wave - W2 - W3 - W0) * RB;
        }
    }
    tile_out(ob, t0 + (ntile - 1) * kXTok, gelu);
}

}  // namespace

// ---------------------------------------------------------------- launchers

namespace {

// waves per workgroup (one workgroup per CU): 8, two per SIMD; binary16 also
// 6, for layers whose 8-wave tiles would leave CUs idle
template <bool SPLIT> constexpr int x16_waves() { return 8; }

// rows per unit of the prepared operands
inline int x16_unit_rows(const nmg_layout *L) {
    return L->dtype == NMG_F32 ? 8 : (L->g % 16 == 0 ? 16 : 8);
}

// staging items per lane (SPLIT) / copy instructions per wave (HALF) and
// window, for workgroups of `nw` waves
inline int x16_nstg(const nmg_layout *L, int nw) {
    const bool split = L->dtype == NMG_F32;
    const int rw = (kXSlots / L->n) * L->m;
    if (split) {
        const int lanes = 64 * nw;
        return (rw * (kXTok / 4) + lanes - 1) / lanes;
    }
    const int inst = rw * (kXTok / 8) / 64;
    return (inst + nw - 1) / nw;
}

}  // namespace

bool nmg_internal::x16_layout_supported(const nmg_layout *L) {
    const bool split = L->dtype == NMG_F32;
    const int64_t ldv = (int64_t)L->C * L->n;
    if (L->n != 1 && L->n != 2) return false;
    if (L->g % 8 != 0) return false;
    if (!split && L->m % 4 != 0) return false;          // whole-wave LDS copies of 4 rows
    const int rowb = split ? 512 : 256;
    if (x16_buffer_bytes(L->n, L->m, rowb) > (split ? x16_buf_cap<true, 1>() : x16_buf_cap<false, 2>()))
        return false;
    if (x16_nstg(L, x16_waves<false>()) > 8) return false;
    return (int64_t)L->M * ldv < ((int64_t)1 << 31);
}

int64_t nmg_internal::x16_prepared_bytes(const nmg_layout *L) {
    if (!x16_layout_supported(L)) return -1;
    return (int64_t)x16_prep_layout(L, x16_unit_rows(L)).bytes;
}

bool nmg_internal::x16_args_supported(const nmg_layout *L, const void *X, int64_t ldx,
                                      const void *Y, int64_t ldy, int64_t N) {
    const bool split = L->dtype == NMG_F32;
    const size_t es = split ? 4 : 2;
    // X rows on 16-byte boundaries; Y rows on 16 (binary32) / 8 (binary16)
    const bool xa = X == nullptr || aligned(X, 16);
    const bool ya = Y == nullptr || aligned(Y, split ? 16 : 8);
    return x16_layout_supported(L) && xa && ya && ldx % (16 / es) == 0 && ldy % 4 == 0 &&
           N % (split ? 4 : 8) == 0 && (int64_t)L->K * ldx < ((int64_t)1 << 31);
}

namespace {

template <bool SPLIT, int NS, int RU>
nmg_status launch_prepare_k(const nmg_layout *L, const void *values, const uint8_t *indices,
                            void *prepared, hipStream_t stream) {
    const XPrep P = x16_prep_layout(L, RU);
    char *base = static_cast<char *>(prepared);
    hipLaunchKernelGGL((k_x16_prepare<SPLIT, NS, RU>), dim3(P.units), dim3(64), 0, stream, values,
                       indices, reinterpret_cast<h8 *>(base + P.frag),
                       reinterpret_cast<uint16_t *>(base + P.offs),
                       reinterpret_cast<int8_t *>(base + P.scale), L->M, L->m, L->g, L->C, P.nwin);
    return launched();
}

struct X16Out {
    void *Y;
    int64_t ldy;
    int epi;
    const void *R;
    int64_t ldr;
};

template <bool SPLIT, int NS, bool U16, int GW, int NW, int NSTG, int DP, int TPW = 1>
nmg_status launch_x16_k(const nmg_layout *L, const void *prepared, const void *X, int64_t ldx,
                        int N, const X16Out &o, hipStream_t stream) {
    using G = XGeom<SPLIT, U16, GW, NW>;
    // GELU only where its table and the outputs share the staging buffers
    if (o.epi == NMG_EPILOGUE_GELU &&
        !x16_gelu_fits(SPLIT, G::rows_wave, NW, x16_buf_cap<SPLIT, DP>(), x16_nbuf<SPLIT, DP>()))
        return NMG_ERR_UNSUPPORTED;
    const XPrep P = x16_prep_layout(L, G::rows_unit);
    const char *base = static_cast<const char *>(prepared);
    const int row_blocks = (L->M + G::rows_wg - 1) / G::rows_wg;
    const int grid = row_blocks * (((N + kXTok - 1) / kXTok + TPW - 1) / TPW);
    const h8 *fr = reinterpret_cast<const h8 *>(base + P.frag);
    const uint16_t *of = reinterpret_cast<const uint16_t *>(base + P.offs);
    const int8_t *sc = reinterpret_cast<const int8_t *>(base + P.scale);
    hipLaunchKernelGGL((k_spmm_x16<SPLIT, NS, U16, GW, NW, NSTG, DP, TPW>), dim3(grid), dim3(64 * NW), 0,
                       stream, fr, of, sc, X, ldx, o.Y, o.ldy,
                       o.epi == NMG_EPILOGUE_ADD ? o.R : nullptr, o.ldr, o.epi, L->M, L->K, N,
                       L->m, P.nwin, row_blocks);
    return launched();
}

// The staging job counts the supported layouts have (x16_nstg, rounded up to
// the instantiated 2, 4, 6, 8): binary16 windows of 32 m / n rows take m / n
// jobs (m = 4 at n = 1; 4, 8, 12 at n = 2), binary32 ones 2 m / n (m = 1..4 at
// n = 1, 2..8 at n = 2)
// With 6-wave workgroups (binary16, 2 units a wave, m <= 8): 3 to 6 jobs.
template <bool SPLIT, int NS, int NW>
constexpr bool x16_nstg_used(int s) {
    if constexpr (SPLIT) return s >= 2;
    if constexpr (NW == 6) return s == 4 || s == 6;
    return NS == 1 ? s == 4 : (s >= 2 && s <= 6);
}

// The pipeline depth of each instantiation: binary16 6-wave workgroups (the
// single-round layers, whose windows all fit 40 KB) copy three windows
// ahead, 8-wave ones two; binary32 one.  Measured on the BERT stack: FFN
// down (24 windows, 6-wave) 22.6 -> 20.6 us at depth 3; at depth 3 the
// 8-wave layers of 6 windows were 0.7 us slower (QKV, FFN up).
template <bool SPLIT, int NS, int NW, int NSTG>
constexpr int x16_dp_of() {
    if constexpr (SPLIT) return 1;
    return NW == 6 ? 3 : 2;
}

// Two token tiles per workgroup (binary16 workgroups of 3 units of 8 rows a
// wave, whose outputs fit one staging buffer; no GELU): when one tile a workgroup would take more than one round of
// workgroups and two tiles a workgroup take one, and every tile's windows end
// a block of the pipeline's static rotation (6 steps at two windows ahead).
// The workgroup's window pipeline then runs on into its second tile while
// the first tile's outputs drain.
template <bool SPLIT, bool U16, int GW, int NW>
constexpr bool x16_two_tile_shape() {
    return !SPLIT && !U16 && GW == 3 && (NW == 8 || NW == 6);
}
inline bool x16_two_tiles(const nmg_layout *L, int64_t N, int rows_wg, int wbytes, int epi) {
    const int nwin = (L->C * L->n + kXSlots - 1) / kXSlots;
    const int64_t tt = (N + kXTok - 1) / kXTok;
    const int64_t rbs = (L->M + rows_wg - 1) / rows_wg;
    const int64_t cus = device_cus();
    return epi != NMG_EPILOGUE_GELU && nwin % 6 == 0 && wbytes <= x16_buf_cap<false, 2>() &&
           rbs * tt > cus && rbs * ((tt + 1) / 2) <= cus;
}

template <bool SPLIT, int NS, bool U16, int GW, int NW = x16_waves<SPLIT>()>
nmg_status launch_x16_s(const nmg_layout *L, const void *prepared, const void *X, int64_t ldx,
                        int N, const X16Out &Y, hipStream_t stream) {
    const int s = x16_nstg(L, NW);
    const int r = s <= 2 ? 2 : s <= 4 ? 4 : s <= 6 ? 6 : 8;
    // a window must fit the buffers of the instantiation's depth
    const int wbytes = x16_buffer_bytes(L->n, L->m, SPLIT ? 512 : 256);
    const bool two = x16_two_tile_shape<SPLIT, U16, GW, NW>() &&
                     x16_two_tiles(L, N, XGeom<SPLIT, U16, GW, NW>::rows_wg, wbytes, Y.epi);
#define X16_CASE(V)                                                                                \
    case V:                                                                                        \
        if constexpr (x16_nstg_used<SPLIT, NS, NW>(V)) {                                           \
            if constexpr (x16_two_tile_shape<SPLIT, U16, GW, NW>()) {                              \
                if (two)                                                                           \
                    return launch_x16_k<SPLIT, NS, U16, GW, NW, V, 2, 2>(L, prepared, X, ldx, N,   \
                                                                         Y, stream);               \
            }                                                                                      \
            constexpr int DPV = x16_dp_of<SPLIT, NS, NW, V>();                                     \
            if (wbytes <= x16_buf_cap<SPLIT, DPV>())                                               \
                return launch_x16_k<SPLIT, NS, U16, GW, NW, V, DPV>(L, prepared, X, ldx, N, Y,     \
                                                                    stream);                       \
        }                                                                                          \
        break;
    switch (r) {
        X16_CASE(2)
        X16_CASE(4)
        X16_CASE(6)
        X16_CASE(8)
        default: break;
    }
#undef X16_CASE
    return NMG_ERR_UNSUPPORTED;
}

// Units per wave.  More rows per workgroup share each staged X window (fewer
// bytes through the CU's load path per instruction); fewer rows give more
// workgroups.  Priced as rounds of workgroups (one per CU) times the rows of
// one plus a fixed share for staging its X; binary32 at most 2 units (its
// registers also hold the X being split), binary16 up to 3.
// 6-wave binary16 workgroups when the window's copies split into at most 6
// per wave (m / n <= 4 at 2 units a wave), the candidate the cost below may
// take for layers whose 8-wave tiles leave CUs idle
inline bool x16_six_ok(const nmg_layout *L) {
    const int s = x16_nstg(L, 6);
    return L->dtype == NMG_F16 && s > 2 && s <= 6;
}

// Waves and units per wave.  More rows per workgroup share each staged X
// window (fewer bytes through the CU's load path per instruction); fewer rows
// give more workgroups.  Priced as rounds of workgroups (one per CU) times
// the rows of one plus a fixed share for staging its X; binary32 at most 2
// units (its registers also hold the X being split), binary16 up to 3, also
// in 6-wave workgroups (2 or 3 units) when the window's copies split into at
// most 6 per wave.  Returns 10 * waves + units.
template <bool SPLIT, bool U16>
int x16_shape(const nmg_layout *L, int64_t N) {
    constexpr int ru = SPLIT ? 8 : (U16 ? 16 : 8);
    const int cands[5][2] = {{8, 3}, {8, 2}, {8, 1}, {6, 3}, {6, 2}};
    const int64_t cus = device_cus();
    const int64_t tt = (N + kXTok - 1) / kXTok;
    int best = 81;
    int64_t best_cost = -1;
    for (const auto &c : cands) {
        const int nw = c[0], gw = c[1];
        if (SPLIT && (gw > 2 || nw != 8)) continue;
        if (nw == 6 && !x16_six_ok(L)) continue;
        const int64_t rows = (int64_t)nw * gw * ru;
        const int64_t wgs = (L->M + rows - 1) / rows * tt;
        const int64_t cost = (wgs + cus - 1) / cus * (rows + 64);
        if (best_cost < 0 || cost < best_cost) {
            best_cost = cost;
            best = 10 * nw + gw;
        }
    }
    return best;
}

template <bool SPLIT, int NS, bool U16>
nmg_status launch_x16_g(const nmg_layout *L, const void *prepared, const void *X, int64_t ldx,
                        int N, const X16Out &Y, hipStream_t stream) {
    switch (x16_shape<SPLIT, U16>(L, N)) {
        case 83:
            if constexpr (!SPLIT) return launch_x16_s<SPLIT, NS, U16, 3>(L, prepared, X, ldx, N, Y, stream);
            return NMG_ERR_UNSUPPORTED;
        case 82: return launch_x16_s<SPLIT, NS, U16, 2>(L, prepared, X, ldx, N, Y, stream);
        case 63:
            if constexpr (!SPLIT) return launch_x16_s<SPLIT, NS, U16, 3, 6>(L, prepared, X, ldx, N, Y, stream);
            return NMG_ERR_UNSUPPORTED;
        case 62:
            if constexpr (!SPLIT) return launch_x16_s<SPLIT, NS, U16, 2, 6>(L, prepared, X, ldx, N, Y, stream);
            return NMG_ERR_UNSUPPORTED;
        default: return launch_x16_s<SPLIT, NS, U16, 1>(L, prepared, X, ldx, N, Y, stream);
    }
}

}  // namespace

nmg_status nmg_internal::x16_prepare(const nmg_layout *L, const void *values, const uint8_t *indices,
                                     void *prepared, hipStream_t stream) {
    const bool split = L->dtype == NMG_F32;
    const int ru = x16_unit_rows(L);
    if (split) return L->n == 1 ? launch_prepare_k<true, 1, 8>(L, values, indices, prepared, stream)
                                : launch_prepare_k<true, 2, 8>(L, values, indices, prepared, stream);
    if (ru == 16) return L->n == 1 ? launch_prepare_k<false, 1, 16>(L, values, indices, prepared, stream)
                                   : launch_prepare_k<false, 2, 16>(L, values, indices, prepared, stream);
    return L->n == 1 ? launch_prepare_k<false, 1, 8>(L, values, indices, prepared, stream)
                     : launch_prepare_k<false, 2, 8>(L, values, indices, prepared, stream);
}

nmg_status nmg_internal::x16_product(const nmg_layout *L, const void *prepared, const void *X,
                                     int64_t ldx, int N, void *Yp, int64_t ldy, int epi,
                                     const void *R, int64_t ldr, hipStream_t stream) {
    const X16Out Y{Yp, ldy, epi, R, ldr};
    if (L->dtype == NMG_F32)
        return L->n == 1 ? launch_x16_g<true, 1, false>(L, prepared, X, ldx, N, Y, stream)
                         : launch_x16_g<true, 2, false>(L, prepared, X, ldx, N, Y, stream);
    const bool u16 = L->g % 16 == 0;
    if (L->n == 1) return u16 ? launch_x16_g<false, 1, true>(L, prepared, X, ldx, N, Y, stream)
                              : launch_x16_g<false, 1, false>(L, prepared, X, ldx, N, Y, stream);
    return u16 ? launch_x16_g<false, 2, true>(L, prepared, X, ldx, N, Y, stream)
               : launch_x16_g<false, 2, false>(L, prepared, X, ldx, N, Y, stream);
}
