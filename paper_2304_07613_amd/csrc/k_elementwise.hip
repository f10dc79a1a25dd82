// k_elementwise.hip -- dense -> n:m:g (Section 5.2) and n:m:g -> dense.
//
//   k_compress_chunk  one thread per (group, chunk) for chunks of at most 32
//               columns: the group scores of the chunk in registers (vector
//               loads when the chunk starts on 16 bytes), ranked in
//               registers; W is read once, every access coalesced across the
//               wave.  HBM-bound.
//   k_compress  one thread per column of a chunk-block (wide chunks, or few
//               (group, chunk) pairs): binary32 group score down the g rows,
//               rank by counting inside the chunk through LDS, then a
//               coalesced copy of the kept weights.
//   k_densify   one thread per output element (k_densify_chunks: one per
//               chunk, for chunks of 4 or 8 columns).
//   k_repack    one thread per kept slot: values from W at given indices.
#include "common.hpp"

namespace {

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
        int i = 0;
        for (; i + 8 <= g; i += 8) {   // the loads of 8 rows in flight, added in row order
            float v[8];
#pragma unroll
            for (int b = 0; b < 8; ++b) v[b] = (float)p[(int64_t)(i + b) * ldw];
#pragma unroll
            for (int b = 0; b < 8; ++b) s = s + fabsf(v[b]);
        }
        for (; i < g; ++i) s = s + fabsf((float)p[(int64_t)i * ldw]);
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

    // copy the kept weights of the g rows, bit for bit, coalesced on output;
    // 8 rows' loads in flight before their stores
    const int nout = min(cpb, C - c_first) * n;
    const B *Wb = reinterpret_cast<const B *>(W);
    B *Vb = reinterpret_cast<B *>(values);
    for (int p = t; p < nout; p += kBlock) {
        const int64_t col = (int64_t)(c_first + p / n) * m + sel[p];
        const int64_t out = (int64_t)c_first * n + p;
        int i = 0;
        for (; i + 8 <= g; i += 8) {
            B v[8];
#pragma unroll
            for (int b = 0; b < 8; ++b) v[b] = Wb[(row0 + i + b) * ldw + col];
#pragma unroll
            for (int b = 0; b < 8; ++b) Vb[(row0 + i + b) * ldv + out] = v[b];
        }
        for (; i < g; ++i) Vb[(row0 + i) * ldv + out] = Wb[(row0 + i) * ldw + col];
    }
}

// --------------------------------------------------- compress, thread per chunk

// For m <= MT (MT = 4, 8, 16 or 32): one thread owns one (group, chunk).  It
// reads the chunk's m columns down the g rows (16-byte vector loads when rows
// and chunks are whole vectors, 4 rows in flight at a time), sums
// the scores in binary32 in row order, selects the n largest in registers
// (the same order as k_compress: key bits, ties to the lower offset; n passes
// of the first maximum for n <= 4, counted ranks otherwise), and writes the
// indices and the kept weights of the g rows.  Adjacent threads own adjacent
// chunks (a row's last chunk is followed by the next group's first), so the
// loads and stores are coalesced across the wave, and W is read exactly once.
template <typename T, int MT>
__global__ __launch_bounds__(kBlock) void k_compress_chunk(
    const T *__restrict__ W, int64_t ldw, T *__restrict__ values,
    uint8_t *__restrict__ indices, int K, int n, int m, int g, int C, bool vec,
    uint32_t pairs) {
    using B = typename Bits<T>::type;
    constexpr int VB = 16 / sizeof(T);            // elements per 16-byte vector
    // pairs > 0: the (group, chunk) pairs are numbered group-major across the
    // whole grid, so every thread owns a chunk however few chunks a row has;
    // pairs == 0 (more pairs than 31 bits hold): a row of groups per grid row
    int G, c;
    if (pairs) {
        const uint32_t p = blockIdx.x * kBlock + threadIdx.x;
        if (p >= pairs) return;
        G = (int)(p / (uint32_t)C);
        c = (int)(p - (uint32_t)G * (uint32_t)C);
    } else {
        G = blockIdx.x;
        c = blockIdx.y * kBlock + threadIdx.x;
        if (c >= C) return;
    }
    const int w = min(m, K - c * m);              // chunk width
    const int64_t ldv = (int64_t)C * n;
    const int64_t row0 = (int64_t)G * g;
    const int64_t col0 = (int64_t)c * m;

    float score[MT];
#pragma unroll
    for (int j = 0; j < MT; ++j) score[j] = 0.0f;
    typedef B BV __attribute__((ext_vector_type(VB)));
    constexpr int NV = MT / VB + (MT % VB != 0);
    // Small groups (g <= RROWS rows of whole 16-byte vectors): every row's
    // chunk is loaded at once and kept in registers, and the kept weights are
    // picked from there -- one round trip to memory.  The pick is an unrolled
    // select over MT offsets per kept slot and row, so RROWS keeps it near
    // 1024 selects (none for MT = 32): larger kernels outgrow the instruction
    // cache and ran 3x slower.
    // With vec, every chunk (the last one too) is whole 16-byte vectors: a
    // vector past a short last chunk's end is loaded from its last vector
    // instead (in bounds), and the scores of columns j >= w are never keys.
    constexpr int RMAX = 16;
    constexpr int RROWS = MT > 16 ? 0 : (RMAX / NV < 1024 / (MT * MT) ? RMAX / NV : 1024 / (MT * MT));
    const bool in_regs = RROWS > 0 && vec && g <= RROWS;
    BV rr[RROWS * NV + (RROWS == 0)];
    if (in_regs) {
#pragma unroll
        for (int q = 0; q < RROWS * NV; ++q) {
            const int i = q / NV, v = q % NV;
            if (i < g && v * VB < m)
                rr[q] = *reinterpret_cast<const BV *>(W + (row0 + i) * ldw + col0 + min(v * VB, w - VB));
        }
#pragma unroll
        for (int q = 0; q < RROWS * NV; ++q) {   // rows in ascending order
            const int i = q / NV, v = q % NV;
            if (i < g && v * VB < m)
#pragma unroll
                for (int e = 0; e < VB; ++e) {
                    const int j = v * VB + e;
                    if (j < MT) score[j] = score[j] + fabsf((float)__builtin_bit_cast(T, (B)rr[q][e]));
                }
        }
        // every row has landed (the scores needed them): said explicitly, so
        // that the stores below are not each preceded by a wait for memory
        wait_all_memory();
    } else if (vec) {
        // Rows come in batches (the loads of a batch in flight together),
        // added in row order.
        auto load_row = [&](int i, BV (&r)[NV]) {
            const T *p = W + (row0 + i) * ldw + col0;
#pragma unroll
            for (int v = 0; v < NV; ++v)
                if (v * VB < m) r[v] = *reinterpret_cast<const BV *>(p + min(v * VB, w - VB));
        };
        auto add_row = [&](const BV (&r)[NV]) {
#pragma unroll
            for (int v = 0; v < NV; ++v)
                if (v * VB < m)
#pragma unroll
                    for (int e = 0; e < VB; ++e) {
                        const int j = v * VB + e;
                        if (j < MT) score[j] = score[j] + fabsf((float)__builtin_bit_cast(T, (B)r[v][e]));
                    }
        };
        // up to 4 rows per batch (16 vectors at most): their loads in flight
        // together
        constexpr int RB = RMAX / NV < 4 ? RMAX / NV : 4;
        int i = 0;
        for (; i + RB <= g; i += RB) {
            BV r[RB][NV];
#pragma unroll
            for (int b = 0; b < RB; ++b) load_row(i + b, r[b]);
#pragma unroll
            for (int b = 0; b < RB; ++b) add_row(r[b]);
        }
        for (; i < g; ++i) {
            BV r0[NV];
            load_row(i, r0);
            add_row(r0);
        }
    } else {
        // element loads, all MT of a row in flight: a column past the chunk's
        // end is loaded from its last column (in bounds) and never becomes a key
        for (int i = 0; i < g; ++i) {
            const T *p = W + (row0 + i) * ldw + col0;
            T e[MT];
#pragma unroll
            for (int j = 0; j < MT; ++j) e[j] = p[min(j, w - 1)];
#pragma unroll
            for (int j = 0; j < MT; ++j) score[j] = score[j] + fabsf((float)e[j]);
        }
    }
    // order keys: non-negative floats order like their bits; NaN above +inf
    uint32_t key[MT];
#pragma unroll
    for (int j = 0; j < MT; ++j)
        key[j] = j < w ? (__builtin_isnan(score[j]) ? 0x7fc00000u : __float_as_uint(score[j])) : 0u;
    // the kept columns as a bit mask
    uint32_t taken = 0;
    if (n <= 4) {
        // n passes of "first maximum among the columns not taken yet" select
        // the same set as ranking (higher score first, ties to the lower
        // offset)
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            if (t >= n) break;
            int best = -1;
            uint32_t bk = 0;
#pragma unroll
            for (int j = 0; j < MT; ++j) {
                const bool cand = j < w && !((taken >> j) & 1u);
                if (cand && (best < 0 || key[j] > bk)) {
                    best = j;
                    bk = key[j];
                }
            }
            taken |= 1u << best;
        }
    } else {
#pragma unroll
        for (int j = 0; j < MT; ++j) {
            if (j < w) {
                int rank = 0;
#pragma unroll
                for (int i = 0; i < MT; ++i)
                    if (i < w) rank += (key[i] > key[j]) || (i < j && key[i] == key[j]);
                if (rank < n) taken |= 1u << j;
            }
        }
    }
    // the kept offsets in ascending order, then the kept weights of every row
    uint8_t *ip = indices + (int64_t)G * ldv + (int64_t)c * n;
    uint32_t t = taken;
    for (int s = 0; s < n; ++s) {
        ip[s] = (uint8_t)__builtin_ctz(t);
        t &= t - 1;
    }
    if (in_regs) {
        // the kept offsets in ascending order (slots s < n), then every row's
        // stores from straight-line code, so that they issue back to back
        int js[MT];
        uint32_t u = taken;
#pragma unroll
        for (int s = 0; s < MT; ++s) {
            js[s] = u ? __builtin_ctz(u) : 0;
            u &= u - 1;
        }
#pragma unroll
        for (int i = 0; i < RROWS; ++i) {
            if (i >= g) continue;
            B *dst = reinterpret_cast<B *>(values + (row0 + i) * ldv) + (int64_t)c * n;
#pragma unroll
            for (int s = 0; s < MT; ++s) {
                if (s >= n) continue;
                B x = 0;
#pragma unroll
                for (int jj = 0; jj < MT; ++jj)
                    if (jj == js[s]) x = (B)rr[i * NV + jj / VB][jj % VB];
                dst[s] = x;
            }
        }
        return;
    }
    for (int i = 0; i < g; ++i) {
        const B *src = reinterpret_cast<const B *>(W + (row0 + i) * ldw + col0);
        B *dst = reinterpret_cast<B *>(values + (row0 + i) * ldv) + (int64_t)c * n;
        uint32_t u = taken;
        for (int s = 0; s < n; ++s) {
            dst[s] = src[__builtin_ctz(u)];
            u &= u - 1;
        }
    }
}

// ------------------------------------------------------------------ densify

template <typename T>
__global__ __launch_bounds__(kBlock) void k_densify(
    const T *__restrict__ values, const uint8_t *__restrict__ indices,
    T *__restrict__ out, int64_t ldw, int K, int n, int m, int g, int C,
    uint8_t *__restrict__ zeros) {
    using B = typename Bits<T>::type;
    const int64_t r = blockIdx.x;
    const int k = blockIdx.y * kBlock + threadIdx.x;
    if (k >= K) return;
    if (zeros != nullptr && r == 0) zeros[k] = 0;  // the expanded weight's index bytes
    const int c = k / m, o = k - c * m;
    const int64_t ldv = (int64_t)C * n;
    const uint8_t *idx = indices + (r / g) * ldv + (int64_t)c * n;
    B v = 0;
    for (int s = 0; s < n; ++s)
        if (idx[s] == o) v = reinterpret_cast<const B *>(values)[r * ldv + (int64_t)c * n + s];
    reinterpret_cast<B *>(out)[r * ldw + k] = v;
}

// The same for layouts whose chunks are all MV columns wide: one thread per
// (row, chunk) writes the chunk's MV outputs in one vector store (the
// expanded product's densify pass writes M K elements at the store rate)
template <typename T, int MV>
__global__ __launch_bounds__(kBlock) void k_densify_chunks(
    const T *__restrict__ values, const uint8_t *__restrict__ indices,
    T *__restrict__ out, int64_t ldw, int n, int g, int C, uint8_t *__restrict__ zeros) {
    using B = typename Bits<T>::type;
    typedef B VB __attribute__((ext_vector_type(MV)));
    const int64_t r = blockIdx.x;
    const int c = blockIdx.y * kBlock + threadIdx.x;
    if (c >= C) return;
    const int64_t ldv = (int64_t)C * n;
    const uint8_t *idx = indices + (r / g) * ldv + (int64_t)c * n;
    const B *val = reinterpret_cast<const B *>(values) + r * ldv + (int64_t)c * n;
    VB o;
#pragma unroll
    for (int j = 0; j < MV; ++j) o[j] = 0;
    for (int s = 0; s < n; ++s) {  // a later slot with the same offset wins, as in k_densify
        const int off = idx[s];
        const B v = val[s];
#pragma unroll
        for (int j = 0; j < MV; ++j)
            if (off == j) o[j] = v;
    }
    if (zeros != nullptr && r == 0)
#pragma unroll
        for (int j = 0; j < MV; ++j) zeros[(int64_t)c * MV + j] = 0;
    *reinterpret_cast<VB *>(reinterpret_cast<B *>(out) + r * ldw + (int64_t)c * MV) = o;
}

// Fixed-mask repack: one thread per kept slot of a row; the offset is clamped
// into its chunk, so malformed indices never read outside the row.
template <typename T>
__global__ __launch_bounds__(kBlock) void k_repack(
    const T *__restrict__ W, int64_t ldw, const uint8_t *__restrict__ indices,
    T *__restrict__ values, int K, int n, int m, int g, int C) {
    using B = typename Bits<T>::type;
    const int64_t r = blockIdx.x;
    const int64_t ldv = (int64_t)C * n;
    const int j = blockIdx.y * kBlock + threadIdx.x;  // kept slot c * n + s
    if (j >= ldv) return;
    const int c = j / n;
    const int w = min(m, K - c * m);
    const int o = min((int)indices[(r / g) * ldv + j], w - 1);
    reinterpret_cast<B *>(values)[r * ldv + j] =
        reinterpret_cast<const B *>(W)[r * ldw + (int64_t)c * m + o];
}

}  // namespace

namespace nmg_internal {

// whole 16-byte vectors: the rows, every chunk and the last chunk
bool chunk_vec(const nmg_layout *L, const void *W, int64_t ldw) {
    const int64_t es = L->dtype == NMG_F32 ? 4 : 2;
    return aligned(W, 16) && (ldw * es) % 16 == 0 && (L->m * es) % 16 == 0 &&
           (L->K * es) % 16 == 0;
}

template <typename T>
nmg_status launch_compress_chunk(const nmg_layout *L, const void *W, int64_t ldw, void *values,
                                 uint8_t *indices, hipStream_t stream) {
    const bool vec = chunk_vec(L, W, ldw);
    const int64_t pairs = (int64_t)(L->M / L->g) * L->C;
    const bool flat = pairs <= INT32_MAX - kBlock;
    const dim3 grid = flat ? dim3((unsigned)((pairs + kBlock - 1) / kBlock))
                           : dim3(L->M / L->g, (L->C + kBlock - 1) / kBlock);
#define NMG_CHUNK(MT)                                                                          \
    hipLaunchKernelGGL((k_compress_chunk<T, MT>), grid, dim3(kBlock), 0, stream, (const T *)W,   \
                       ldw, (T *)values, indices, L->K, L->n, L->m, L->g, L->C, vec,           \
                       flat ? (uint32_t)pairs : 0u)
    if (L->m <= 4) NMG_CHUNK(4);
    else if (L->m <= 8) NMG_CHUNK(8);
    else if (L->m <= 16) NMG_CHUNK(16);
    else NMG_CHUNK(32);
#undef NMG_CHUNK
    return launched();
}

nmg_status launch_compress(const nmg_layout *L, const void *W, int64_t ldw, void *values,
                           uint8_t *indices, hipStream_t stream) {
    // up to 32 columns per chunk and enough (group, chunk) pairs to fill the
    // GPU: one thread per chunk, in registers; otherwise one thread per column.
    // Groups of at most 4 rows take the thread per chunk from 16K pairs, when
    // its loads are vectors or at most 16 per row (a thread walks its rows in
    // turn, so more rows favour a thread per column).
    const int64_t pairs = (int64_t)(L->M / L->g) * L->C;
    const bool few_rows = L->g <= 4 && pairs >= 16384 && (L->m <= 16 || chunk_vec(L, W, ldw));
    if (L->m <= 32 && (pairs >= 65536 || few_rows))
        return L->dtype == NMG_F32
                   ? launch_compress_chunk<float>(L, W, ldw, values, indices, stream)
                   : launch_compress_chunk<_Float16>(L, W, ldw, values, indices, stream);
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

nmg_status launch_densify(const nmg_layout *L, const void *values, const uint8_t *indices,
                          void *W_out, int64_t ldw, hipStream_t stream, uint8_t *zeros) {
    const int64_t es = (int64_t)elem_size(L->dtype);
    const int64_t vb = L->m * es;  // bytes of one chunk's vector store
    if ((L->m == 4 || L->m == 8) && L->K % L->m == 0 && (vb & (vb - 1)) == 0 &&
        aligned(W_out, (size_t)vb) && (ldw * es) % vb == 0) {
        dim3 grid(L->M, (L->C + kBlock - 1) / kBlock);
#define NMG_DENSIFY_CHUNKS(T, MV)                                                             \
    hipLaunchKernelGGL((k_densify_chunks<T, MV>), grid, dim3(kBlock), 0, stream,             \
                       (const T *)values, indices, (T *)W_out, ldw, L->n, L->g, L->C, zeros)
        if (L->dtype == NMG_F32) {
            if (L->m == 4) NMG_DENSIFY_CHUNKS(float, 4);
            else NMG_DENSIFY_CHUNKS(float, 8);
        } else {
            if (L->m == 4) NMG_DENSIFY_CHUNKS(_Float16, 4);
            else NMG_DENSIFY_CHUNKS(_Float16, 8);
        }
#undef NMG_DENSIFY_CHUNKS
        return launched();
    }
    dim3 grid(L->M, (L->K + kBlock - 1) / kBlock);
    if (L->dtype == NMG_F32)
        hipLaunchKernelGGL((k_densify<float>), grid, dim3(kBlock), 0, stream, (const float *)values,
                           indices, (float *)W_out, ldw, L->K, L->n, L->m, L->g, L->C, zeros);
    else
        hipLaunchKernelGGL((k_densify<_Float16>), grid, dim3(kBlock), 0, stream,
                           (const _Float16 *)values, indices, (_Float16 *)W_out, ldw, L->K, L->n,
                           L->m, L->g, L->C, zeros);
    return launched();
}

nmg_status launch_repack(const nmg_layout *L, const void *W, int64_t ldw, const uint8_t *indices,
                         void *values, hipStream_t stream) {
    const int64_t ldv = (int64_t)L->C * L->n;
    dim3 grid(L->M, (unsigned)((ldv + kBlock - 1) / kBlock));
    if (L->dtype == NMG_F32)
        hipLaunchKernelGGL((k_repack<float>), grid, dim3(kBlock), 0, stream, (const float *)W, ldw,
                           indices, (float *)values, L->K, L->n, L->m, L->g, L->C);
    else
        hipLaunchKernelGGL((k_repack<_Float16>), grid, dim3(kBlock), 0, stream,
                           (const _Float16 *)W, ldw, indices, (_Float16 *)values, L->K, L->n,
                           L->m, L->g, L->C);
    return launched();
}

}  // namespace nmg_internal
