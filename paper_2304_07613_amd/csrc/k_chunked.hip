// k_chunked.hip -- the paper's own chunked n:m:g layout (Section 5): chunks
// of S = C(m,n) * g blocks that use every pattern exactly g times, in
// revolving-door order, with the blocks reordered by pattern and an index of
// their rows; the CPU converter of Section 5.2; the product; the conversion
// back to dense.
//
//   k_p_compress  one workgroup per chunk: the magnitude every pattern keeps
//                 for every row (binary32, the pattern's offsets ascending) in
//                 LDS, then the greedy: S times, the largest pair whose row is
//                 free and whose pattern has room (a workgroup max-reduction
//                 of 64-bit keys: magnitude bits, then lower pattern, then
//                 lower row) -- the same pairs, in the same order, as scanning
//                 the sorted list of all pairs, since a pair that is not
//                 eligible never becomes eligible again.
//   k_p_compress_w the same greedy for chunks of at most 1536 (row, pattern)
//                 pairs: one wave per chunk, each lane holding up to 24 pairs'
//                 keys in registers with a mask of the pairs still eligible;
//                 every step is a wave-wide maximum by shuffles, the pattern
//                 counts live in registers (pattern p with lane p % 64), so a
//                 workgroup of 4 waves converts 4 chunks with 24 KB of LDS.
//   k_p_refine_w  the same swap search for chunks of at most 1536 pairs: one
//                 wave per chunk, each lane owning up to 4 rows, the round's
//                 flag a wave vote.
//   k_p_spmm      vector FMAs: the rows of a group are scattered over the
//                 chunk, so rows share no operands; each wave owns 16 rows of
//                 one chunk and 256 tokens, and finds each row's position in
//                 every block column through an inverse table built in LDS.
//                 When m <= 32 and the chunk has at least 64 rows, the X rows
//                 of a window of block columns are staged in LDS (binary32, 32
//                 rows) and every row reads the rows its pattern selects from
//                 there, instead of gathering them from global memory.
//   k_p_spmm_mfma matrix cores on the expanded blocks: in one block column a
//                 row's block is an m-vector with m - n zeros, and all S rows
//                 of the chunk read the same m rows of X there, so the chunk
//                 times X is a dense contraction over K of which n / m of the
//                 products are useful.  Each workgroup owns 64 rows x 256
//                 tokens; per window of up to 32 k-columns every stored block
//                 writes its expanded m values into a k-major LDS tile at its
//                 chunk row (no inverse table), and each wave runs 4 x 4
//                 v_mfma_f32_16x16x4f32 tiles (64 rows x 64 tokens) with its
//                 X operands loaded from global memory straight into
//                 registers, one window ahead.
//   k_p_densify   one thread per stored block.
//   k_p_refine    the swap search of the paper's GPU converter (Section 5.2),
//                 in a fixed order: one workgroup per chunk, one thread per
//                 row; each round every row finds its best improving partner
//                 (binary64 gains of the binary32 magnitudes, ties to the lower
//                 row) and mutual best partners swap, until no swap improves
//                 (at most 8 * S rounds).  Gains are symmetric, so while a swap
//                 improves there is a mutual pair.
#include "common.hpp"

namespace {

constexpr int kPMaxS = 256;        // rows per chunk
constexpr int kPMaxPairs = 8192;   // S * P scores held in LDS by the converter
constexpr int kPMaxWblk = 8192;    // S * m weights of a chunk held in LDS
constexpr int kPMaxPat = 4096;     // P * n pattern offsets held in LDS
constexpr int kPRowsWave = 16;
constexpr int kPTokens = 256;      // 4 per lane
constexpr int kPWin = 32;          // block columns per inverse table
constexpr int kPStageRows = 32;    // X rows staged per window by k_p_spmm (256 tokens each)

__host__ __device__ inline int p_binom(int m, int n) {
    int64_t v = 1;
    for (int i = 1; i <= n; ++i) {
        v = v * (m - n + i) / i;
        if (v > 4096) return 4097;
    }
    return (int)v;
}

// Offsets (ascending) of pattern `idx` of the revolving-door list of the
// n-subsets of {0 .. m-1}: the list of (m, n) is the list of (m-1, n)
// followed by the list of (m-1, n-1) reversed, each with m-1 added; (m, m)
// holds the single full set.  Unranked from the top: every binomial on the way
// is at most C(m, n).
__device__ void p_unrank(int m, int n, int idx, uint8_t *out) {
    while (n > 0) {
        if (n == m) {
            for (int i = 0; i < n; ++i) out[i] = (uint8_t)i;
            return;
        }
        const int first = p_binom(m - 1, n);
        if (idx >= first) {  // in the second half: m-1 is in the pattern
            idx = p_binom(m - 1, n - 1) - 1 - (idx - first);
            out[n - 1] = (uint8_t)(m - 1);
            --n;
        }
        --m;
    }
}

template <typename T>
__device__ __forceinline__ float p_abs(const T *p) { return fabsf((float)*p); }

template <typename T>
__global__ __launch_bounds__(kBlock) void k_p_compress(const T *__restrict__ W, int64_t ldw,
                                                       T *__restrict__ values,
                                                       uint8_t *__restrict__ index, int n, int m,
                                                       int g, int P, int S, int B) {
    using Bt = typename Bits<T>::type;
    __shared__ float wabs[kPMaxWblk];
    __shared__ float score[kPMaxPairs];
    __shared__ uint8_t pat[kPMaxPat];
    __shared__ int assigned[kPMaxS];
    __shared__ int count[kPMaxS];
    __shared__ unsigned long long best[kBlock / 64];
    const int c = blockIdx.x, b = blockIdx.y, t = threadIdx.x;
    const int64_t row0 = (int64_t)c * S, ldv = (int64_t)B * n;

    for (int i = t; i < S * m; i += kBlock)
        wabs[i] = p_abs(W + (row0 + i / m) * ldw + (int64_t)b * m + i % m);
    for (int p = t; p < P; p += kBlock) p_unrank(m, n, p, pat + p * n);
    for (int r = t; r < S; r += kBlock) assigned[r] = -1;
    for (int p = t; p < P; p += kBlock) count[p] = 0;
    __syncthreads();
    for (int i = t; i < S * P; i += kBlock) {
        const int r = i / P, p = i % P;
        float s = 0.f;  // binary32, the pattern's offsets ascending, from +0
        for (int k = 0; k < n; ++k) s = s + wabs[r * m + pat[p * n + k]];
        score[i] = s;
    }
    __syncthreads();

    // key of pair (r, p): larger magnitude (NaN above all), then lower p, then lower r
    auto key = [&](int i) -> unsigned long long {
        const int r = i / P, p = i % P;
        const float s = score[i];
        const uint32_t bits = isnan(s) ? 0x7fc00000u : __builtin_bit_cast(uint32_t, s);
        return ((unsigned long long)bits << 17) | (1ull << 16) | ((uint64_t)(255 - p) << 8) |
               (uint64_t)(255 - r);
    };
    for (int it = 0; it < S; ++it) {
        unsigned long long k = 0;
        for (int i = t; i < S * P; i += kBlock) {
            const int r = i / P, p = i % P;
            if (assigned[r] < 0 && count[p] < g) k = max(k, key(i));
        }
        for (int off = 32; off > 0; off >>= 1) k = max(k, (unsigned long long)__shfl_xor(k, off));
        if ((t & 63) == 0) best[t >> 6] = k;
        __syncthreads();
        if (t == 0) {
            unsigned long long w = best[0];
            for (int i = 1; i < kBlock / 64; ++i) w = max(w, best[i]);
            // every step has a pair: the free rows equal the free pattern places
            const int r = 255 - (int)(w & 0xff), p = 255 - (int)((w >> 8) & 0xff);
            assigned[r] = p;
            ++count[p];
        }
        __syncthreads();
    }

    // positions: patterns in order, rows of a group ascending; bit copies of W
    for (int r = t; r < S; r += kBlock) {
        const int p = assigned[r];
        int pos = p * g;
        for (int q = 0; q < r; ++q) pos += assigned[q] == p;
        index[(row0 + pos) * B + b] = (uint8_t)r;
        for (int k = 0; k < n; ++k)
            reinterpret_cast<Bt *>(values)[(row0 + pos) * ldv + (int64_t)b * n + k] =
                reinterpret_cast<const Bt *>(W)[(row0 + r) * ldw + (int64_t)b * m + pat[p * n + k]];
    }
}

// One wave per chunk, for chunks of at most kPwPairs * 64 pairs (see the
// file comment); the same keys, eligibility and order as k_p_compress.
constexpr int kPwWaves = 4;
constexpr int kPwPairs = 24;       // pairs per lane, at most (the live mask is 32 bits)
constexpr int kPwWblk = 1024;      // S * m weights per chunk
constexpr int kPwPat = 1024;       // P * n pattern offsets per chunk

__device__ __forceinline__ void p_wave_sync() {
    // this wave's LDS writes are done before its later LDS reads
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// PP pairs per lane (16 for chunks of up to 1024 pairs, else kPwPairs: every
// step scans all PP, so small chunks take the smaller PP).
template <typename T, int PP>
__global__ __launch_bounds__(64 * kPwWaves) void k_p_compress_w(const T *__restrict__ W, int64_t ldw,
                                                                T *__restrict__ values,
                                                                uint8_t *__restrict__ index, int n,
                                                                int m, int g, int P, int S, int B,
                                                                int chunks) {
    using Bt = typename Bits<T>::type;
    __shared__ float wabs_all[kPwWaves][kPwWblk];
    __shared__ uint8_t pat_all[kPwWaves][kPwPat];
    __shared__ int assigned_all[kPwWaves][kPMaxS];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int id = blockIdx.x * kPwWaves + wave;
    if (id >= chunks) return;  // whole waves; no workgroup barrier follows
    float *wabs = wabs_all[wave];
    uint8_t *pat = pat_all[wave];
    int *assigned = assigned_all[wave];
    const int c = id / B, b = id % B;
    const int64_t row0 = (int64_t)c * S, ldv = (int64_t)B * n;

    for (int i = lane; i < S * m; i += 64)
        wabs[i] = p_abs(W + (row0 + i / m) * ldw + (int64_t)b * m + i % m);
    for (int p = lane; p < P; p += 64) p_unrank(m, n, p, pat + p * n);
    p_wave_sync();

    // this lane's pairs j = lane + 64 q: key as in k_p_compress, row and pattern
    unsigned long long key[PP];
    uint32_t rp[PP];
    uint32_t alive = 0;
#pragma unroll
    for (int q = 0; q < PP; ++q) {
        const int j = lane + 64 * q;
        key[q] = 0;
        rp[q] = 0xffffu;
        if (j < S * P) {
            const int r = j / P, p = j - r * P;
            float sc = 0.f;  // binary32, the pattern's offsets ascending, from +0
            for (int k = 0; k < n; ++k) sc = sc + wabs[r * m + pat[p * n + k]];
            const uint32_t bits = isnan(sc) ? 0x7fc00000u : __builtin_bit_cast(uint32_t, sc);
            key[q] = ((unsigned long long)bits << 17) | (1ull << 16) | ((uint64_t)(255 - p) << 8) |
                     (uint64_t)(255 - r);
            rp[q] = ((uint32_t)r << 8) | (uint32_t)p;
            alive |= 1u << q;
        }
    }
    // pattern p's count lives in register p / 64 of lane p % 64 (P <= 256)
    int cnt[4] = {0, 0, 0, 0};
    for (int it = 0; it < S; ++it) {
        unsigned long long k = 0;
#pragma unroll
        for (int q = 0; q < PP; ++q)
            if ((alive >> q) & 1u) k = max(k, key[q]);
        for (int off = 32; off > 0; off >>= 1) k = max(k, (unsigned long long)__shfl_xor(k, off));
        // every step has a pair: the free rows equal the free pattern places
        const int rw = 255 - (int)(k & 0xff), pw = 255 - (int)((k >> 8) & 0xff);
        const int slot = pw >> 6;
        int now = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i)
            if (i == slot) now = __builtin_amdgcn_readlane(cnt[i], pw & 63) + 1;
        if (lane == (pw & 63)) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (i == slot) cnt[i] = now;
        }
        if (lane == 0) assigned[rw] = pw;
        const bool full = now >= g;
#pragma unroll
        for (int q = 0; q < PP; ++q) {
            const uint32_t r = rp[q] >> 8, p = rp[q] & 0xffu;
            if (r == (uint32_t)rw || (full && p == (uint32_t)pw)) alive &= ~(1u << q);
        }
    }
    p_wave_sync();

    // positions: patterns in order, rows of a group ascending; bit copies of W
    for (int r = lane; r < S; r += 64) {
        const int p = assigned[r];
        int pos = p * g;
        for (int q = 0; q < r; ++q) pos += assigned[q] == p;
        index[(row0 + pos) * B + b] = (uint8_t)r;
        for (int k = 0; k < n; ++k)
            reinterpret_cast<Bt *>(values)[(row0 + pos) * ldv + (int64_t)b * n + k] =
                reinterpret_cast<const Bt *>(W)[(row0 + r) * ldw + (int64_t)b * m + pat[p * n + k]];
    }
}

// The swap search with one wave per chunk (at most kPwPairs * 64 pairs): the
// same rounds, gains and tie rules as k_p_refine.
template <typename T>
__global__ __launch_bounds__(64 * kPwWaves) void k_p_refine_w(const T *__restrict__ W, int64_t ldw,
                                                              T *__restrict__ values,
                                                              uint8_t *__restrict__ index, int n,
                                                              int m, int g, int P, int S, int B,
                                                              int chunks) {
    using Bt = typename Bits<T>::type;
    __shared__ float wabs_all[kPwWaves][kPwWblk];
    __shared__ float score_all[kPwWaves][64 * kPwPairs];
    __shared__ uint8_t pat_all[kPwWaves][kPwPat];
    __shared__ int pa_all[kPwWaves][kPMaxS];
    __shared__ int best_all[kPwWaves][kPMaxS];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int id = blockIdx.x * kPwWaves + wave;
    if (id >= chunks) return;  // whole waves; no workgroup barrier follows
    float *wabs = wabs_all[wave], *score = score_all[wave];
    uint8_t *pat = pat_all[wave];
    int *pa = pa_all[wave], *best = best_all[wave];
    const int c = id / B, b = id % B;
    const int64_t row0 = (int64_t)c * S, ldv = (int64_t)B * n;

    for (int i = lane; i < S * m; i += 64)
        wabs[i] = p_abs(W + (row0 + i / m) * ldw + (int64_t)b * m + i % m);
    for (int p = lane; p < P; p += 64) p_unrank(m, n, p, pat + p * n);
    // the packing to start from (a malformed index leaves rows on pattern 0
    // and never reads outside the tables)
    for (int r = lane; r < S; r += 64) pa[r] = 0;
    p_wave_sync();
    for (int j = lane; j < S; j += 64) pa[min((int)index[(row0 + j) * B + b], S - 1)] = j / g;
    p_wave_sync();
    for (int i = lane; i < S * P; i += 64) {
        const int r = i / P, p = i % P;
        float sc = 0.f;  // binary32, the pattern's offsets ascending, from +0
        for (int k = 0; k < n; ++k) sc = sc + wabs[r * m + pat[p * n + k]];
        score[i] = sc;
    }
    p_wave_sync();
    for (int round = 0; round < 8 * S; ++round) {
        bool found = false;
        for (int r = lane; r < S; r += 64) {
            const int a = pa[r];
            int bq = -1;
            double bg = 0.0;
            for (int q = 0; q < S; ++q) {
                const int e = pa[q];
                if (e == a) continue;
                const double gain = ((double)score[r * P + e] + (double)score[q * P + a]) -
                                    ((double)score[r * P + a] + (double)score[q * P + e]);
                if (gain > bg) {  // strictly larger: ties keep the lower q
                    bg = gain;
                    bq = q;
                }
            }
            best[r] = bq;
            found = found || bq >= 0;
        }
        if (!__any(found)) break;  // uniform across the wave
        p_wave_sync();
        for (int r = lane; r < S; r += 64) {
            const int q = best[r];
            if (q > r && best[q] == r) {  // mutual best partners: disjoint pairs
                const int a = pa[r];
                pa[r] = pa[q];
                pa[q] = a;
            }
        }
        p_wave_sync();
    }
    p_wave_sync();

    // stored like nmg_p_compress's result: patterns in order, rows of a group ascending
    for (int r = lane; r < S; r += 64) {
        const int p = pa[r];
        int pos = p * g;
        for (int q = 0; q < r; ++q) pos += pa[q] == p;
        index[(row0 + pos) * B + b] = (uint8_t)r;
        for (int k = 0; k < n; ++k)
            reinterpret_cast<Bt *>(values)[(row0 + pos) * ldv + (int64_t)b * n + k] =
                reinterpret_cast<const Bt *>(W)[(row0 + r) * ldw + (int64_t)b * m + pat[p * n + k]];
    }
}

template <typename T>
__global__ __launch_bounds__(kBlock) void k_p_densify(const T *__restrict__ values,
                                                      const uint8_t *__restrict__ index,
                                                      T *__restrict__ out, int64_t ldw, int M,
                                                      int n, int m, int g, int P, int S, int B) {
    using Bt = typename Bits<T>::type;
    __shared__ uint8_t pat[kPMaxPat];
    for (int p = threadIdx.x; p < P; p += kBlock) p_unrank(m, n, p, pat + p * n);
    __syncthreads();
    const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;  // (stored row, block column)
    if (i >= (int64_t)M * B) return;
    const int64_t R = i / B;
    const int b = (int)(i % B);
    const int j = (int)(R % S);
    const int64_t r = R - j + min((int)index[R * B + b], S - 1);  // chunk row, clamped
    const uint8_t *off = pat + (j / g) * n;
    Bt *o = reinterpret_cast<Bt *>(out) + r * ldw + (int64_t)b * m;
    for (int k = 0; k < m; ++k) o[k] = 0;
    const Bt *v = reinterpret_cast<const Bt *>(values) + R * ((int64_t)B * n) + (int64_t)b * n;
    for (int k = 0; k < n; ++k) o[off[k]] = v[k];
}

template <typename T>
__global__ __launch_bounds__(kBlock) void k_p_refine(const T *__restrict__ W, int64_t ldw,
                                                     T *__restrict__ values, uint8_t *__restrict__ index,
                                                     int n, int m, int g, int P, int S, int B) {
    using Bt = typename Bits<T>::type;
    __shared__ float wabs[kPMaxWblk];
    __shared__ float score[kPMaxPairs];
    __shared__ uint8_t pat[kPMaxPat];
    __shared__ int pa[kPMaxS];     // pattern of each chunk row
    __shared__ int best[kPMaxS];   // best improving partner, or -1
    __shared__ int any;
    const int c = blockIdx.x, b = blockIdx.y, t = threadIdx.x;
    const int64_t row0 = (int64_t)c * S, ldv = (int64_t)B * n;

    for (int i = t; i < S * m; i += kBlock)
        wabs[i] = p_abs(W + (row0 + i / m) * ldw + (int64_t)b * m + i % m);
    for (int p = t; p < P; p += kBlock) p_unrank(m, n, p, pat + p * n);
    // the packing to start from (a malformed index leaves rows on pattern 0
    // and never reads outside the tables)
    for (int r = t; r < S; r += kBlock) pa[r] = 0;
    __syncthreads();
    for (int j = t; j < S; j += kBlock) pa[min((int)index[(row0 + j) * B + b], S - 1)] = j / g;
    __syncthreads();
    for (int i = t; i < S * P; i += kBlock) {
        const int r = i / P, p = i % P;
        float s = 0.f;  // binary32, the pattern's offsets ascending, from +0
        for (int k = 0; k < n; ++k) s = s + wabs[r * m + pat[p * n + k]];
        score[i] = s;
    }
    for (int round = 0; round < 8 * S; ++round) {
        if (t == 0) any = 0;
        __syncthreads();  // scores, patterns and the flag are ready
        for (int r = t; r < S; r += kBlock) {
            const int a = pa[r];
            int bq = -1;
            double bg = 0.0;
            for (int q = 0; q < S; ++q) {
                const int e = pa[q];
                if (e == a) continue;
                const double gain = ((double)score[r * P + e] + (double)score[q * P + a]) -
                                    ((double)score[r * P + a] + (double)score[q * P + e]);
                if (gain > bg) {  // strictly larger: ties keep the lower q
                    bg = gain;
                    bq = q;
                }
            }
            best[r] = bq;
            if (bq >= 0) any = 1;
        }
        __syncthreads();
        if (any == 0) break;  // uniform: read after the barrier
        for (int r = t; r < S; r += kBlock) {
            const int q = best[r];
            if (q > r && best[q] == r) {  // mutual best partners: disjoint pairs
                const int a = pa[r];
                pa[r] = pa[q];
                pa[q] = a;
            }
        }
        __syncthreads();  // the flag is reset only after every thread has read it
    }
    __syncthreads();

    // stored like nmg_p_compress's result: patterns in order, rows of a group ascending
    for (int r = t; r < S; r += kBlock) {
        const int p = pa[r];
        int pos = p * g;
        for (int q = 0; q < r; ++q) pos += pa[q] == p;
        index[(row0 + pos) * B + b] = (uint8_t)r;
        for (int k = 0; k < n; ++k)
            reinterpret_cast<Bt *>(values)[(row0 + pos) * ldv + (int64_t)b * n + k] =
                reinterpret_cast<const Bt *>(W)[(row0 + r) * ldw + (int64_t)b * m + pat[p * n + k]];
    }
}

constexpr int kPMaxWaves = kPMaxS / kPRowsWave;  // 16 waves cover the largest chunk

template <typename T, bool STAGED>
__global__ __launch_bounds__(64 * kPMaxWaves) void k_p_spmm(const T *__restrict__ values,
                                                   const uint8_t *__restrict__ index,
                                                   const T *__restrict__ X, int64_t ldx,
                                                   T *__restrict__ Y, int64_t ldy, int N, int n,
                                                   int m, int g, int P, int S, int B, int tok_tiles,
                                                   bool xvec) {
    __shared__ uint8_t pat[kPMaxPat];
    __shared__ uint8_t inv[kPWin * kPMaxS];  // position of chunk row rr in block column w
    __shared__ v4f xs[STAGED ? kPStageRows * 64 : 1];  // staged X rows, 4 tokens per lane
    const int c = blockIdx.x / tok_tiles, tt = blockIdx.x % tok_tiles;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t row0 = (int64_t)c * S, ldv = (int64_t)B * n;
    const int tok = tt * kPTokens + 4 * lane;
    const int valid = N - tok;
    const int rr0 = wave * kPRowsWave;  // this wave's first chunk row

    for (int p = threadIdx.x; p < P; p += blockDim.x) p_unrank(m, n, p, pat + p * n);

    float acc[kPRowsWave][4];
#pragma unroll
    for (int r = 0; r < kPRowsWave; ++r)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[r][j] = 0.f;

    // block columns per window (host checked for STAGED: m <= kPStageRows)
    const int nbw = STAGED ? min(kPWin, kPStageRows / m) : kPWin;
    for (int b0 = 0; b0 < B; b0 += nbw) {
        const int nb = min(nbw, B - b0);
        __syncthreads();  // the previous window's table and rows are no longer read
        for (int i = threadIdx.x; i < nb * S; i += blockDim.x) {
            const int w = i / S, jpos = i % S;
            const int rr = min((int)index[(row0 + jpos) * B + b0 + w], S - 1);
            inv[w * kPMaxS + rr] = (uint8_t)jpos;
        }
        if constexpr (STAGED) {
            // X rows b0 m .. (b0 + nb) m - 1 (all inside K = B m), this tile's tokens
            for (int i = threadIdx.x; i < nb * m * 64; i += blockDim.x) {
                const int xr = i >> 6, l = i & 63;
                const int t4 = tt * kPTokens + 4 * l;
                xs[i] = load4<T>(X + ((int64_t)b0 * m + xr) * ldx + t4, N - t4, xvec);
            }
        }
        __syncthreads();
        for (int w = 0; w < nb; ++w) {
            const int b = b0 + w;
#pragma unroll
            for (int r = 0; r < kPRowsWave; ++r) {
                const int rr = rr0 + r;
                if (rr >= S) continue;
                const int jpos = min((int)inv[w * kPMaxS + rr], S - 1);  // clamped: malformed
                                                                          // indices stay inside
                const uint8_t *off = pat + (jpos / g) * n;
                const T *v = values + (row0 + jpos) * ldv + (int64_t)b * n;
                for (int k = 0; k < n; ++k) {
                    const float wv = (float)v[k];
                    const v4f x = STAGED ? xs[(w * m + off[k]) * 64 + lane]
                                         : load4<T>(X + ((int64_t)b * m + off[k]) * ldx + tok, valid, xvec);
#pragma unroll
                    for (int j = 0; j < 4; ++j) acc[r][j] = fmaf(wv, x[j], acc[r][j]);
                }
            }
        }
    }
#pragma unroll
    for (int r = 0; r < kPRowsWave; ++r) {
        const int rr = rr0 + r;
        if (rr >= S) continue;
        T *y = Y + (row0 + rr) * ldy + tok;
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (j < valid) y[j] = (T)acc[r][j];
    }
}

bool p_fits(const nmg_p_layout *L) {
    return L->S * L->P <= kPMaxPairs && L->S * L->m <= kPMaxWblk && L->P * L->n <= kPMaxPat &&
           L->S <= kPMaxS;
}

// ------------------------------------------------ product on matrix cores

constexpr int kPmRows = 64;               // rows per workgroup
constexpr int kPmTok = 256;               // tokens per workgroup (64 per wave)
constexpr int kPmKw = 32;                 // k columns per window, at most
constexpr int kPmLda = kPmRows + 16;      // padded: the 4 k rows of an A read
                                          // fall on 4 disjoint sets of 16 banks
constexpr int kPmLdr = kPmKw + 4;         // row path, A[row][k]: 16 rows' 16-byte
                                          // reads cover the 256 bytes of banks once
constexpr int kPmPre = 8;                 // kept weights prefetched per thread and window

// Division of e < 2^16 by 1 <= d < 2^16 through a multiply-high: with
// mul = ceil(2^32 / d), floor(e mul / 2^32) = floor(e / d) since e d < 2^32.
__device__ __forceinline__ uint32_t magic_u16(uint32_t d) {
    return d > 1 ? (uint32_t)(0xffffffffu / d + 1u) : 0u;
}
__device__ __forceinline__ uint32_t div_u16(uint32_t e, uint32_t mul, uint32_t d) {
    return d > 1 ? __umulhi(e, mul) : e;
}

// N4 > 0: m = 4 and n = N4 <= 3 with whole windows (B % 8 == 0), values on
// 16-byte and the index on 4-byte boundaries, and at most 256 stored rows per
// tile: thread j owns stored row j of the tile's chunks for the whole K loop
// (its chunk slot, target rows and pattern fixed), loads its window of kept
// weights as 16-byte vectors and its 8 index bytes as 2 words, and scatters
// them with register indices known at compile time.  N4 = 0: any m <= 32,
// element by element.
template <typename T, int N4, bool XFULL>
__global__ __launch_bounds__(256, 3) void k_p_spmm_mfma(const T *__restrict__ values,
                                                     const uint8_t *__restrict__ index,
                                                     const T *__restrict__ X, int64_t ldx,
                                                     T *__restrict__ Y, int64_t ldy, int M, int N,
                                                     int n, int m, int g, int P, int S, int B,
                                                     int row_tiles, int tok_tiles, bool xvec) {
    __shared__ uint8_t pat[kPMaxPat];
    // expanded weights: As[k][row] (element path), As[row][k] (row path)
    __shared__ __align__(16) float As[kPmKw * kPmLda];
    const int tile = xcd_tile(blockIdx.x, row_tiles * tok_tiles);
    const int tt = tile / row_tiles, rt = tile - tt * row_tiles;
    const int R0 = rt * kPmRows, t0 = tt * kPmTok;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lr = lane & 15, lk = lane >> 4;
    const int64_t ldv = (int64_t)B * n;
    // the stored rows whose blocks can land in this tile: its chunks'
    const int s_lo = (R0 / S) * S;
    const int s_hi = min(M, (min(M, R0 + kPmRows) + S - 1) / S * S);
    const int ns = s_hi - s_lo;
    // XFULL: every tile is 256 whole tokens of 16-byte aligned X rows (vector
    // loads, no tail); otherwise each load is checked

    for (int p = tid; p < P; p += 256) p_unrank(m, n, p, pat + p * n);

    v4f acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

    const int nbw = kPmKw / m;   // block columns per window (m <= kPmKw, host checked)
    // A window's kept weights: ns stored rows x nb * n values, element e of
    // stored row e / (nb n).  Thread tid prefetches elements tid + 256 q
    // (q < kPmPre) and their index bytes into registers while the previous
    // window is multiplied; elements past 256 kPmPre are read when scattered.
    // (kept in their loaded types, converted where they are written to LDS,
    // so that nothing waits for them before the multiplications)
    // X goes from global memory straight into the B operands: column c of this
    // wave's token tile j is token t0 + 64 wave + 4 c + j, so lane (lr, lk)
    // needs tokens 4 lr .. 4 lr + 3 of row k0 + lk for its 4 tiles -- one
    // 16-byte load per k-step.  x[q] holds k-step q of the current window and
    // is reloaded with k-step q of the next one as soon as it is read.
    const int tx = t0 + 64 * wave + 4 * lr;
    typedef typename std::conditional<std::is_same<T, float>::value, v4f, h4>::type XV;
    XV x[kPmKw / 4];
    auto load_x = [&](int b0, int q) {
        // rows past kw re-read row kw - 1 (multiplied by zero weights and
        // masked at use)
        const int kw = min(nbw, B - b0) * m;
        // k-step q of lane group lk: column 4 q + lk, or 8 lk + q on the row
        // path (whole windows), where a lane's A values are then contiguous
        const int k = N4 > 0 ? 8 * lk + q : min(4 * q + lk, kw - 1);
        const T *src = X + ((int64_t)b0 * m + k) * ldx + tx;
        if constexpr (XFULL) {
            x[q] = *reinterpret_cast<const XV *>(src);
        } else {
            const v4f v = load4<T>(src, N - tx, xvec);   // binary16 back exactly
            x[q] = XV{(T)v[0], (T)v[1], (T)v[2], (T)v[3]};
        }
    };
    constexpr int kRowPre = N4 > 0 ? 1 : kPmPre;   // element path only
    T pv[kRowPre];
    uint8_t pi[kRowPre];
    // row path: this thread's stored row, its vectors and index words
    typedef unsigned int u4 __attribute__((ext_vector_type(4)));
    constexpr int kRowVec = N4 > 0 ? 8 * N4 * (int)sizeof(T) / 16 : 1;
    u4 rv[kRowVec];
    uint32_t ri[2];
    const int jrow = min(tid, ns - 1);
    const T *vrow = values + (int64_t)(s_lo + jrow) * ldv;
    const uint8_t *irow = index + (int64_t)(s_lo + jrow) * B;
    const int jslot = jrow % S;
    const int rbase = s_lo + jrow - jslot - R0;   // tile row of chunk row 0
    auto prefetch = [&](int b0) {
        const int nb = min(nbw, B - b0), kw = nb * m, nvw = nb * n, total = ns * nvw;
        const uint32_t mv = magic_u16(nvw), mn = magic_u16(n);
        if constexpr (N4 > 0) {
            (void)total;
#pragma unroll
            for (int q = 0; q < kRowVec; ++q)
                rv[q] = *reinterpret_cast<const u4 *>(vrow + (int64_t)b0 * N4 + q * (16 / (int)sizeof(T)));
            ri[0] = *reinterpret_cast<const uint32_t *>(irow + b0);
            ri[1] = *reinterpret_cast<const uint32_t *>(irow + b0 + 4);
            return;
        }
#pragma unroll
        for (int q = 0; q < kRowPre; ++q) {
            const uint32_t e = (uint32_t)min(tid + 256 * q, total - 1);   // clamped: in bounds
            const uint32_t j = div_u16(e, mv, nvw), qq = e - j * nvw;
            const uint32_t w = div_u16(qq, mn, n);
            const int64_t Rs = s_lo + (int64_t)j;
            pv[q] = values[Rs * ldv + (int64_t)b0 * n + qq];
            pi[q] = index[Rs * B + b0 + w];
        }
    };
    prefetch(0);
#pragma unroll
    for (int q = 0; q < kPmKw / 4; ++q) load_x(0, q);
    const int b_last = (B - 1) / nbw * nbw;   // the last window's first block column
    for (int b0 = 0; b0 < B; b0 += nbw) {
        const int nb = min(nbw, B - b0);
        const int kw = nb * m, kw4 = (kw + 3) & ~3;
        const int nvw = nb * n, total = ns * nvw;
        const uint32_t mv = magic_u16(nvw), mn = magic_u16(n), mg = magic_u16(g),
                       ms = magic_u16(S);
        __syncthreads();  // the previous window is no longer read
        if constexpr (N4 == 0) {
            // A's k columns 0 .. kw4 - 1 to zero
            for (int i = tid; i < kw4 * (kPmRows / 4); i += 256) {
                const int k = i / (kPmRows / 4), c4 = i % (kPmRows / 4);
                *reinterpret_cast<v4f *>(As + k * kPmLda + 4 * c4) = v4f{0.f, 0.f, 0.f, 0.f};
            }
            __syncthreads();
        }
        // every kept weight to its chunk row (A[w m + offset][row])
        auto scatter = [&](uint32_t e, float v, int rho) {
            const uint32_t j = div_u16(e, mv, nvw), qq = e - j * nvw;
            const uint32_t w = div_u16(qq, mn, n), sl = qq - w * n;
            const uint32_t js = j - div_u16(j, ms, S) * S;             // slot in the chunk
            const int r = s_lo + (int)(j - js) + min(rho, S - 1) - R0;  // row in the tile
            if (r >= 0 && r < kPmRows)
                As[(w * m + pat[div_u16(js, mg, g) * n + sl]) * kPmLda + r] = v;
        };
        if constexpr (N4 > 0) {
            if (tid < ns) {
                const T *vals = reinterpret_cast<const T *>(rv);
                const uint8_t *off = pat + (jslot / g) * N4;
                int o[N4];
#pragma unroll
                for (int sl = 0; sl < N4; ++sl) o[sl] = off[sl];
#pragma unroll
                for (int w = 0; w < 8; ++w) {
                    // the whole block, zeros included: with a permutation index
                    // every (row, block) of the tile is written once
                    const int rho = (ri[w >> 2] >> (8 * (w & 3))) & 0xff;
                    const int r = rbase + min(rho, S - 1);
                    v4f blk = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int k = 0; k < 4; ++k)
#pragma unroll
                        for (int sl = 0; sl < N4; ++sl)
                            if (o[sl] == k) blk[k] = (float)vals[w * N4 + sl];
                    if ((unsigned)r < (unsigned)kPmRows)
                        *reinterpret_cast<v4f *>(As + r * kPmLdr + 4 * w) = blk;
                }
            }
        } else {
#pragma unroll
        for (int q = 0; q < kRowPre; ++q) {
            const int e = tid + 256 * q;
            if (e < total) scatter((uint32_t)e, (float)pv[q], (int)pi[q]);
        }
        }
        for (int e = tid + 256 * kRowPre; N4 == 0 && e < total; e += 256) {
            const uint32_t j = div_u16((uint32_t)e, mv, nvw), qq = (uint32_t)e - j * nvw;
            const int64_t Rs = s_lo + (int64_t)j;
            scatter((uint32_t)e, (float)values[Rs * ldv + (int64_t)b0 * n + qq],
                    index[Rs * B + b0 + div_u16(qq, mn, n)]);
        }
        __syncthreads();
        if (b0 + nbw < B) prefetch(b0 + nbw);
        // 16 x 16 x 4 steps: lane (lr, lk) brings A[row lr][k lk] and
        // B[k lk][token lr]; row tiles i and token tiles j of this wave
        v4f ar[4];   // row path: A[16 i + lr][8 lk + 4 h .. + 3] for h = q / 4
#pragma unroll
        for (int q = 0; q < kPmKw / 4; ++q) {
            if (4 * q >= kw4) break;
            float a[4];
            if constexpr (N4 > 0) {
                if (q % 4 == 0)
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        ar[i] = *reinterpret_cast<const v4f *>(As + (16 * i + lr) * kPmLdr + 8 * lk + q);
#pragma unroll
                for (int i = 0; i < 4; ++i) a[i] = ar[i][q % 4];
            } else {
#pragma unroll
                for (int i = 0; i < 4; ++i) a[i] = As[(4 * q + lk) * kPmLda + 16 * i + lr];
            }
            const bool kin = N4 > 0 || 4 * q + lk < kw;   // padded k rows: zero operands
            float bx[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) bx[j] = kin ? (float)x[q][j] : 0.f;
            load_x(min(b0 + nbw, b_last), q);   // the last window reloads itself
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], bx[j], acc[i][j], 0, 0, 0);
        }
    }
    // acc[i][j][e] = Y[R0 + 16 i + 4 lk + e][t0 + 64 wave + 4 lr + j]: the 4
    // tiles give 4 consecutive tokens, one 16-byte store when whole
    const bool yvec = XFULL && (uintptr_t)Y % (4 * sizeof(T)) == 0 && ldy % 4 == 0;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int row = R0 + 16 * i + 4 * lk + e;
            if (row >= M) continue;
            T *y = Y + (int64_t)row * ldy + tx;
            if (yvec) {
                *reinterpret_cast<XV *>(y) =
                    XV{(T)acc[i][0][e], (T)acc[i][1][e], (T)acc[i][2][e], (T)acc[i][3][e]};
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (tx + j < N) y[j] = (T)acc[i][j][e];
            }
        }
}

}  // namespace

namespace nmg_internal {

nmg_status check_p_layout(const nmg_p_layout *L) {
    if (!L) return NMG_ERR_NULL;
    if (L->dtype != NMG_F32 && L->dtype != NMG_F16) return NMG_ERR_DTYPE;
    if (L->M < 1 || L->K < 1 || L->n < 1 || L->m < L->n || L->m > 255 || L->g < 1)
        return NMG_ERR_PARAM;
    const int P = p_binom(L->m, L->n);
    if (P > 256 || L->P != P || L->S != P * L->g || L->B != L->K / L->m) return NMG_ERR_PARAM;
    if (L->S > kPMaxS || L->K % L->m != 0 || L->M % L->S != 0) return NMG_ERR_SHAPE;
    return NMG_OK;
}

int p_pattern_count(int m, int n) { return p_binom(m, n); }

nmg_status launch_p_compress(const nmg_p_layout *L, const void *W, int64_t ldw, void *values,
                             uint8_t *index, hipStream_t stream) {
    if (!p_fits(L)) return NMG_ERR_UNSUPPORTED;
    const int64_t chunks = (int64_t)(L->M / L->S) * L->B;
    if (L->S * L->P <= 64 * kPwPairs && L->S * L->m <= kPwWblk && L->P * L->n <= kPwPat &&
        chunks <= INT32_MAX - kPwWaves) {
        const unsigned blocks = (unsigned)((chunks + kPwWaves - 1) / kPwWaves);
        const bool small = L->S * L->P <= 64 * 16;
#define NMG_P_W(T, PP)                                                                            \
    hipLaunchKernelGGL((k_p_compress_w<T, PP>), dim3(blocks), dim3(64 * kPwWaves), 0, stream,      \
                       (const T *)W, ldw, (T *)values, index, L->n, L->m, L->g, L->P, L->S, L->B,  \
                       (int)chunks)
        if (L->dtype == NMG_F32) {
            if (small) NMG_P_W(float, 16);
            else NMG_P_W(float, kPwPairs);
        } else {
            if (small) NMG_P_W(_Float16, 16);
            else NMG_P_W(_Float16, kPwPairs);
        }
#undef NMG_P_W
        return launched();
    }
    dim3 grid(L->M / L->S, L->B);
    if (L->dtype == NMG_F32)
        hipLaunchKernelGGL((k_p_compress<float>), grid, dim3(kBlock), 0, stream, (const float *)W,
                           ldw, (float *)values, index, L->n, L->m, L->g, L->P, L->S, L->B);
    else
        hipLaunchKernelGGL((k_p_compress<_Float16>), grid, dim3(kBlock), 0, stream,
                           (const _Float16 *)W, ldw, (_Float16 *)values, index, L->n, L->m, L->g,
                           L->P, L->S, L->B);
    return launched();
}

nmg_status launch_p_refine(const nmg_p_layout *L, const void *W, int64_t ldw, void *values,
                           uint8_t *index, hipStream_t stream) {
    if (!p_fits(L)) return NMG_ERR_UNSUPPORTED;
    const int64_t chunks = (int64_t)(L->M / L->S) * L->B;
    if (L->S * L->P <= 64 * kPwPairs && L->S * L->m <= kPwWblk && L->P * L->n <= kPwPat &&
        chunks <= INT32_MAX - kPwWaves) {
        const unsigned blocks = (unsigned)((chunks + kPwWaves - 1) / kPwWaves);
        if (L->dtype == NMG_F32)
            hipLaunchKernelGGL((k_p_refine_w<float>), dim3(blocks), dim3(64 * kPwWaves), 0, stream,
                               (const float *)W, ldw, (float *)values, index, L->n, L->m, L->g,
                               L->P, L->S, L->B, (int)chunks);
        else
            hipLaunchKernelGGL((k_p_refine_w<_Float16>), dim3(blocks), dim3(64 * kPwWaves), 0,
                               stream, (const _Float16 *)W, ldw, (_Float16 *)values, index, L->n,
                               L->m, L->g, L->P, L->S, L->B, (int)chunks);
        return launched();
    }
    dim3 grid(L->M / L->S, L->B);
    if (L->dtype == NMG_F32)
        hipLaunchKernelGGL((k_p_refine<float>), grid, dim3(kBlock), 0, stream, (const float *)W,
                           ldw, (float *)values, index, L->n, L->m, L->g, L->P, L->S, L->B);
    else
        hipLaunchKernelGGL((k_p_refine<_Float16>), grid, dim3(kBlock), 0, stream,
                           (const _Float16 *)W, ldw, (_Float16 *)values, index, L->n, L->m, L->g,
                           L->P, L->S, L->B);
    return launched();
}

nmg_status launch_p_densify(const nmg_p_layout *L, const void *values, const uint8_t *index,
                            void *W_out, int64_t ldw, hipStream_t stream) {
    if (!p_fits(L)) return NMG_ERR_UNSUPPORTED;
    const int64_t blocks = ((int64_t)L->M * L->B + kBlock - 1) / kBlock;
    if (blocks > INT32_MAX) return NMG_ERR_PARAM;
    if (L->dtype == NMG_F32)
        hipLaunchKernelGGL((k_p_densify<float>), dim3((unsigned)blocks), dim3(kBlock), 0, stream,
                           (const float *)values, index, (float *)W_out, ldw, L->M, L->n, L->m,
                           L->g, L->P, L->S, L->B);
    else
        hipLaunchKernelGGL((k_p_densify<_Float16>), dim3((unsigned)blocks), dim3(kBlock), 0,
                           stream, (const _Float16 *)values, index, (_Float16 *)W_out, ldw, L->M,
                           L->n, L->m, L->g, L->P, L->S, L->B);
    return launched();
}

nmg_status launch_p_spmm(const nmg_p_layout *L, nmg_kernel kernel, const void *values,
                         const uint8_t *index, const void *X, int64_t ldx, int N, void *Y,
                         int64_t ldy, hipStream_t stream) {
    if (!p_fits(L)) return NMG_ERR_UNSUPPORTED;
    const size_t es = elem_size(L->dtype);
    const bool xvec = aligned(X, 4 * es) && ldx % 4 == 0;
    // matrix cores when a quarter or more of the expanded products are useful
    if (kernel == NMG_KERNEL_AUTO) kernel = 4 * L->n >= L->m && L->m <= kPmKw ? NMG_KERNEL_MFMA
                                                                          : NMG_KERNEL_VALU;
    if (kernel == NMG_KERNEL_MFMA) {
        if (L->m > kPmKw) return NMG_ERR_UNSUPPORTED;
        const int row_tiles = (L->M + kPmRows - 1) / kPmRows;
        const int tok_tiles = (N + kPmTok - 1) / kPmTok;
        const int64_t grid = (int64_t)row_tiles * tok_tiles;
        if (grid > INT32_MAX) return NMG_ERR_PARAM;
        // the row path (see k_p_spmm_mfma): m = 4, whole windows, aligned
        // rows, and a tile's chunks hold at most 256 stored rows (S <= 128, or
        // tiles that never straddle two chunks)
        const bool rows = L->m == 4 && L->n <= 3 && L->B % 8 == 0 && aligned(values, 16) &&
                          aligned(index, 4) && (L->S <= 128 || L->S % kPmRows == 0);
        const int n4 = rows ? L->n : 0;
        // every token tile whole and X rows on 16-byte boundaries
        const bool xfull = xvec && N % kPmTok == 0;
#define NMG_P_MFMA(T, N4)                                                                         \
    if (xfull)                                                                                    \
        hipLaunchKernelGGL((k_p_spmm_mfma<T, N4, true>), dim3((unsigned)grid), dim3(256), 0,       \
                           stream, (const T *)values, index, (const T *)X, ldx, (T *)Y, ldy, L->M, \
                           N, L->n, L->m, L->g, L->P, L->S, L->B, row_tiles, tok_tiles, xvec);     \
    else                                                                                          \
        hipLaunchKernelGGL((k_p_spmm_mfma<T, N4, false>), dim3((unsigned)grid), dim3(256), 0,      \
                           stream, (const T *)values, index, (const T *)X, ldx, (T *)Y, ldy, L->M, \
                           N, L->n, L->m, L->g, L->P, L->S, L->B, row_tiles, tok_tiles, xvec)
#define NMG_P_MFMA_N(T)                                                                           \
    switch (n4) {                                                                                 \
        case 1: NMG_P_MFMA(T, 1); break;                                                          \
        case 2: NMG_P_MFMA(T, 2); break;                                                          \
        case 3: NMG_P_MFMA(T, 3); break;                                                          \
        default: NMG_P_MFMA(T, 0); break;                                                         \
    }
        if (L->dtype == NMG_F32) {
            NMG_P_MFMA_N(float);
        } else {
            NMG_P_MFMA_N(_Float16);
        }
#undef NMG_P_MFMA_N
#undef NMG_P_MFMA
        return launched();
    }
    if (kernel != NMG_KERNEL_VALU) return NMG_ERR_UNSUPPORTED;
    const int tok_tiles = (N + kPTokens - 1) / kPTokens;
    const int64_t grid = (int64_t)(L->M / L->S) * tok_tiles;
    if (grid > INT32_MAX) return NMG_ERR_PARAM;
    const int waves = (L->S + kPRowsWave - 1) / kPRowsWave;
    // staging pays when the chunk has enough rows (4 waves or more) to share
    // each staged row; small chunks gather (measured on the 3072 x 768 sweep)
    const bool staged = L->m <= kPStageRows && L->S >= 64;
#define NMG_P_SPMM(T, ST)                                                                         \
    hipLaunchKernelGGL((k_p_spmm<T, ST>), dim3((unsigned)grid), dim3(64 * waves), 0, stream,       \
                       (const T *)values, index, (const T *)X, ldx, (T *)Y, ldy, N, L->n, L->m,    \
                       L->g, L->P, L->S, L->B, tok_tiles, xvec)
    if (L->dtype == NMG_F32) {
        if (staged) NMG_P_SPMM(float, true);
        else NMG_P_SPMM(float, false);
    } else {
        if (staged) NMG_P_SPMM(_Float16, true);
        else NMG_P_SPMM(_Float16, false);
    }
#undef NMG_P_SPMM
    return launched();
}

}  // namespace nmg_internal
