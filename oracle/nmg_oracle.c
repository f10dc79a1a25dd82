/*
 * CPU oracle for the grouped n:m (n:m:g) sparsity layout.
 *
 * TEST INFRASTRUCTURE ONLY.  This is a deliberately plain, slow reference of
 * what the GPU library computes.  Only the test suite, the package smoke check
 * and the CPU-baseline leg of the benchmark load it; the product path never
 * does.  It shares no source, header, table or helper with the GPU library.
 *
 * Paper: Hoefler et al., "STen: Productive and Efficient Sparsity in PyTorch"
 * (arXiv 2304.07613), Section 5 "Grouped n:m Sparsity".
 *
 * Layout (Section 5, opening paragraph: an n:m pattern that is shared by g
 * rows, which form a group).  A dense M x K weight W (row-major, leading
 * dimension ldw) is cut along K into C = ceil(K/m) chunks of m consecutive
 * columns; the last chunk has width r = K - (C-1)*m, which may be below m.
 * Rows [G*g, G*g+g) form group G; every row of a group keeps the same n column
 * offsets inside a chunk.
 *   values  : M x (C*n), row-major, W's element type.  values[r][c*n+s] is
 *             the s-th kept element of row r in chunk c (a bit copy of W).
 *   indices : (M/g) x (C*n) bytes.  indices[G][c*n+s] is the in-chunk offset
 *             of that element; offsets are strictly ascending in s.
 *
 * Selection (Section 5.2: the converter maximises the L1 norm of the pruned
 * tensor over all n:m:g-valid tensors).  For a group and a chunk the kept L1
 * mass is the sum of the kept columns' scores
 *     score[j] = sum over i < g of |W[G*g+i][c*m+j]|,
 * and different (group, chunk) pairs do not constrain each other, so the
 * maximiser keeps the n columns with the largest scores.  Readings taken where
 * the paper is silent:
 *   - scores are summed in binary32, rows in ascending order, from +0;
 *     binary16 weights are first widened exactly to binary32;
 *   - equal scores go to the lower offset;
 *   - a NaN score orders above every number; NaN scores tie with each other;
 *   - a tail chunk narrower than n is rejected.
 *
 * Product (Section 5.1, and the dense conversion at the end of Section 5.2):
 * Y = densify(values, indices) * X, with X K x N row-major.  The oracle sums,
 * for every output, the products of the kept weights with their X entries in
 * ascending column order (the dense dot product with its zero terms left
 * out), in binary64.  Every product of two binary32 (or binary16) numbers is
 * exact in binary64.  It also returns the error scale
 *     B[r][t] = sum over kept k of |W_s[r][k]| * |X[k][t]|.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORC_F32 = 0, ORC_F16 = 1 };
enum { ORC_OK = 0, ORC_EPARAM = 1, ORC_ESHAPE = 2, ORC_EINDEX = 3 };

/* ---------------------------------------------------------------- binary16 */

/* Exact binary16 -> binary32 widening, from the IEEE 754 binary16 encoding:
 * 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits. */
float oracle_half_to_float(uint16_t h)
{
    unsigned sign = h >> 15, e = (h >> 10) & 0x1fu, f = h & 0x3ffu;
    double v;
    if (e == 0)
        v = ldexp((double)f, -24);              /* subnormal: f * 2^-24 */
    else if (e == 31)
        v = f ? NAN : INFINITY;
    else
        v = ldexp((double)(f | 0x400u), (int)e - 25); /* (1024+f) * 2^(e-25) */
    return (float)(sign ? -v : v);
}

/* binary64 -> binary16, round to nearest, ties to even (one rounding). */
uint16_t oracle_double_to_half(double x)
{
    uint16_t sign = signbit(x) ? 0x8000u : 0u;
    if (isnan(x))
        return (uint16_t)(sign | 0x7e00u);
    double a = fabs(x);
    if (isinf(a))
        return (uint16_t)(sign | 0x7c00u);
    if (a == 0.0)
        return sign;
    int e2;
    frexp(a, &e2);              /* a in [2^(e2-1), 2^e2) */
    int ue = e2 - 1;            /* unbiased binade exponent */
    if (ue < -14)
        ue = -14;               /* subnormals share the spacing 2^-24 */
    /* In the binade 2^ue the binary16 spacing is 2^(ue-10). */
    double q = nearbyint(ldexp(a, 10 - ue)); /* default mode: ties to even */
    double v = ldexp(q, ue - 10);
    if (v > 65504.0)
        return (uint16_t)(sign | 0x7c00u);
    if (v < ldexp(1.0, -14))                  /* still subnormal */
        return (uint16_t)(sign | (uint16_t)ldexp(v, 24));
    int ev;
    frexp(v, &ev);
    int E = ev - 1;                           /* v = (1024 + f) * 2^(E-10) */
    unsigned k = (unsigned)ldexp(v, 10 - E);  /* 1024 <= k < 2048 */
    return (uint16_t)(sign | (unsigned)((E + 15) << 10) | (k - 1024u));
}

uint16_t oracle_float_to_half(float x) { return oracle_double_to_half((double)x); }

void oracle_round_to_half(const double *in, uint16_t *out, int64_t count)
{
    for (int64_t i = 0; i < count; ++i)
        out[i] = oracle_double_to_half(in[i]);
}

/* --------------------------------------------------------------- elements */

static double elem(int dtype, const void *p, int64_t ld, int64_t r, int64_t k)
{
    if (dtype == ORC_F32)
        return (double)((const float *)p)[r * ld + k];
    return (double)oracle_half_to_float(((const uint16_t *)p)[r * ld + k]);
}

static float abs_elem32(int dtype, const void *p, int64_t ld, int64_t r, int64_t k)
{
    if (dtype == ORC_F32)
        return fabsf(((const float *)p)[r * ld + k]);
    return fabsf(oracle_half_to_float(((const uint16_t *)p)[r * ld + k]));
}

static void copy_elem(int dtype, void *dst, int64_t ldd, int64_t rd, int64_t kd,
                      const void *src, int64_t lds, int64_t rs, int64_t ks)
{
    size_t sz = dtype == ORC_F32 ? 4 : 2;
    memcpy((char *)dst + (size_t)(rd * ldd + kd) * sz,
           (const char *)src + (size_t)(rs * lds + ks) * sz, sz);
}

/* ------------------------------------------------------------- validation */

static int64_t n_chunks(int64_t K, int m) { return (K + m - 1) / m; }

static int check_layout(int dtype, int64_t M, int64_t K, int n, int m, int g)
{
    if (dtype != ORC_F32 && dtype != ORC_F16)
        return ORC_EPARAM;
    if (M < 1 || K < 1 || n < 1 || m < n || m > 255 || g < 1)
        return ORC_EPARAM;
    if (M % g != 0)
        return ORC_ESHAPE;
    int64_t tail = K - (n_chunks(K, m) - 1) * m;
    if (tail < n)
        return ORC_ESHAPE;
    return ORC_OK;
}

/* Every (group, chunk) must list n strictly ascending offsets inside the
 * chunk. */
static int check_indices(int64_t M, int64_t K, int n, int m, int g,
                         const uint8_t *idx)
{
    int64_t C = n_chunks(K, m), groups = M / g;
    for (int64_t G = 0; G < groups; ++G)
        for (int64_t c = 0; c < C; ++c) {
            int64_t w = K - c * m < m ? K - c * m : m;
            for (int s = 0; s < n; ++s) {
                int o = idx[G * C * n + c * n + s];
                if (o >= w)
                    return ORC_EINDEX;
                if (s > 0 && o <= idx[G * C * n + c * n + s - 1])
                    return ORC_EINDEX;
            }
        }
    return ORC_OK;
}

/* ---------------------------------------------------------------- compress */

/* a ranks strictly above b: NaN above every number, else numeric order. */
static int score_above(float a, float b)
{
    if (isnan(a))
        return !isnan(b);
    if (isnan(b))
        return 0;
    return a > b;
}

static int score_equal(float a, float b)
{
    if (isnan(a) || isnan(b))
        return isnan(a) && isnan(b);
    return a == b;
}

int oracle_compress(int dtype, int64_t M, int64_t K, int n, int m, int g,
                    const void *W, int64_t ldw, void *values, uint8_t *indices)
{
    int st = check_layout(dtype, M, K, n, m, g);
    if (st != ORC_OK)
        return st;
    if (ldw < K)
        return ORC_EPARAM;
    int64_t C = n_chunks(K, m), groups = M / g, ldv = C * n;
    float score[256];
    for (int64_t G = 0; G < groups; ++G)
        for (int64_t c = 0; c < C; ++c) {
            int64_t w = K - c * m < m ? K - c * m : m;
            /* group score of every column of the chunk */
            for (int64_t j = 0; j < w; ++j) {
                float s = 0.0f;
                for (int i = 0; i < g; ++i)
                    s = s + abs_elem32(dtype, W, ldw, G * g + i, c * m + j);
                score[j] = s;
            }
            /* keep column j iff fewer than n columns rank above it */
            int slot = 0;
            for (int64_t j = 0; j < w; ++j) {
                int64_t rank = 0;
                for (int64_t i = 0; i < w; ++i)
                    if (score_above(score[i], score[j]) ||
                        (i < j && score_equal(score[i], score[j])))
                        ++rank;
                if (rank < n)
                    indices[G * ldv + c * n + slot++] = (uint8_t)j;
            }
            if (slot != n)
                abort(); /* a strict total order keeps exactly n */
            /* copy the kept elements of the g rows */
            for (int i = 0; i < g; ++i)
                for (int s = 0; s < n; ++s)
                    copy_elem(dtype, values, ldv, G * g + i, c * n + s, W, ldw,
                              G * g + i, c * m + indices[G * ldv + c * n + s]);
        }
    return ORC_OK;
}

/* ------------------------------------------------------------------ repack */

/* The fixed-mask path after a weight update (Section 5.3: a sparsifier that
 * keeps the tensor's existing format; the STen converters re-pack new dense
 * values into the pattern already chosen).  The indices are given; values get
 * W's entries at the kept positions:
 *     values[r][c*n+s] = W[r][c*m + indices[r/g][c*n+s]]   (a bit copy). */
int oracle_repack(int dtype, int64_t M, int64_t K, int n, int m, int g,
                  const void *W, int64_t ldw, const uint8_t *indices, void *values)
{
    int st = check_layout(dtype, M, K, n, m, g);
    if (st != ORC_OK)
        return st;
    if (ldw < K)
        return ORC_EPARAM;
    st = check_indices(M, K, n, m, g, indices);
    if (st != ORC_OK)
        return st;
    int64_t C = n_chunks(K, m), ldv = C * n;
    for (int64_t r = 0; r < M; ++r)
        for (int64_t c = 0; c < C; ++c)
            for (int s = 0; s < n; ++s)
                copy_elem(dtype, values, ldv, r, c * n + s, W, ldw, r,
                          c * m + indices[(r / g) * ldv + c * n + s]);
    return ORC_OK;
}

/* ----------------------------------------------------------------- densify */

/* W_out (M x K, leading dimension ldw) gets the kept values at their original
 * columns and zeros elsewhere; mask (M x K bytes, optional) gets 1 at the kept
 * positions, taken from the indices alone. */
int oracle_densify(int dtype, int64_t M, int64_t K, int n, int m, int g,
                   const void *values, const uint8_t *indices, void *W_out,
                   int64_t ldw, uint8_t *mask)
{
    int st = check_layout(dtype, M, K, n, m, g);
    if (st != ORC_OK)
        return st;
    if (ldw < K)
        return ORC_EPARAM;
    st = check_indices(M, K, n, m, g, indices);
    if (st != ORC_OK)
        return st;
    int64_t C = n_chunks(K, m), ldv = C * n;
    size_t sz = dtype == ORC_F32 ? 4 : 2;
    for (int64_t r = 0; r < M; ++r) {
        memset((char *)W_out + (size_t)(r * ldw) * sz, 0, (size_t)K * sz);
        if (mask)
            memset(mask + r * K, 0, (size_t)K);
    }
    for (int64_t r = 0; r < M; ++r)
        for (int64_t c = 0; c < C; ++c)
            for (int s = 0; s < n; ++s) {
                int64_t k = c * m + indices[(r / g) * ldv + c * n + s];
                copy_elem(dtype, W_out, ldw, r, k, values, ldv, r, c * n + s);
                if (mask)
                    mask[r * K + k] = 1;
            }
    return ORC_OK;
}

/* -------------------------------------------------------------------- spmm */

static void spmm_one(int dtype, int64_t K, int n, int m, int g,
                     const void *values, const uint8_t *indices, const void *X,
                     int64_t ldx, int64_t r, int64_t t, double *y, double *b)
{
    int64_t C = n_chunks(K, m), ldv = C * n;
    double acc = 0.0, scale = 0.0;
    for (int64_t c = 0; c < C; ++c)
        for (int s = 0; s < n; ++s) {
            int64_t k = c * m + indices[(r / g) * ldv + c * n + s];
            double v = elem(dtype, values, ldv, r, c * n + s);
            double x = elem(dtype, X, ldx, k, t);
            acc += v * x;
            scale += fabs(v) * fabs(x);
        }
    *y = acc;
    *b = scale;
}

/* Y, B: M x N binary64, row-major.  nthreads <= 0 lets OpenMP decide. */
int oracle_spmm(int dtype, int64_t M, int64_t K, int n, int m, int g,
                const void *values, const uint8_t *indices, const void *X,
                int64_t ldx, int64_t N, double *Y, double *B, int nthreads)
{
    int st = check_layout(dtype, M, K, n, m, g);
    if (st != ORC_OK)
        return st;
    if (N < 1 || ldx < N)
        return ORC_EPARAM;
    st = check_indices(M, K, n, m, g, indices);
    if (st != ORC_OK)
        return st;
    int64_t C = n_chunks(K, m), ldv = C * n;
#ifdef _OPENMP
    int nt = nthreads > 0 ? nthreads : omp_get_max_threads();
#else
    (void)nthreads;
#endif
#pragma omp parallel for schedule(dynamic, 1) num_threads(nt)
    for (int64_t r = 0; r < M; ++r) {
        double *yr = Y + r * N, *br = B + r * N;
        for (int64_t t = 0; t < N; ++t) {
            yr[t] = 0.0;
            br[t] = 0.0;
        }
        /* ascending (chunk, slot) = ascending column, as in the dense
         * product with its zero terms left out */
        for (int64_t c = 0; c < C; ++c)
            for (int s = 0; s < n; ++s) {
                int64_t k = c * m + indices[(r / g) * ldv + c * n + s];
                double v = elem(dtype, values, ldv, r, c * n + s);
                for (int64_t t = 0; t < N; ++t) {
                    double x = elem(dtype, X, ldx, k, t);
                    yr[t] += v * x;
                    br[t] += fabs(v) * fabs(x);
                }
            }
    }
    return ORC_OK;
}

/* The same sums at npts sampled outputs (rows[i], cols[i]). */
int oracle_spmm_points(int dtype, int64_t M, int64_t K, int n, int m, int g,
                       const void *values, const uint8_t *indices,
                       const void *X, int64_t ldx, int64_t N, int64_t npts,
                       const int64_t *rows, const int64_t *cols, double *Y,
                       double *B)
{
    int st = check_layout(dtype, M, K, n, m, g);
    if (st != ORC_OK)
        return st;
    if (N < 1 || ldx < N)
        return ORC_EPARAM;
    st = check_indices(M, K, n, m, g, indices);
    if (st != ORC_OK)
        return st;
    for (int64_t i = 0; i < npts; ++i) {
        if (rows[i] < 0 || rows[i] >= M || cols[i] < 0 || cols[i] >= N)
            return ORC_EPARAM;
        spmm_one(dtype, K, n, m, g, values, indices, X, ldx, rows[i], cols[i],
                 &Y[i], &B[i]);
    }
    return ORC_OK;
}

/* --------------------------------------------- elementwise glue (binary16) */

/* GELU in its erf form, 0.5 x (1 + erf(x / sqrt 2)), evaluated in binary64
 * and rounded once to binary16. */
void oracle_gelu_f16(const uint16_t *in, uint16_t *out, int64_t count)
{
    for (int64_t i = 0; i < count; ++i) {
        double x = (double)oracle_half_to_float(in[i]);
        out[i] = oracle_double_to_half(0.5 * x * (1.0 + erf(x / sqrt(2.0))));
    }
}

/* Residual sum a + b, exact in binary64, rounded once to binary16. */
void oracle_add_f16(const uint16_t *a, const uint16_t *b, uint16_t *out,
                    int64_t count)
{
    for (int64_t i = 0; i < count; ++i)
        out[i] = oracle_double_to_half((double)oracle_half_to_float(a[i]) +
                                       (double)oracle_half_to_float(b[i]));
}

/* ============================================ the paper's chunked layout */

/* Section 5 of the paper, read literally ("Reading P"): besides repeating a
 * pattern over a group, groups are combined into chunks that hold every one
 * of the P = C(m, n) patterns in a fixed order, and the blocks of a chunk may
 * be reordered, with an index recording each block's original place.
 *   block    : m consecutive weights of one row along K; row r has K/m blocks
 *              (K % m == 0 is required);
 *   chunk    : the S = P*g blocks of S consecutive rows in one block column
 *              (M % S == 0 and S <= 256 are required);
 *   pattern  : an n-subset of the m offsets; the P patterns are listed in
 *              revolving-door order, so adjacent patterns differ in one
 *              position (Section 5.1: one register changes between groups);
 *   group    : the g blocks of a chunk that use one pattern -- every pattern
 *              is used by exactly g blocks of every chunk.
 * Storage, with B = K/m block columns and the rows of a chunk in pattern
 * order (positions j = 0 .. S-1, pattern j / g, rows of a group ascending):
 *   values[c*S + j][b*n + s] = W[c*S + index[c*S + j][b]][b*m + pattern_{j/g}[s]]
 *   index[c*S + j][b]        = the chunk row whose block sits at position j.
 * Converter (Section 5.2, the CPU algorithm): every (row, pattern) pair of a
 * chunk gets the magnitude its pattern keeps, summed in binary32 over the
 * pattern's offsets in ascending order; the pairs are taken from the largest
 * magnitude down (a NaN sum above every number; equal sums: lower pattern,
 * then lower row, first), and a pair is used when its row has no pattern yet
 * and its pattern has fewer than g rows. */

static int64_t binom(int m, int n)
{
    int64_t v = 1;
    for (int i = 1; i <= n; ++i) {
        v = v * (m - n + i) / i;
        if (v > 4096)
            return 4097; /* more than any admissible layout */
    }
    return v;
}

/* Writes the revolving-door list of the n-subsets of {0 .. m-1} (each
 * ascending) from `out`, returns the count:
 *   list(m, n) = list(m-1, n), then list(m-1, n-1) reversed, each with m-1 added;
 *   list(m, 0) = { {} };  list(m, m) = { {0 .. m-1} }. */
static int64_t revolving_door(int m, int n, uint8_t *out)
{
    if (n == 0)
        return 1;
    if (n == m) {
        for (int i = 0; i < n; ++i)
            out[i] = (uint8_t)i;
        return 1;
    }
    int64_t a = revolving_door(m - 1, n, out);
    uint8_t *tail = out + a * n;
    int64_t b = revolving_door(m - 1, n - 1, tail);
    /* reverse the second list in place (patterns of n-1 offsets) and append m-1 */
    uint8_t *tmp = (uint8_t *)malloc((size_t)(b * (n - 1) + 1));
    memcpy(tmp, tail, (size_t)(b * (n - 1)));
    for (int64_t i = 0; i < b; ++i) {
        const uint8_t *src = tmp + (b - 1 - i) * (n - 1);
        for (int s = 0; s < n - 1; ++s)
            tail[i * n + s] = src[s];
        tail[i * n + n - 1] = (uint8_t)(m - 1);
    }
    free(tmp);
    return a + b;
}

int oracle_p_patterns(int m, int n, uint8_t *out)
{
    if (n < 1 || m < n || m > 255 || binom(m, n) > 256)
        return ORC_EPARAM;
    revolving_door(m, n, out);
    return ORC_OK;
}

static int check_p_layout(int dtype, int64_t M, int64_t K, int n, int m, int g,
                          int64_t *P, int64_t *S)
{
    if (dtype != ORC_F32 && dtype != ORC_F16)
        return ORC_EPARAM;
    if (M < 1 || K < 1 || n < 1 || m < n || m > 255 || g < 1)
        return ORC_EPARAM;
    *P = binom(m, n);
    if (*P > 256)
        return ORC_EPARAM;
    *S = *P * g;
    if (*S > 256 || K % m != 0 || M % *S != 0)
        return ORC_ESHAPE;
    return ORC_OK;
}

/* every chunk's index column is a permutation of 0 .. S-1 */
static int check_p_index(int64_t M, int64_t B, int64_t S, const uint8_t *index)
{
    for (int64_t c = 0; c < M / S; ++c)
        for (int64_t b = 0; b < B; ++b) {
            uint8_t seen[256] = {0};
            for (int64_t j = 0; j < S; ++j) {
                int r = index[(c * S + j) * B + b];
                if (r >= S || seen[r])
                    return ORC_EINDEX;
                seen[r] = 1;
            }
        }
    return ORC_OK;
}

struct p_pair {
    float score;
    int p, r;
};

static int p_pair_order(const void *x, const void *y)
{
    const struct p_pair *a = (const struct p_pair *)x, *b = (const struct p_pair *)y;
    if (score_above(a->score, b->score))
        return -1;
    if (score_above(b->score, a->score))
        return 1;
    if (a->p != b->p)
        return a->p < b->p ? -1 : 1;
    return a->r < b->r ? -1 : (a->r > b->r);
}

int oracle_p_compress(int dtype, int64_t M, int64_t K, int n, int m, int g,
                      const void *W, int64_t ldw, void *values, uint8_t *index)
{
    int64_t P, S;
    int st = check_p_layout(dtype, M, K, n, m, g, &P, &S);
    if (st != ORC_OK)
        return st;
    if (ldw < K)
        return ORC_EPARAM;
    int64_t B = K / m, ldv = B * n;
    uint8_t pat[256 * 255];
    revolving_door(m, n, pat);
    struct p_pair *pairs = (struct p_pair *)malloc(sizeof(struct p_pair) * (size_t)(S * P));
    for (int64_t c = 0; c < M / S; ++c)
        for (int64_t b = 0; b < B; ++b) {
            /* the magnitude each pattern keeps for each row of the chunk */
            for (int64_t r = 0; r < S; ++r)
                for (int64_t p = 0; p < P; ++p) {
                    float s = 0.0f;
                    for (int i = 0; i < n; ++i)
                        s = s + abs_elem32(dtype, W, ldw, c * S + r, b * m + pat[p * n + i]);
                    pairs[r * P + p] = (struct p_pair){s, (int)p, (int)r};
                }
            qsort(pairs, (size_t)(S * P), sizeof(struct p_pair), p_pair_order);
            int assigned[256], count[256];
            for (int i = 0; i < 256; ++i) {
                assigned[i] = -1;
                count[i] = 0;
            }
            for (int64_t i = 0; i < S * P; ++i) {
                const struct p_pair *q = &pairs[i];
                if (assigned[q->r] < 0 && count[q->p] < g) {
                    assigned[q->r] = q->p;
                    ++count[q->p];
                }
            }
            /* positions: patterns in order, rows of a group ascending */
            int64_t j = 0;
            for (int64_t p = 0; p < P; ++p)
                for (int64_t r = 0; r < S; ++r)
                    if (assigned[r] == p) {
                        index[(c * S + j) * B + b] = (uint8_t)r;
                        for (int i = 0; i < n; ++i)
                            copy_elem(dtype, values, ldv, c * S + j, b * n + i, W, ldw, c * S + r,
                                      b * m + pat[p * n + i]);
                        ++j;
                    }
        }
    free(pairs);
    return ORC_OK;
}

int oracle_p_densify(int dtype, int64_t M, int64_t K, int n, int m, int g,
                     const void *values, const uint8_t *index, void *W_out, int64_t ldw,
                     uint8_t *mask)
{
    int64_t P, S;
    int st = check_p_layout(dtype, M, K, n, m, g, &P, &S);
    if (st != ORC_OK)
        return st;
    if (ldw < K)
        return ORC_EPARAM;
    int64_t B = K / m, ldv = B * n;
    st = check_p_index(M, B, S, index);
    if (st != ORC_OK)
        return st;
    uint8_t pat[256 * 255];
    revolving_door(m, n, pat);
    size_t sz = dtype == ORC_F32 ? 4 : 2;
    for (int64_t r = 0; r < M; ++r) {
        memset((char *)W_out + (size_t)(r * ldw) * sz, 0, (size_t)K * sz);
        if (mask)
            memset(mask + r * K, 0, (size_t)K);
    }
    for (int64_t c = 0; c < M / S; ++c)
        for (int64_t b = 0; b < B; ++b)
            for (int64_t j = 0; j < S; ++j) {
                int64_t r = c * S + index[(c * S + j) * B + b], p = j / g;
                for (int i = 0; i < n; ++i) {
                    int64_t k = b * m + pat[p * n + i];
                    copy_elem(dtype, W_out, ldw, r, k, values, ldv, c * S + j, b * n + i);
                    if (mask)
                        mask[r * K + k] = 1;
                }
            }
    return ORC_OK;
}

/* Y = W_s X in binary64 for the chunked layout (the dense product with its
 * zero terms left out, ascending column order per output row) and
 * B = |W_s| |X|. */
int oracle_p_spmm(int dtype, int64_t M, int64_t K, int n, int m, int g,
                  const void *values, const uint8_t *index, const void *X, int64_t ldx,
                  int64_t N, double *Y, double *Bnd)
{
    int64_t P, S;
    int st = check_p_layout(dtype, M, K, n, m, g, &P, &S);
    if (st != ORC_OK)
        return st;
    if (N < 1 || ldx < N)
        return ORC_EPARAM;
    int64_t B = K / m, ldv = B * n;
    st = check_p_index(M, B, S, index);
    if (st != ORC_OK)
        return st;
    uint8_t pat[256 * 255];
    revolving_door(m, n, pat);
    /* the position of every (row, block column) */
    int64_t *pos = (int64_t *)malloc(sizeof(int64_t) * (size_t)(M * B));
    for (int64_t c = 0; c < M / S; ++c)
        for (int64_t b = 0; b < B; ++b)
            for (int64_t j = 0; j < S; ++j)
                pos[(c * S + index[(c * S + j) * B + b]) * B + b] = j;
    for (int64_t r = 0; r < M; ++r) {
        double *yr = Y + r * N, *br = Bnd + r * N;
        for (int64_t t = 0; t < N; ++t) {
            yr[t] = 0.0;
            br[t] = 0.0;
        }
        int64_t c = r / S;
        for (int64_t b = 0; b < B; ++b) {
            int64_t j = pos[r * B + b], p = j / g;
            for (int i = 0; i < n; ++i) {
                int64_t k = b * m + pat[p * n + i];
                double v = elem(dtype, values, ldv, c * S + j, b * n + i);
                for (int64_t t = 0; t < N; ++t) {
                    double x = elem(dtype, X, ldx, k, t);
                    yr[t] += v * x;
                    br[t] += fabs(v) * fabs(x);
                }
            }
        }
    }
    free(pos);
    return ORC_OK;
}

/* The paper's GPU converter (Section 5.2) as a refinement of a packing: the
 * blocks of a chunk hold patterns; a swap of the patterns of two blocks with
 * different patterns is made when it raises the magnitude the pair keeps,
 * until no swap does.  The paper lets threads race for swaps; this reading
 * fixes an order.  In every round each row finds its best partner -- the
 * largest gain s(r,b) + s(r',a) - s(r,a) - s(r',b) > 0, sums in binary64 of
 * the binary32 magnitudes, ties to the lower partner row; every pair of
 * mutual best partners swaps.  (Gains are symmetric, so while any swap
 * improves there is a mutual pair: the lowest row of a pair with the largest
 * gain and its lowest such partner.)  Rounds end when no swap improves, or
 * after 8 * S rounds.  The
 * result is stored like nmg_p_compress's (patterns in order, rows of a group
 * ascending), values copied from W. */
static double p_gain(const float *sc, int64_t P, int r, int a, int q, int b)
{
    return ((double)sc[r * P + b] + (double)sc[q * P + a]) -
           ((double)sc[r * P + a] + (double)sc[q * P + b]);
}

int oracle_p_refine(int dtype, int64_t M, int64_t K, int n, int m, int g, const void *W,
                    int64_t ldw, void *values, uint8_t *index, int *rounds_out)
{
    int64_t P, S;
    int st = check_p_layout(dtype, M, K, n, m, g, &P, &S);
    if (st != ORC_OK)
        return st;
    if (ldw < K)
        return ORC_EPARAM;
    int64_t B = K / m, ldv = B * n;
    st = check_p_index(M, B, S, index);
    if (st != ORC_OK)
        return st;
    uint8_t pat[256 * 255];
    revolving_door(m, n, pat);
    float *sc = (float *)malloc(sizeof(float) * (size_t)(S * P));
    int max_rounds = 0;
    for (int64_t c = 0; c < M / S; ++c)
        for (int64_t b = 0; b < B; ++b) {
            for (int64_t r = 0; r < S; ++r)
                for (int64_t p = 0; p < P; ++p) {
                    float s = 0.0f;
                    for (int i = 0; i < n; ++i)
                        s = s + abs_elem32(dtype, W, ldw, c * S + r, b * m + pat[p * n + i]);
                    sc[r * P + p] = s;
                }
            int pa[256], best[256];
            double bg[256];
            for (int64_t j = 0; j < S; ++j)
                pa[index[(c * S + j) * B + b]] = (int)(j / g);
            int round = 0;
            for (; round < 8 * S; ++round) {
                int any = 0;
                for (int r = 0; r < S; ++r) {
                    best[r] = -1;
                    bg[r] = 0.0;
                    for (int q = 0; q < S; ++q) {
                        if (pa[q] == pa[r])
                            continue;
                        double gq = p_gain(sc, P, r, pa[r], q, pa[q]);
                        if (gq > bg[r]) { /* strictly larger: ties keep the lower q */
                            bg[r] = gq;
                            best[r] = q;
                        }
                    }
                    any |= best[r] >= 0;
                }
                if (!any)
                    break;
                int newpa[256];
                memcpy(newpa, pa, sizeof(int) * (size_t)S);
                for (int r = 0; r < S; ++r) {
                    int q = best[r];
                    if (q > r && best[q] == r) { /* mutual best partners: disjoint pairs */
                        newpa[r] = pa[q];
                        newpa[q] = pa[r];
                    }
                }
                memcpy(pa, newpa, sizeof(int) * (size_t)S);
            }
            if (round > max_rounds)
                max_rounds = round;
            int64_t j = 0;
            for (int64_t p = 0; p < P; ++p)
                for (int64_t r = 0; r < S; ++r)
                    if (pa[r] == p) {
                        index[(c * S + j) * B + b] = (uint8_t)r;
                        for (int i = 0; i < n; ++i)
                            copy_elem(dtype, values, ldv, c * S + j, b * n + i, W, ldw, c * S + r,
                                      b * m + pat[p * n + i]);
                        ++j;
                    }
        }
    free(sc);
    if (rounds_out)
        *rounds_out = max_rounds;
    return ORC_OK;
}
