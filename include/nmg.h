/*
 * nmg.h -- C ABI of the grouped n:m (n:m:g) sparse-weight library for AMD
 * Instinct MI355X (gfx950).
 *
 * Paper: STen (arXiv 2304.07613), Section 5 "Grouped n:m Sparsity".
 *
 * LAYOUT (Section 5, opening paragraph: the n:m nonzero pattern is repeated
 * over the g rows of a group).  A dense weight W is M x K, row-major, with
 * leading dimension ldw >= K (elements).  Along K it is cut into
 * C = ceil(K / m) chunks of m consecutive columns; the last chunk has width
 * r = K - (C - 1) * m and must satisfy r >= n.  Rows [G*g, G*g + g) form group
 * G (M must be a multiple of g).  Inside every chunk all rows of a group keep
 * the same n columns.
 *
 *   values  : M x (C*n) elements of the layout's type, row-major, contiguous.
 *             values[r*(C*n) + c*n + s] is the s-th kept weight of row r in
 *             chunk c.
 *   indices : (M/g) x (C*n) bytes, row-major, contiguous.
 *             indices[G*(C*n) + c*n + s] is the in-chunk offset o of that
 *             weight (absolute column c*m + o); the n offsets of a chunk are
 *             strictly ascending.
 *
 * SELECTION (Section 5.2: the converter keeps the n:m:g-valid tensor of
 * largest L1 norm).  Groups and chunks do not constrain one another, so the
 * optimum keeps, per (group, chunk), the n columns of largest group score
 *     score[j] = |W[G*g][c*m+j]| + |W[G*g+1][c*m+j]| + ... + |W[G*g+g-1][c*m+j]|
 * summed in binary32 in that row order, starting from +0 (binary16 weights
 * are widened exactly first; no flush of subnormals).  Equal scores go to the
 * lower offset; a NaN score orders above every number and NaNs tie.
 *
 * PRODUCT (Section 5.1, the sparse x dense GEMM): Y = W_s * X, where W_s is
 * the dense matrix the layout represents, X is K x N (row-major, leading
 * dimension ldx >= N) and Y is M x N (row-major, leading dimension ldy >= N).
 * Accumulation is binary32; binary16 outputs are rounded to nearest even.
 *
 * CONVENTIONS FOR EVERY CALL
 *   - All data pointers are device pointers (HIP global memory) of the current
 *     device.  The caller allocates and owns every buffer; the library keeps
 *     no pointer after a call returns.  The only device memory it allocates
 *     is the scratch memory of three product families (NMG_KERNEL_MFMA_WIDE /
 *     _SPLIT and NMG_KERNEL_MFMA_EXPAND, the last also an NMG_KERNEL_AUTO
 *     choice), allocated and freed in stream order on the call's stream;
 *     nmg_spmm_epilogue_noalloc uses a fixed per-GPU array instead.
 *   - Work is enqueued on `stream` (0 = the null stream) and runs
 *     asynchronously; a call returns after validation and launch.  Calls are
 *     thread-safe (nmg_spmm_epilogue_noalloc: see there).  The only mutable
 *     global state is host-side tables filled once and never changed: the
 *     compute-unit count per device and the resident-workgroup count per
 *     (device, kernel, workgroup size), which pick launch shapes, and the
 *     address of each device's fixed scratch array.  Each entry is filled on
 *     first use under a lock, so a call's launch shape -- and with it the
 *     order of its sums and its output bits -- depends only on its arguments
 *     and the device, whichever thread makes it.
 *   - Launch failures are read with hipGetLastError right after the launch;
 *     an error that earlier runtime calls left pending on the calling thread
 *     is cleared first (and not reported by this library).
 *   - Arguments are validated on the host before anything is launched; on an
 *     error nothing is enqueued and no output is written.
 *   - Floating-point inputs must be finite for the product; the selection is
 *     defined for every input, NaN included.
 */
#ifndef NMG_H
#define NMG_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum nmg_status {
    NMG_OK = 0,
    NMG_ERR_NULL = 1,        /* a required pointer is NULL                     */
    NMG_ERR_PARAM = 2,       /* n, m, g, a size or a leading dimension invalid */
    NMG_ERR_SHAPE = 3,       /* M % g != 0, or the tail chunk is narrower than n */
    NMG_ERR_DTYPE = 4,       /* unknown element type                           */
    NMG_ERR_ALIGN = 5,       /* a pointer or leading dimension is misaligned   */
    NMG_ERR_LAUNCH = 6,      /* the HIP runtime reported an error on launch    */
    NMG_ERR_UNSUPPORTED = 7, /* the requested kernel cannot run this layout    */
    NMG_ERR_CAPACITY = 8     /* a fixed-size working buffer is too small for
                                the layout                                    */
} nmg_status;

typedef enum nmg_dtype {
    NMG_F32 = 0,             /* IEEE binary32 */
    NMG_F16 = 1              /* IEEE binary16 (accumulation stays binary32) */
} nmg_dtype;

/* Shape of one n:m:g weight.  Fill it with nmg_layout_init. */
typedef struct nmg_layout {
    int32_t M, K;            /* dense weight is M x K                   */
    int32_t n, m, g;         /* n kept of every m columns, g rows/group */
    int32_t C;               /* number of chunks, ceil(K / m)           */
    nmg_dtype dtype;         /* element type of W, values, X and Y      */
} nmg_layout;

/* Kernel family for the product (the choice is recorded, not guessed). */
typedef enum nmg_kernel {
    NMG_KERNEL_AUTO = 0,         /* the library's choice for this layout       */
    NMG_KERNEL_VALU = 1,         /* vector-ALU FMA; runs every valid layout     */
    NMG_KERNEL_MFMA = 2,         /* the best binary32 matrix-core kernel below
                                    that takes this layout                      */
    NMG_KERNEL_MFMA_GENERAL = 3, /* matrix cores on the gathered g x n sub-tiles;
                                    needs g % 4 == 0 and a window of 2..16
                                    k-slots (a power of two that n divides)
                                    whose chunks fit its staging buffer         */
    NMG_KERNEL_MFMA_SCALAR = 4,  /* the same product with the index words of a
                                    window moved to scalar registers and wider
                                    token tiles; additionally needs n a power of
                                    two and a window of 4..16 k-slots          */
    NMG_KERNEL_MFMA_F16 = 5,     /* binary16 layouts on the binary16 matrix
                                    cores, 4 k-slots per instruction (binary32
                                    accumulation); needs g % 4 == 0, n a power
                                    of two, the chunks of max(4, n) k-slots
                                    within 512 staged X rows (m <= 128 for
                                    n <= 4), X and ldx on 16-byte boundaries
                                    and N % 8 == 0                            */
    NMG_KERNEL_MFMA_DIRECT = 6,  /* binary32 matrix cores fed by gathering each
                                    group's selected X rows straight from
                                    global memory (no staging of whole
                                    windows), with the k-slots split over the
                                    waves of a workgroup when the layer alone
                                    cannot fill the GPU; needs g % 4 == 0 and
                                    n a power of two                          */
    NMG_KERNEL_SMFMAC_F16 = 7,   /* binary16 layouts on gfx950's sparse matrix
                                    instruction (2 stored of every aligned 4
                                    columns): X read as contiguous rows, no
                                    gather; needs n in {1, 2}, m in {4, 8,
                                    16}, C * n % 8 == 0, values, indices, X and
                                    ldx on 16-byte boundaries, N % 8 == 0     */
    NMG_KERNEL_VALU_STAGED = 8,  /* vector-ALU FMA on X windows staged in LDS
                                    (the choice for binary32 layouts the
                                    grouped matrix-core kernels decline when m
                                    > 8 n); needs binary32, m <= 32, n <= 16,
                                    X and ldx on 16-byte boundaries, N % 4 == 0 */
    NMG_KERNEL_MFMA_WIDE = 9,    /* binary16 layouts on the 16 x 16 x 32
                                    binary16 matrix instruction (32 gathered
                                    k-slots of a group per instruction, binary32
                                    accumulation) from prepared operands: made
                                    on every call by nmg_spmm_with, once per
                                    weight with nmg_x16_prepare +
                                    nmg_spmm_x16; the layouts and arguments
                                    nmg_spmm_x16 takes                        */
    NMG_KERNEL_MFMA_SPLIT = 10,  /* binary32 layouts on the same binary16
                                    instruction, each operand carried as two
                                    binary16 parts (see nmg_spmm_x16)         */
    NMG_KERNEL_MFMA_EXPAND = 11  /* the matrix cores for groups they cannot
                                    share (g % 4 != 0, n not a power of two):
                                    W_s written out dense (zeros elsewhere)
                                    into scratch memory (M K elements + K
                                    bytes, stream-ordered on every call), then
                                    multiplied as one dense group by the
                                    MFMA_SCALAR kernel -- m / n times the
                                    useful work, and a non-finite X entry
                                    reaches every output of its token, as in a
                                    dense product; needs M % 4 == 0 and
                                    M K < 2^31                               */
} nmg_kernel;
/* With n == m every column is kept and every index row is 0 .. m-1, so the
 * matrix-core kernels treat the weight as one group whatever g is. */

/* Checks 1 <= n <= m <= 255, g >= 1, M >= 1, K >= 1 (NMG_ERR_PARAM),
 * M % g == 0 and tail width >= n (NMG_ERR_SHAPE), a known dtype
 * (NMG_ERR_DTYPE), and fills *layout (C included).  Pure host code. */
nmg_status nmg_layout_init(nmg_layout *layout, int32_t M, int32_t K, int32_t n,
                           int32_t m, int32_t g, nmg_dtype dtype);

/* Element count of `values` (M * C * n) and byte count of `indices`
 * ((M / g) * C * n); -1 for an invalid layout.  Pure host code. */
int64_t nmg_values_numel(const nmg_layout *layout);
int64_t nmg_indices_numel(const nmg_layout *layout);

/* Dense -> n:m:g (Section 5.2, the L1-maximising converter, here exact).
 * W: M x K, leading dimension ldw >= K, element-aligned.  Writes every entry
 * of values (a bit copy of the kept weights, sign of zero included) and of
 * indices. */
nmg_status nmg_compress(const nmg_layout *layout, const void *W, int64_t ldw,
                        void *values, uint8_t *indices, hipStream_t stream);

/* Fixed-mask repack (Section 5.3: the sparsifier that keeps a tensor's
 * existing format, used when updated weights are sparsified again): values
 * get W's entries at the positions `indices` selects, a bit copy; indices are
 * only read.  W: M x K, leading dimension ldw >= K, element-aligned.  Indices
 * must hold n strictly ascending in-chunk offsets per (group, chunk); other
 * contents give unspecified values, but no read leaves W's row. */
nmg_status nmg_repack(const nmg_layout *layout, const void *W, int64_t ldw,
                      const uint8_t *indices, void *values, hipStream_t stream);

/* Y = W_s * X (Section 5.1).  X: K x N, leading dimension ldx; Y: M x N,
 * leading dimension ldy; N >= 1, ldx >= N, ldy >= N; values, X and Y aligned
 * to their element size (NMG_ERR_ALIGN).  X rows that start on 16-byte (fp32)
 * or 8-byte (fp16) boundaries are read with vector loads; other X is read
 * element by element, more slowly.  `indices` must hold n
 * strictly ascending in-chunk offsets per (group, chunk), as nmg_compress
 * writes them; other contents are not detected and give unspecified Y (the
 * kernels still never read outside X's K rows).  Uses NMG_KERNEL_AUTO, which
 * takes NMG_KERNEL_MFMA_EXPAND (scratch memory in stream order, dense-product
 * treatment of non-finite X) for binary32 layouts the grouped matrix-core
 * kernels cannot take when m <= 8 n. */
nmg_status nmg_spmm(const nmg_layout *layout, const void *values,
                    const uint8_t *indices, const void *X, int64_t ldx,
                    int64_t N, void *Y, int64_t ldy, hipStream_t stream);

/* nmg_spmm with an explicit kernel family; NMG_ERR_UNSUPPORTED when that
 * family cannot run this layout.  NMG_KERNEL_MFMA_WIDE / _SPLIT (prepared
 * operands) and NMG_KERNEL_MFMA_EXPAND (the dense weight) keep their scratch
 * memory in device memory allocated and freed in stream order on `stream`
 * (hipMallocAsync / hipFreeAsync; NMG_ERR_LAUNCH when the allocation fails). */
nmg_status nmg_spmm_with(const nmg_layout *layout, nmg_kernel kernel,
                         const void *values, const uint8_t *indices,
                         const void *X, int64_t ldx, int64_t N, void *Y,
                         int64_t ldy, hipStream_t stream);

/* What happens to the product before it is stored (the glue of a BERT
 * encoder block folded into the product; not part of the paper's format).
 * P is W_s * X rounded to the element type, exactly what nmg_spmm writes. */
typedef enum nmg_epilogue {
    NMG_EPILOGUE_NONE = 0,   /* Y = P                                      */
    NMG_EPILOGUE_GELU = 1,   /* Y = GELU(P), as nmg_gelu computes it        */
    NMG_EPILOGUE_ADD = 2     /* Y = P + R, as nmg_add computes it           */
} nmg_epilogue;

/* nmg_spmm_with followed by an epilogue; the result equals nmg_spmm_with
 * followed by nmg_gelu or nmg_add bit for bit.  NMG_KERNEL_MFMA_F16 and
 * NMG_KERNEL_SMFMAC_F16 apply the epilogue in the product kernel (no second pass over Y), and so
 * do NMG_KERNEL_MFMA_WIDE / _SPLIT for ADD when R and ldr sit on 16-byte
 * boundaries and NMG_KERNEL_MFMA_WIDE for GELU where nmg_spmm_x16_epilogue
 * folds it in; the other cases run the elementwise kernel on Y afterwards.  R (ADD only; ignored
 * otherwise, may be NULL) is M x N with leading dimension ldr >= N, the
 * layout's element type, element-aligned, and must not overlap Y. */
nmg_status nmg_spmm_epilogue(const nmg_layout *layout, nmg_kernel kernel, nmg_epilogue epilogue,
                             const void *values, const uint8_t *indices, const void *X,
                             int64_t ldx, int64_t N, const void *R, int64_t ldr, void *Y,
                             int64_t ldy, hipStream_t stream);

/* nmg_spmm_epilogue for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): same arguments, same results bit for bit, and no allocation.
 * The families with scratch memory (NMG_KERNEL_MFMA_WIDE / _SPLIT, their
 * prepared operands; NMG_KERNEL_MFMA_EXPAND, chosen explicitly or by
 * NMG_KERNEL_AUTO, the dense weight) keep it in a fixed 16 MiB array in
 * device memory instead of a stream-ordered allocation (one array per GPU,
 * held until the process ends; NMG_ERR_CAPACITY for a layout whose scratch
 * memory -- nmg_x16_prepared_bytes, or M K elements + K bytes -- exceeds it).  Every call on
 * a GPU shares that GPU's array: calls that overlap on one GPU (from several
 * threads or on several streams) race, so serialise them.  `stream` must
 * belong to the current device (NMG_ERR_PARAM).  The other families use no
 * scratch memory and run exactly as in nmg_spmm_epilogue. */
nmg_status nmg_spmm_epilogue_noalloc(const nmg_layout *layout, nmg_kernel kernel,
                                     nmg_epilogue epilogue, const void *values,
                                     const uint8_t *indices, const void *X, int64_t ldx,
                                     int64_t N, const void *R, int64_t ldr, void *Y,
                                     int64_t ldy, hipStream_t stream);

/* The kernel family NMG_KERNEL_AUTO picks for this layout and N, assuming
 * 16-byte aligned X, 4-byte aligned indices and ldx = N (never
 * NMG_KERNEL_MFMA; NMG_KERNEL_AUTO only for an invalid layout). */
nmg_kernel nmg_spmm_auto_kernel(const nmg_layout *layout, int64_t N);

/* ------------------------------------------------------------------------
 * THE 16 x 16 x 32 PRODUCTS (Section 5.1's product on gfx950's
 * v_mfma_f32_16x16x32_f16; families NMG_KERNEL_MFMA_WIDE and
 * NMG_KERNEL_MFMA_SPLIT).  One instruction contracts 32 gathered k-slots of a
 * group for 16 tokens; its per-window operands -- each lane's weight fragment
 * and the in-chunk offsets of the X rows it reads -- are arranged once per
 * packed weight ("prepared operands", a pure function of values and indices)
 * and then reused by every product with that weight.
 *
 * Layouts taken: n in {1, 2}; g % 8 == 0; the staging of one window (32
 * k-slots = 32 / n chunks of m X rows, 128 tokens per row) within the LDS
 * buffers: binary16 needs m % 4 == 0 and (32 / n) (256 m + 32) <= 53248
 * (m = 4 at n = 1; m = 4, 8 or 12 at n = 2); binary32 needs (32 / n) (512 m +
 * 32) <= 81920 and m <= 8 (m <= 4 at n = 1, m <= 8 at n = 2); M * C * n <
 * 2^31.
 *
 * Binary32 (MFMA_SPLIT) is not binary32 arithmetic: every weight w (scaled by
 * a power of two per 8 rows that puts the largest |w| of those rows into
 * [2^13, 2^14)) is carried as hi = fp16(w), lo = fp16(w - hi), every X entry
 * x as hi = fp16(x), lo = fp16((x - hi) 2^11), and all four products of the
 * parts are summed in binary32 (the products with x's lo part against weight
 * parts scaled by 2^-11); the output is scaled back exactly.  Per output,
 * |Y - W_s X| is at most about 2^-21 B + 2^-36 sum_k |w_k| + 2^-37 w_max
 * sum_k |x_k| + (binary32 summation error), B = sum_k |w_k x_k| over the
 * kept k and w_max the largest |w| of the output's 8-row block, for finite X
 * with |x| < 65504 -- within the 1e-5 B of the binary32 families unless
 * nearly all of B comes from a few k.  NMG_KERNEL_AUTO never chooses it.
 */

/* Bytes of the prepared operands of a layout; -1 for an invalid layout or one
 * these products do not take.  Pure host code. */
int64_t nmg_x16_prepared_bytes(const nmg_layout *layout);

/* Prepared operands from a packed weight (values, indices as nmg_compress
 * writes them; binary16 layouts give MFMA_WIDE operands, binary32 MFMA_SPLIT
 * operands).  `prepared` (device, 16-byte aligned, nmg_x16_prepared_bytes
 * long) is written whole; values and indices are only read.
 * NMG_ERR_UNSUPPORTED for a layout these products do not take. */
nmg_status nmg_x16_prepare(const nmg_layout *layout, const void *values, const uint8_t *indices,
                           void *prepared, hipStream_t stream);

/* Y = W_s X from prepared operands.  X: K x N, leading dimension ldx; Y: M x
 * N, leading dimension ldy; layout dtype for both.  Needs X and ldx on 16-byte
 * boundaries, Y and ldy on 16-byte (binary32) / 8-byte (binary16) boundaries,
 * N % 4 == 0 (binary32) / N % 8 == 0 (binary16), K * ldx < 2^31; else
 * NMG_ERR_UNSUPPORTED. */
nmg_status nmg_spmm_x16(const nmg_layout *layout, const void *prepared, const void *X,
                        int64_t ldx, int64_t N, void *Y, int64_t ldy, hipStream_t stream);

/* nmg_spmm_x16 with an epilogue, bit for bit what nmg_spmm_x16 followed by
 * nmg_add / nmg_gelu gives (P the product rounded to the element type):
 * NMG_EPILOGUE_NONE (= nmg_spmm_x16), NMG_EPILOGUE_ADD (Y = P + R; R is M x
 * N, leading dimension ldr >= N, 16-byte aligned with ldr a multiple of 16
 * bytes, else NMG_ERR_UNSUPPORTED, and must not overlap Y, else
 * NMG_ERR_PARAM; added as the outputs are stored) or NMG_EPILOGUE_GELU
 * (looked up as the outputs are stored for binary16 layouts whose tile
 * leaves room in LDS for the table -- units of 8 rows, and of 16 rows at
 * most 2 per wave -- else a second pass over Y). */
nmg_status nmg_spmm_x16_epilogue(const nmg_layout *layout, const void *prepared,
                                 nmg_epilogue epilogue, const void *X, int64_t ldx, int64_t N,
                                 const void *R, int64_t ldr, void *Y, int64_t ldy,
                                 hipStream_t stream);

/* n:m:g -> dense (end of Section 5.2): W_out (M x K, leading dimension
 * ldw >= K) gets the kept weights at their columns and +0 elsewhere. */
nmg_status nmg_densify(const nmg_layout *layout, const void *values,
                       const uint8_t *indices, void *W_out, int64_t ldw,
                       hipStream_t stream);

/* Elementwise glue between the layers of a linear stack (not in the paper's
 * format; BERT's encoder block).  `count` elements, contiguous, same dtype.
 *   nmg_gelu: out = 0.5 x (1 + erf(x / sqrt 2)).  binary16: looked up in a
 *             table of every binary16 input, built from a binary64 evaluation
 *             rounded to nearest even (NaN and -inf give NaN, +inf gives
 *             +inf).  binary32: evaluated in binary32 as 0.5 x erfc(-x / sqrt 2)
 *             (no cancellation for negative x).
 *   nmg_add : out = a + b, computed in binary32 (exactly rounded for
 *             binary16 operands).
 * In-place use (out == in / out == a) is allowed. */
nmg_status nmg_gelu(nmg_dtype dtype, const void *in, void *out, int64_t count,
                    hipStream_t stream);
nmg_status nmg_add(nmg_dtype dtype, const void *a, const void *b, void *out,
                   int64_t count, hipStream_t stream);

/* ------------------------------------------------------------------------
 * THE PAPER'S CHUNKED LAYOUT (Section 5, read literally).  Besides sharing a
 * pattern over a group, blocks are combined into chunks that use every one of
 * the P = C(m, n) patterns exactly g times, in revolving-door order (adjacent
 * patterns differ in one position), and the blocks of a chunk are reordered
 * by pattern with an index recording each block's row.
 *   block   : m consecutive weights of a row along K (K % m == 0 required);
 *   chunk   : the S = P * g blocks of S consecutive rows in one block column
 *             (M % S == 0, S <= 256, P <= 256 required);
 *   values  : M x (B * n), B = K / m; row c*S + j of chunk row-set c holds, in
 *             block column b, the kept weights of the block at position j,
 *             which uses pattern j / g (positions in pattern order, the rows of
 *             a group ascending);
 *   index   : M x B bytes; index[c*S + j][b] is the chunk row (0 .. S-1) of
 *             the block at position j of block column b.
 * nmg_p_compress follows the paper's CPU converter (Section 5.2): every
 * (row, pattern) pair of a chunk is scored by the magnitude the pattern keeps
 * (binary32, the pattern's offsets ascending, binary16 widened exactly), and
 * pairs are taken from the largest down -- NaN above every number, equal
 * scores to the lower pattern, then the lower row -- when the row has no
 * pattern yet and the pattern has fewer than g rows.  A heuristic: it need not
 * reach the largest kept magnitude.  The product and the conversion back follow
 * the layout.  NMG_ERR_UNSUPPORTED when a chunk does not fit the kernels'
 * LDS: S * P <= 8192, S * m <= 8192, P * n <= 4096. */
typedef struct nmg_p_layout {
    int32_t M, K;            /* dense weight is M x K                      */
    int32_t n, m, g;
    int32_t P, S, B;         /* patterns, rows per chunk, block columns    */
    nmg_dtype dtype;
} nmg_p_layout;

/* Checks the parameters (NMG_ERR_PARAM), the shape rules above
 * (NMG_ERR_SHAPE) and the dtype, and fills *layout.  Pure host code. */
nmg_status nmg_p_layout_init(nmg_p_layout *layout, int32_t M, int32_t K, int32_t n,
                             int32_t m, int32_t g, nmg_dtype dtype);

/* Dense W (M x K, leading dimension ldw >= K, element-aligned) -> values and
 * index; writes every entry of both. */
nmg_status nmg_p_compress(const nmg_p_layout *layout, const void *W, int64_t ldw, void *values,
                          uint8_t *index, hipStream_t stream);

/* The swap search of the paper's GPU converter (Section 5.2), from the
 * packing `index` already holds (nmg_p_compress's, or any valid one): within a
 * chunk, blocks with different patterns exchange them when that raises the
 * magnitude the pair keeps.  The paper lets threads race; here each round
 * every row takes its best improving partner (the largest gain, sums of the
 * binary32 magnitudes in binary64, ties to the lower row) and mutual best
 * partners swap, until no swap improves or 8 * S rounds have run.  Rewrites
 * index (stored as nmg_p_compress stores it) and values (copied from W). */
nmg_status nmg_p_refine(const nmg_p_layout *layout, const void *W, int64_t ldw, void *values,
                        uint8_t *index, hipStream_t stream);

/* Y = W_s * X for the chunked layout (the product of Section 5 on this
 * layout): X K x N (ldx >= N), Y M x N (ldy >= N), element-aligned; binary32
 * accumulation (binary16 inputs widened exactly).  An index that is not a
 * permutation in every chunk column gives unspecified Y, but no read leaves
 * the buffers.  Uses NMG_KERNEL_AUTO. */
nmg_status nmg_p_spmm(const nmg_p_layout *layout, const void *values, const uint8_t *index,
                      const void *X, int64_t ldx, int64_t N, void *Y, int64_t ldy,
                      hipStream_t stream);

/* nmg_p_spmm with an explicit kernel:
 *   NMG_KERNEL_VALU  vector FMAs, each row's kept products in ascending column
 *                    order; every valid layout.
 *   NMG_KERNEL_MFMA  binary32 matrix cores on the blocks expanded to m values
 *                    (n / m of the products useful); m <= 32, else
 *                    NMG_ERR_UNSUPPORTED.
 *   NMG_KERNEL_AUTO  MFMA when 4 n >= m and m <= 32, else VALU.
 * Any other kernel: NMG_ERR_UNSUPPORTED.  Arguments as nmg_p_spmm. */
nmg_status nmg_p_spmm_with(const nmg_p_layout *layout, nmg_kernel kernel, const void *values,
                           const uint8_t *index, const void *X, int64_t ldx, int64_t N, void *Y,
                           int64_t ldy, hipStream_t stream);

/* Chunked layout -> dense W_out (M x K, leading dimension ldw >= K). */
nmg_status nmg_p_densify(const nmg_p_layout *layout, const void *values, const uint8_t *index,
                         void *W_out, int64_t ldw, hipStream_t stream);

/* Static description of a status code; never NULL. */
const char *nmg_status_str(nmg_status status);

/* Library version string, e.g. "nmg 0.1.0 gfx950". */
const char *nmg_version(void);

#ifdef __cplusplus
}
#endif

#endif /* NMG_H */
