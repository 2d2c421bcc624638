/*
 * us.h - C-ABI of the UnionSparse W4A4 IE-BME SpMM library for MI355X (gfx950).
 *
 * The library encodes a masked INT4 weight matrix into the paper's
 * Index-Efficient Bitmap Encoding (IE-BME, Section V-A), multiplies it on the
 * GPU by dense INT4 activations into INT32 (the kernel of Section VI,
 * "UnionSparse Kernel" algorithm), and accounts its bytes by the
 * Payload-to-Metadata Ratio (Eq. 1) and effective compute intensity (Eq. 2).
 *
 * Conventions for every call:
 *   - arguments are checked before any work; a negative us_status means
 *     nothing was written and nothing was launched;
 *   - device pointers are plain HIP device addresses owned by the caller;
 *   - a stream argument is a hipStream_t passed as void * (NULL = the null
 *     stream); GPU calls are asynchronous on that stream, never synchronise
 *     and never allocate device memory;
 *   - the only state the library keeps is a per-device cache (the compute-unit
 *     count, kernel attributes applied once); every call is thread-safe.
 */
#ifndef UNIONSPARSE_US_H
#define UNIONSPARSE_US_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    US_OK = 0,
    US_ERR_ARG = -1,     /* null pointer, bad option value, misaligned pointer */
    US_ERR_SHAPE = -2,   /* M % 16, K % 64, N outside [1, US_N_LIMIT], size limits */
    US_ERR_RANGE = -3,   /* a weight outside the signed INT4 range [-8, 7] */
    US_ERR_NOMEM = -4,   /* host allocation failed (encoder only) */
    US_ERR_DEVICE = -5,  /* the HIP launch reported an error */
    US_ERR_FORMAT = -6   /* encoded arrays are inconsistent with each other */
} us_status;

/* Fixed IE-BME geometry of the hot path (Section V-A; the LT size is given in
 * the caption of the encoding figure, R_A = C_A = 2 in every illustration). */
#define US_LT_H 16          /* H_L: rows of a local tile (LT)              */
#define US_LT_W 64          /* K_L: columns of an LT                       */
#define US_RA 2             /* R_A: area rows per LT                       */
#define US_CA 2             /* C_A: area columns per LT (Q = R_A C_A = 4)  */
#define US_WORDS_PER_LT 4   /* 8 x 32 union-mask bits = four 64-bit words  */
#define US_PAYLOAD_PAD 16   /* zero bytes after the payload                */
#define US_N_MAX 32         /* widest activation matrix of one kernel pass */
#define US_N_LIMIT 1024     /* widest activation matrix; N > US_N_MAX runs as
                               slabs of US_N_MAX columns, each streaming W */
#define US_K_MAX 130048     /* K bound: int32 headroom of the kernel's scaled sums */

/*
 * Host IE-BME matrix (Section V-A, "IE-BME Storage Layout").
 *
 * LT t = mb * (K/64) + kb covers rows [16 mb, 16 mb + 16) and columns
 * [64 kb, 64 kb + 64). Area q = a * 2 + c holds LT rows [8a, 8a + 8) and
 * columns [32c, 32c + 32). Union-mask bit (i, j), i < 8, j < 32, is set when
 * any area is nonzero at (i, j); it is bit (32 i + j) % 64 of word
 * 4 t + (32 i + j) / 64 of `bitmaps`. offsets[t] = sum over tau < t of 4 P_tau
 * (P = active union-mask bits), in INT4 values, with offsets[n_lt] the total.
 * Payload: area q = 2 a + c's value at (i, j), for every active (i, j) of
 * rank rho (its place among the LT's active bits, row-major), is value
 * o_t + 4 a P_t + 2 rho + c: the two areas of an area row alternate by rank,
 * so one read at a rank fetches both. (The paper lists each area's values in
 * turn, o_t + q P_t + rho; the values of an LT, the offsets and the byte
 * count are the same.) Value n is the low nibble of byte n / 2 when n is
 * even, the high nibble when odd, in two's complement.
 *
 * With bits = 2 (W2A4, us_encode_w2) the weights are signed 2-bit values in
 * [-2, 1] and payload value n sits at bits 2 (n mod 4) .. 2 (n mod 4) + 1 of
 * byte n / 4; the bitmaps, the offsets (still counted in values) and the
 * value order are those of the 4-bit format.
 *
 * Row reordering (Section V-B) is recorded in `perm`. When it is NULL the
 * LTs keep their row order. Otherwise bits 4p .. 4p + 3 of perm[t] hold
 * pi_t[p], the row of LT t that was moved to row p before encoding. The
 * bitmaps, offsets and payload then describe the reordered LTs: rows
 * pi_t[i] and pi_t[8 + i] of the original LT share union-mask row i.
 *
 * The arrays are allocated by us_encode / us_encode_reordered and freed by
 * us_iebme_free.
 */
typedef struct {
    int32_t M, K;                 /* weight matrix is M x K                 */
    int32_t lt_h, lt_w, ra, ca;   /* 16, 64, 2, 2                           */
    int64_t n_lt;                 /* (M/16) * (K/64)                        */
    int64_t nnz;                  /* nonzero weights                        */
    int64_t n_payload;            /* stored INT4 values = offsets[n_lt]     */
    int64_t payload_bytes;        /* ceil(n_payload bits / 8) + US_PAYLOAD_PAD */
    uint64_t *bitmaps;            /* n_lt * 4 words                         */
    uint32_t *offsets;            /* n_lt + 1 entries                       */
    uint8_t *payload;             /* payload_bytes bytes, zeroed padding    */
    uint64_t *perm;               /* NULL, or n_lt row permutations         */
    int32_t bits;                 /* bits per payload value: 4, or 2 (W2A4) */
} us_iebme;

/*
 * us_encode - IE-BME encoding of a masked INT4 matrix (Section V-A: area
 * partitioning, shared union mask, the three storage arrays).
 *   w    : host int8, M rows of `ldw` elements, values in [-8, 7], 0 = pruned
 *   M, K : M % 16 == 0, K % 64 == 0, M * K < 2^32
 *   ldw  : row stride of w in elements, >= K
 *   out  : filled on success; on error it is left untouched
 * Returns US_ERR_ARG, US_ERR_SHAPE, US_ERR_RANGE or US_ERR_NOMEM on failure.
 */
us_status us_encode(const int8_t *w, int32_t M, int32_t K, int64_t ldw, us_iebme *out);

/*
 * us_encode_w2 - IE-BME encoding of a masked signed 2-bit matrix, the W2A4
 * setting of the evaluation (Section VII): as us_encode, with weights in
 * [-2, 1] (US_ERR_RANGE otherwise) packed four to a byte; out->bits = 2.
 */
us_status us_encode_w2(const int8_t *w, int32_t M, int32_t K, int64_t ldw, us_iebme *out);

/*
 * us_encode_reordered - bitmap-aware row reordering followed by IE-BME
 * (Section V-B, then Section V-A). Each LT's 16 rows are split into 8 pairs
 * that activate the fewest union-mask entries in total (Eq. 3-5, solved
 * exactly by the grouped subset DP). The result is deterministic:
 *   - ties keep the first optimal partner, in increasing row order, of the
 *     smallest remaining row;
 *   - the pairs are sorted, and pi_t lists the first rows of all pairs,
 *     then the second rows (the canonical permutation of Section V-B).
 * Same arguments and errors as us_encode; `out->perm` is allocated. Offline
 * work: about 20 us of one CPU thread per LT, spread over all threads.
 */
us_status us_encode_reordered(const int8_t *w, int32_t M, int32_t K, int64_t ldw, us_iebme *out);

/* us_iebme_free - release the arrays of an encoded matrix and zero it. */
void us_iebme_free(us_iebme *m);

/*
 * Byte accounting of an encoded matrix (Section III-B, Eq. 1; Section III-C,
 * Eq. 2). Metadata is bitmaps (32 B per LT) plus offsets (4 B per LT; the
 * sentinel is not counted). B_w = bits / 8 bytes per weight.
 */
typedef struct {
    int64_t nnz;                  /* nonzero weights                           */
    int64_t stored_values;        /* n_payload: nnz plus zeros of active groups */
    int64_t n_lt;
    int64_t payload_stored_bytes; /* ceil(stored_values bits / 8)              */
    int64_t bitmap_bytes;         /* 32 n_lt                                   */
    int64_t offset_bytes;         /* 4 n_lt                                    */
    int64_t meta_bytes;           /* Stor_meta of Eq. 1                        */
    double payload_useful_bytes;  /* B_w * nnz                                 */
    double pmr;                   /* Eq. 1: payload_useful_bytes / meta_bytes  */
    double pmr_stored;            /* stored payload bytes / meta_bytes         */
    double ci_eff;                /* Eq. 2 for activation width N, as printed  */
    int64_t perm_bytes;           /* 8 n_lt with row reordering, else 0; not
                                     part of Stor_meta (Eq. 1 predates it)     */
} us_pmr_report;

/*
 * us_pmr - fill `out` for `m`; N > 0 also evaluates Eq. 2 (N = 0 leaves
 * ci_eff at 0). Checks that offsets agree with the bitmaps (US_ERR_FORMAT).
 */
us_status us_pmr(const us_iebme *m, int32_t N, us_pmr_report *out);

/*
 * Cross-format byte accounting (Section III-B, Eq. 1 and the PMR comparison
 * across precisions and formats; Section III-C, Eq. 2 and the roofline view).
 * For the sparsity pattern of an encoded matrix and a value width, each
 * format's metadata and payload bytes:
 *   US_FMT_DENSE       : every weight stored, no metadata;
 *   US_FMT_CSR         : nonzeros only, a 32-bit column index per nonzero and
 *                        M + 1 32-bit row pointers;
 *   US_FMT_AREA_BITMAP : every 8 x 32 area of every LT with its own 256-bit
 *                        bitmap and 32-bit payload offset (IE-BME with one
 *                        area per mask), nonzeros only;
 *   US_FMT_IEBME       : the union mask shared by Q = 4 areas (32 B + 4 B
 *                        per LT), payload with the zeros of active groups.
 */
typedef enum { US_FMT_DENSE = 0, US_FMT_CSR = 1, US_FMT_AREA_BITMAP = 2, US_FMT_IEBME = 3 } us_format;
#define US_NUM_FORMATS 4

typedef struct {
    int32_t format;               /* us_format                                   */
    int32_t value_bits;           /* 16, 8, 4 or 2: B_w = value_bits / 8         */
    int64_t meta_bytes;           /* Stor_meta of Eq. 1 (0 for dense)            */
    double payload_useful_bytes;  /* B_w NNZ (B_w M K for dense)                 */
    double payload_stored_bytes;  /* what the format stores as values            */
    double pmr;                   /* Eq. 1 (0 for dense: no metadata)            */
    double ci_eff;                /* Eq. 2 for N columns, as printed (dense: s = 0,
                                     no metadata term)                           */
    double total_bytes;           /* metadata + stored payload                   */
    double ci_stored;             /* Eq. 2's form on the bytes actually stored:
                                     2 NNZ N / (total_bytes + B_w N K), useful
                                     MACs only (dense: all M K)                  */
} us_format_report;

/*
 * us_pmr_formats - fill out[f] for every format f in us_format (in that
 * order) for the mask of `m` at `value_bits` bits per value (16, 8, 4, 2)
 * and N >= 1 activation columns. Host only. US_ERR_ARG for other widths or
 * N < 1; US_ERR_FORMAT as us_pmr.
 */
us_status us_pmr_formats(const us_iebme *m, int32_t value_bits, int32_t N, us_format_report out[US_NUM_FORMATS]);

/*
 * An IE-BME matrix whose three arrays the caller has copied to the GPU
 * (Section V-A, "IE-BME Storage Layout"). The arrays must be those an
 * us_encode* call produced (bitmaps and offsets consistent, offsets
 * non-decreasing and ending at n_payload); the GPU does not check them. For
 * arrays that are not, Y is unspecified, but every payload read stays inside
 * the payload array: the kernels clamp each slice's range to it.
 */
typedef struct {
    const uint64_t *bitmaps;      /* device, n_lt * 4 words, 8-byte aligned  */
    const uint32_t *offsets;      /* device, n_lt + 1 entries, 4-byte aligned */
    const uint8_t *payload;       /* device, ceil(n_payload bits / 8) + US_PAYLOAD_PAD bytes */
    int32_t M, K;
    int64_t n_lt, n_payload;
    const uint64_t *perm;         /* device, n_lt words, 8-byte aligned, or NULL
                                     (see us_iebme); words that are not
                                     permutations give unspecified Y       */
    int32_t bits;                 /* 4 (0 reads as 4) or 2; 2-bit matrices
                                     cannot be row-reordered (US_ERR_ARG)  */
} us_iebme_dev;

/* Most K blocks a row block's K range can be split into across workgroups. */
#define US_K_BLOCKS_MAX 64

/*
 * Launch options (all zero = automatic). The split-K of the paper's kernel
 * (Section VI-C, "UnionSparse Kernel" algorithm: a grid of split-K batches by
 * row tiles, each batch storing its partial tile to a reduction workspace,
 * then a reduction) is realised at two levels: the wavefronts of a workgroup
 * split one row block's K range and combine in LDS (split_k), and with
 * k_blocks > 1 several workgroups split it and combine through the workspace.
 */
typedef struct {
    int32_t split_k;  /* K slices per workgroup, one wavefront each:
                         0 = automatic, else 1, 2, 4, 8 or 16; halved
                         while it exceeds K / 64 (one LT per slice);
                         required with variant 3                         */
    int32_t variant;  /* payload staging: 0 = automatic, 1 = whole chunk,
                         2 = 4 KB ring (N <= 16 only), 3 = single pass:
                         each wavefront requests its whole slice at once
                         (N <= 16 only); a choice that fits no
                         configuration returns US_ERR_ARG                */
    int32_t chunk_lts; /* LTs per chunk: 0 = automatic, else 4, 8, 11 or
                         16 (4 or 8 when N > 16); with variant 3 the most
                         LTs per wavefront slice: 4, 8, 11, 16, 22 or 32;
                         for tuning and tests                            */
    int32_t k_blocks; /* workgroups per row block, each taking a
                         contiguous K block: 0 or 1 = one (no workspace),
                         2 .. US_K_BLOCKS_MAX with variant 3 only; needs
                         the workspace (us_spmm_workspace_size)          */
} us_spmm_opts;

/*
 * us_spmm_plan - the launch configuration us_spmm would use for this shape
 * and options on the current device (a 256-CU MI355X when no device is
 * visible), given a workspace: the paper's split-K (Section VI-C, the
 * "UnionSparse Kernel" algorithm's split-K batches) as K slices per
 * workgroup (one wavefront each) and, in k_blocks (may be NULL), K blocks
 * across workgroups; LTs per chunk or single-pass slice; and payload staging
 * (1 whole chunk, 2 ring, 3 single pass) of the first slab of
 * min(N, US_N_MAX) columns, for a matrix of `bits`-bit values (4 or 2) that
 * is row-reordered when `reordered` != 0 (its stages are larger). The
 * paper claims a shape-aware kernel selection (Section I, contributions)
 * without describing it; this is ours. Host only; for tuning and reporting.
 * Same argument errors as us_spmm; US_ERR_ARG if no configuration fits.
 */
us_status us_spmm_plan(int32_t M, int32_t K, int32_t N, int32_t bits, int32_t reordered, const us_spmm_opts *opts,
                       int32_t *split_k, int32_t *chunk_lts, int32_t *staging, int32_t *k_blocks);

/*
 * us_spmm_workspace_size - device workspace bytes us_spmm needs for this
 * shape and options: the reduction workspace of the paper's split-K
 * (Section VI-C, "UnionSparse Kernel" algorithm: StoreTile into the
 * ReductionWorkspace, then Reduction), used when a row block's K range is
 * split across workgroups (k_blocks > 1): 4 M min(N, 16) bytes of int32
 * accumulators, then 4 M / 16 bytes of tickets. 0 when no such split is
 * requested. The workspace must be zero-filled before its first use; every
 * call leaves it zero-filled again. Calls that may overlap (other streams,
 * other threads) need workspaces of their own.
 */
us_status us_spmm_workspace_size(int32_t M, int32_t K, int32_t N, const us_spmm_opts *opts,
                                 size_t *bytes);

/*
 * us_spmm - Y = W X on the GPU: W in IE-BME (device copy), X dense INT4,
 * INT32 accumulation (Section VI, "UnionSparse Kernel" algorithm: the kernel
 * takes the IE-BME matrix, the activations and a split-K count, and returns Y).
 *   w      : encoded matrix, device arrays; with w->perm the LTs are
 *            row-reordered (Section V-B) and Y is still in original row order;
 *            w->bits = 2 multiplies a W2A4 matrix
 *   x      : device, N x K row-major INT4, two values per byte along K
 *            (even k in the low nibble), 16-byte aligned
 *   N      : 1..US_N_LIMIT activation columns; beyond US_N_MAX (32) the
 *            call runs one pass per slab of 32 columns (the last one
 *            narrower), each with its own configuration and each reading W
 *            again: prefill-sized N at decode-kernel cost per slab
 *   y      : device int32, N x M row-major (y[n * M + m] = Y[m][n])
 *   scale  : device float32[M] or NULL; with it, y_f32[n * M + m] =
 *            fl32(fl32(Y[m][n]) * scale[m]) is written too (the dequant
 *            epilogue is not part of the paper)
 *   y_f32  : device float32, N x M row-major; NULL exactly when scale is NULL
 *   ws     : device workspace of ws_bytes, 4-byte aligned (may be NULL when
 *            us_spmm_workspace_size reports 0); see us_spmm_workspace_size
 *            for its contents between calls
 *   opts   : NULL for automatic choices
 *   stream : hipStream_t
 * Argument errors return before launch; a launch error returns US_ERR_DEVICE.
 * The call never allocates, clears memory or synchronises, so it can be
 * captured in a HIP graph. Call each shape once outside the capture first:
 * the first call of a kernel configuration on a device sets its LDS limit.
 */
us_status us_spmm(const us_iebme_dev *w, const uint8_t *x, int32_t N, int32_t *y,
                  const float *scale, float *y_f32, void *ws, size_t ws_bytes,
                  const us_spmm_opts *opts, void *stream);

/* Bytes of the array us_spmm_noalloc uses as its workspace. */
#define US_NOALLOC_SCRATCH_BYTES (4u << 20)

/*
 * us_spmm_noalloc - us_spmm for callers that cannot allocate device memory
 * or pass a workspace: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc. Same arguments, results and errors as
 * us_spmm, without ws / ws_bytes: the reduction workspace of a K range split
 * across workgroups (us_spmm_opts.k_blocks > 1) is a fixed array of
 * US_NOALLOC_SCRATCH_BYTES bytes inside the library, one per GPU, held until
 * the process ends. A split whose workspace (us_spmm_workspace_size) exceeds
 * it returns US_ERR_SHAPE before any launch; US_ERR_DEVICE if the array's
 * address cannot be obtained. The array is zero when the library is loaded
 * and every call leaves it zero again, so no call clears it. All calls on
 * one GPU share that GPU's array: calls that may overlap (several streams or
 * threads) race on it and must not be issued concurrently. The call itself
 * allocates nothing.
 */
us_status us_spmm_noalloc(const us_iebme_dev *w, const uint8_t *x, int32_t N, int32_t *y,
                          const float *scale, float *y_f32, const us_spmm_opts *opts, void *stream);

/*
 * us_gemm_i8 - dense INT8 GEMM, Y = W X with INT32 accumulation, on the int8
 * matrix cores: the in-library dense comparison point (the paper compares
 * against dense Tensor-Core GEMMs, Section VII-A "Baselines and Fairness").
 *   w : device int8, M x K row-major, 16-byte aligned
 *   x : device int8, N x K row-major (row n is activation column n), 16-byte aligned
 *   y : device int32, N x M row-major
 * M % 16 == 0, K % 64 == 0, K <= US_K_MAX, 1 <= N <= US_N_LIMIT (slabs of 32
 * columns beyond 32, as in us_spmm).
 */
us_status us_gemm_i8(const int8_t *w, const int8_t *x, int32_t M, int32_t K, int32_t N,
                     int32_t *y, void *stream);

/* us_status_string - static text naming a status code. */
const char *us_status_string(us_status s);

#ifdef __cplusplus
}
#endif

#endif /* UNIONSPARSE_US_H */
