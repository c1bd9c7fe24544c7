/*
 * nsd.h -- C ABI of libnsd, sparse tensor expressions and their gradients on
 * AMD MI355X (gfx950), keeping sparsity.
 *
 * The problem statement follows the paper's `gradient e x` (Section 4.3, the
 * gradient API figure): a sparse tensor, dense operands and an upstream
 * gradient go in; the loss and the gradients come out.  The gradient with
 * respect to a sparse operand lives only on that operand's stored keys,
 * because `onehot` iterates the stored keys alone; it is returned as a value
 * array aligned 1:1 with the operand's own storage order, so its pattern is
 * the input pattern by construction.  Gradients with respect to dense operands
 * are transposed sparse x dense products.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Pointers.  Every array argument is a DEVICE pointer unless the comment says
 *   "host".  The caller owns all memory; the library never allocates, never
 *   frees, and keeps no pointer after the call returns.
 * Outputs.  Destination-passing style (Section 5.5): outputs are caller
 *   buffers that are fully overwritten.  An output element that receives no
 *   contribution (an empty row or column, nnz = 0) is written as 0, the value
 *   of an empty sum.
 * Formats (the physical storage of Section 5.3).  Indices are int32, values
 *   fp32, dense operands row-major with leading dimension equal to their
 *   width k (element (i, c) at i * k + c).  A CSR holds unique keys sorted by
 *   (row, col); its `rowidx` is the row of every stored entry (the COO row
 *   array of the same order), produced by nsd_csr_expand_rows or
 *   nsd_coo_to_csr.  A CSC is the stable column order of a CSR plus `perm`,
 *   the CSR slot of every CSC slot.
 * Streams.  `stream` is a hipStream_t passed as void* (NULL: the default
 *   stream).  Hot-path calls are asynchronous on it: they only enqueue
 *   kernels (no copy, fill, allocation or synchronisation), so a sequence of
 *   them can be captured in a HIP graph and replayed.  Builders, validators
 *   and nsd_batax_jacobian synchronise it before returning, because they
 *   report counts or errors.
 * Workspace.  Calls that need scratch take `ws` (device, 256-byte aligned) and
 *   `ws_bytes`; the size queries say how much.  Contents need no initial value.
 * Errors.  The status is the return value; nothing is thrown across the ABI.
 *   Argument errors are detected before any launch and leave outputs
 *   untouched.  Malformed formats are detected only by the validators and
 *   builders; passing a malformed CSR/CSC to a hot-path call is undefined.
 *   nsd_last_error() gives a thread-local message for the last failure.
 * Determinism.  Every entry point is bitwise reproducible run to run: no
 *   floating-point atomics; every reduction has a fixed order.
 * Limits.  nnz and every dimension are < 2^31; dense offsets use 64-bit
 *   arithmetic.  Any k >= 1 works; k in {1, 32, 64, 128, 256} and other
 *   multiples of 4 up to 256 take the vector paths.
 */
#ifndef NSD_H
#define NSD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum nsd_status {
    NSD_OK = 0,
    NSD_ERR_INVALID_ARG = 1, /* null pointer, negative size, k < 1, ... */
    NSD_ERR_BAD_FORMAT = 2,  /* validator/builder: malformed indices */
    NSD_ERR_DUPLICATE = 3,   /* builder: duplicate coordinate under NSD_DUP_ERROR */
    NSD_ERR_TOO_LARGE = 4,   /* a size at or above 2^31 */
    NSD_ERR_WORKSPACE = 5,   /* ws_bytes below the queried size */
    NSD_ERR_UNSUPPORTED = 6,
    NSD_ERR_HIP = 7          /* a HIP runtime error; see nsd_last_error() */
} nsd_status;

/* Duplicate coordinates in a COO input: summed (the "+=" of a singleton
 * inserted inside a sum, Section 5.5) or rejected (the `unique` annotation of
 * the storage formats, Section 5.3). */
typedef enum nsd_dup_policy { NSD_DUP_SUM = 0, NSD_DUP_ERROR = 1 } nsd_dup_policy;

/*
 * Work plan of a sorted sparse operand (the rows of a CSR or the columns of a
 * CSC), built once per sparsity pattern by nsd_plan_build.  Entries are cut
 * into work items of about item_len (L) entries: a segment of at most
 * S = L + min(L, 32) entries is never split (consecutive ones are packed into
 * one item, at most L + S entries), a longer segment is cut into chunks of L
 * entries whose partial sums are added in chunk order afterwards, and empty
 * segments are listed for a zero fill.
 * It balances power-law segment lengths without atomics.  A long segment with
 * more than 64 chunks is "huge" (listed in huge_idx): the combine gives a whole
 * workgroup to each that still has more than 64 partial rows once the chunks
 * computed by one wave have been added together.  Chunk partials are kept in
 * a compact array with one row per chunk item (chunk_ord), so the scratch of
 * a reduction grows with the entries of long segments only.
 */
typedef struct nsd_plan {
    int32_t item_len;          /* L: entries per chunk; segments above
                                  L + min(L, 32) are long */
    int32_t nitems, nlong, nhuge, nchunks, nempty;
    const int32_t *item_ptr;   /* [nitems+1] first entry of every item; [nitems] = nnz */
    const int32_t *long_seg;   /* [nlong] segment id of every long segment */
    const int32_t *long_first; /* [nlong] first item of every long segment */
    const int32_t *huge_idx;   /* [nhuge] positions in the long lists of huge segments */
    const int32_t *chunk_item; /* [nchunks] every item that is a chunk of a long segment */
    const int32_t *chunk_ord;  /* [nitems] position of a chunk item in chunk_item (the
                                  row of its partial sum), -1 for other items */
    const int32_t *empty_seg;  /* [nempty] segments without entries */
    int32_t longest_chunks;    /* chunks of the longest segment (0: none is long) */
} nsd_plan;

/*
 * A fixed permutation of n values split into two coalesced passes
 * (nsd_permute_f32): dst[q] = src[perm[q]].  Built once per permutation by
 * nsd_perm_plan_build into three caller arrays of n elements.
 */
typedef struct nsd_perm_plan {
    int32_t n;                  /* elements */
    int32_t tile;               /* span of either pass (source tile, destination bucket) */
    const int32_t *stage;       /* [n] staging position of pass 1's output slot */
    const uint16_t *src_local;  /* [n] source index within its tile of that slot */
    const uint16_t *dst_local;  /* [n] destination offset within its bucket of staging slot */
} nsd_perm_plan;

/* Matrix CSR (Section 5.3, the matrix CSR storage `(len,pos,idx,val)`). */
typedef struct nsd_csr {
    int32_t nrows, ncols, nnz;
    const int32_t *rowptr; /* [nrows+1], rowptr[0] = 0, rowptr[nrows] = nnz */
    const int32_t *rowidx; /* [nnz], row of every entry, non-decreasing */
    const int32_t *colind; /* [nnz], strictly increasing within a row */
    const float *val;      /* [nnz] */
    nsd_plan plan;         /* plan over the rows (for reductions into rows) */
} nsd_csr;

/* Matrix CSC of the same matrix (Section 5.3: expressed like CSR). */
typedef struct nsd_csc {
    int32_t nrows, ncols, nnz;
    const int32_t *colptr; /* [ncols+1] */
    const int32_t *colidx; /* [nnz], column of every CSC slot, non-decreasing */
    const int32_t *rowind; /* [nnz], strictly increasing within a column */
    const int32_t *perm;   /* [nnz], CSR slot holding the same entry */
    nsd_plan plan;         /* plan over the columns (for reductions into columns) */
    /* Optional (n = 0: absent) two-pass forms of perm, built once per pattern
     * with nsd_perm_plan_build: to_csc moves values from CSR to CSC order
     * (valT[q] = val[perm[q]], inverse = 0), to_csr moves them back
     * (g[perm[q]] = gT[q], inverse = 1).  When both are present the column
     * pass of nsd_loss_bilinear reads A's values and writes its sparse
     * gradient in CSC order, moved by them, instead of one 4-byte access per
     * entry through perm; its workspace then holds 3 nnz more floats. */
    nsd_perm_plan to_csc, to_csr;
} nsd_csc;

/*
 * A COO 3-tensor seen through one mode n: its entries stably sorted by the
 * mode-n coordinate (nsd_coo_mode_index), with the other coordinates and the
 * values gathered into that order, and the work plan over the mode-n slices.
 * "Input order" is the order of the coordinate arrays the mode indexes were
 * built from.  Holding the tensor in lexicographic coordinate order (a stable
 * sort by the last coordinate, then each earlier one) makes mode 0's perm the
 * identity, so the gradient on X's keys is written sequentially.
 */
typedef struct nsd_coo3_mode {
    int32_t mode;          /* n in {0, 1, 2} */
    const int32_t *segptr; /* [dims[n]+1] */
    const int32_t *segidx; /* [nnz] mode-n coordinate, non-decreasing */
    const int32_t *idx_a;  /* [nnz] coordinate of mode (n+1) % 3 */
    const int32_t *idx_b;  /* [nnz] coordinate of mode (n+2) % 3 */
    const float *val;      /* [nnz] values in this order */
    const int32_t *perm;   /* [nnz] input position of every sorted entry */
    nsd_plan plan;         /* plan over the mode-n slices */
} nsd_coo3_mode;

/* Sparse 3-tensor (the order-3 `tensor` of Section 3) in its three mode orders. */
typedef struct nsd_coo3 {
    int32_t dims[3];
    int32_t nnz;
    nsd_coo3_mode mode[3];
} nsd_coo3;

/* Highest tensor order of the order-N entry points. */
#define NSD_MAX_ORDER 6

/*
 * Projection of a sparse order-N tensor X (3 <= N <= NSD_MAX_ORDER) along
 * one mode n, the layout of its mode-n products (nsd_ttv, nsd_ttm): X's
 * entries in lexicographic order of their other coordinates with the
 * distinct projected keys numbered (the keys of Y = X x_n U), and X's
 * entries in mode-n order, each view with its work plan.  Built by
 * nsd_ttv_build; the two plans by nsd_plan_build on yptr and lptr.  "l"
 * below is the mode-n coordinate.
 */
typedef struct nsd_ttv_plan {
    int32_t order;         /* N */
    int32_t mode;          /* n, the contracted mode */
    int32_t dims[NSD_MAX_ORDER];
    int32_t nnz, ny;       /* entries of X; distinct projected keys of Y */
    const int32_t *ykey[NSD_MAX_ORDER - 1];  /* [ny] coordinate of every key in
                                                each other mode (modes in
                                                increasing order), keys in
                                                lexicographic order */
    const int32_t *yptr;   /* [ny+1] entries of every key in the key-sorted order */
    const int32_t *yseg;   /* [nnz] key of every key-sorted entry */
    const int32_t *yperm;  /* [nnz] input position of every key-sorted entry */
    const int32_t *ykidx;  /* [nnz] l of every key-sorted entry */
    nsd_plan yplan;        /* plan over the keys */
    const int32_t *lptr;   /* [dims[mode]+1] entries of every l in the l-sorted order */
    const int32_t *lseg;   /* [nnz] l of every l-sorted entry, non-decreasing */
    const int32_t *lperm;  /* [nnz] input position of every l-sorted entry */
    const int32_t *lpair;  /* [nnz] key of every l-sorted entry */
    nsd_plan lplan;        /* plan over l */
} nsd_ttv_plan;


/* ----------------------------------------------------------------- info */

/* Static string naming a status code. */
const char *nsd_status_string(int status);
/* Thread-local detail message of this thread's last failing call ("" if none). */
const char *nsd_last_error(void);
/* Library ABI version (major * 10000 + minor * 100 + patch). */
int nsd_version(void);

/* ------------------------------------------------------- timing probe */

/* Kernels that a timing probe can bracket. */
typedef enum nsd_kernel_id {
    NSD_KERNEL_NONE = 0,
    NSD_KERNEL_SGR_MAIN = 1,   /* gather-reduce over a plan (SpMV/SpMM/A^T G) */
    NSD_KERNEL_SGR_FIX = 2,    /* long-segment combine */
    NSD_KERNEL_SDDMM = 3,      /* SDDMM over equal entry ranges */
    NSD_KERNEL_FROB_ROW = 4,   /* SpMM-gradient row pass */
    NSD_KERNEL_FROB_COL = 5,   /* SpMM-gradient column pass */
    NSD_KERNEL_MF = 6,         /* factorisation row + column passes */
    NSD_KERNEL_CP = 7,         /* CP three mode passes */
    NSD_KERNEL_LOSS = 8,       /* loss total */
    NSD_KERNEL_TTV = 9,        /* TTV entry kernels */
    NSD_KERNEL_DUAL = 10,      /* one column pass giving dA, A^T G and the loss
                                  (bilinear and SMVM losses) */
    NSD_KERNEL_SORT = 11,      /* radix-sort scatter pass of the builders */
    NSD_KERNEL_JVP = 12,       /* forward-mode tangent of the matrix product */
    NSD_KERNEL_CPN = 13,       /* order-N CP mode passes */
    NSD_KERNEL_PERM = 14,      /* the two passes of a value permutation */
    NSD_KERNEL_BATAX_ROWS = 15 /* rows of the BATAX Jacobian built in LDS */
} nsd_kernel_id;

/*
 * Instrumentation for callers that measure kernel durations (benchmarks).
 * While a probe is set on the calling thread, the library records the
 * caller's hipEvent_t start[i % n] on the launching stream right before the
 * i-th launch of the given kernel and stop[i % n] right after it, so that
 * hipEventElapsedTime(start[i], stop[i]) is that launch's duration.  The
 * probe keeps the n event handles (host arrays copied at the call) until
 * nsd_probe_clear; the events themselves stay owned by the caller.
 */
nsd_status nsd_probe_set(int kernel_id, void *const *start_events, void *const *stop_events,
                         int32_t n);
/* Launches recorded since nsd_probe_set (host output). */
nsd_status nsd_probe_count(int32_t *count);
nsd_status nsd_probe_clear(void);

/* ------------------------------------------------------------ workspace */

/* Bytes of `ws` that any hot-path entry point below needs for the operand A
 * (with its row plan), its CSC At (with its column plan; may be NULL when only
 * row-side calls are made) and dense width k.  Writes *bytes (host). */
nsd_status nsd_workspace_size(const nsd_csr *A, const nsd_csc *At, int32_t k, size_t *bytes);

/* Bytes of `ws` that the builders need to sort n entries whose keys are below
 * max_key (max_key >= 1).  Writes *bytes (host). */
nsd_status nsd_build_workspace_size(int32_t n, int32_t max_key, size_t *bytes);

/* ------------------------------------------------------------- builders */

/* Suggested item length L for a plan of an operand with nnz entries used at
 * dense width k (enough items to fill the GPU; 16 <= L <= 256, shorter, down
 * to 2, for inputs too small to give every SIMD a wave of 16-entry items). */
nsd_status nsd_plan_item_len(int32_t nnz, int32_t k, int32_t *item_len);

/* Array sizes for nsd_plan_build: item_ptr needs *max_items + 1 entries,
 * chunk_ord *max_items, long_seg, long_first and huge_idx *max_long each,
 * chunk_item *max_chunks,
 * empty_seg nseg; *ws_bytes of workspace.  Host outputs.
 * NSD_ERR_TOO_LARGE when 2 nnz + nseg >= 2^31. */
nsd_status nsd_plan_bounds(int32_t nseg, int32_t nnz, int32_t item_len, int32_t *max_items,
                           int32_t *max_long, int32_t *max_chunks, size_t *ws_bytes);

/*
 * Builds the work plan of a segment pointer array segptr [nseg+1] (a CSR
 * rowptr or a CSC colptr) into the caller's arrays and fills *plan (host):
 * counts and device pointers.  Deterministic.  Synchronous.
 */
nsd_status nsd_plan_build(int32_t nseg, int32_t nnz, const int32_t *segptr, int32_t item_len,
                          int32_t *item_ptr, int32_t *long_seg, int32_t *long_first,
                          int32_t *huge_idx, int32_t *chunk_item, int32_t *chunk_ord,
                          int32_t *empty_seg, nsd_plan *plan, void *ws, size_t ws_bytes,
                          void *stream);

/* rowidx[p] = the row r with rowptr[r] <= p < rowptr[r+1].  Async. */
nsd_status nsd_csr_expand_rows(int32_t nrows, int32_t nnz, const int32_t *rowptr,
                               int32_t *rowidx, void *stream);

/*
 * COO -> CSR (Section 5.3: vector/matrix COO and CSR storage; the CSR keeps
 * unique keys).  Entries are stably sorted by (row, col); a coordinate given
 * several times is merged under NSD_DUP_SUM (values added in input order, the
 * semi-ring "+=") or rejected with NSD_ERR_DUPLICATE under NSD_DUP_ERROR.
 * Inputs row/col/val: [nnz].  Outputs (each sized for nnz, the first
 * *nnz_out entries are written): rowptr [nrows+1], rowidx, colind, val_out,
 * perm (input position of the first occurrence of each output entry).
 * *nnz_out is a host int32.  Index outputs are bit-exact; a merged value is
 * the fp32 sum of its duplicates in input order.  Coordinates out of range
 * give NSD_ERR_BAD_FORMAT.  After NSD_ERR_BAD_FORMAT or NSD_ERR_DUPLICATE
 * the outputs hold unspecified values.
 * Synchronous.  ws: nsd_build_workspace_size(nnz, max(nrows, ncols)).
 */
nsd_status nsd_coo_to_csr(int32_t nrows, int32_t ncols, int32_t nnz, const int32_t *row,
                          const int32_t *col, const float *val, int policy,
                          int32_t *rowptr, int32_t *rowidx, int32_t *colind,
                          float *val_out, int32_t *perm, int32_t *nnz_out,
                          void *ws, size_t ws_bytes, void *stream);

/*
 * CSR -> CSC by a stable counting sort on the column index (Section 5.3, CSC
 * "expressed similarly" to CSR).  Outputs: colptr [ncols+1]; colidx, rowind,
 * perm [nnz] with perm[q] the CSR slot of CSC slot q; rows ascend within every
 * column.  Bit-exact.  A column index outside [0, ncols) gives
 * NSD_ERR_BAD_FORMAT (the outputs then hold unspecified values).
 * Synchronous.  ws: nsd_build_workspace_size(nnz, ncols).
 */
nsd_status nsd_csr_to_csc(const nsd_csr *A, int32_t *colptr, int32_t *colidx,
                          int32_t *rowind, int32_t *perm, void *ws, size_t ws_bytes,
                          void *stream);

/*
 * Mode index of a COO 3-tensor (or any int32 key array): a stable counting
 * sort of positions 0..nnz-1 by key[p] in [0, dim).  Outputs: segptr [dim+1],
 * segidx [nnz] (sorted keys), perm [nnz] (input position of sorted slot q).
 * Bit-exact.  A key outside [0, dim) gives NSD_ERR_BAD_FORMAT (the outputs
 * then hold unspecified values).  Synchronous.  ws:
 * nsd_build_workspace_size(nnz, dim).
 */
nsd_status nsd_coo_mode_index(int32_t nnz, int32_t dim, const int32_t *key,
                              int32_t *segptr, int32_t *segidx, int32_t *perm,
                              void *ws, size_t ws_bytes, void *stream);

/* Bytes of `ws` nsd_perm_plan_build needs for n elements (host output). */
nsd_status nsd_perm_plan_workspace_size(int32_t n, size_t *bytes);

/*
 * Plan of dst[q] = src[perm[q]] (inverse = 0) or of dst[perm[q]] = src[q]
 * (inverse = 1), perm a permutation of [0, n) (device), for
 * nsd_permute_f32: the permutation factored into two of bounded span (a
 * two-digit radix permutation with digits of `tile` elements): pass 1 moves
 * each source tile's values into the staging runs of their destination
 * buckets, pass 2 places each bucket's values at their destinations.
 * Outputs stage [n], src_local [n], dst_local [n] (caller arrays) and *plan
 * (host).  NSD_ERR_BAD_FORMAT when perm is not a permutation.  Synchronous.
 */
nsd_status nsd_perm_plan_build(int32_t n, const int32_t *perm, int inverse, int32_t *stage,
                               uint16_t *src_local, uint16_t *dst_local, nsd_perm_plan *plan,
                               void *ws, size_t ws_bytes, void *stream);

/* The plan's permutation applied to src: an exact fp32 copy in two
 * coalesced passes; staging [n] is caller scratch; src and dst must not
 * alias.  Async. */
nsd_status nsd_permute_f32(const nsd_perm_plan *plan, const float *src, float *dst,
                           float *staging, void *stream);

/* dst[q] = src[perm[q]] for q < n: an exact fp32 copy (values into CSC or
 * mode order).  Async. */
nsd_status nsd_gather_f32(int32_t n, const int32_t *perm, const float *src, float *dst,
                          void *stream);

/* dst[q] = src[perm[q]] for q < n, int32 (coordinates into mode order).  Async. */
nsd_status nsd_gather_i32(int32_t n, const int32_t *perm, const int32_t *src, int32_t *dst,
                          void *stream);

/* Checks a CSR: rowptr[0] = 0, non-decreasing, rowptr[nrows] = nnz; colind in
 * [0, ncols) and, when check_sorted, strictly increasing within each row;
 * rowidx (if not NULL) consistent with rowptr.  NSD_OK or NSD_ERR_BAD_FORMAT.
 * Synchronous.  ws: at least 256 bytes. */
nsd_status nsd_validate_csr(const nsd_csr *A, int check_sorted, void *ws, size_t ws_bytes,
                            void *stream);

/* Bytes of `ws` for nsd_validate_coo.  dims: host array of `order` sizes. */
nsd_status nsd_validate_coo_workspace_size(int32_t order, const int32_t *dims, int32_t nnz,
                                           size_t *bytes);

/* Checks a COO tensor of order 2 to NSD_MAX_ORDER (the dictionary of
 * Section 2 stores each key once): every coordinate of mode m in
 * [0, dims[m]) (else NSD_ERR_BAD_FORMAT) and, when check_unique, no key
 * twice (else NSD_ERR_DUPLICATE; found by sorting the entries
 * lexicographically).  dims and coords are HOST arrays of `order` sizes /
 * device pointers to [nnz] int32 coordinates.  Synchronous. */
nsd_status nsd_validate_coo(int32_t order, const int32_t *dims, int32_t nnz,
                            const int32_t *const *coords, int check_unique, void *ws,
                            size_t ws_bytes, void *stream);

/* ------------------------------------------------------------- forward */

/* y = A x (SpMV: the matrix-vector product of Logical SDQLite, Section 3,
 * a sum over each row's stored entries).  x [ncols], y [nrows].  Async. */
nsd_status nsd_spmv(const nsd_csr *A, const float *x, float *y, void *ws, size_t ws_bytes,
                    void *stream);

/* C = A B (SpMM; the matrix-matrix product of Logical SDQLite, Section 3).
 * B [ncols x k], C [nrows x k].  Async. */
nsd_status nsd_spmm(const nsd_csr *A, const float *B, int32_t k, float *C, void *ws,
                    size_t ws_bytes, void *stream);

/* ---------------------------------------------------- VJP primitives */

/*
 * SDDMM on A's pattern, the gradient w.r.t. a sparse operand.  The gradient
 * API seeds a sparse input with a one-hot over its own stored keys
 * (Sections 4.2 and 4.3), so its gradient is keyed by those keys only:
 *   out[p] = alpha * <X[rowidx[p], :], Y[colind[p], :]>   for p < nnz,
 * aligned with A's CSR order (A's values are not read).  X [nrows x k]
 * (NULL: all ones), Y [ncols x k], out [nnz].  Async.
 */
nsd_status nsd_sddmm(const nsd_csr *A, const float *X, const float *Y, int32_t k,
                     float alpha, float *out, void *stream);

/*
 * Transposed product, the gradient w.r.t. a dense right operand of the
 * matrix product (Sections 4.2 and 4.3; the "+=" of singletons inside a sum,
 * Section 5.5, computed as a gather over the CSC so every output is written
 * once):
 *   out[j, :] = alpha * sum over stored (i, j) of A(i, j) * G[i, :]
 * read through the CSC At of A (values taken from A->val via At->perm).
 * G [nrows x k] (NULL: all ones, e.g. column sums for k = 1), out [ncols x k].
 * Async.
 */
nsd_status nsd_spmm_t(const nsd_csr *A, const nsd_csc *At, const float *G, int32_t k,
                      float alpha, float *out, void *ws, size_t ws_bytes, void *stream);

/*
 * Vector-Jacobian product of C = A X (the reverse-mode result the paper's
 * tensorized forward mode computes for the matrix product, Sections 4.2
 * and 6.4) for an upstream gradient G = dL/dC [nrows x k] (NULL: all ones):
 *   dA[p] = <G[i,:], X[j,:]> on A's pattern (SDDMM, A's storage order),
 *   dX = A^T G  [ncols x k].
 * X [ncols x k].  One fused pass over the columns when k fits it (see
 * nsd_loss_bilinear), else SDDMM then the transposed product.  Workspace:
 * nsd_workspace_size(A, At, k).  Async.
 */
nsd_status nsd_spmm_vjp(const nsd_csr *A, const nsd_csc *At, const float *X, const float *G,
                        int32_t k, float *dA, float *dX, void *ws, size_t ws_bytes, void *stream);

/* The same for y = A x: gy [nrows] (NULL: ones), dA [nnz], dx [ncols]. */
nsd_status nsd_spmv_vjp(const nsd_csr *A, const nsd_csc *At, const float *x, const float *gy,
                        float *dA, float *dx, void *ws, size_t ws_bytes, void *stream);

/* -------------------------------------------------------- fused losses */
/* `seed` is the upstream gradient dL_out/dL (1 for plain training); it scales
 * every gradient and never the loss.  `loss` is one device double. */

/*
 * L = sum(A x): the SMVM kernel of Section 7.1 (the sum of a matrix-vector
 * product), differentiated with respect to both operands (Section 4.3).
 * dA[p] = seed * x[colind[p]] on A's pattern; dx = seed * A^T 1.
 * x [ncols]; dA [nnz]; dx [ncols].  Async.
 */
nsd_status nsd_loss_sum_spmv(const nsd_csr *A, const nsd_csc *At, const float *x, float seed,
                             double *loss, float *dA, float *dx, void *ws, size_t ws_bytes,
                             void *stream);

/*
 * L = 1/2 ||A B||_F^2: a loss over the matrix product of Section 3, its
 * gradients those of the gradient API (Section 4.3), the sparse one on A's
 * keys (Section 4.2).  C = A B (written to C [nrows x k]);
 * dA[p] = seed * <C[i,:], B[j,:]> on A's pattern (SDDMM);
 * dB = seed * A^T C.  B, dB [ncols x k]; dA [nnz].  Async.
 */
nsd_status nsd_loss_frob_spmm(const nsd_csr *A, const nsd_csc *At, const float *B, int32_t k,
                              float seed, float *C, double *loss, float *dA, float *dB,
                              void *ws, size_t ws_bytes, void *stream);

/*
 * GNN layer: L = sum((A H) o G) = sum over stored (i, j) of A(i,j) <G[i,:], H[j,:]>
 * (the matrix product of Section 3 weighted by the upstream gradient G;
 * gradients as in Sections 4.2 and 4.3).
 * dA[p] = seed * <G[i,:], H[j,:]> on A's pattern (SDDMM); dH = seed * A^T G.
 * H, dH [ncols x k]; G [nrows x k]; dA [nnz].  Async.
 */
nsd_status nsd_loss_bilinear(const nsd_csr *A, const nsd_csc *At, const float *H,
                             const float *G, int32_t k, float seed, double *loss, float *dA,
                             float *dH, void *ws, size_t ws_bytes, void *stream);

/*
 * nsd_loss_bilinear without a workspace, for callers that cannot allocate
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the same kernels and results, bit for bit, with the scratch
 * (the column plan's chunk partials and the loss partials) taken from a
 * static device array of 64 MiB that the library holds on every GPU it runs
 * on until the process ends.  It calls no allocator.  Operands that need more
 * scratch than that (about 64 MiB / (4 k) chunk items of long columns, or
 * some 8M fused-pass blocks) give NSD_ERR_WORKSPACE before any launch; use
 * nsd_loss_bilinear then.  Every call on a GPU uses that GPU's one array, so
 * calls that overlap on one GPU (other streams, other threads) race: order
 * them on one stream.  Arguments and results as nsd_loss_bilinear.  Async.
 */
nsd_status nsd_loss_bilinear_noalloc(const nsd_csr *A, const nsd_csc *At, const float *H,
                                     const float *G, int32_t k, float seed, double *loss,
                                     float *dA, float *dH, void *stream);

/*
 * Sparse matrix factorisation, a sum over A's stored keys (the dictionary
 * iteration of Section 2.2; gradients by Sections 4.2 and 4.3):
 *   L = sum over stored (i, j) of r_ij^2,  r_ij = A(i,j) - <U[i,:], V[j,:]>
 *   dU[i,:] = -2 seed sum_j r_ij V[j,:];  dV[j,:] = -2 seed sum_i r_ij U[i,:]
 * A's CSR gives the row pass (values A->val), its CSC the column pass with
 * the values in CSC order valT [nnz] (nsd_gather_f32 of A->val by At->perm,
 * made once when A is data; NULL: read A->val through At->perm each call).
 * U, dU [nrows x k]; V, dV [ncols x k].  Any k >= 1: up to 256 (multiple of
 * 4, 16-byte aligned rows) or up to 64 otherwise, both passes run fused in
 * one launch; a wider k forms r once per stored entry in the workspace (its
 * size query counts nnz floats for every k > 64) and runs the two
 * gather-reduces with r as weights.  Async.
 */
nsd_status nsd_loss_mf(const nsd_csr *A, const nsd_csc *At, const float *valT, const float *U,
                       const float *V, int32_t k, float seed, double *loss, float *dU, float *dV,
                       void *ws, size_t ws_bytes, void *stream);

/* Bytes of `ws` nsd_loss_cp needs for X (with its three plans) at the given
 * rank.  Writes *bytes (host). */
nsd_status nsd_cp_workspace_size(const nsd_coo3 *X, int32_t rank, size_t *bytes);

/*
 * CP decomposition of a sparse 3-tensor X (an order-3 tensor of nested
 * dictionaries, Section 3; its loss a sum over X's stored keys, gradients by
 * Sections 4.2 and 4.3) with factors F1 [dims[0] x rank],
 * F2 [dims[1] x rank], F3 [dims[2] x rank]:
 *   R = X - m on X's keys, m_ijl = sum_r F1[i,r] F2[j,r] F3[l,r]
 *   L = 1/2 sum R^2
 *   dX [nnz] = seed * R, aligned with X's input order (X->mode[n].perm)
 *   dF1[i,:] = -seed sum R_ijl (F2[j,:] o F3[l,:]), cyclically dF2, dF3
 *   (the negated mode-n MTTKRPs of R).
 * Any rank >= 1: up to 256 (multiple of 4, 16-byte aligned rows) or up to 64
 * otherwise, the three mode passes run fused in one launch; a wider rank
 * forms R once in the workspace (counted by nsd_cp_workspace_size for every
 * rank > 64) and runs one gather-reduce per mode with R as weights.  Async.
 */
nsd_status nsd_loss_cp(const nsd_coo3 *X, const float *F1, const float *F2, const float *F3,
                       int32_t rank, float seed, double *loss, float *dX, float *dF1,
                       float *dF2, float *dF3, void *ws, size_t ws_bytes, void *stream);

/* Bytes of workspace nsd_ttv_build needs; dims is a host array of `order`. */
nsd_status nsd_ttv_build_workspace_size(int32_t order, const int32_t *dims, int32_t nnz,
                                        size_t *bytes);

/*
 * Projection of an order-N COO tensor along mode n (3 <= N <= NSD_MAX_ORDER,
 * 0 <= n < N): coords is a HOST array of N device pointers to [nnz] int32
 * coordinates (input order), dims a host array of N sizes.  The entries are
 * stably sorted by their other coordinates in lexicographic order (mode 0
 * most significant, ties in input order) and the distinct projected keys
 * numbered in that order: ykey is a HOST array of N - 1 device pointers
 * (capacity nnz each) receiving the keys' coordinates in the other modes,
 * yptr [nnz+1] their entry ranges; yseg, yperm, ykidx [nnz] as in
 * nsd_ttv_plan.  The mode-n view: lptr [dims[n]+1], lseg, lperm, lpair
 * [nnz] (stable by the mode-n coordinate).  *ny (host) = number of keys.
 * Coordinates out of range give NSD_ERR_BAD_FORMAT.  Bit-exact.
 * Synchronous.
 */
nsd_status nsd_ttv_build(int32_t order, const int32_t *dims, int32_t nnz,
                         const int32_t *const *coords, int32_t mode, int32_t *const *ykey,
                         int32_t *yptr, int32_t *yseg, int32_t *yperm, int32_t *ykidx,
                         int32_t *lptr, int32_t *lseg, int32_t *lperm, int32_t *lpair,
                         int32_t *ny, void *ws, size_t ws_bytes, void *stream);

/* Bytes of `ws` for nsd_ttv and nsd_ttv_vjp.  Writes *bytes (host). */
nsd_status nsd_ttv_workspace_size(const nsd_ttv_plan *T, size_t *bytes);

/*
 * Tensor-times-vector along the plan's mode n: y[s] = sum over the stored
 * entries whose other coordinates form key s of x * v(l), Y = X x_n v on the
 * projected keys (a sum over X's keys inserting singletons with "+=",
 * Section 3 and Section 5.5).  x [nnz] in X's input order, v [dims[n]],
 * y [ny].  Async.
 */
nsd_status nsd_ttv(const nsd_ttv_plan *T, const float *x, const float *v, float *y, void *ws,
                   size_t ws_bytes, void *stream);

/*
 * Vector-Jacobian product of nsd_ttv for the upstream gy [ny]:
 * dx[p] = gy[key(p)] * v(l_p) on X's keys (input order, [nnz]);
 * dv(l) = sum over the stored entries with mode-n coordinate l of
 * x * gy[key]  (dv [dims[n]]).  Async.
 */
nsd_status nsd_ttv_vjp(const nsd_ttv_plan *T, const float *x, const float *v, const float *gy,
                       float *dx, float *dv, void *ws, size_t ws_bytes, void *stream);

/* Bytes of `ws` for nsd_ttm and nsd_ttm_vjp at width R (R >= 1).  Writes
 * *bytes (host). */
nsd_status nsd_ttm_workspace_size(const nsd_ttv_plan *T, int32_t R, size_t *bytes);

/*
 * Tensor-times-matrix along the plan's mode n, the matrix form of nsd_ttv
 * (the n-mode product of Section 3's tensor algebra, kept sparse on the
 * projected keys): Y[s, :] = sum over the stored entries of key s of
 * x * U[l, :].  x [nnz] in X's input order, U row-major [dims[n] x R], Y
 * row-major [ny x R], every row written.  T is X's projection along n.
 * Async.
 */
nsd_status nsd_ttm(const nsd_ttv_plan *T, const float *x, const float *U, int32_t R, float *Y,
                   void *ws, size_t ws_bytes, void *stream);

/*
 * Vector-Jacobian product of nsd_ttm for the upstream gY row-major [ny x R]:
 * dx[p] = <gY[key(p), :], U[l_p, :]> on X's keys (input order, [nnz]);
 * dU[l, :] = sum over the stored entries with mode-n coordinate l of
 * x * gY[key, :]  (dU [dims[n] x R], every row written).  Async.
 */
nsd_status nsd_ttm_vjp(const nsd_ttv_plan *T, const float *x, const float *U, int32_t R,
                       const float *gY, float *dx, float *dU, void *ws, size_t ws_bytes,
                       void *stream);

/*
 * *out = alpha * sum_{i < n} x[i] * y[i] (y NULL: ones), accumulated in fp64
 * in a fixed order, plus the previous *out when `accumulate` is nonzero: the
 * full contraction of two dense tensors, or of a sparse operand's values with
 * a sampled product on its keys (the scalar `sum` of Logical SDQLite,
 * Section 3).  `out` is one device double.  Workspace: 16 KiB suffice (one
 * double per block, at most 2048 blocks).  Async.
 */
nsd_status nsd_dot(int64_t n, const float *x, const float *y, double alpha, int accumulate,
                   double *out, void *ws, size_t ws_bytes, void *stream);

/*
 * y = alpha * x + beta * y over n elements (x NULL: ones; beta == 0: y is
 * overwritten without being read): the sum and scalar product of tensors
 * that share one layout (Logical SDQLite `+` and real `*`, Section 3).
 * Async.
 */
nsd_status nsd_axpby(int64_t n, float alpha, const float *x, float beta, float *y,
                     void *stream);

/*
 * out[p] = alpha where A's stored key p is diagonal (row = column), else 0,
 * over A's nnz entries in its storage order: the gradient of the trace
 * sum_i A(i, i) with respect to A on its stored keys, scaled by alpha.  It is
 * the identity restricted to the stored diagonal keys (the trace example of
 * Section 4.3, Example 3): a diagonal key that is not stored gets no
 * gradient, and the value array is aligned 1:1 with A's keys like every
 * sparse gradient.  Needs A's rowidx and colind (not its values or plan).
 * Async.
 */
nsd_status nsd_diag_keys(const nsd_csr *A, float alpha, float *out, void *stream);

/*
 * A product taken key by key (Section 5: what multiplication normalisation
 * leaves of a term in which no index is summed): for i in [0, n)
 *     y[yi] = alpha * s1 * s2 * x1[i] * x2[x2i] + beta * y[yi],
 *     yi = y_idx ? y_idx[i] : i,   x2i = x2_idx ? x2_idx[i] : i.
 * s1, s2: device doubles, reals of a program (inputs or results; NULL: 1).
 * x1, x2: device floats (NULL: ones), x1 aligned with the n keys; x2_idx
 * gathers x2 (a dense operand read at each key's row, column or index).
 * y_idx scatters into a dense y and must hold n distinct indices (each
 * output is written once); the indices are not checked (out of range or
 * repeated ones are undefined, as a malformed operand of any hot-path call
 * is).  beta == 0: y is not read.  The product is formed in double and
 * rounded once.  The Jacobians of the vector kernels
 * of Section 7.1 and of matrix-valued programs on a matrix's keys reduce to
 * this.  Async.
 */
nsd_status nsd_scale(int64_t n, double alpha, const double *s1, const double *s2,
                     const float *x1, const float *x2, const int32_t *x2_idx, float beta,
                     float *y, const int32_t *y_idx, void *stream);

/*
 * The same for one real: y[0] = alpha * s1 * s2 * x + beta * y[0] on device
 * doubles (s1, s2, x NULL: 1; beta == 0: y is not read).  Async.
 */
nsd_status nsd_scale_real(double alpha, const double *s1, const double *s2, const double *x,
                          double beta, double *y, void *stream);

/* ---------------------------------------------------------------------------
 * Order-N sparse tensors and the CP gradient for orders 3 to NSD_MAX_ORDER
 * (the order-N form of the nested-dictionary tensor of Section 3).
 *
 * nsd_coon holds one mode index per mode n: the stored entries sorted
 * stably by coordinate n (nsd_coo_mode_index), segptr / segidx over the
 * mode's slices, idx[o] = the coordinate of mode (n + 1 + o) mod order of
 * every entry in that order (o = 0 .. order - 2), val in that order, perm =
 * input position of every slot, and the slices' work plan.
 */
typedef struct nsd_coon_mode {
    int32_t mode;
    const int32_t *segptr;                  /* [dims[mode] + 1] */
    const int32_t *segidx;                  /* [nnz] */
    const int32_t *idx[NSD_MAX_ORDER - 1];  /* [order - 1][nnz] other coordinates */
    const float *val;                       /* [nnz] */
    const int32_t *perm;                    /* [nnz] */
    nsd_plan plan;
    /* Second level of the compressed-fiber tree (0: none).  With 1, the
     * slices' entries are taken as fibers: runs of equal coordinate of the
     * fiber mode (mode 1 for mode 0, else mode 0), as lexicographic storage
     * gives them.  The pass then gathers that mode's factor row once per
     * fiber, keeps the fiber's partial product with the slice's own row and
     * adds the fiber's sum once into the slice, instead of per entry.  Any
     * order of entries gives the same values (up to rounding); long runs
     * give the savings. */
    int32_t fiber;
} nsd_coon_mode;

typedef struct nsd_coon {
    int32_t order;                  /* 3 .. NSD_MAX_ORDER */
    int32_t dims[NSD_MAX_ORDER];
    int32_t nnz;
    nsd_coon_mode mode[NSD_MAX_ORDER];
} nsd_coon;

/* Bytes of `ws` for nsd_loss_cpn.  Writes *bytes (host). */
nsd_status nsd_cpn_workspace_size(const nsd_coon *X, int32_t rank, size_t *bytes);

/*
 * Rank-R CP model of an order-N sparse tensor X:
 *   m = sum_r prod_n F_n(c_n, r),  R = x - m on X's keys,  L = 1/2 sum R^2,
 *   dX = seed * R on X's keys (X's input order, [nnz]),
 *   dF_n(c_n, :) = -seed sum R * (o_{m != n} F_m(c_m, :))  (negated MTTKRPs).
 * F and dF are HOST arrays of `order` device pointers to [dims[n] x rank]
 * row-major factors.  *loss (device fp64) is not scaled by seed.  Any
 * rank >= 1; ranks above 256 (above 64 without 16-byte aligned rows of a
 * multiple of 4) form R once in the workspace and run one gather-reduce per
 * mode.  Async.
 */
nsd_status nsd_loss_cpn(const nsd_coon *X, const float *const *F, int32_t rank, float seed,
                        double *loss, float *dX, float *const *dF, void *ws, size_t ws_bytes,
                        void *stream);

/* ---------------------------------------------------------------------------
 * Forward-mode tangent of C = A B, the paper's mode of differentiation
 * (Section 4.1: values carried with their tangents; Section 4.2: tensors of
 * tangents): for a tangent dA on A's stored keys and a dense tangent dB,
 *     C  = A B,     dC = dA B + A dB.
 * A: CSR with rowidx and the row plan.  dAval [nnz]: the tangent of A's
 * values in A's storage order.  B, dB [ncols x k], C, dC [nrows x k],
 * row-major, fully overwritten (0 for empty rows).  Any k >= 1.
 * Workspace: at least nsd_workspace_size(A, NULL, 2k, ...) bytes.  Async.
 */
nsd_status nsd_spmm_jvp(const nsd_csr *A, const float *dAval, const float *B, const float *dB,
                        int32_t k, float *C, float *dC, void *ws, size_t ws_bytes,
                        void *stream);

/*
 * A batch of m tangents of C = A B at once (Section 4.2: the tangent is a
 * tensor with one more key, the batch index t; this is J V for the m
 * columns of V):
 *     dC_t = dA_t B + A dB_t,   t = 0 .. m - 1.
 * Tangents are taken in groups of four: each group reads A and the rows of
 * B once for all of its tangents.  dAval: [m x nnz], tangent t's values in
 * A's storage order (NULL: every dA_t = 0).  dB: [m x ncols x k] (NULL:
 * every dB_t = 0).  C: [nrows x k], computed when not NULL.  dC:
 * [m x nrows x k], fully overwritten.  Any k >= 1, m >= 0.
 * Workspace: nsd_spmm_jvp_batch_workspace_size bytes (independent of m).
 * Async.
 */
nsd_status nsd_spmm_jvp_batch_workspace_size(const nsd_csr *A, int32_t k, size_t *bytes);
nsd_status nsd_spmm_jvp_batch(const nsd_csr *A, int32_t m, const float *dAval, const float *B,
                              const float *dB, int32_t k, float *C, float *dC, void *ws,
                              size_t ws_bytes, void *stream);

/* ---------------------------------------------------------------------------
 * Jacobian of the BATAX kernel f(j) = sum_{i,k} beta A(i,j) A(i,k) x(k) with
 * respect to x (Example 5; the matrix kernels of Section 7):
 *     J = beta A^T A,  J(j, k) = beta sum_i A(i, j) A(i, k),
 * an ncols x ncols sparse matrix whose pattern is not an input's: a key
 * (j, k) for every pair of stored entries of A that share a row (the
 * normalised program of Example 5 inserts the outer product of every row
 * with itself).  Keys are structural: a pair whose product is 0 keeps its
 * key.  A is a CSR (rowptr, colind, val; sorted unique columns per row; no
 * plan needed; rowidx may be NULL, else it must be A's row index).
 *
 * Three calls:
 *   nsd_batax_pairs          *npairs (host) = sum over rows of length^2, the
 *                            number of products and an upper bound on the
 *                            keys of J.  `ws`: at least 256 device bytes.
 *                            Synchronous.
 *   nsd_batax_workspace_size bytes of `ws` for nsd_batax_jacobian.
 *   nsd_batax_jacobian       J as a CSR: jrowptr [ncols + 1], jcolind / jval
 *                            [npairs capacity]; *nnz_out (host) = its keys,
 *                            in (row, col) order.  Values are the sums of
 *                            the products in row order of A, accumulated in
 *                            fp64 and rounded once (reproducible).
 *                            Synchronous.
 * Two ways give the same bits.  When every row of J has at most 512 terms,
 * J is built row by row (row j gathers the rows of A storing column j, its
 * terms sorted by column in LDS); otherwise every term is expanded and
 * sorted twice through HBM.  The environment variable NSD_BATAX_ROW_CAP
 * lowers the 512 (0: always the second way).
 * Errors: NSD_ERR_TOO_LARGE when npairs >= 2^30; NSD_ERR_INVALID_ARG when
 * npairs differs from A's (nothing is written then but workspace).
 */
nsd_status nsd_batax_pairs(const nsd_csr *A, int64_t *npairs, void *ws, size_t ws_bytes,
                           void *stream);
nsd_status nsd_batax_workspace_size(const nsd_csr *A, int64_t npairs, size_t *bytes);
nsd_status nsd_batax_jacobian(const nsd_csr *A, float beta, int64_t npairs, int32_t *jrowptr,
                              int32_t *jcolind, float *jval, int32_t *nnz_out, void *ws,
                              size_t ws_bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* NSD_H */
