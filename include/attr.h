/*
 * attr.h -- C ABI of the MI355X (gfx950) gradient-attribution hot path.
 *
 * The library implements the data-parallel core of gradient-based data
 * attribution as described in "Bergson: An Open Source Library for Data
 * Attribution":
 *   (1) per-example double-sided random projection of linear-layer
 *       gradients (Figure 1 caption; Appendix B, paragraph "Gradients");
 *   (2) unit normalisation and second-moment preconditioning of the
 *       compressed rows (section "Attribution Pipelines": processing may
 *       include unit normalisation and preconditioning; the flat
 *       autocorrelation / empirical Fisher of the method-family table);
 *   (3) exact top-k lookup of a query against the gradient store (section
 *       "Attribution Pipelines": every store supports exact top-k).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Plain C99.  Pointers are DEVICE pointers (HIP device memory of the
 *   current device) unless marked (host).  Sizes and strides are in
 *   ELEMENTS, row-major, int64.
 * - `stream` is a hipStream_t passed as void*; NULL means the null stream.
 *   Every call only enqueues work on `stream` and returns; results are
 *   valid once the stream has completed.  No call synchronises.
 * - The caller owns every buffer, including the workspace `ws` whose
 *   minimum size the matching *_workspace_size() function returns (0 means
 *   no workspace is needed; `ws` may then be NULL).  The library keeps no
 *   per-call state between calls and never allocates device memory; the one
 *   exception is the static per-GPU scratch array of attr_project_noalloc.
 * - Errors: arguments are validated on the host before anything is
 *   enqueued.  On any error the call enqueues nothing, leaves every output
 *   untouched and returns a non-zero attr_status; attr_last_error() then
 *   describes it.  ATTR_ERR_DEVICE reports a failed kernel launch (which may
 *   also surface an earlier asynchronous error).  No C++ exception crosses
 *   this boundary.  Values inside device arrays (lengths, offsets) cannot be
 *   checked on the host; their documented clamping applies instead.
 * - Calls that share a workspace or an output must be ordered by the
 *   caller (same stream, or events); concurrent calls on different
 *   workspaces are independent.
 */
#ifndef ATTR_H_
#define ATTR_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ATTR_ABI_VERSION 3

typedef enum {
  ATTR_OK = 0,
  ATTR_ERR_INVALID_ARG = 1,  /* null pointer with non-zero size, negative size, bad stride, overlap */
  ATTR_ERR_UNSUPPORTED = 2,  /* dtype / k / mode combination not implemented */
  ATTR_ERR_ALIGNMENT = 3,    /* pointer not 16-byte aligned, width or stride not a multiple of 8 elements */
  ATTR_ERR_WORKSPACE = 4,    /* ws_bytes below the queried size, or ws NULL when needed */
  ATTR_ERR_DEVICE = 5        /* HIP launch / runtime error */
} attr_status;

typedef enum { ATTR_F32 = 0, ATTR_BF16 = 1, ATTR_F16 = 2 } attr_dtype;

typedef enum {
  ATTR_PRECOND_NONE = 0,  /* identity */
  ATTR_PRECOND_DIAG = 1,  /* per-coordinate scale m (diagonal of H^{-1/2}) */
  ATTR_PRECOND_FULL = 2   /* full matrix M (H^{-1/2}), y = M x */
} attr_precond;

/* ------------------------------------------------------------------------ */
/* (1) attr_project: per-example compressed gradients of linear modules.    */
/* ------------------------------------------------------------------------ */

/* One linear module y = W x with W of shape [d_out, d_in].  Read only during
 * the call (host struct; the pointers inside are device pointers). */
typedef struct {
  const void* a;     /* input activations, rows of d_in elements, row stride lda */
  const void* g;     /* output gradients dL/dy, rows of d_out elements, row stride ldg */
  const void* R;     /* [d_out, k] row-major, same dtype as a/g (output-side projection) */
  const void* S;     /* [d_in,  k] row-major, same dtype as a/g (input-side projection) */
  int64_t lda, ldg;  /* row strides in elements, >= d_in / d_out, multiples of 8 */
  int64_t d_in, d_out;  /* multiples of 64 (bf16) or 32 (fp32); at most 65536 */
  int64_t out_col;   /* first column of this module's k*k block in `out` */
  /* Optional optimizer-state normalisation (Figure 1 caption: Adafactor
   * second moments): the factored second moment v_ij = v_out[i] v_in[j] /
   * sum(v_out) of the module's weight; each per-example gradient is divided
   * elementwise by sqrt(v) before projection (entries where v is 0 or a
   * factor is not positive become 0; no epsilon).  Device fp32 [d_out] and
   * [d_in], both NULL for no normalisation.  Applied by scaling the rows of
   * R and S while they are packed, so the projection itself costs the same. */
  const float* v_out;
  const float* v_in;
} attr_module;

/* Double-sided projection (Figure 1 caption; Appendix B "Gradients"): for
 * every example i and module m, with len_i valid tokens,
 *     P_{i,m} = sum_{t < len_i} (R^T g_t)(S^T a_t)^T          (k x k)
 * which equals R^T G_i S for the per-example weight gradient
 * G_i = sum_t g_t a_t^T, without ever forming G_i.  The result is written
 * row-major into out[i * ldo + out_col + r * k + c] (r: column of R,
 * c: column of S) as fp32; other columns of `out` are not touched.
 *
 * Token t of example i is row (row_offset ? row_offset[i] : i * T) + t of
 * both a and g.  Tokens t >= len_i are never read, so padding may hold any
 * bit pattern including NaN.  Modules that pass the same a pointer with the
 * same lda and d_in (the q/k/v or gate/up projections of one layer) have
 * their shared rows read once for up to three of them (two at k = 64); the
 * results are the same bits as with separate copies of a.
 *
 *   mods       (host) [n_mods] module descriptors; 1 <= n_mods <= 4096
 *   in_dtype   ATTR_BF16 (bf16 MFMA, fp32 accumulate) or ATTR_F32 (fp32 MFMA)
 *   k          16, 32 or 64
 *   n_examples examples in this call (0 is a no-op)
 *   T          tokens per example slot, >= 1
 *   row_offset device int64 [n_examples] or NULL (then i * T)
 *   length     device int32 [n_examples] or NULL (then T); values are
 *              clamped to [0, T]; len 0 gives a zero block
 *   out, ldo   device fp32 [n_examples, ldo]; out_col + k*k <= ldo per module
 *   ws         device workspace of at least
 *              attr_project_workspace_size(mods, n_mods, in_dtype, n_examples, T, k)
 *              bytes, 256-byte aligned; contents on entry are ignored.
 * The module blocks of `out` must not overlap each other.
 */
size_t attr_project_workspace_size(const attr_module* mods, int32_t n_mods,
                                   attr_dtype in_dtype, int64_t n_examples, int64_t T,
                                   int32_t k);
attr_status attr_project(const attr_module* mods, int32_t n_mods, attr_dtype in_dtype,
                         int32_t k, int64_t n_examples, int64_t T,
                         const int64_t* row_offset, const int32_t* length,
                         float* out, int64_t ldo, void* ws, size_t ws_bytes,
                         void* stream);

/* Per-token compressed gradients (Figure 1 caption: attribution scores are
 * per-token or per-sequence): the same projection without the token sum.
 * For every valid token t of example i and module m the k x k block
 *     P_{i,t,m} = (R^T g_t)(S^T a_t)^T
 * is written row-major into out[row * ldo + out_col + r * k + c], where row
 * = (row_offset ? row_offset[i] : i * T) + t is the token's own row in a
 * and g.  Rows of tokens t >= len_i and columns outside the module blocks
 * are not touched; rows >= n_rows are not written (size `out` to cover
 * every valid token's row).  Summing a token's blocks over t gives
 * attr_project's row; unit normalisation and scoring of the token rows use
 * attr_precond_apply and attr_score_topk.  Arguments as attr_project, plus
 *   out, ldo, n_rows  device fp32 [n_rows, ldo]
 *   ws        attr_project_workspace_size(...) bytes (the same query)
 */
attr_status attr_project_tokens(const attr_module* mods, int32_t n_mods, attr_dtype in_dtype,
                                int32_t k, int64_t n_examples, int64_t T,
                                const int64_t* row_offset, const int32_t* length, float* out,
                                int64_t ldo, int64_t n_rows, void* ws, size_t ws_bytes,
                                void* stream);

/* attr_project without a workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops
 * and harnesses that forbid allocation.  It computes exactly what
 * attr_project computes (same kernels, same bits) and makes no allocating
 * call: its scratch is a static device array of ATTR_PROJECT_NOALLOC_SCRATCH
 * bytes, one per GPU, created when the library's code first runs on that
 * GPU and held until the process ends.  Every call on a GPU shares that
 * GPU's array, so calls that overlap on one GPU (different streams or host
 * threads without ordering) race and give undefined results; order them.
 * A call whose workspace would exceed the array (attr_project_workspace_size
 * above ATTR_PROJECT_NOALLOC_SCRATCH) returns ATTR_ERR_WORKSPACE and
 * enqueues nothing.  Arguments and other errors as attr_project.
 */
#define ATTR_PROJECT_NOALLOC_SCRATCH (64ull << 20)
attr_status attr_project_noalloc(const attr_module* mods, int32_t n_mods, attr_dtype in_dtype,
                                 int32_t k, int64_t n_examples, int64_t T,
                                 const int64_t* row_offset, const int32_t* length, float* out,
                                 int64_t ldo, void* stream);

/* ------------------------------------------------------------------------ */
/* (2a) attr_precond_accumulate: second-moment statistics of store rows.    */
/* ------------------------------------------------------------------------ */

/* Accumulates the (unscaled) second moment of the rows of X, the
 * autocorrelation / empirical Fisher preconditioner of the method-family
 * table, restricted to its diagonal (DIAG) or in full (FULL):
 *   DIAG: H[j]       += sum_i X[i,j]^2                    (H: fp32 [D])
 *   FULL: H[p*D + q] += sum_i X[i,p] * X[i,q]  for p <= q (H: fp32 [D, D];
 *         the upper triangle including the diagonal is updated, the strict
 *         lower triangle is never read or written)
 * Accumulation is additive across calls, so a store can be processed in
 * chunks; divide by the total row count afterwards.  Within a call, partial
 * sums are formed in fp32 (DIAG: 8-row groups; FULL: matrix-core products
 * over at most 32768 rows), combined in fp64 in a fixed order and rounded
 * once into H, so results are deterministic.
 *
 *   X, ldx   device [n_rows, D] rows: DIAG takes ATTR_F16, ATTR_BF16 or
 *            ATTR_F32, FULL takes ATTR_F16 or ATTR_BF16; ldx >= D (FULL:
 *            ldx <= 65536, so that 16384 rows span at most 2 GiB)
 *   D        multiple of 8 (DIAG) or of 64 (FULL); FULL needs D <= 32768
 *   mode     ATTR_PRECOND_DIAG or ATTR_PRECOND_FULL
 *   ws       attr_precond_accumulate_workspace_size(n_rows, D, x_dtype, mode)
 */
size_t attr_precond_accumulate_workspace_size(int64_t n_rows, int64_t D, attr_dtype x_dtype,
                                              attr_precond mode);
attr_status attr_precond_accumulate(const void* X, attr_dtype x_dtype, int64_t n_rows,
                                    int64_t D, int64_t ldx, attr_precond mode, float* H,
                                    void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* (2b) attr_precond_apply: precondition, unit-normalise, cast.             */
/* ------------------------------------------------------------------------ */

/* For every row x of X (processing step of section "Attribution Pipelines";
 * grad-cosine when unit_normalize is set):
 *   y = x (NONE), y = M .* x (DIAG, M: fp32 [D]) or y = M x (FULL, M: fp32
 *   [D, D] row-major, symmetric in use: y_p = sum_q M[p*D+q] x_q);
 *   if unit_normalize, y /= ||y||_2 over the whole row (a zero row stays 0);
 *   Y = y cast to y_dtype (round to nearest even).
 * FULL evaluates M as a scaled fp16 pair, A = 2^s M (max|A| <= 2^15),
 * A_hi = fp16(A), A_lo = fp16(A - A_hi), y = 2^-s X (A_hi + A_lo)^T on fp16
 * MFMA with fp32 accumulation (about 22 significant bits of M).
 *
 *   X, ldx   device [n_rows, D], x_dtype ATTR_F32 or ATTR_F16
 *            (FULL: ATTR_F16 only)
 *   Y, ldy   device [n_rows, D], y_dtype ATTR_F16 or ATTR_F32
 *   D        multiple of 8 (NONE/DIAG), of 64 (FULL)
 *   In-place (Y == X) is allowed for NONE/DIAG when dtype and stride match;
 *   any other overlap of X and Y is ATTR_ERR_INVALID_ARG.
 *   ws       attr_precond_apply_workspace_size(n_rows, D, mode)
 */
size_t attr_precond_apply_workspace_size(int64_t n_rows, int64_t D, attr_precond mode);
attr_status attr_precond_apply(const void* X, attr_dtype x_dtype, int64_t n_rows, int64_t D,
                               int64_t ldx, attr_precond mode, const float* M,
                               int32_t unit_normalize, void* Y, attr_dtype y_dtype,
                               int64_t ldy, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* (3) attr_score_topk: query x store scores with exact streaming top-k.    */
/* ------------------------------------------------------------------------ */

/* For every query q: s_qj = <Q_q, G_j> (fp32 accumulation; the cosine when
 * both sides are unit rows) over the n_g store rows, and the k best
 * (index_base + j) ordered by (score desc, index asc); NaN and -inf scores
 * are never selected; missing slots are (-inf, -1).  Exact top-k lookup,
 * section "Attribution Pipelines".  With few queries the scan streams the
 * store once and the score matrix never reaches memory (on stores of
 * 262144 rows or more a first pass over 16384 rows finds, per query, a
 * lower bound on its k-th best score, and rows below it are skipped by the
 * selection: a few KB of workspace); with many fp16
 * queries (n_q >= 128) it is computed chunk by chunk into the workspace
 * (~256 MB per chunk, plus one maximum per 64 rows) and selected exactly
 * from there; after the first chunk only 64-row segments that can still
 * beat a query's running k-th best score are written and read.
 *
 *   Q, ldq       device [n_q, D];  G, ldg: device [n_g, D]; both `dtype`
 *                (ATTR_F16 or ATTR_F32); D a multiple of 64 (fp16) or 32
 *                (fp32); n_q, n_g below 2^31; 256 rows of either operand
 *                must span less than 2 GiB (ld * 256 * element size)
 *   k            1..128
 *   index_base   added to the local row index j (store offset of G), >= 0
 *   merge        0: overwrite top_*;  1: top_* hold a previous sorted
 *                result which is merged with this chunk (streaming over
 *                stores larger than one call)
 *   top_score    device fp32 [n_q, k];  top_index: device int64 [n_q, k]
 *   ws           attr_score_topk_workspace_size(n_q, n_g, D, k)
 * n_q == 0 is a no-op; n_g == 0 leaves top_* unchanged when merge == 1 and
 * fills them with (-inf, -1) when merge == 0.
 */
size_t attr_score_topk_workspace_size(int64_t n_q, int64_t n_g, int64_t D, int32_t k);
attr_status attr_score_topk(const void* Q, int64_t n_q, int64_t ldq, const void* G,
                            int64_t n_g, int64_t ldg, attr_dtype dtype, int64_t D,
                            int32_t k, int64_t index_base, int32_t merge,
                            float* top_score, int64_t* top_index,
                            void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Calibration (not part of the method): the rates this GPU sustains, used  */
/* as measured peaks beside the nominal ones.                               */
/* ------------------------------------------------------------------------ */

/* Streams `bytes` (a multiple of 16, x 16-byte aligned) from device memory
 * once with non-temporal 16-byte loads and no write stream (the result is
 * folded into registers; `sink`, a device word, is written only on an
 * improbable value).  Time it to get the achievable HBM read bandwidth. */
attr_status attr_probe_read(const void* x, size_t bytes, void* sink, void* stream);
/* Runs n_mfma (a multiple of 8, > 0) fp16 16x16x32 MFMAs per wave on 512
 * workgroups of four waves (two waves per SIMD on 256 CUs), operands in
 * registers: 2 * 16 * 16 * 32 * n_mfma * 2048 flops.  Time it to get the
 * achievable dense fp16 matrix-core rate.  `sink`: a device float. */
attr_status attr_probe_mfma(int64_t n_mfma, void* sink, void* stream);

/* ------------------------------------------------------------------------ */
/* Diagnostics.                                                             */
/* ------------------------------------------------------------------------ */

/* Message of the last failed call on this thread ("" if none); valid until
 * the next call on this thread. */
const char* attr_last_error(void);
/* Static name of a status code. */
const char* attr_status_string(attr_status status);
/* ATTR_ABI_VERSION of the loaded library. */
int attr_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* ATTR_H_ */
