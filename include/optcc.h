/*
 * liboptcc -- low-rank power-iteration compressor with error feedback on one
 * AMD Instinct MI355X (gfx950).
 *
 * The compressor is the one Optimus-CC (arXiv 2301.09830) applies to
 * inter-stage activation gradients (Sec. 5, compressed backpropagation),
 * embedding gradients (Sec. 6) and data-parallel weight gradients (Sec. 7):
 * PowerSGD-style power iteration warm-started from the previous factor
 * (Sec. 2.3, Sec. 8), with the compression residual kept in memory and added
 * to the next input (Sec. 5.1, lazy error propagation, Eq. (star2)).
 *
 * One call of the fused entry point computes, for an m x n input M:
 *
 *     A     = M + err_prev                        (error-feedback add)
 *     repeat `iters` times:
 *         P     = A Q                             (left product, m x r)
 *         P_hat = orthonormal basis of P          (CholeskyQR, thin-QR factor)
 *         Q     = A^T P_hat                       (right product, n x r)
 *     M_hat = P_hat Q^T                           (decompression)
 *     err   = A - M_hat                           (residual for the next call)
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Every array pointer is a DEVICE pointer owned by the caller.  No call
 *   allocates or frees device memory; the library keeps no per-call state
 *   outside the workspace the caller passes in.
 * - Matrices are row-major.  ld* is the leading dimension in elements
 *   (>= cols).  P is m x rank and Q is n x rank, both contiguous (ld = rank).
 *   err, P, Q and M_hat are fp32.  M is fp32 or bf16 (occ_dtype_t).
 * - Any alignment is accepted; 16-byte aligned bases with ld a multiple of 4
 *   select the vectorised load path.
 * - Argument errors are detected on the host before anything is enqueued and
 *   are returned as occ_status_t; nothing aborts.  A failed kernel launch
 *   returns OCC_E_HIP.
 * - Numeric conditions never fail a call.  They set sticky bits in the
 *   workspace header, read with occ_get_flags: a non-finite input propagates
 *   into the outputs and sets OCC_F_NONFINITE; a direction of P that is
 *   numerically dependent on the previous ones (Cholesky pivot below 1e-12 of
 *   the largest Gram diagonal) gives a zero column of P_hat and sets
 *   OCC_F_RANK_DEFICIENT.
 * - Work is enqueued on `stream` (a hipStream_t; NULL = the null stream) and
 *   runs asynchronously.  Only occ_get_flags and occ_profile_end synchronise.
 * - Calls that share one workspace must not overlap in time (same stream, or
 *   caller-side ordering); overlapping calls on one workspace race.
 */
#ifndef OPTCC_H
#define OPTCC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define OCC_ABI_VERSION 2
#define OCC_MAX_RANK 128
#define OCC_MAX_ITERS 64

typedef void* occ_stream_t; /* a hipStream_t */

typedef enum {
  OCC_OK = 0,
  OCC_E_NULL = 1,      /* a required pointer is NULL */
  OCC_E_SHAPE = 2,     /* rows/cols < 1, ld < cols, count < 1, or sizes overflow */
  OCC_E_RANK = 3,      /* rank < 1, rank > min(rows, cols) or rank > OCC_MAX_RANK */
  OCC_E_ITERS = 4,     /* iters < 1 or iters > OCC_MAX_ITERS */
  OCC_E_DTYPE = 5,     /* unknown dtype, or mixed dtypes in one batch */
  OCC_E_ALIGN = 6,     /* a pointer is not aligned to its element size */
  OCC_E_ALIAS = 7,     /* two buffers overlap (only err_new == err_prev may) */
  OCC_E_WORKSPACE = 8, /* workspace NULL, too small, or not 256-byte aligned */
  OCC_E_HIP = 9,       /* a HIP runtime call or kernel launch failed */
  OCC_E_FLAGS = 10     /* unknown bit in the flags argument */
} occ_status_t;

typedef enum { OCC_F32 = 0, OCC_BF16 = 1 } occ_dtype_t;

/* sticky numeric flags, read with occ_get_flags; OCC_F_BAD_ROWS: the row list
 * of occ_step_rows was not strictly increasing inside [0, rows) (the results
 * of that call are then unspecified, but no memory outside the arguments is
 * touched) */
enum { OCC_F_NONFINITE = 1u, OCC_F_RANK_DEFICIENT = 2u, OCC_F_BAD_ROWS = 4u };

/* call flags for occ_step / occ_step_batched */
enum { OCC_NO_MHAT = 1u }; /* sender side: do not write M_hat (err is still updated) */

/* flags of occ_decompress_ex */
enum {
  /* run the products occ_step runs for a bf16 M: at padded ranks 32..128 on
   * bf16 matrix cores with each factor split into two bf16 parts (about 2^-16
   * of |M_hat| per element); at padded rank <= 16 the products are fp32 either
   * way and the flag changes nothing */
  OCC_DEC_SPLIT_BF16 = 1u,
  /* store M_hat as bf16 (round to nearest even from the fp32 result) */
  OCC_DEC_OUT_BF16 = 2u
};

/* One matrix and its compressor state.
 *   M      input gradient, rows x cols, leading dimension ldm, dtype m_dtype
 *   err    fp32 error buffer rows x cols (ld lde): read as err_prev, then
 *          overwritten with err_new by occ_step (in place)
 *   P      fp32 rows x rank: output P_hat (orthonormal columns)
 *   Q      fp32 cols x rank: input warm start, output A^T P_hat
 *   M_hat  fp32 rows x cols (ld ldh): output reconstruction P_hat Q^T;
 *          may be NULL when OCC_NO_MHAT is passed */
typedef struct {
  const void* M;
  int32_t m_dtype; /* occ_dtype_t */
  int32_t reserved;
  int64_t rows, cols, ldm;
  float* err;
  int64_t lde;
  float* P;
  float* Q;
  float* M_hat;
  int64_t ldh;
} occ_mat_t;

/* Library ABI version (OCC_ABI_VERSION). */
int occ_abi_version(void);

/* Static description of a status code; never NULL. */
const char* occ_status_str(int status);

/* Workspace bytes that occ_step_batched (count matrices) or occ_step
 * (count = 1) needs for these shapes, rank and iters.  The value does not
 * depend on the pointers.  Returns 0 for invalid arguments. */
size_t occ_workspace_bytes(const occ_mat_t* mats, int count, int rank, int iters);

/* Workspace bytes occ_compress needs for one m x n matrix whose M has dtype
 * m_dtype (the tiling of the large-rank passes depends on it).  Returns 0 for
 * invalid arguments. */
size_t occ_compress_workspace_bytes(int64_t m, int64_t n, int m_dtype, int rank, int iters);

/* Clear the workspace header (sticky flags) on `stream`.  Call once after
 * allocating a workspace; the rest of the workspace needs no initialisation. */
occ_status_t occ_workspace_init(void* ws, size_t ws_bytes, occ_stream_t stream);

/* Compression only (Sec. 2.3 power iteration with the Sec. 5.1 error add):
 * A = M + err_prev (err_prev is read, not modified; NULL means zero);
 * Q (n x rank) is the warm start on entry and A^T P_hat on return;
 * P (m x rank) receives P_hat. */
occ_status_t occ_compress(const void* M, int m_dtype, int64_t m, int64_t n, int64_t ldm,
                          const float* err_prev, int64_t lde, float* P, float* Q,
                          int rank, int iters, void* ws, size_t ws_bytes,
                          occ_stream_t stream);

/* Decompression (Sec. 9.6): M_hat = P Q^T with P m x rank and Q n x rank,
 * fp32 products with fp32 accumulation, M_hat fp32 (m x n, ld ldh). */
occ_status_t occ_decompress(const float* P, const float* Q, int64_t m, int64_t n, int rank,
                            float* M_hat, int64_t ldh, occ_stream_t stream);

/* Decompression on the receiving side of compressed backpropagation (Sec. 5:
 * the next pipeline stage rebuilds the activation gradient from the two
 * factors it received and continues its backward pass with it).  As
 * occ_decompress, with `flags` (OCC_DEC_*):
 *   OCC_DEC_SPLIT_BF16  the products occ_step runs for a bf16 M, so that
 *                       M_hat is bitwise the one the fused step writes;
 *   OCC_DEC_OUT_BF16    M_hat is stored as bf16 (M_hat points to uint16 bf16
 *                       bit patterns, ld ldh elements): each element is the
 *                       fp32 result rounded to nearest even, relative error
 *                       at most 2^-9 per element.
 * Unknown flag bits return OCC_E_FLAGS. */
occ_status_t occ_decompress_ex(const float* P, const float* Q, int64_t m, int64_t n, int rank,
                               unsigned flags, void* M_hat, int64_t ldh, occ_stream_t stream);

/* Error update (Sec. 5.1): err_new = (M + err_prev) - M_hat, elementwise.
 * err_prev and err_new share the leading dimension lde; err_new may equal
 * err_prev (in place); err_prev NULL means zero (lde is then err_new's). */
occ_status_t occ_err_update(const void* M, int m_dtype, int64_t m, int64_t n, int64_t ldm,
                            const float* err_prev, int64_t lde, const float* M_hat,
                            int64_t ldh, float* err_new, occ_stream_t stream);

/* Fused compress + decompress + error update of one matrix; err is updated
 * in place.  Bitwise equal to occ_compress, occ_decompress_ex (with
 * OCC_DEC_SPLIT_BF16 when M is bf16) and occ_err_update called in sequence on
 * the same inputs. */
occ_status_t occ_step(const occ_mat_t* mat, int rank, int iters, unsigned flags,
                      void* ws, size_t ws_bytes, occ_stream_t stream);

/* occ_step on `count` independent matrices (all of one pipeline stage,
 * Sec. 7), one kernel launch per pass for the whole batch.  All matrices
 * share rank, iters and M dtype.  Each result is bitwise equal to occ_step
 * on that matrix alone. */
occ_status_t occ_step_batched(const occ_mat_t* mats, int count, int rank, int iters,
                              unsigned flags, void* ws, size_t ws_bytes,
                              occ_stream_t stream);

/* Row-sparse step for embedding gradients.  The first pipeline stage's copy
 * of the embedding converts the batch's words into embedding values (Sec. 6),
 * so the gradient of that lookup is zero outside the rows of the words the
 * batch contains.  `rows` (DEVICE pointer, n_rows int32 entries, strictly
 * increasing, each in [0, mat->rows)) lists the rows to compress; the call
 * compresses the n_rows x cols matrix of those rows of M + err and reads and
 * writes nothing else of M, err and M_hat: every other row of err and M_hat
 * is left untouched.  When M and err are zero outside the listed rows (the
 * list is the union of the nonzero rows of both), the result equals
 * occ_step on the whole matrix with M_hat zero in the unlisted rows.
 *   mat->P   receives P_hat in compact form: n_rows x rank, row i belonging to
 *            matrix row rows[i];
 *   mat->Q   warm start in, A^T P_hat out (cols x rank), as in occ_step.
 * Requires n_rows >= rank, except n_rows == 0 (then A is zero: Q is set to
 * zero and OCC_F_RANK_DEFICIENT raised); a caller with fewer live rows than
 * `rank` can list additional zero rows.  The list is checked on the device:
 * a violation raises OCC_F_BAD_ROWS.  Workspace: occ_step_rows_workspace_bytes. */
occ_status_t occ_step_rows(const occ_mat_t* mat, const int32_t* rows, int64_t n_rows, int rank,
                           int iters, unsigned flags, void* ws, size_t ws_bytes,
                           occ_stream_t stream);

/* Workspace bytes occ_step_rows needs for n_rows listed rows of a matrix with
 * `cols` columns and M dtype m_dtype.  Returns 0 for invalid arguments. */
size_t occ_step_rows_workspace_bytes(int64_t n_rows, int64_t cols, int m_dtype, int rank,
                                     int iters);

/* occ_step_batched without a workspace argument and without any device
 * allocation, for callers that cannot allocate: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  The
 * workspace is a static device array of OCC_NOALLOC_MAX_BYTES inside the
 * library (one per GPU, held until the process ends); a call whose
 * occ_workspace_bytes exceeds it returns OCC_E_WORKSPACE before anything is
 * enqueued.  Every call on one GPU shares that GPU's array: calls that
 * overlap in time on one GPU (other streams, other threads) race, so callers
 * order them.  Numeric flags are OR-ed into *flags_out (a DEVICE word the
 * caller owns and clears), or dropped when flags_out is NULL.  Results are
 * bitwise those of occ_step_batched on the same arguments. */
#define OCC_NOALLOC_MAX_BYTES ((size_t)64 << 20)
occ_status_t occ_step_batched_noalloc(const occ_mat_t* mats, int count, int rank, int iters,
                                      unsigned flags, uint32_t* flags_out, occ_stream_t stream);

/* Selective stage compression (Sec. 7), host-side model.  With pipeline
 * parallelism the later stages finish their backward passes first and start
 * their data-parallel gradient exchange early; the exchange of the earliest
 * stage is left exposed.  Compressing the exchanges of chosen stages,
 * starting from the earliest, trades compression error for time; each choice
 * moves the bottleneck to another stage.  Times are in one unit of the
 * caller's choice; no device is touched. */

/* When each stage's last backward pass ends under the one-forward-one-
 * backward pipeline schedule (Sec. 2.2), by event simulation: n_stages
 * uniform stages, n_micro micro-batches, t_fwd / t_bwd per micro-batch and
 * stage, t_p2p per hop between adjacent stages.  bwd_done receives n_stages
 * values; *t_end (if not NULL) the end of the schedule.  Invalid counts or
 * negative / non-finite times return OCC_E_SHAPE. */
occ_status_t occ_pipeline_1f1b(int n_stages, int n_micro, double t_fwd, double t_bwd,
                               double t_p2p, double* bwd_done, double* t_end);

/* One stage for occ_sc_select. */
typedef struct {
  double bwd_done;        /* end of the stage's last backward pass */
  double comm;            /* its data-parallel gradient exchange, uncompressed */
  double comm_compressed; /* the exchange of the low-rank factors instead */
  double compress;        /* compressor time on the stage's gradients (e.g. a
                             measured occ_step_batched over the stage) */
} occ_stage_t;

/* Chooses the stages to compress: the exchange of stage s ends at
 * bwd_done + comm, or bwd_done + compress + comm_compressed when compressed.
 * Starting with none compressed, while fewer than max_compressed are, the
 * stage whose exchange ends last is compressed if that ends it earlier; the
 * selection stops at the first bottleneck that is compressed already or would
 * not gain.  selected[s] = 1 for a chosen stage, else 0; *n_selected (if not
 * NULL) the count; *t_end (if not NULL) the end of the last exchange, the
 * least that any choice of at most max_compressed stages reaches. */
occ_status_t occ_sc_select(const occ_stage_t* stages, int n_stages, int max_compressed,
                           uint8_t* selected, int* n_selected, double* t_end);

/* Read (and optionally clear) the sticky numeric flags of a workspace.
 * Synchronises `stream`. */
occ_status_t occ_get_flags(void* ws, uint32_t* flags_out, int clear, occ_stream_t stream);

/* Per-kernel timing with HIP events, for benchmarks.  Between
 * occ_profile_begin and occ_profile_end every kernel the library launches is
 * bracketed by events on its stream.  occ_profile_end synchronises those
 * events and fills up to `max` records (kernel name, launches, total
 * milliseconds), returning the number of distinct kernels in *n_out.  Not
 * thread-safe; intended for single-threaded measurement. */
typedef struct {
  char name[48];
  int32_t launches;
  int32_t reserved;
  double total_ms;
} occ_kernel_time_t;

occ_status_t occ_profile_begin(void);
occ_status_t occ_profile_end(occ_kernel_time_t* out, int max, int* n_out);

#ifdef __cplusplus
}
#endif

#endif /* OPTCC_H */
