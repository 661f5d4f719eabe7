/*
 * turbomuon.h - C ABI of the MI355X (gfx950) Turbo-Muon orthogonalizer.
 *
 * The library approximates the polar factor of gradient matrices with the
 * pre-conditioned Newton-Schulz iteration of arXiv 2512.04632:
 *
 *   Algorithm 2 (Turbo-Muon): A0 = Gram of X0; AOL vector
 *     s_i = 1 / sqrt(sum_j |A0_ij|)                       (eq. (aol), Sec. 4.1)
 *   X1 = X0 scaled by s, A1 = diag(s) A0 diag(s) (no second product), then for
 *   k = 1..t:  A_k = Gram(X_k) (k >= 2), B_k = b_k A_k + c_k A_k^2,
 *              X_{k+1} = a_k X_k + X_k B_k                (Algorithm 1, eq. (ns_quintic))
 *   Algorithm 1 (Muon) instead scales by 1 / ||X0||_F (precond FROBENIUS); the
 *   Schatten-4 variant of the paper's appendix on other pre-conditionings scales
 *   by (sum_i sigma_i^4)^(-1/4) = ||A0||_F^(-1/2), again from the first Gram.
 *
 * Orientation.  For an m x n input with m <= n (square included) the Gram is
 * the m x m matrix X X^T and the AOL vector scales rows; for m > n it is the
 * n x n matrix X^T X and scales columns.  The Gram is always min(m, n) square
 * (Sec. 4.1 keeps the extra memory at O(min(m, n))).  The output keeps the
 * input's layout.
 *
 * Arithmetic.  bf16 entry points store X, A and B in bfloat16 (round to
 * nearest even) and accumulate every product in fp32 on the matrix cores; the
 * AOL row sums are taken from the fp32 Gram accumulators.  f32 entry points
 * store and multiply in fp32.  Results are deterministic: no float atomics.
 *
 * Small matrices.  A bf16 call with iters >= 1 whose every matrix has
 * min(m, n) <= 128 and fits, zero padded to multiples of 32, in one compute
 * unit's 160 KB of LDS (min(m, n) = 64: max(m, n) <= 1088; 128: <= 320) runs
 * as a single launch, one workgroup per matrix, with no workspace.  Its
 * results are bit for bit those of the tiled kernels that other calls use
 * (the same products in the same order, the same roundings); setting
 * TM_DISABLE_FUSED in the environment sends such calls to the tiled kernels.
 *
 * Streams and memory.  All work is enqueued on `stream` (a hipStream_t passed
 * as void*, NULL = the legacy default stream) without host synchronisation;
 * results are valid once the stream has passed the call.  Matrix pointers are
 * device pointers owned by the caller.  The library owns a workspace per
 * (device, stream), grown on first use with hipMalloc and kept until
 * tm_release_workspaces() or process exit; growing it synchronises `stream`.
 * Calls on different streams may run concurrently; calls that overlap on the
 * same stream are ordered by the stream.  The cache is keyed by the stream
 * handle: synchronise a stream before destroying it, since a stream created
 * later may receive the same handle and reuse that workspace.
 *
 * Graph capture.  A call on a stream whose workspace is already large enough
 * (an earlier call of the same or larger shapes on that stream) allocates
 * nothing and synchronises nothing, so it can be captured into a HIP graph;
 * the captured kernels keep that workspace's address.  A call under capture
 * whose workspace is too small returns TM_ERR_UNSUPPORTED (nothing can be
 * allocated during capture).  A workspace once used under capture is never
 * freed or reused in place by a larger call: a later, larger eager call on the
 * same stream handle (torch hands out pooled stream handles, so another stream
 * object may share it) gets a new workspace and the captured one stays valid
 * until tm_release_workspaces(), which must not be called while such a graph
 * is in use.  Graphs captured on one stream share its workspace: do not replay
 * them concurrently (on different streams) with each other or with eager calls
 * on that stream.  tm_orthogonalize_noalloc needs no workspace at all.
 *
 * Errors.  Arguments are validated before anything is enqueued; an invalid
 * call returns a negative status and leaves memory untouched.  Failures of the
 * HIP runtime return TM_ERR_HIP.  tm_last_error() gives a thread-local message
 * for the last failure.  Input values are not checked: NaN/Inf propagate.
 */
#ifndef TURBOMUON_H
#define TURBOMUON_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int tm_status;

#define TM_OK               0
#define TM_ERR_INVALID_ARG  (-1) /* null pointer, size or iteration count out of range, unknown precond */
#define TM_ERR_UNSUPPORTED  (-2) /* pointer not element aligned, no gfx950 device, launch too large */
#define TM_ERR_NO_MEMORY    (-3) /* workspace allocation failed */
#define TM_ERR_HIP          (-4) /* a HIP runtime call or kernel launch failed */

/* Pre-conditioning of the first iteration. */
#define TM_PRECOND_NONE       0  /* X1 = X0 */
#define TM_PRECOND_FROBENIUS  1  /* X1 = X0 / ||X0||_F: Algorithm 1 (Muon); zero stays zero */
#define TM_PRECOND_AOL        2  /* X1 = AOL(X0), eq. (aol): Algorithm 2 (Turbo-Muon) */
#define TM_PRECOND_SCHATTEN4  3  /* X1 = X0 / ||X0||_S4 with ||X0||_S4 = ||A0||_F^(1/2) from the
                                    first Gram (appendix on other pre-conditionings) */

/* Limits checked by every entry point. */
#define TM_MAX_DIM    65536      /* m, n <= TM_MAX_DIM */
#define TM_MAX_ITERS  64         /* 0 <= iters <= TM_MAX_ITERS */

/*
 * tm_orthogonalize - Algorithm 2 (precond AOL) or Algorithm 1 (FROBENIUS/NONE)
 * on `batch` bf16 matrices, in place.
 *
 *   X       device pointer, `batch` row-major m x n bfloat16 matrices stored
 *           back to back (matrix b starts at X + b*m*n); aligned to the
 *           element size (16-byte alignment and n % 8 == 0 enable vector loads).
 *           Overwritten with the result X_{iters+1}.
 *   m, n    1 <= m, n <= TM_MAX_DIM.
 *   batch   >= 0; 0 is a no-op returning TM_OK.
 *   iters   number t of (Gram, polynomial, update) triples, 0..TM_MAX_ITERS.
 *           iters = 0 returns the pre-conditioned X1.  Turbo-Muon's default
 *           is 4 (Sec. 2), Muon's 5.
 *   coeffs  host array of iters*3 floats (a_k, b_k, c_k) in iteration order,
 *           read during the call only; NULL selects the constant triple
 *           (3.4445, -4.7750, 2.0315) for every iteration.
 *   precond TM_PRECOND_*.
 *   stream  hipStream_t as void*.
 */
tm_status tm_orthogonalize(void* X, int64_t m, int64_t n, int64_t batch, int iters,
                           const float* coeffs, int precond, void* stream);

/* Same contract with fp32 storage and fp32 matrix-core arithmetic. */
tm_status tm_orthogonalize_f32(float* X, int64_t m, int64_t n, int64_t batch, int iters,
                               const float* coeffs, int precond, void* stream);

/*
 * tm_orthogonalize_grouped - `count` independent bf16 matrices of arbitrary
 * shapes, processed together: every phase of the iteration (Gram, AOL
 * vector, polynomial, update) is one launch over the tiles of all matrices.
 *
 *   X       host array of `count` device pointers (element aligned, pairwise
 *           non-overlapping); matrix g is row-major m[g] x n[g].
 *   m, n    host arrays of `count` sizes, each in 1..TM_MAX_DIM.
 *   count   >= 0; 0 is a no-op.
 *   other arguments as tm_orthogonalize; the same coefficients and
 *   pre-conditioning apply to every matrix.  The host arrays are read during
 *   the call only.
 */
tm_status tm_orthogonalize_grouped(void* const* X, const int64_t* m, const int64_t* n,
                                   int64_t count, int iters, const float* coeffs,
                                   int precond, void* stream);

/* Grouped variant with fp32 storage. */
tm_status tm_orthogonalize_grouped_f32(float* const* X, const int64_t* m, const int64_t* n,
                                       int64_t count, int iters, const float* coeffs,
                                       int precond, void* stream);

/*
 * tm_muon_step_grouped - one optimizer step over `count` fp32 parameter
 * matrices: Muon's step with its orthogonalization done by this library (the
 * paper uses Turbo-Muon as a drop-in replacement of Muon's orthogonalization;
 * its steepest-descent appendix writes the update as -eta PolarFactor(G S)).
 * Per matrix g (rows m[g], columns n[g], row-major):
 *
 *   M <- momentum M + G
 *   U  = G + momentum M   if nesterov, else U = M      (rounded to bf16)
 *   O  = the bf16 orthogonalization of U (tm_orthogonalize_grouped semantics:
 *        iters, coeffs, precond as there)
 *   W <- W (1 - lr weight_decay) - lr scale O,
 *        scale = sqrt(max(1, m[g] / n[g])) if shape_scale, else 1
 *
 *   W, G, M  host arrays of `count` device pointers to fp32 matrices (4-byte
 *            aligned; W and M updated in place, G read only; no two of all
 *            these matrices may overlap).
 *   m, n     host arrays of sizes, each in 1..TM_MAX_DIM.
 * U lives in a second library-owned buffer per (device, stream), grown like
 * the workspace.  Errors as tm_orthogonalize_grouped.
 */
tm_status tm_muon_step_grouped(float* const* W, const float* const* G, float* const* M,
                               const int64_t* m, const int64_t* n, int64_t count, float lr,
                               float momentum, int nesterov, float weight_decay, int shape_scale,
                               int iters, const float* coeffs, int precond, void* stream);

/*
 * tm_schedule_tail - fewer iterations from a coefficient schedule designed for
 * more (appendix on the tuning of Newton-Schulz coefficients: a schedule
 * computed for a fixed number of iterations runs fewer by keeping its last
 * rows).
 *
 *   schedule  host array of rows*3 floats (a_k, b_k, c_k) in iteration order.
 *   rows      rows of the schedule, 1..TM_MAX_ITERS.
 *   iters     iterations to run, 0..rows.
 * Returns schedule + 3*(rows - iters): the last `iters` rows, to pass as the
 * `coeffs` of a call with that many iterations.  Reads no element and
 * allocates nothing; NULL (detail in tm_last_error) for a NULL schedule or
 * rows / iters out of range.
 */
const float* tm_schedule_tail(const float* schedule, int rows, int iters);

/*
 * tm_orthogonalize_noalloc - tm_orthogonalize for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc.  Same arguments, kernels and launch plan as
 * tm_orthogonalize (results are bitwise equal to it), but the workspace is a
 * static device array of TM_NOALLOC_SCRATCH_BYTES per GPU, placed with the
 * library's code object and held until the process ends, instead of the
 * per-stream cache.  The call allocates nothing, frees nothing and
 * synchronises nothing; the timing hooks do not apply to it.
 *
 *   Limit   the call's workspace (tm_workspace_bytes over `batch` copies of
 *           the shape m x n, dtype_bytes 2) must fit in
 *           TM_NOALLOC_SCRATCH_BYTES: e.g. one 2048 x 2048 matrix (48 MiB),
 *           one 1024 x 4096 (24 MiB) or a batch of 4 of 768 x 3072 (54 MiB);
 *           a larger call returns TM_ERR_UNSUPPORTED before anything is
 *           enqueued.
 *   Sharing every call on one GPU uses that GPU's one array: calls that
 *           overlap in time on a GPU (other streams or host threads) race and
 *           must be serialised by the caller.  The array keeps the last call's
 *           contents; nothing in it needs to start at zero.
 */
#define TM_NOALLOC_SCRATCH_BYTES 67108864   /* 64 MiB */
tm_status tm_orthogonalize_noalloc(void* X, int64_t m, int64_t n, int64_t batch, int iters,
                                   const float* coeffs, int precond, void* stream);

/* Bytes of workspace a call with these shapes needs (0 on invalid shapes).
 * dtype_bytes is 2 (bf16) or 4 (fp32).  An upper bound: a bf16 call that the
 * fused small-matrix kernel serves uses none. */
uint64_t tm_workspace_bytes(const int64_t* m, const int64_t* n, int64_t count,
                            int dtype_bytes);

/* Free every cached workspace.  Synchronises the device first; must not be
 * called while another thread is inside a tm_* call. */
tm_status tm_release_workspaces(void);

/* Kernel phases, as counted by the timing hooks below. */
#define TM_PHASE_TRANSPOSE_IN  0  /* tall input: W = X^T */
#define TM_PHASE_FROB          1  /* partial sums of squares of X0 (Algorithm 1, first line) or of A0 (Schatten-4) */
#define TM_PHASE_GRAM          2  /* A = X X^T, upper tiles (+ AOL row sums at iteration 1) */
#define TM_PHASE_AOL_VECTOR    3  /* s_i = 1/sqrt(row sum) (Algorithm 2, second line) */
#define TM_PHASE_POLY          4  /* B = b A + c A^2 */
#define TM_PHASE_UPDATE        5  /* X <- a X + B X */
#define TM_PHASE_APPLY_SCALE   6  /* iters = 0: X1 = diag(s) X0 */
#define TM_PHASE_COPY_OUT      7  /* iters = 1: result copied into the caller's buffer */
#define TM_PHASE_LOAD_IN       8  /* bf16: X (or X^T) copied into the zero-padded workspace */
#define TM_PHASE_SCALE_A       9  /* bf16: A1 = diag(s) A0 diag(s) (X1 is never stored: the first
                                    polynomial keeps B~ diag(s) and the update reads X0) */
#define TM_PHASE_OPT_MOMENTUM 10  /* optimizer step: momentum and the bf16 matrix to orthogonalize */
#define TM_PHASE_OPT_APPLY    11  /* optimizer step: parameter update */
#define TM_PHASE_FUSED        12  /* bf16 calls of small matrices: every iteration in one launch */
#define TM_NUM_PHASES         13

/* Timing hooks (a profiling aid for benchmarks).  While enabled, every kernel
 * launch of later calls is bracketed by a pair of HIP events recorded on the
 * call's stream.  tm_timing_read synchronises the recorded events and returns
 * the summed event time (ms) and launch count of one phase since the last
 * reset; tm_timing_reset drops the records.  Not thread-safe with concurrent
 * tm_* calls on other threads. */
tm_status tm_timing_enable(int enable);
tm_status tm_timing_read(int phase, double* total_ms, int64_t* launches);
tm_status tm_timing_reset(void);

/* Static description of a status code. */
const char* tm_status_string(tm_status s);

/* Thread-local detail of the last failure in this thread ("" if none). */
const char* tm_last_error(void);

/* Library version, "major.minor.patch". */
const char* tm_version(void);

#ifdef __cplusplus
}
#endif

#endif /* TURBOMUON_H */
