/*
 * ff.h -- C ABI of the FlipFlop Hessian engine for AMD MI355X (gfx950).
 *
 * The engine estimates the Kronecker-factored Hessian H ~ A (x) B of one
 * linear layer W (m x n) from N samples G_i (m x n), with
 * H = E[vec(G) vec(G)^T] and column-major vec (paper, Section 2 notation and
 * Section 5).  A (n x n) is the input-side factor, B (m x m) the output-side
 * factor.  The estimate is the flip-flop iteration of Section 5, i.e. the
 * matrix-normal maximum-likelihood iteration:
 *
 *     B <- (1/(N n)) sum_i G_i A^-1 G_i^T          (update of B for fixed A)
 *     A <- (1/(N m)) sum_i G_i^T B^-1 G_i          (update of A for fixed B)
 *     c = tr(A)/n;  A <- A/c;  B <- B c            (scale fixed: tr(A) = n)
 *
 * started from A = I_n with B updated first (Appendix B convention; one
 * iteration = one update of B and one of A).  Optional damping (Appendix B)
 * adds kappa * tr(X)/dim * I to each factor right after its update.
 *
 * Conventions shared by every entry point
 *  - Every call returns an ff_status; no C++ exception crosses this ABI.
 *    On error, out-parameters are left untouched (except *iters_done, which
 *    ff_iterate always writes).  ff_last_error() gives a message for the
 *    most recent failure on the calling thread.
 *  - The library never allocates device memory.  G, the workspace, A0/B0,
 *    X/Y and the output buffers are owned by the caller.  Host memory for
 *    the handle itself is allocated by ff_init and freed by ff_destroy.
 *  - Device pointers must be 256-byte aligned where stated, otherwise
 *    16-byte aligned.  All matrices are dense row-major.
 *  - Work is enqueued on cfg.stream (a hipStream_t; NULL = default stream).
 *    ff_iterate, ff_factors(on_host=1), ff_kron_apply and ff_objective
 *    synchronise that stream once before returning; the others return
 *    without waiting.
 *  - A handle is not thread-safe; distinct handles are independent.  The
 *    device that is current at ff_init must be current for every later
 *    call on the handle.
 */
#ifndef FF_H
#define FF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ff_handle_s* ff_handle;

typedef enum {
  FF_OK = 0,
  FF_ERR_INVALID_ARG = 1, /* bad shape, dtype, pointer, alignment or option */
  FF_ERR_NOT_SPD = 2,     /* a factor to be inverted had a pivot <= 0 or NaN */
  FF_ERR_WORKSPACE = 3,   /* workspace missing, too small or misaligned */
  FF_ERR_HIP = 4,         /* a HIP runtime call failed */
  FF_ERR_STATE = 5        /* call not valid in the handle's state */
} ff_status;

/* Element type of the samples G.  The factors are always fp32.
 * FF_F32: every product runs in fp32 (fp32 matrix cores, fp32 accumulate).
 * FF_BF16: G is bf16; the whitening operand L^-1 and the whitened samples
 * are rounded to bf16 (round to nearest even) and all products accumulate
 * in fp32 on the bf16 matrix cores; factorisations stay in fp32. */
typedef enum { FF_F32 = 0, FF_BF16 = 1 } ff_dtype;

/* Update order.  B_FIRST (default; Appendix B): start from A0 (I_n if NULL),
 * each iteration updates B then A.  A_FIRST (Section 5 indexing): start from
 * B0 (I_m if NULL), each iteration updates A then B.  Both end each
 * iteration with the trace normalisation tr(A) = n and share the same fixed
 * point; their iterates differ. */
typedef enum { FF_ORDER_B_FIRST = 0, FF_ORDER_A_FIRST = 1 } ff_order;

/* ff_kron_apply modes: (A (x) B) vec(X) = vec(B X A) (A symmetric), and
 * its inverse vec(B^-1 X A^-1). */
typedef enum { FF_APPLY = 0, FF_APPLY_INV = 1 } ff_apply_mode;

/* How the samples are given.  FF_SAMPLES_DENSE: N matrices G_i (m x n).
 * FF_SAMPLES_RANK1: N tokens, sample t being the rank-one matrix
 * G_t = g_t x_t^T of an output gradient g_t (m) and an input x_t (n), the
 * form the paper runs (Section 5 writes both half steps for it:
 * A <- E[(g^T B^-1 g) x x^T], B <- E[(x^T A^-1 x) g g^T]; Table 1, FlipFlop
 * row).  The iteration, scalings and outputs are those of the dense form
 * applied to these G_t; the cost per iteration is 2 N (m^2 + n^2). */
typedef enum { FF_SAMPLES_DENSE = 0, FF_SAMPLES_RANK1 = 1 } ff_sample_form;

/* Which Kronecker approximation A (x) B of H = E[x x^T (x) g g^T] the
 * iteration computes (Table 1).  Every estimator ends each iteration with
 * the trace normalisation tr(A) = n and applies the damping option after
 * each update.
 *   FF_EST_FLIPFLOP: the flip-flop iteration (Section 5), the default.
 *   FF_EST_FROBENIUS: the same iteration with the factors in place of their
 *     inverses, B <- (1/(N n)) sum_i G_i A G_i^T, A <- (1/(N m)) sum_i G_i^T B G_i
 *     (rank-one form: weights x^T A x and g^T B g), a power iteration for
 *     min ||H - A (x) B||_F (Section 5).  Nothing is factorised or
 *     inverted: each half step forms P_i = G_i F (dense, twice the
 *     triangular whitening's work; the bf16 path rounds F and P to bf16)
 *     and sums the upper tiles of P_i G_i^T, so a factor of any condition
 *     number (the undamped iteration's estimates lose rank on few samples)
 *     is handled.  Only FF_ORDER_B_FIRST: with A first, the trace
 *     normalisation leaves B's scale growing doubly exponentially.
 *   FF_EST_MARGINAL: A = E[x x^T], B = E[g g^T] (means over the tokens).
 *   FF_EST_INPUT: A = E[x x^T], B = I_m.
 * MARGINAL and INPUT need the rank-one form (they are functions of the
 * tokens, not of G_t); every iteration recomputes the same estimate.  The
 * per-iteration log-likelihood of ff_iterate is the matrix-normal one for
 * FLIPFLOP only; the other estimators report NaN. */
typedef enum {
  FF_EST_FLIPFLOP = 0,
  FF_EST_FROBENIUS = 1,
  FF_EST_MARGINAL = 2,
  FF_EST_INPUT = 3
} ff_estimator;

typedef struct {
  int64_t m, n, N;        /* G is [N][m][n], row-major, contiguous; all >= 1
                             (RANK1: N = number of tokens) */
  ff_dtype dtype;         /* element type of G */
  const void* G;          /* DEVICE pointer, 16-byte aligned, BORROWED: must
                             stay valid and unmodified until ff_destroy */
  void* stream;           /* hipStream_t for all work of this handle */
  ff_order order;
  double damping;         /* kappa >= 0 (0 for the plain iteration) */
  const float* A0;        /* optional DEVICE n x n SPD start for A (B_FIRST);
                             NULL = I_n.  Copied at ff_init */
  const float* B0;        /* optional DEVICE m x m SPD start for B (A_FIRST);
                             NULL = I_m.  Copied at ff_init */
  int whiten_split;       /* FF_BF16 only.  0 = automatic (the default of a
                             zeroed config): each factorisation computes on
                             the device the rounding sensitivity
                             s = (1/dim) sum_j F_jj (F^-1)_jj of its factor F
                             (from the column norms of L^-1; rms whitening
                             distortion 2^-9 sqrt(s/3)); the whitenings use
                             two passes while the latest s of A or of B
                             exceeds 16, and always when fewer than 16
                             samples per dimension determine a factor
                             (min(N m / n, N n / m); rank-one form:
                             N / max(m, n)), one pass otherwise;
                             1 = L^-1 rounded to bf16 once;
                             2 = L^-1 split as hi + lo bf16 parts (two passes,
                             smaller whitening error).  The Frobenius
                             estimator's operand is not an inverse: automatic
                             means one pass there.  Ignored for FF_F32 */
  void* workspace;        /* DEVICE scratch, 256-byte aligned, owned by the
                             caller, >= ff_workspace_size() bytes; must stay
                             valid until ff_destroy */
  size_t workspace_bytes;
  ff_sample_form form;    /* 0 = FF_SAMPLES_DENSE (a zeroed config is dense) */
  const void* x;          /* RANK1: DEVICE [N][n] token inputs, row-major,
                             dtype, 16-byte aligned, BORROWED like G.  G is
                             ignored (may be NULL) */
  const void* g;          /* RANK1: DEVICE [N][m] token output gradients */
  ff_estimator estimator; /* 0 = FF_EST_FLIPFLOP; FROBENIUS needs B_FIRST,
                             MARGINAL and INPUT need FF_SAMPLES_RANK1 */
} ff_config;

/* Bytes of device workspace ff_init needs for cfg (only the shape, dtype and
 * whiten_split fields are read).  Errors: FF_ERR_INVALID_ARG. */
ff_status ff_workspace_size(const ff_config* cfg, size_t* bytes);

/* Validate cfg, lay out the workspace and enqueue the set-up on cfg->stream:
 * the starting factor (A0/B0 or identity) and the internal copies of G
 * (a transposed copy used by the A update; a zero-padded copy when m or n is
 * not a multiple of the tile size).  Does not wait for the stream.
 * Errors: FF_ERR_INVALID_ARG, FF_ERR_WORKSPACE, FF_ERR_HIP. */
ff_status ff_init(const ff_config* cfg, ff_handle* out);

/* Run up to `iters` (>= 0) flip-flop iterations (Section 5) continuing from
 * the handle's current factors, then synchronise the stream.
 * *iters_done receives the number of iterations completed by this call.
 * loglik (host array of `iters` doubles, may be NULL) receives, per completed
 * iteration, the matrix-normal log-likelihood of the samples under the new
 * A (x) B, -(N/2)(m log|A| + n log|B|) - T/2 - (N m n/2) log 2 pi, with the
 * log-determinants from the Cholesky pivots and the trace term
 * T = sum_i tr(B^-1 G_i A^-1 G_i^T) in closed form: N m n after a
 * maximum-likelihood half step (Section 5 trace identity); with damping
 * kappa > 0 (Appendix B), N d' (d - kappa/(1 + kappa) (tr(F)/d) ||L_F^-1||_F^2)
 * for the second-updated factor F (dimension d, the other one d') and its
 * Cholesky factor L_F, which the next iteration needs anyway.  The other
 * estimators report NaN.
 * FF_ERR_NOT_SPD: a factor to be inverted was not positive definite (the
 * paper assumes invertibility, Section 2; use damping > 0).  The handle then
 * keeps the factors of the last completed iteration and stays usable.  An
 * iteration whose new factor is singular still completes (its log-likelihood
 * entry is NaN); the next iteration, which must invert it, fails.
 * Errors: FF_ERR_INVALID_ARG, FF_ERR_NOT_SPD, FF_ERR_HIP. */
ff_status ff_iterate(ff_handle h, int iters, int* iters_done, double* loglik);

/* ff_iterate with the convergence diagnostic of the iteration.  After each
 * iteration g the device evaluates, in fp64, the relative change of the
 * normalised Kronecker product
 *   delta_g = ||A_g (x) B_g - A_{g-1} (x) B_{g-1}||_F / (||A_{g-1}||_F ||B_{g-1}||_F)
 * from ||X (x) Y - X' (x) Y'||^2 = ||dX||^2 ||Y||^2 + ||X'||^2 ||dY||^2
 * + 2 <dX, X'> <Y, dY> (dX = X - X', dY = Y - Y'; the mn x mn product is
 * never formed; for the first iteration of a handle the previous iterate is
 * the start A0 / B0 or identity).  delta (host array of max_iters doubles,
 * may be NULL) receives delta_g per completed iteration.  tol > 0 stops after
 * the first iteration with delta_g <= tol; that iteration is complete (its
 * factors, log-likelihood and the factorisation the next one needs) and
 * *iters_done counts it.  tol == 0 runs all max_iters.  No host round trip
 * per iteration: later iterations already enqueued return at once on the
 * device.  Errors: as ff_iterate, and FF_ERR_INVALID_ARG for a negative or
 * non-finite tol. */
ff_status ff_iterate_tol(ff_handle h, int max_iters, double tol, int* iters_done, double* loglik,
                         double* delta);

/* One half step of Section 5 with the other factor held fixed, unscaled and
 * undamped: FF_HALF_B: out (m x m) = (1/(N n)) sum_i G_i F^-1 G_i^T with
 * F (n x n); FF_HALF_A: out (n x n) = (1/(N m)) sum_i G_i^T F^-1 G_i with
 * F (m x m).  (The Frobenius estimator uses F in place of F^-1.)  F: DEVICE
 * fp32 row-major SPD (lower triangle read), or NULL for the handle's current
 * factor; out: DEVICE fp32, 16-byte aligned.  Same path as an iteration's
 * update (factorisation, whitening, symmetric product).  The handle's factors
 * are untouched; the next ff_iterate refactorises them.  Synchronises the
 * stream.  Errors: FF_ERR_INVALID_ARG (also for the Marginal and Input
 * estimators), FF_ERR_NOT_SPD (F not positive definite), FF_ERR_HIP. */
typedef enum { FF_HALF_B = 0, FF_HALF_A = 1 } ff_half;
ff_status ff_half_step(ff_handle h, ff_half which, const float* F, float* out);

/* Copy the current factors: A (n x n) and B (m x m), fp32 row-major,
 * normalised to tr(A) = n.  on_host = 0: A and B are device pointers and the
 * copy is enqueued on the stream; on_host = 1: host pointers, the call waits.
 * Either pointer may be NULL to skip that factor.
 * Errors: FF_ERR_INVALID_ARG, FF_ERR_HIP. */
ff_status ff_factors(ff_handle h, float* A, float* B, int on_host);

/* Apply the current Kronecker factors to `batch` matrices X_b (m x n):
 * FF_APPLY: Y_b = B X_b A  (= (A (x) B) vec(X_b), column-major vec);
 * FF_APPLY_INV: Y_b = B^-1 X_b A^-1.  X and Y are DEVICE fp32 [batch][m][n],
 * 16-byte aligned and must not overlap.  Computed in fp32.
 * Errors: FF_ERR_INVALID_ARG, FF_ERR_NOT_SPD (INV with a singular factor),
 * FF_ERR_HIP. */
ff_status ff_kron_apply(ff_handle h, const float* X, float* Y, int64_t batch,
                        ff_apply_mode mode);

/* The Kronecker-Hessian mismatch objective of the factors A (n x n) and
 * B (m x m), Section 4: with H = (1/N) sum_i vec(G_i) vec(G_i)^T the samples'
 * second moment, the mismatch factor Phi(H, A (x) B) is the ratio of
 * tr(H (A (x) B)^-1) / (m n) to |H|^(1/(m n)) |A|^(-1/n) |B|^(-1/m).  *psi
 * receives its log without the H-only term,
 *   psi = log( (1/(N m n)) sum_i tr(B^-1 G_i A^-1 G_i^T) ) + log|A|/n + log|B|/m
 *       = log Phi(H, A (x) B) + log|H| / (m n),
 * invariant under A -> c A, B -> B / c and minimised by the flip-flop fixed
 * point (Section 5).  A and B are DEVICE fp32 row-major symmetric positive
 * definite matrices (lower triangles read); either may be NULL to use the
 * handle's current factor.  The trace term runs through the handle's path
 * (bf16 whitening on a bf16 handle), the log-determinants come from its fp32
 * Cholesky factorisations.  Synchronises the stream.  The handle's factors
 * are untouched; the next ff_iterate refactorises them.
 * Errors: FF_ERR_INVALID_ARG, FF_ERR_NOT_SPD (A or B not positive definite),
 * FF_ERR_HIP. */
ff_status ff_objective(ff_handle h, const float* A, const float* B, double* psi);

/* Scales of the quantisation grid for ff_quantize.  FF_SCALES_WATERFILL:
 * computed by Corollary 3.2, alpha_j = sqrt(gamma) |A|^(1/2n) / L^A_jj and
 * beta_i = sqrt(gamma) |B|^(1/2m) / L^B_ii with L = RevCholesky (the lower
 * triangular L with positive diagonal and L^T L = M, Section 2), and written
 * to alpha and beta.  FF_SCALES_GIVEN: alpha and beta are inputs (Algorithm 2
 * takes them as given). */
typedef enum { FF_SCALES_WATERFILL = 0, FF_SCALES_GIVEN = 1 } ff_scale_mode;

/* Bytes of the device workspace ff_quantize needs for an m x n weight
 * matrix.  Errors: FF_ERR_INVALID_ARG (m or n < 1 or > 1048576, bytes NULL). */
ff_status ff_quantize_workspace_size(int64_t m, int64_t n, size_t* bytes);

/* WaterKron (Section 3): two-sided GPTQ, Algorithm 2, of the weights W
 * (m x n) under the Kronecker Hessian A (x) B, on the grid
 * V = beta alpha^T (.) Z (Section 2.1).  Entry by entry (columns in order,
 * rows in order within a column) the current value is rounded to the nearest
 * grid point (ties to even) and the error is spread over the entries below
 * and to the right with the outer product of the columns of the normalised
 * inverse factors, L^-1 with each column divided by its diagonal entry, of
 * L^B = RevCholesky(B) and L^A = RevCholesky(A).  The result is the one whose
 * transformed error E = (L~B)^-1 (V - W) (L~A)^-T lies in the cell
 * |E_ij| <= alpha_j beta_i / 2 (L~ the normalised inverses), unique up to ties.
 *
 * h: the handle whose shape (m, n) is used.  W: DEVICE fp32 m x n row-major.
 * A (n x n), B (m x m): DEVICE fp32 symmetric positive definite (lower
 * triangles read); NULL means the handle's current factor.  gamma > 0: the
 * step parameter of FF_SCALES_WATERFILL (ignored for FF_SCALES_GIVEN).
 * alpha (n), beta (m): DEVICE fp32, outputs or inputs by mode; given scales
 * must be finite and > 0.  Z: DEVICE int32 m x n, the integer codes (exact
 * while |Z| < 2^24).  V: DEVICE fp32 m x n, the quantised weights, or NULL.
 * distortion: HOST, receives D_{A,B} = ||L^B (V - W) L^A^T||_F^2 / (m n)
 * (Section 2.3), or NULL.  workspace: DEVICE, 256-byte aligned, at least
 * ff_quantize_workspace_size(m, n) bytes, owned by the caller, contents
 * undefined afterwards.  The factorisations run in fp32, B's on a second
 * stream the handle creates on first use (ordered after the work already on
 * the handle's stream and joined back into it); the handle's factors are
 * untouched (the next ff_iterate refactorises them).  Synchronises the
 * stream.
 * Errors: FF_ERR_INVALID_ARG, FF_ERR_WORKSPACE, FF_ERR_NOT_SPD (A or B not
 * positive definite), FF_ERR_HIP. */
ff_status ff_quantize(ff_handle h, const float* W, const float* A, const float* B,
                      double gamma, ff_scale_mode mode, float* alpha, float* beta, int32_t* Z,
                      float* V, double* distortion, void* workspace, size_t workspace_bytes);

/* For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  One call
 * does what ff_init + ff_iterate + ff_factors(on_host = 0) do, with the same
 * kernels and results, but takes its scratch from a static device array of
 * FF_NOALLOC_SCRATCH_BYTES that the library holds on each device it runs on
 * (until the process ends) instead of a caller workspace, and creates no
 * streams or events (the factorisation's inverse products run on cfg->stream).
 * It calls no allocating routine.  cfg: as for ff_init; cfg->workspace and
 * cfg->workspace_bytes are ignored.  A (n x n) and B (m x m): DEVICE fp32
 * outputs, tr(A) = n.  iters_done / loglik: as ff_iterate.  The call
 * synchronises cfg->stream.  Every call on one device shares that device's
 * array and the set-up rewrites everything it reads, so a call depends on no
 * earlier one; calls that overlap in time on one device (several host
 * threads or streams) race and give undefined results.
 * Errors: FF_ERR_WORKSPACE when ff_workspace_size(cfg) exceeds
 * FF_NOALLOC_SCRATCH_BYTES (the message gives both sizes), and the errors of
 * ff_init and ff_iterate. */
#define FF_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
ff_status ff_fit_noalloc(const ff_config* cfg, int iters, int* iters_done, double* loglik,
                         float* A, float* B);

/* Release the handle (host memory only; waits for the handle's stream).
 * NULL is accepted. */
ff_status ff_destroy(ff_handle h);

/* State of the automatic whitening split (whiten_split = 0): the statistic
 * s of the latest factorisation of A and of B (NaN when not computed: fp32
 * path, forced split, Frobenius estimator, or no factorisation of that side
 * yet) and the passes (1 or 2) the next whitening with each side's operand
 * uses (the same for both sides under the automatic rule; as configured for
 * a forced split).  Synchronises the handle's stream.  Any pointer may be
 * NULL.  Errors: FF_ERR_INVALID_ARG, FF_ERR_HIP. */
ff_status ff_whiten_split_state(ff_handle h, double* s_A, double* s_B, int* passes_A,
                                int* passes_B);

/* Measurement hook (not needed for estimation).  With timing enabled,
 * ff_iterate and ff_quantize bracket each launch of the main kernels with HIP
 * events on the handle's stream and accumulate their durations and
 * algorithmic flop counts; enabling resets the counters.  Kernel ids: 0 = whitening
 * (N m n^2 or N m^2 n flop per launch), 1 = symmetric product over the
 * stacked samples (N n m^2 or N m n^2), 2 = reduction of its partial sums
 * (0 flop), 3 = Cholesky + inverse of one factor (dim^3 / 3 flop), 4 = one
 * launch (one anti-diagonal of 64 x 64 tiles) of the ff_quantize sweep; the
 * m^2 n + m n^2 flop of the products that spread the rounding errors are
 * shared evenly over its ceil(m/64) + ceil(n/64) - 1 launches.
 * Errors: FF_ERR_INVALID_ARG, FF_ERR_HIP. */
ff_status ff_set_timing(ff_handle h, int enable);
ff_status ff_kernel_timing(ff_handle h, int kernel, int64_t* launches, double* total_ms,
                           double* alg_flop);

/* Static description of a status code. */
const char* ff_status_string(ff_status s);

/* Message of the most recent failing call on this thread ("" if none). */
const char* ff_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* FF_H */
