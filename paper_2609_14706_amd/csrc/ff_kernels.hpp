// Host-side launchers of the FlipFlop kernels.  Every launcher enqueues on
// the given stream, checks its shape preconditions on the host and returns
// the launch status; none allocates memory.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ff {

typedef uint16_t bf16_t;

// ---------------------------------------------------------------- bf16 path
// Tile of the bf16 matrix-core kernels; every padded dimension is a multiple.
constexpr int kTileBF16 = 256;

// Whitening (triangular product, bf16 matrix cores, fp32 accumulation):
//   C[r][c] = sum_{k <= c} X[r][k] * Y[c][k]  (+ same with Y2 when non-null
//   and, if use2 is non-null, *use2 != 0 or *use2b != 0 (use2b may be null):
//   flags read on the device at launch)
// X: rows x Kp, Y/Y2: Kp x Kp lower triangular, C: rows x Kp, all row-major
// bf16 with leading dimension Kp.  rows and Kp are multiples of 256.  With
// full = true, Y/Y2 are dense and k runs over all of Kp (C = X Y^T).
hipError_t launch_whiten_bf16(const bf16_t* X, const bf16_t* Y, const bf16_t* Y2, const int* use2,
                              const int* use2b, bf16_t* C, int64_t rows, int64_t Kp, const int* st,
                              hipStream_t s, bool full = false);

// Row norms of the whitened rows without storing them: part[r][2 cj + h]
// (2 Kp / 256 floats per row) = sum of squares of (X Y^T (+ X Y2^T))[r][.]
// over the 128 columns h of column tile cj.  Same shape and Y2 rules as above.
hipError_t launch_whiten_norm_bf16(const bf16_t* X, const bf16_t* Y, const bf16_t* Y2,
                                   const int* use2, const int* use2b, float* part, int64_t rows,
                                   int64_t Kp, const int* st, hipStream_t s);

// Symmetric rank-k product over segmented rows, split over k:
//   P[z][tile] = partial sums of X X^T for upper tiles (ti <= tj),
// where row r of X is the concatenation over segments s < nseg of
// X[s * seg_stride + r * ld .. + ld).  dim_p (rows) and ld are multiples of
// 256 and 64.  P holds splits * T(T+1)/2 tiles of 256 x 256 fp32 in the
// matrix-core fragment order (decoded by launch_reduce_frag).  With Xb
// non-null (same layout), the upper tiles of X Xb^T instead (for a product
// the caller knows to be symmetric).
hipError_t launch_syrk_bf16(const bf16_t* X, int64_t dim_p, int64_t ld, int64_t seg_stride,
                            int64_t nseg, int splits, float* P, const int* st, hipStream_t s,
                            const bf16_t* Xb = nullptr);

// F (dim x dim, fp32, row-major) = scale * sum_z P[z]  (upper tiles mirrored).
hipError_t launch_reduce_frag(const float* P, int splits, int64_t dim_p, float* F, int64_t dim,
                              double scale, const int* st, hipStream_t s);

// ---------------------------------------------------------------- fp32 path
enum GemmFlags : int {
  kKHiRow = 1,   // k < i0 + 64   (left operand lower triangular)
  kKLoRow = 2,   // k >= i0       (left operand upper triangular)
  kKHiCol = 4,   // k < j0 + 64   (right operand upper triangular)
  kKLoCol = 8,   // k >= j0       (right operand lower triangular)
  kCLower = 16,  // write only C[i][j] with i >= j
};

struct GemmF32 {
  const float* A;
  const float* B;
  float* C;
  int64_t lda, ldb, ldc;
  int64_t sA, sB, sC;  // batch strides (grid z = batch when ksplit == 1)
  int64_t M, N, K;
  int transA;          // 0: A(i,k) = A[i*lda + k]; 1: A(i,k) = A[k*lda + i]
  int transB;          // 0: B(k,j) = B[k*ldb + j]; 1: B(k,j) = B[j*ldb + k]
  float alpha, beta;
  int flags;
  int64_t kseg;        // segmented k: k -> (k / kseg) * seg + k % kseg (kseg = K: plain)
  int64_t segA, segB;
  int ksplit;          // > 1: grid z splits k, C += z * sC, beta ignored
  const int* st;
  int tile;            // 0: chosen by size; 64: 64 x 64 tiles; 128: 128 x 128 tiles (a
                       // workgroup reads all of its rows of op(A) before it writes, so C
                       // may alias A when N <= 128)
};
// C = alpha * op(A) op(B) + beta * C on the fp32 matrix cores (64 x 64 tiles).
hipError_t launch_gemm_f32(const GemmF32& p, int batch, hipStream_t s);

// F (dim x dim) = scale * sum_z P[z] with P[z] row-major dim_p x dim_p, lower
// triangle read, mirrored.
hipError_t launch_reduce_rowmajor(const float* P, int splits, int64_t dim_p, float* F,
                                  int64_t dim, double scale, const int* st, hipStream_t s);

// ------------------------------------------------------ factorisation / misc
constexpr int kLeaf = 128;  // diagonal block factorised inside one workgroup

// One step of the right-looking blocked factorisation of the dim x dim
// matrix L (row-major, lower triangle; L^-1 blocks into Li): the diagonal
// block at d0 (a multiple of 128) is factored and inverted in one workgroup
// (pivots d0.., log-determinant share into logdet[d0 / 128], factor written
// in place, L^-1 block into Li; a non-positive or NaN pivot sets the status
// word to {iteration, side, pivot}), after the update of panel ok (columns
// [ok, ok + 128), already holding L below ok + 128) when ok >= 0; that panel's
// update is also applied to every other 128 x 128 block of the trailing lower
// triangle at or below d0 with block column below jend, by up to
// kStepWorkers further workgroups.  ok < 0: the diagonal block only.
constexpr int kStepWorkers = 255;
// Panel of the blocked factorisation, in place: P (rows x 128, leading
// dimension ld) <- P Xkk^T with Xkk the 128 x 128 inverse of the diagonal
// block (lower, zeros above; leading dimension ld).
hipError_t launch_panel_solve(float* P, const float* Xkk, int64_t ld, int64_t rows, const int* st,
                              hipStream_t s);
hipError_t launch_chol_step(float* L, float* Li, int64_t dim, int64_t d0, int64_t ok, int64_t jend,
                            double* logdet, int iteration, int side, int* st, hipStream_t s);

// out[s][r][c] (rows_p x cols_p) from G[s] (m x n): copy (transpose = 0,
// rows_p >= m, cols_p >= n) or transpose (transpose = 1, rows_p >= n,
// cols_p >= m), zero padding.  elem_bytes = 2 (bf16) or 4 (fp32).
hipError_t launch_pack(const void* G, void* out, int64_t N, int64_t m, int64_t n, int64_t rows_p,
                       int64_t cols_p, int transpose, int elem_bytes, hipStream_t s);

// Lw (dim_p x dim_p, elem) = lower(Li) (all of Li with full = 1) rounded
// (bf16: hi part; Lw2: lo part if non-null), zero elsewhere.  elem_bytes = 2
// or 4.  With part non-null (and full = 0),
// convert_parts(dim_p) partial sums of sum_j F_jj ||column j of lower(Li)||^2
// go to part (F: the dim x dim factor whose inverse factor Li is; the input
// of launch_split_decide).
constexpr int64_t kConvertChunks = 64;
int64_t convert_parts(int64_t dim_p);
hipError_t launch_convert_inverse(const float* Li, int64_t dim, void* Lw, void* Lw2, int64_t dim_p,
                                  int elem_bytes, const float* F, double* part, const int* st,
                                  hipStream_t s, int full = 0);

// From those partials: out[0] = s = (1/dim) sum_j F_jj (F^-1)_jj and
// flag[0] = (s > threshold).
hipError_t launch_split_decide(const double* part, int64_t dim, int64_t dim_p, double threshold,
                               int* flag, double* out, const int* st, hipStream_t s);

// tr = trace(F); with kappa > 0, F += kappa * tr/dim * I first and tr is the
// trace after damping.  fp64 accumulation, one workgroup, fixed order.
hipError_t launch_trace_damp(float* F, int64_t dim, double kappa, double* tr, const int* st,
                             hipStream_t s);

// c = trA / n; FA /= c; FB *= c; *c_out = c.
hipError_t launch_normalise(float* FA, int64_t n, float* FB, int64_t m, const double* trA,
                            double* c_out, const int* st, hipStream_t s);

// ll = -(N/2)(m logdetA + n logdetB) - T/2 - (N m n / 2) log 2 pi, with
// logdet = 2 * sum of slots (the side factorised before the normalisation
// gets its log-determinant corrected by -+ dim * log c) and T the trace
// term: N m n when kappa = 0, otherwise from the kDiagBlocks partials of
// launch_sumsq_trace on the second-updated factor (exact under damping).
constexpr int kDiagBlocks = 256;
hipError_t launch_loglik(const double* slotsA, int nA, const double* slotsB, int nB,
                         const double* c, int first_is_B, double m, double n, double N,
                         double kappa, const double* part, double* ll_out, const int* st,
                         hipStream_t s);

// part[2 b] / part[2 b + 1]: fixed-order partial sums of Li^2 (dim x dim)
// and of diag(F), b < kDiagBlocks.
hipError_t launch_sumsq_trace(const float* Li, const float* F, int64_t dim, double* part,
                              const int* st, hipStream_t s);

// *delta_out = ||A (x) B - Ap (x) Bp||_F / (||Ap||_F ||Bp||_F) in fp64 (part:
// 8 kDiagBlocks doubles of scratch); with tol > 0 and delta <= tol, st[3] =
// iteration (the rest of the enqueued pipeline halts).
hipError_t launch_delta(const float* A, const float* Ap, int64_t nA, const float* B,
                        const float* Bp, int64_t nB, double* part, double* delta_out, double tol,
                        int iteration, int* st, hipStream_t s);

// w[r] = sum_j P[r][j] V[r][j], rows x cols, elem_bytes 2 (bf16) or 4.
hipError_t launch_row_dot(const void* P, const void* V, int64_t rows, int64_t cols, int elem_bytes,
                          float* w, const int* st, hipStream_t s);

// w[r] = sum_j P[r][j] (square = 0) or sum_j P[r][j]^2 (square = 1), rows x cols.
hipError_t launch_row_sums(const float* P, int64_t rows, int64_t cols, int square, float* w,
                           const int* st, hipStream_t s);

// transpose(diag(sqrt(w)) M) for M rows_p x cols_p, stored as rows_p / seg
// segments of cols_p x seg (element (c, r) at
// (r / seg) * cols_p * seg + c * seg + r % seg); seg | rows_p, 64 | seg.
hipError_t launch_scale_transpose(const void* M, const float* w, int64_t rows_p, int64_t cols_p,
                                  int64_t seg, void* out, int elem_bytes, const int* st,
                                  hipStream_t s);

// out[0] = sum_i a[i] b[i] (fp64, fixed order), out[1] = 2 sum(slotsA),
// out[2] = 2 sum(slotsB).  scratch: 512 doubles.
hipError_t launch_objective_terms(const float* a, const float* b, int64_t count,
                                  const double* slotsA, int nA, const double* slotsB, int nB,
                                  double* scratch, double* out, const int* st, hipStream_t s);

hipError_t launch_copy_f32(const float* src, float* dst, int64_t count, const int* st,
                           hipStream_t s);
// dst[r][c] = src[r][c] for r < rows, c < cols (leading dimensions lds, ldd).
hipError_t launch_copy2d_f32(const float* src, int64_t lds, float* dst, int64_t ldd, int64_t rows,
                             int64_t cols, const int* st, hipStream_t s);
hipError_t launch_fill_f32(float* dst, int64_t count, float v, hipStream_t s);
hipError_t launch_identity_f32(float* dst, int64_t dim, hipStream_t s);
hipError_t launch_set_int(int* dst, int64_t count, int v, hipStream_t s);

// ------------------------------------------------------------ WaterKron
// Tile edge of the quantiser sweep; padded dimensions are multiples of it.
constexpr int kTileWK = 64;

// Device operands of one quantiser sweep.  La (nq x nq) and Lb (mq x mq) are
// the padded normalised inverse factors (identity in the padding); alpha
// (nq) and beta (mq) the padded scales (1 in the padding); dA, dB the
// RevCholesky diagonals.  Racc, Pre, X, E: MT * NT tiles of 64 x 64 floats
// each (tile (I, J) at offset (I * NT + J) * 4096; Racc and Pre zeroed
// before the first diagonal).  Z: mq x nq codes (padded, leading dimension
// nq); dpart: MT * NT doubles.
struct WkParams {
  const float* W;
  int64_t m, n;
  const float* La;
  const float* Lb;
  const float* alpha;
  const float* beta;
  const float* dA;
  const float* dB;
  float* Racc;
  float* Pre;
  float* X;
  float* E;
  int32_t* Z;
  double* dpart;
  int64_t mq, nq;
  int MT, NT;
  const int* st;
};

// J M J for M d x d.
hipError_t launch_wk_reverse(const float* M, int64_t d, float* out, const int* st, hipStream_t s);
// Normalised inverse of RevCholesky(M) (padded dq x dq) and its diagonal,
// from Ci = Cholesky(J M J)^-1.
hipError_t launch_wk_normalise(const float* Ci, int64_t d, int64_t dq, float* Lt, float* diag,
                               const int* st, hipStream_t s);
// Padded scales; given = 0: waterfilling from diag and the log-pivot slots
// (also written to user), given = 1: copied from user.
hipError_t launch_wk_scales(const float* diag, int64_t d, int64_t dq, const double* slots,
                            int nslots, double gamma, int given, float* user, float* scale,
                            const int* st, hipStream_t s);
// Workgroups pushing the tiles of diagonal d - 1 forward.
int64_t wk_push_units(int d, int MT, int NT);
// Anti-diagonal d (0 <= d <= MT + NT - 2) of the sweep.
hipError_t launch_wk_diagonal(const WkParams& p, int d, hipStream_t s);
// Z (m x n) from the padded codes Zp (leading dimension nq) and, when V is
// non-null, V = beta alpha^T (.) Z.
hipError_t launch_wk_finish(const int32_t* Zp, int64_t nq, int64_t m, int64_t n,
                           const float* alpha, const float* beta, int32_t* Z, float* V,
                           const int* st, hipStream_t s);
// *out = scale * sum part[0..count), fixed order.
hipError_t launch_wk_sum(const double* part, int64_t count, double scale, double* out,
                         const int* st, hipStream_t s);

}  // namespace ff
