// Bandwidth-bound helper kernels of the flip-flop iteration: sample packing
// (zero-padded copy / transpose), inverse conversion for the whitening
// operand, trace + damping, the trace normalisation, the per-iteration
// log-likelihood, and plain fills and copies.
#include <math.h>

#include "ff_common.hpp"
#include "ff_kernels.hpp"

namespace ff {
namespace {

// ------------------------------------------------------------------ packing
// out[s][r][c], r < rows_p, c < cols_p.  transpose = 0: G[s][r][c] when
// r < m, c < n.  transpose = 1: G[s][c][r] when r < n, c < m.  64 x 64 tiles
// through LDS so that both the read and the write are coalesced.
template <typename T>
__global__ __launch_bounds__(256) void k_pack(const T* __restrict__ G, T* __restrict__ out,
                                              int64_t m, int64_t n, int64_t rows_p, int64_t cols_p,
                                              int transpose) {
  __shared__ T tile[64][65];
  const int64_t s = blockIdx.z;
  const int64_t r0 = (int64_t)blockIdx.y * 64, c0 = (int64_t)blockIdx.x * 64;
  const T* g = G + s * m * n;
  T* o = out + s * rows_p * cols_p;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  if (!transpose) {
    for (int y = ty; y < 64; y += 4) {
      const int64_t r = r0 + y, c = c0 + tx;
      if (r < rows_p && c < cols_p) o[r * cols_p + c] = (r < m && c < n) ? g[r * n + c] : T(0);
    }
    return;
  }
  // tile of the source: source rows c0.. (m side), source cols r0.. (n side)
  for (int y = ty; y < 64; y += 4) {
    const int64_t sr = c0 + y, sc = r0 + tx;
    tile[y][tx] = (sr < m && sc < n) ? g[sr * n + sc] : T(0);
  }
  __syncthreads();
  for (int y = ty; y < 64; y += 4) {
    const int64_t r = r0 + y, c = c0 + tx;
    if (r < rows_p && c < cols_p) o[r * cols_p + c] = tile[tx][y];
  }
}

// Transposing bf16 copy with 8-byte accesses: out[s][r][c] = G[s][c][r] (r < n,
// c < m), zero padding; a 64 x 64 tile per workgroup, rows of 16 four-element
// chunks.  Requires n % 4 == 0 and cols_p % 4 == 0 (the caller checks).
__global__ __launch_bounds__(256) void k_pack_t16(const bf16_t* __restrict__ G, bf16_t* __restrict__ out,
                                                  int64_t m, int64_t n, int64_t rows_p, int64_t cols_p) {
  __shared__ bf16_t tile[64][72];
  const int64_t s = blockIdx.z;
  const int64_t r0 = (int64_t)blockIdx.y * 64, c0 = (int64_t)blockIdx.x * 64;
  const bf16_t* g = G + s * m * n;
  bf16_t* o = out + s * rows_p * cols_p;
  const int tid = threadIdx.x, q = tid & 15, y0 = tid >> 4;
  // source rows c0.. (m side), 4 consecutive source columns r0 + 4 q .. (n side)
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int y = y0 + 16 * t;
    const int64_t sr = c0 + y, sc = r0 + 4 * q;
    uint2 v = {0u, 0u};
    if (sr < m && sc < n) v = *reinterpret_cast<const uint2*>(g + sr * n + sc);
    *reinterpret_cast<uint2*>(&tile[y][4 * q]) = v;
  }
  __syncthreads();
  // output rows r0.. , 4 consecutive output columns c0 + 4 q ..
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int y = y0 + 16 * t;
    const int64_t r = r0 + y, c = c0 + 4 * q;
    if (r < rows_p && c < cols_p) {
      const uint32_t a = tile[4 * q][y], b = tile[4 * q + 1][y], d = tile[4 * q + 2][y],
                     e = tile[4 * q + 3][y];
      const uint2 v = {a | (b << 16), d | (e << 16)};
      *reinterpret_cast<uint2*>(o + r * cols_p + c) = v;
    }
  }
}

// ------------------------------------------- rank-one (per-token) weights
// w[r] = sum_j v(r, j) over cols entries of row r (square = 0: v = P[r][j];
// square = 1: v = P[r][j]^2), one wave per row, fixed reduction order.
__global__ __launch_bounds__(256) void k_row_sums(const float* __restrict__ P, int64_t rows,
                                                  int64_t cols, int square, float* __restrict__ w,
                                                  const int* st) {
  if (ff_halted(st)) return;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= rows) return;
  const float* p = P + r * cols;
  double s = 0.0;
  for (int64_t j = lane; j < cols; j += 64) {
    const double v = p[j];
    s += square ? v * v : v;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o);
  if (lane == 0) w[r] = (float)s;
}

// w[r] = sum_j P[r][j] V[r][j] (rows x cols, row-major, elem T, fp64 sum per
// row): the quadratic forms v_r^T F v_r from P = V F.
template <typename T>
__global__ __launch_bounds__(256) void k_row_dot(const T* __restrict__ P, const T* __restrict__ V,
                                                 int64_t rows, int64_t cols, float* __restrict__ w,
                                                 const int* st) {
  if (ff_halted(st)) return;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= rows) return;
  const T* p = P + r * cols;
  const T* v = V + r * cols;
  double s = 0.0;
  for (int64_t j = lane; j < cols; j += 64)
    s += (double)Elem<T>::to_f32(p[j]) * (double)Elem<T>::to_f32(v[j]);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o);
  if (lane == 0) w[r] = (float)s;
}

// sqrt(w[r]) * M[r][c] for the rows_p x cols_p matrix M: the rows of M
// (tokens) weighted and turned into the k axis of a symmetric product, in
// segments of seg tokens: element (c, r) goes to
// out[(r / seg) * cols_p * seg + c * seg + r % seg], so that the product reads
// short rows (seg elements) instead of rows_p-long ones.  64 x 64 tiles
// through LDS; seg is a multiple of 64.
template <typename T>
__global__ __launch_bounds__(256) void k_scale_transpose(const T* __restrict__ M,
                                                         const float* __restrict__ w,
                                                         int64_t rows_p, int64_t cols_p, int64_t seg,
                                                         T* __restrict__ out, const int* st) {
  if (ff_halted(st)) return;
  __shared__ float tile[64][65];
  const int64_t r0 = (int64_t)blockIdx.y * 64, c0 = (int64_t)blockIdx.x * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int y = ty; y < 64; y += 4) {
    const int64_t r = r0 + y, c = c0 + tx;
    float v = 0.0f;
    if (r < rows_p && c < cols_p) v = sqrtf(w[r]) * Elem<T>::to_f32(M[r * cols_p + c]);
    tile[y][tx] = v;
  }
  __syncthreads();
  T* o = out + (r0 / seg) * cols_p * seg + (r0 % seg);
  for (int y = ty; y < 64; y += 4) {
    const int64_t c = c0 + y, r = r0 + tx;
    if (c < cols_p && r < rows_p) o[c * seg + tx] = Elem<T>::from_f32(tile[tx][y]);
  }
}

// The same for bf16 with 8-byte accesses (four consecutive elements per
// thread on both sides; the tile lies within one segment since 64 | seg).
// Requires cols_p % 4 == 0.
__global__ __launch_bounds__(256) void k_scale_transpose_16(const bf16_t* __restrict__ M,
                                                            const float* __restrict__ w,
                                                            int64_t rows_p, int64_t cols_p, int64_t seg,
                                                            bf16_t* __restrict__ out, const int* st) {
  if (ff_halted(st)) return;
  __shared__ float tile[64][65];
  const int64_t r0 = (int64_t)blockIdx.y * 64, c0 = (int64_t)blockIdx.x * 64;
  const int tid = threadIdx.x, q = tid & 15, y0 = tid >> 4;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int y = y0 + 16 * t;
    const int64_t r = r0 + y, c = c0 + 4 * q;
    float v[4] = {0.f, 0.f, 0.f, 0.f};
    if (r < rows_p && c < cols_p) {
      const uint2 u = *reinterpret_cast<const uint2*>(M + r * cols_p + c);
      const float sw = sqrtf(w[r]);
      v[0] = sw * bf16_to_f32((bf16_t)(u.x & 0xffffu));
      v[1] = sw * bf16_to_f32((bf16_t)(u.x >> 16));
      v[2] = sw * bf16_to_f32((bf16_t)(u.y & 0xffffu));
      v[3] = sw * bf16_to_f32((bf16_t)(u.y >> 16));
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) tile[y][4 * q + e] = v[e];
  }
  __syncthreads();
  bf16_t* o = out + (r0 / seg) * cols_p * seg + (r0 % seg);
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int y = y0 + 16 * t;
    const int64_t c = c0 + y, r = r0 + 4 * q;
    if (c < cols_p && r < rows_p) {
      const uint32_t a = f32_to_bf16(tile[4 * q][y]), b = f32_to_bf16(tile[4 * q + 1][y]),
                     d = f32_to_bf16(tile[4 * q + 2][y]), e = f32_to_bf16(tile[4 * q + 3][y]);
      const uint2 v = {a | (b << 16), d | (e << 16)};
      *reinterpret_cast<uint2*>(o + c * seg + 4 * q) = v;
    }
  }
}

// --------------------------------------------------------- inverse convert
// Thread (column j, row chunk y) converts rows [y rch, (y + 1) rch) of
// column j: coalesced along each row.  With part non-null it also writes,
// per workgroup, part[y][x] = sum over its 256 columns j of
// F_jj * (sum over its rows of Li[i][j]^2): the chunk's share of
// sum_j F_jj (F^-1)_jj, since (F^-1)_jj is the squared norm of column j of
// L^-1.
template <typename T>
__global__ __launch_bounds__(256) void k_convert_inverse(const float* __restrict__ Li, int64_t dim,
                                                         T* __restrict__ Lw, T* __restrict__ Lw2,
                                                         int64_t dim_p, int64_t rch, int full,
                                                         const float* __restrict__ F,
                                                         double* __restrict__ part, const int* st) {
  if (ff_halted(st)) return;
  __shared__ double red[256];
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  float acc = 0.0f;
  if (j < dim_p) {
    const int64_t i0 = (int64_t)blockIdx.y * rch, i1 = i0 + rch < dim_p ? i0 + rch : dim_p;
    constexpr int U = 8;
    for (int64_t i = i0; i < i1; i += U) {
      float v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t r = i + u;
        v[u] = (r < i1 && r < dim && j < dim && (full || j <= r)) ? Li[r * dim + j] : 0.0f;
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t r = i + u;
        if (r >= i1) break;
        acc += v[u] * v[u];
        const T hi = Elem<T>::from_f32(v[u]);
        Lw[r * dim_p + j] = hi;
        if (Lw2 != nullptr) Lw2[r * dim_p + j] = Elem<T>::from_f32(v[u] - Elem<T>::to_f32(hi));
      }
    }
  }
  if (part == nullptr) return;
  red[threadIdx.x] = j < dim ? (double)F[j * dim + j] * (double)acc : 0.0;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) part[(int64_t)blockIdx.y * gridDim.x + blockIdx.x] = red[0];
}

// Rounding sensitivity of the whitening operand L^-1 of F:
//   s = (1/dim) sum_j F_jj (F^-1)_jj   (the sum of the npart partials).
// Rounding L^-1 to bf16 with independent relative errors of rms u/sqrt(3)
// (u = 2^-9) perturbs L^-1 L = I by R with E||R||_F^2 = (u^2/3) sum_j
// F_jj (F^-1)_jj, an rms distortion of the whitened metric of
// u sqrt(s/3) per direction.  flag = 1 (whiten with the hi + lo parts) when
// s > threshold; out[0] = s.  One workgroup, fixed summation order.
__global__ __launch_bounds__(256) void k_split_decide(const double* __restrict__ part, int64_t npart,
                                                      int64_t dim, double threshold, int* flag,
                                                      double* out, const int* st) {
  if (ff_halted(st)) return;
  __shared__ double red[256];
  double acc = 0.0;
  for (int64_t k = threadIdx.x; k < npart; k += 256) acc += part[k];
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const double sv = red[0] / (double)dim;
    out[0] = sv;
    flag[0] = sv > threshold ? 1 : 0;
  }
}

// ---------------------------------------------------------- trace, damping
__device__ double block_sum_256(double v, double* red) {
  const int tid = threadIdx.x;
  red[tid] = v;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (tid < w) red[tid] += red[tid + w];
    __syncthreads();
  }
  const double r = red[0];
  __syncthreads();
  return r;
}

__global__ __launch_bounds__(256) void k_trace_damp(float* F, int64_t dim, double kappa,
                                                    double* tr_out, const int* st) {
  if (ff_halted(st)) return;
  __shared__ double red[256];
  double s = 0.0;
  for (int64_t i = threadIdx.x; i < dim; i += 256) s += (double)F[i * dim + i];
  double tr = block_sum_256(s, red);
  if (kappa > 0.0) {
    const float add = (float)(kappa * tr / (double)dim);
    s = 0.0;
    for (int64_t i = threadIdx.x; i < dim; i += 256) {
      const float v = F[i * dim + i] + add;
      F[i * dim + i] = v;
      s += (double)v;
    }
    tr = block_sum_256(s, red);
  }
  if (threadIdx.x == 0) *tr_out = tr;
}

__global__ __launch_bounds__(256) void k_normalise(float* __restrict__ FA, int64_t nA,
                                                   float* __restrict__ FB, int64_t nB,
                                                   const double* trA, int64_t n, double* c_out,
                                                   const int* st) {
  if (ff_halted(st)) return;
  const double c = *trA / (double)n;
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < nA; i += stride)
    FA[i] = (float)((double)FA[i] / c);
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < nB; i += stride)
    FB[i] = (float)((double)FB[i] * c);
  if (blockIdx.x == 0 && threadIdx.x == 0) *c_out = c;
}

// Trace term of the log-likelihood, sum_i tr(B^-1 G_i A^-1 G_i^T).  After
// the second update of an iteration, F_d = F_h + kappa t I with F_h the
// maximum-likelihood half step (dimension d, scaled by 1 / (N d_o)) and
// t = tr(F_h) / d; the term is N d_o tr(F_d^-1 F_h) = N d_o (d - kappa t tr(F_d^-1)),
// which the normalisation (F_n = F_d / c or c F_d, the other factor scaled
// the other way) leaves unchanged.  In terms of the normalised factor and
// its Cholesky factor L_n: N d_o (d - kappa / (1 + kappa) (tr(F_n) / d) ||L_n^-1||_F^2).
// part holds per-workgroup (sum of squares of L_n^-1, diagonal sum of F_n).
__global__ __launch_bounds__(256) void k_loglik(const double* slotsA, int nA, const double* slotsB,
                                                int nB, const double* cptr, int first_is_B,
                                                double m, double n, double N, double kappa,
                                                const double* part, int nparts, double* ll_out,
                                                const int* st) {
  if (ff_halted(st)) return;
  if (threadIdx.x != 0) return;
  double la = 0.0, lb = 0.0;
  for (int i = 0; i < nA; ++i) la += slotsA[i];
  for (int i = 0; i < nB; ++i) lb += slotsB[i];
  la *= 2.0;
  lb *= 2.0;
  const double logc = log(*cptr);
  // The side updated first was factorised before the normalisation
  // (B <- c B, or A <- A / c in the A-first order).
  if (first_is_B) lb += m * logc;
  else la -= n * logc;
  double trace_term = N * m * n;
  if (kappa > 0.0 && part != nullptr) {
    double ss = 0.0, tf = 0.0;
    for (int b = 0; b < nparts; ++b) {
      ss += part[2 * b];
      tf += part[2 * b + 1];
    }
    const double d = first_is_B ? n : m, d_o = first_is_B ? m : n;
    trace_term = N * d_o * (d - kappa / (1.0 + kappa) * (tf / d) * ss);
  }
  const double log2pi = 1.8378770664093454835606594728112;
  *ll_out = -0.5 * N * (m * la + n * lb) - 0.5 * trace_term - 0.5 * N * m * n * log2pi;
}

// Per-workgroup partial sums (fixed strided subsets, fixed-order reduction)
// of sum Li^2 over dim x dim and of the diagonal of F.
__global__ __launch_bounds__(256) void k_sumsq_trace(const float* __restrict__ Li,
                                                     const float* __restrict__ F, int64_t dim,
                                                     double* __restrict__ part, const int* st) {
  if (ff_halted(st)) return;
  __shared__ double red[256];
  const int64_t stride = (int64_t)kDiagBlocks * 256;
  const int64_t first = (int64_t)blockIdx.x * 256 + threadIdx.x;
  double ss = 0.0, tf = 0.0;
  for (int64_t i = first; i < dim * dim; i += stride) {
    const double v = (double)Li[i];
    ss += v * v;
  }
  for (int64_t i = first; i < dim; i += stride) tf += (double)F[i * dim + i];
  ss = block_sum_256(ss, red);
  tf = block_sum_256(tf, red);
  if (threadIdx.x == 0) {
    part[2 * blockIdx.x] = ss;
    part[2 * blockIdx.x + 1] = tf;
  }
}

// Relative change of the Kronecker product between two iterates, in fp64,
// from the differences themselves (no cancellation floor):
//   ||A (x) B - Ap (x) Bp||_F^2 = ||dA||^2 ||B||^2 + ||Ap||^2 ||dB||^2 + 2 <dA, Ap> <B, dB>,
// dA = A - Ap, dB = B - Bp, divided by ||Ap||_F ||Bp||_F.  Partials per
// workgroup: [||dA||^2, <dA,Ap>, ||Ap||^2, ||B||^2, ||dB||^2, <B,dB>, ||Bp||^2, 0].
__global__ __launch_bounds__(256) void k_delta_partial(const float* __restrict__ A,
                                                       const float* __restrict__ Ap, int64_t nA,
                                                       const float* __restrict__ B,
                                                       const float* __restrict__ Bp, int64_t nB,
                                                       double* __restrict__ part, const int* st) {
  if (ff_halted(st)) return;
  __shared__ double red[256];
  const int64_t stride = (int64_t)kDiagBlocks * 256;
  const int64_t first = (int64_t)blockIdx.x * 256 + threadIdx.x;
  double v[7] = {0, 0, 0, 0, 0, 0, 0};
  for (int64_t i = first; i < nA; i += stride) {
    const double a = A[i], ap = Ap[i], d = a - ap;
    v[0] += d * d;
    v[1] += d * ap;
    v[2] += ap * ap;
  }
  for (int64_t i = first; i < nB; i += stride) {
    const double b = B[i], bp = Bp[i], d = b - bp;
    v[3] += b * b;
    v[4] += d * d;
    v[5] += b * d;
    v[6] += bp * bp;
  }
  for (int k = 0; k < 7; ++k) {
    const double r = block_sum_256(v[k], red);
    if (threadIdx.x == 0) part[8 * blockIdx.x + k] = r;
  }
}

// delta_out = the relative change; with tol > 0 and delta <= tol, st[3] =
// iteration, which halts the rest of the pipeline (the iterate is complete).
__global__ __launch_bounds__(64) void k_delta_final(const double* __restrict__ part,
                                                    double* delta_out, double tol, int iteration,
                                                    int* st) {
  if (ff_halted(st)) return;
  if (threadIdx.x != 0) return;
  double v[7] = {0, 0, 0, 0, 0, 0, 0};
  for (int b = 0; b < kDiagBlocks; ++b)
    for (int k = 0; k < 7; ++k) v[k] += part[8 * b + k];
  const double sq = v[0] * v[3] + v[2] * v[4] + 2.0 * v[1] * v[5];
  const double den = sqrt(v[2] * v[6]);
  const double delta = sqrt(sq > 0.0 ? sq : 0.0) / den;
  *delta_out = delta;
  if (tol > 0.0 && delta <= tol) st[3] = iteration;
}

// Partial sums of a[i] * b[i] in fp64: block z sums a fixed strided subset
// and reduces it in a fixed order, so the result does not depend on timing.
constexpr int kDotBlocks = 512;
__global__ __launch_bounds__(256) void k_dot_partial(const float* __restrict__ a,
                                                     const float* __restrict__ b, int64_t count,
                                                     double* __restrict__ part, const int* st) {
  if (ff_halted(st)) return;
  __shared__ double red[256];
  double s = 0.0;
  const int64_t stride = (int64_t)kDotBlocks * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < count; i += stride)
    s += (double)a[i] * (double)b[i];
  s = block_sum_256(s, red);
  if (threadIdx.x == 0) part[blockIdx.x] = s;
}

// out[0] = sum of the partials, out[1] = 2 sum(slotsA), out[2] = 2 sum(slotsB).
__global__ __launch_bounds__(256) void k_dot_final(const double* __restrict__ part,
                                                   const double* slotsA, int nA,
                                                   const double* slotsB, int nB, double* out,
                                                   const int* st) {
  if (ff_halted(st)) return;
  __shared__ double red[256];
  double s = 0.0;
  for (int i = threadIdx.x; i < kDotBlocks; i += 256) s += part[i];
  s = block_sum_256(s, red);
  if (threadIdx.x == 0) {
    double la = 0.0, lb = 0.0;
    for (int i = 0; i < nA; ++i) la += slotsA[i];
    for (int i = 0; i < nB; ++i) lb += slotsB[i];
    out[0] = s;
    out[1] = 2.0 * la;
    out[2] = 2.0 * lb;
  }
}

__global__ __launch_bounds__(256) void k_copy_f32(const float* __restrict__ src,
                                                  float* __restrict__ dst, int64_t count,
                                                  const int* st) {
  if (ff_halted(st)) return;
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < count; i += stride) dst[i] = src[i];
}

__global__ __launch_bounds__(256) void k_copy2d_f32(const float* __restrict__ src, int64_t lds,
                                                    float* __restrict__ dst, int64_t ldd,
                                                    int64_t rows, int64_t cols, const int* st) {
  if (ff_halted(st)) return;
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < rows * cols; i += stride) {
    const int64_t r = i / cols, c = i % cols;
    dst[r * ldd + c] = src[r * lds + c];
  }
}

__global__ __launch_bounds__(256) void k_fill_f32(float* dst, int64_t count, float v) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < count; i += stride) dst[i] = v;
}

__global__ __launch_bounds__(256) void k_identity_f32(float* dst, int64_t dim) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < dim * dim; i += stride)
    dst[i] = (i / dim == i % dim) ? 1.0f : 0.0f;
}

__global__ void k_set_int(int* dst, int64_t count, int v) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < count) dst[i] = v;
}

uint32_t grid_for(int64_t count) {
  int64_t b = (count + 255) / 256;
  if (b > 8192) b = 8192;
  if (b < 1) b = 1;
  return (uint32_t)b;
}

}  // namespace

hipError_t launch_pack(const void* G, void* out, int64_t N, int64_t m, int64_t n, int64_t rows_p,
                       int64_t cols_p, int transpose, int elem_bytes, hipStream_t s) {
  if (N < 1 || N > 65535 || rows_p < 1 || cols_p < 1) return hipErrorInvalidValue;
  if (transpose ? (rows_p < n || cols_p < m) : (rows_p < m || cols_p < n))
    return hipErrorInvalidValue;
  dim3 grid((uint32_t)((cols_p + 63) / 64), (uint32_t)((rows_p + 63) / 64), (uint32_t)N);
  if (elem_bytes == 2 && transpose && n % 4 == 0 && cols_p % 4 == 0 &&
      (reinterpret_cast<uintptr_t>(G) & 7) == 0 && (reinterpret_cast<uintptr_t>(out) & 7) == 0) {
    hipLaunchKernelGGL(k_pack_t16, grid, dim3(256), 0, s, (const bf16_t*)G, (bf16_t*)out, m, n,
                       rows_p, cols_p);
  } else if (elem_bytes == 2)
    hipLaunchKernelGGL(k_pack<bf16_t>, grid, dim3(256), 0, s, (const bf16_t*)G, (bf16_t*)out, m, n,
                       rows_p, cols_p, transpose);
  else if (elem_bytes == 4)
    hipLaunchKernelGGL(k_pack<float>, grid, dim3(256), 0, s, (const float*)G, (float*)out, m, n,
                       rows_p, cols_p, transpose);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_row_sums(const float* P, int64_t rows, int64_t cols, int square, float* w,
                           const int* st, hipStream_t s) {
  if (rows < 0 || cols < 1) return hipErrorInvalidValue;
  if (rows == 0) return hipSuccess;
  const int64_t blocks = (rows + 3) / 4;
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_row_sums, dim3((uint32_t)blocks), dim3(256), 0, s, P, rows, cols, square, w,
                     st);
  return hipGetLastError();
}

hipError_t launch_row_dot(const void* P, const void* V, int64_t rows, int64_t cols, int elem_bytes,
                          float* w, const int* st, hipStream_t s) {
  const int64_t blocks = (rows + 3) / 4;
  if (elem_bytes == 2)
    hipLaunchKernelGGL(k_row_dot<bf16_t>, dim3((uint32_t)blocks), dim3(256), 0, s, (const bf16_t*)P,
                       (const bf16_t*)V, rows, cols, w, st);
  else if (elem_bytes == 4)
    hipLaunchKernelGGL(k_row_dot<float>, dim3((uint32_t)blocks), dim3(256), 0, s, (const float*)P,
                       (const float*)V, rows, cols, w, st);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_scale_transpose(const void* M, const float* w, int64_t rows_p, int64_t cols_p,
                                  int64_t seg, void* out, int elem_bytes, const int* st,
                                  hipStream_t s) {
  if (rows_p < 1 || cols_p < 1 || seg < 64 || seg % 64 || rows_p % seg) return hipErrorInvalidValue;
  const int64_t gx = (cols_p + 63) / 64, gy = (rows_p + 63) / 64;
  if (gx > 0x7fffffff || gy > 65535) return hipErrorInvalidValue;
  const dim3 grid((uint32_t)gx, (uint32_t)gy);
  if (elem_bytes == 2 && cols_p % 4 == 0 && (reinterpret_cast<uintptr_t>(M) & 7) == 0 &&
      (reinterpret_cast<uintptr_t>(out) & 7) == 0)
    hipLaunchKernelGGL(k_scale_transpose_16, grid, dim3(256), 0, s, (const bf16_t*)M, w, rows_p,
                       cols_p, seg, (bf16_t*)out, st);
  else if (elem_bytes == 2)
    hipLaunchKernelGGL(k_scale_transpose<bf16_t>, grid, dim3(256), 0, s, (const bf16_t*)M, w,
                       rows_p, cols_p, seg, (bf16_t*)out, st);
  else if (elem_bytes == 4)
    hipLaunchKernelGGL(k_scale_transpose<float>, grid, dim3(256), 0, s, (const float*)M, w, rows_p,
                       cols_p, seg, (float*)out, st);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

int64_t convert_parts(int64_t dim_p) {
  const int64_t nchunk = dim_p < kConvertChunks ? dim_p : kConvertChunks;
  const int64_t rch = (dim_p + nchunk - 1) / nchunk;
  return ((dim_p + 255) / 256) * ((dim_p + rch - 1) / rch);
}

hipError_t launch_convert_inverse(const float* Li, int64_t dim, void* Lw, void* Lw2, int64_t dim_p,
                                  int elem_bytes, const float* F, double* part, const int* st,
                                  hipStream_t s, int full) {
  if (dim < 1 || dim_p < dim) return hipErrorInvalidValue;
  const int64_t nchunk = dim_p < kConvertChunks ? dim_p : kConvertChunks;
  const int64_t rch = (dim_p + nchunk - 1) / nchunk;
  const dim3 grid((uint32_t)((dim_p + 255) / 256), (uint32_t)((dim_p + rch - 1) / rch));
  if (elem_bytes == 2)
    hipLaunchKernelGGL(k_convert_inverse<bf16_t>, grid, dim3(256), 0, s, Li, dim, (bf16_t*)Lw,
                       (bf16_t*)Lw2, dim_p, rch, full, F, part, st);
  else if (elem_bytes == 4)
    hipLaunchKernelGGL(k_convert_inverse<float>, grid, dim3(256), 0, s, Li, dim, (float*)Lw,
                       (float*)Lw2, dim_p, rch, full, F, part, st);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_split_decide(const double* part, int64_t dim, int64_t dim_p, double threshold,
                               int* flag, double* out, const int* st, hipStream_t s) {
  hipLaunchKernelGGL(k_split_decide, dim3(1), dim3(256), 0, s, part, convert_parts(dim_p), dim,
                     threshold, flag, out, st);
  return hipGetLastError();
}

hipError_t launch_trace_damp(float* F, int64_t dim, double kappa, double* tr, const int* st,
                             hipStream_t s) {
  hipLaunchKernelGGL(k_trace_damp, dim3(1), dim3(256), 0, s, F, dim, kappa, tr, st);
  return hipGetLastError();
}

hipError_t launch_normalise(float* FA, int64_t n, float* FB, int64_t m, const double* trA,
                            double* c_out, const int* st, hipStream_t s) {
  hipLaunchKernelGGL(k_normalise, dim3(grid_for(n * n > m * m ? n * n : m * m)), dim3(256), 0, s,
                     FA, n * n, FB, m * m, trA, n, c_out, st);
  return hipGetLastError();
}

hipError_t launch_loglik(const double* slotsA, int nA, const double* slotsB, int nB,
                         const double* c, int first_is_B, double m, double n, double N,
                         double kappa, const double* part, double* ll_out, const int* st,
                         hipStream_t s) {
  hipLaunchKernelGGL(k_loglik, dim3(1), dim3(64), 0, s, slotsA, nA, slotsB, nB, c, first_is_B, m,
                     n, N, kappa, part, kDiagBlocks, ll_out, st);
  return hipGetLastError();
}

hipError_t launch_sumsq_trace(const float* Li, const float* F, int64_t dim, double* part,
                              const int* st, hipStream_t s) {
  if (dim < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_sumsq_trace, dim3(kDiagBlocks), dim3(256), 0, s, Li, F, dim, part, st);
  return hipGetLastError();
}

hipError_t launch_delta(const float* A, const float* Ap, int64_t nA, const float* B,
                        const float* Bp, int64_t nB, double* part, double* delta_out, double tol,
                        int iteration, int* st, hipStream_t s) {
  if (nA < 1 || nB < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_delta_partial, dim3(kDiagBlocks), dim3(256), 0, s, A, Ap, nA, B, Bp, nB,
                     part, st);
  hipLaunchKernelGGL(k_delta_final, dim3(1), dim3(64), 0, s, part, delta_out, tol, iteration, st);
  return hipGetLastError();
}

hipError_t launch_objective_terms(const float* a, const float* b, int64_t count,
                                  const double* slotsA, int nA, const double* slotsB, int nB,
                                  double* scratch, double* out, const int* st, hipStream_t s) {
  if (count < 0 || nA < 0 || nB < 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_dot_partial, dim3(kDotBlocks), dim3(256), 0, s, a, b, count, scratch, st);
  hipLaunchKernelGGL(k_dot_final, dim3(1), dim3(256), 0, s, scratch, slotsA, nA, slotsB, nB, out,
                     st);
  return hipGetLastError();
}

hipError_t launch_copy_f32(const float* src, float* dst, int64_t count, const int* st,
                           hipStream_t s) {
  hipLaunchKernelGGL(k_copy_f32, dim3(grid_for(count)), dim3(256), 0, s, src, dst, count, st);
  return hipGetLastError();
}

hipError_t launch_copy2d_f32(const float* src, int64_t lds, float* dst, int64_t ldd, int64_t rows,
                             int64_t cols, const int* st, hipStream_t s) {
  if (rows < 0 || cols < 0 || lds < cols || ldd < cols) return hipErrorInvalidValue;
  if (rows == 0 || cols == 0) return hipSuccess;
  hipLaunchKernelGGL(k_copy2d_f32, dim3(grid_for(rows * cols)), dim3(256), 0, s, src, lds, dst, ldd,
                     rows, cols, st);
  return hipGetLastError();
}

hipError_t launch_fill_f32(float* dst, int64_t count, float v, hipStream_t s) {
  hipLaunchKernelGGL(k_fill_f32, dim3(grid_for(count)), dim3(256), 0, s, dst, count, v);
  return hipGetLastError();
}

hipError_t launch_identity_f32(float* dst, int64_t dim, hipStream_t s) {
  hipLaunchKernelGGL(k_identity_f32, dim3(grid_for(dim * dim)), dim3(256), 0, s, dst, dim);
  return hipGetLastError();
}

hipError_t launch_set_int(int* dst, int64_t count, int v, hipStream_t s) {
  hipLaunchKernelGGL(k_set_int, dim3((uint32_t)((count + 255) / 256)), dim3(256), 0, s, dst, count,
                     v);
  return hipGetLastError();
}

}  // namespace ff
