// Cholesky factorisation and inverse of one diagonal block (fp32).
//
// The factors' inverses enter every flip-flop update (Section 5: A^-1 and
// B^-1 in the two half steps); the iteration whitens with the inverse of the
// lower Cholesky factor, L^-1 (Section 2 notation: Cholesky(M) is the lower
// L with positive diagonal and L L^T = M).  Blocks of up to 128 rows are
// handled here by one workgroup; larger factors are assembled by the host
// recursion from these blocks and fp32 matrix-core products.
//
// Register-blocked: thread (ti, tj), tid = 16 tj + ti, holds the 8 x 8 block
// (ti, tj) of the lower triangle.  The 16 threads of block column p are
// consecutive lanes of one wave, so the panel factorisation of block column p
// needs only lane shuffles; the panel is then published in LDS and every
// thread applies the rank-8 update to its own block (one barrier per block
// column).  The inverse follows right-looking by block rows from the stored
// panels.  A ragged block (b < 128) is padded with the identity.
#include <math.h>

#include "ff_common.hpp"
#include "ff_kernels.hpp"

namespace ff {
namespace {

constexpr int NB = 128;  // block size
constexpr int TB = 8;    // per-thread block
constexpr int NT = NB / TB;

__global__ __launch_bounds__(256) void k_chol_leaf(const float* __restrict__ Lblk,
                                                   float* __restrict__ Liblk, int64_t ld, int b,
                                                   int64_t pivot_base, double* logdet, int slot,
                                                   int iteration, int side, int* st) {
  if (ff_halted(st)) return;
  __shared__ __align__(16) float Pn[NT][TB][NB + 4];  // panel p = block column p of L, transposed
  __shared__ float Ld[NT][TB][TB + 1];  // inverses of the diagonal 8 x 8 blocks
  __shared__ __align__(16) float Xr[2][TB][NB + 4];  // finished block row of L^-1
  __shared__ double ldp[NT];
  __shared__ int bad;
  const int tid = threadIdx.x;
  const int ti = tid & 15, tj = tid >> 4;
  const bool lower = ti >= tj;
  float blk[TB][TB];
#pragma unroll
  for (int r = 0; r < TB; ++r)
#pragma unroll
    for (int c = 0; c < TB; ++c) {
      const int i = ti * TB + r, j = tj * TB + c;
      float v = 0.0f;
      if (lower) {
        if (i < b && j < b) v = j <= i ? Lblk[(int64_t)i * ld + j] : 0.0f;
        else if (i == j) v = 1.0f;
      }
      blk[r][c] = v;
    }
  if (tid == 0) bad = -1;
  __syncthreads();

  // ---------------------------------------------------------- factorisation
  for (int p = 0; p < NT; ++p) {
    if (tj == p) {  // the 16 lanes of block column p; (p, p) is lane (17 p) mod 64
      const int dl = (17 * p) & 63;
      bool ok = true;
#pragma unroll
      for (int c = 0; c < TB; ++c) {
        const float d = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(blk[c][c]), dl));
        if (!(d > 0.0f) || !(d < INFINITY)) ok = false;
        const float s = sqrtf(d), rs = 1.0f / s;
#pragma unroll
        for (int r = 0; r < TB; ++r) {
          if (ti == p) blk[r][c] = r > c ? blk[r][c] * rs : (r == c ? s : 0.0f);
          else blk[r][c] *= rs;
        }
#pragma unroll
        for (int c2 = c + 1; c2 < TB; ++c2) {
          const float lc =
              __int_as_float(__builtin_amdgcn_readlane(__float_as_int(blk[c2][c]), dl));
#pragma unroll
          for (int r = 0; r < TB; ++r) blk[r][c2] -= blk[r][c] * lc;
        }
      }
      if (!ok && ti == p) {  // first failing column of this block
        int c0 = 0;
        for (; c0 < TB; ++c0)
          if (!(blk[c0][c0] > 0.0f) || !(blk[c0][c0] < INFINITY)) break;
        bad = p * TB + (c0 < TB ? c0 : 0);
      }
      if (ti >= p) {
#pragma unroll
        for (int c = 0; c < TB; ++c) {
          f32x4* dst = reinterpret_cast<f32x4*>(&Pn[p][c][ti * TB]);
          dst[0] = f32x4{blk[0][c], blk[1][c], blk[2][c], blk[3][c]};
          dst[1] = f32x4{blk[4][c], blk[5][c], blk[6][c], blk[7][c]};
        }
      }
    }
    __syncthreads();
    if (bad >= 0) break;
    if (tj > p && lower) {
      float a[TB][TB], bb[TB][TB];  // a[r][k] = L(8 ti + r, 8 p + k), bb likewise for tj
#pragma unroll
      for (int k = 0; k < TB; ++k) {
        const f32x4* sa = reinterpret_cast<const f32x4*>(&Pn[p][k][ti * TB]);
        const f32x4* sb = reinterpret_cast<const f32x4*>(&Pn[p][k][tj * TB]);
        const f32x4 a0 = sa[0], a1 = sa[1], b0 = sb[0], b1 = sb[1];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          a[q][k] = a0[q];
          a[q + 4][k] = a1[q];
          bb[q][k] = b0[q];
          bb[q + 4][k] = b1[q];
        }
      }
#pragma unroll
      for (int r = 0; r < TB; ++r)
#pragma unroll
        for (int c = 0; c < TB; ++c) {
          float acc = blk[r][c];
#pragma unroll
          for (int k = 0; k < TB; ++k) acc -= a[r][k] * bb[c][k];
          blk[r][c] = acc;
        }
    }
  }
  if (bad >= 0) {
    if (tid == 0) {
      st[1] = side;
      st[2] = (int)(pivot_base + bad);
      __threadfence();
      st[0] = iteration;
    }
    return;
  }
  // Diagonal blocks, in parallel: log-determinant share and 8 x 8 inverse.
  if (ti == tj) {
    double lsum = 0.0;
#pragma unroll
    for (int c = 0; c < TB; ++c) lsum += log((double)blk[c][c]);
    ldp[ti] = lsum;
    float inv[TB][TB];
#pragma unroll
    for (int c = 0; c < TB; ++c) {
#pragma unroll
      for (int r = 0; r < TB; ++r) {
        float acc = r == c ? 1.0f : 0.0f;
#pragma unroll
        for (int k = 0; k < TB; ++k)
          if (k >= c && k < r) acc -= blk[r][k] * inv[k][c];
        inv[r][c] = r >= c ? acc / blk[r][r] : 0.0f;
      }
    }
#pragma unroll
    for (int r = 0; r < TB; ++r)
#pragma unroll
      for (int c = 0; c < TB; ++c) Ld[ti][r][c] = inv[r][c];
  }
  __syncthreads();
  if (tid == 0) {
    double s = 0.0;
    for (int p = 0; p < NT; ++p) s += ldp[p];
    logdet[slot] = s;
  }

  // ---------------------------------------------------------------- inverse
  // acc(ti, tj) = E - sum_{k < p} L(ti, k) X(k, tj); block row p is final at step p.
#pragma unroll
  for (int r = 0; r < TB; ++r)
#pragma unroll
    for (int c = 0; c < TB; ++c) blk[r][c] = (lower && ti == tj && r == c) ? 1.0f : 0.0f;
  for (int p = 0; p < NT; ++p) {
    const int buf = p & 1;
    if (ti == p && tj <= p) {
      float x[TB][TB];
#pragma unroll
      for (int r = 0; r < TB; ++r)
#pragma unroll
        for (int c = 0; c < TB; ++c) {
          float acc = 0.0f;
#pragma unroll
          for (int k = 0; k < TB; ++k) acc += Ld[p][r][k] * blk[k][c];
          x[r][c] = acc;
        }
#pragma unroll
      for (int r = 0; r < TB; ++r) {
#pragma unroll
        for (int c = 0; c < TB; ++c) blk[r][c] = x[r][c];
        f32x4* dst = reinterpret_cast<f32x4*>(&Xr[buf][r][tj * TB]);
        dst[0] = f32x4{x[r][0], x[r][1], x[r][2], x[r][3]};
        dst[1] = f32x4{x[r][4], x[r][5], x[r][6], x[r][7]};
      }
    }
    __syncthreads();
    if (ti > p && tj <= p) {
      float a[TB][TB], xb[TB][TB];
#pragma unroll
      for (int k = 0; k < TB; ++k) {
        const f32x4* sa = reinterpret_cast<const f32x4*>(&Pn[p][k][ti * TB]);
        const f32x4* sx = reinterpret_cast<const f32x4*>(&Xr[buf][k][tj * TB]);
        const f32x4 a0 = sa[0], a1 = sa[1], x0 = sx[0], x1 = sx[1];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          a[q][k] = a0[q];
          a[q + 4][k] = a1[q];
          xb[k][q] = x0[q];
          xb[k][q + 4] = x1[q];
        }
      }
#pragma unroll
      for (int r = 0; r < TB; ++r)
#pragma unroll
        for (int c = 0; c < TB; ++c) {
          float acc = blk[r][c];
#pragma unroll
          for (int k = 0; k < TB; ++k) acc -= a[r][k] * xb[k][c];
          blk[r][c] = acc;
        }
    }
  }
#pragma unroll
  for (int r = 0; r < TB; ++r)
#pragma unroll
    for (int c = 0; c < TB; ++c) {
      const int i = ti * TB + r, j = tj * TB + c;
      if (i < b && j < b) Liblk[(int64_t)i * ld + j] = (lower && j <= i) ? blk[r][c] : 0.0f;
    }
}

}  // namespace

hipError_t launch_chol_leaf(const float* Lblk, float* Liblk, int64_t ld, int b, int64_t pivot_base,
                            double* logdet, int slot, int iteration, int side, int* st,
                            hipStream_t s) {
  if (b < 1 || b > kLeaf || ld < b) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_chol_leaf, dim3(1), dim3(256), 0, s, Lblk, Liblk, ld, b, pivot_base, logdet,
                     slot, iteration, side, st);
  return hipGetLastError();
}

}  // namespace ff
