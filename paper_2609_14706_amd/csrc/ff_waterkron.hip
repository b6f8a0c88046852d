// WaterKron: two-sided GPTQ (Algorithm 2) with the waterfilling scales of
// Corollary 3.2.
//
// Algorithm 2 visits the entries of W column by column (j outer, i inner)
// and spreads the rounding error of entry (i, j) over the entries i' >= i,
// j' >= j with the outer product of column i of the normalised inverse
// output factor Lb and column j of the normalised inverse input factor La.
// The value entry (i, j) is rounded from is therefore
//     c_ij = W_ij + sum over (i', j') <= (i, j), (i', j') != (i, j),
//                   of Lb[i][i'] e[i'][j'] La[j][j'],
// with e = v - c the rounding residuals: it depends only on the entries
// above and to the left of it.  Any order that respects that partial order
// gives the same codes, so 64 x 64 tiles on one anti-diagonal I + J = d are
// independent.  The engine makes one launch per anti-diagonal:
//
// * one "tile" workgroup per tile (I, J) of the diagonal completes its
//   outside contributions (the two coming from the diagonal just finished),
//   then one wave runs the in-tile recurrence: columns in order; in a
//   column, lane i holds row i and row k's residual is broadcast with
//   v_readlane at step k;
// * "push" workgroups add each tile of the previous diagonal into the
//   accumulators of the tiles two or more steps below or right of it.
//
// Accumulators, per 64 x 64 tile (tile-blocked storage, 4096 floats each):
//   X[I][J]    = sum_{J' <= J} E[I][J'] La[J][J']^T        (row-block prefix)
//   Pre[I][J]  = sum_{J' <  J} E[I][J'] La[J][J']^T
//   Racc[I][J] = sum_{I' <  I} Lb[I][I'] X[I'][J]
// so that the tile's input is R = W + Racc + Lb[I][I] Pre.  Each push is
// one 64 x 64 x 64 fp32 matrix-core product; every accumulator receives its
// terms in a fixed order (one per diagonal), so results are deterministic.
//
// In-tile arithmetic is scaled by the step s_ij = alpha_j beta_i: lane i
// carries q = c / s_ij, the rounding is q -> rint(q) (ties to even), the row
// coupling uses Lb[i][k] beta_k / beta_i and the column coupling
// La[j][j'] alpha_j' / alpha_j on the scaled column updates
// u'_ij = (v_ij - c_start_ij) / s_ij.
#include <math.h>

#include "ff_common.hpp"
#include "ff_kernels.hpp"

namespace ff {
namespace {

constexpr int WT = 64;   // tile edge
constexpr int WTT = WT * WT;
constexpr int OP = 96;   // operand pitch: rows k and k + 1 fall in opposite bank halves

__device__ __forceinline__ float bcastf(float v, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

// ------------------------------------------------------------ preparation
// out[i][j] = M[d-1-i][d-1-j]  (J M J)
__global__ __launch_bounds__(256) void k_wk_reverse(const float* __restrict__ M, int64_t d,
                                                    float* __restrict__ out, const int* st) {
  if (ff_halted(st)) return;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= d * d) return;
  const int64_t i = idx / d, j = idx % d;
  out[idx] = M[(d - 1 - i) * d + (d - 1 - j)];
}

// Ci = C^-1 with C = Cholesky(J M J) (d x d, ld d).  RevCholesky(M) = J C^T J,
// its inverse is J C^-T J, whose entry (i, j) is Ci[d-1-j][d-1-i]; dividing
// column j by its diagonal entry gives the normalised inverse
//   Lt[i][j] = Ci[d-1-j][d-1-i] / Ci[d-1-j][d-1-j]   (i >= j),
// written padded to dq x dq with the identity outside d x d.  diag[j] =
// RevCholesky(M)_jj = 1 / Ci[d-1-j][d-1-j] (0 in the padding).
__global__ __launch_bounds__(256) void k_wk_normalise(const float* __restrict__ Ci, int64_t d,
                                                      int64_t dq, float* __restrict__ Lt,
                                                      float* __restrict__ diag, const int* st) {
  if (ff_halted(st)) return;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= dq * dq) return;
  const int64_t i = idx / dq, j = idx % dq;
  float v;
  if (i < d && j < d) {
    const int64_t r = d - 1 - j;
    const float dj = Ci[r * d + r];
    v = i >= j ? Ci[r * d + (d - 1 - i)] / dj : 0.0f;
    if (i == j) diag[j] = 1.0f / dj;
  } else {
    v = i == j ? 1.0f : 0.0f;
    if (i == j) diag[j] = 0.0f;
  }
  Lt[idx] = v;
}

// Padded scales (1 in the padding).  given == 0: Corollary 3.2,
// scale[j] = sqrt(gamma) |M|^(1/2d) / diag[j] with log |M|^(1/2d) = the sum of
// the factorisation's log-pivot slots / d, also written to user[0..d);
// given == 1: scale[j] = user[j].
__global__ __launch_bounds__(256) void k_wk_scales(const float* __restrict__ diag, int64_t d,
                                                   int64_t dq, const double* slots, int nslots,
                                                   double gamma, int given, float* __restrict__ user,
                                                   float* __restrict__ scale, const int* st) {
  if (ff_halted(st)) return;
  double g = 0.0;
  if (!given) {
    double ls = 0.0;
    for (int k = 0; k < nslots; ++k) ls += slots[k];
    g = sqrt(gamma) * exp(ls / (double)d);
  }
  for (int64_t j = threadIdx.x; j < dq; j += 256) {
    float v = 1.0f;
    if (j < d) {
      if (given) {
        v = user[j];
      } else {
        v = (float)(g / (double)diag[j]);
        user[j] = v;
      }
    }
    scale[j] = v;
  }
}

// ------------------------------------------------------------- the sweep
struct WkLDS {
  float sa[WT][OP];  // left operand, [k][row]; the tile's residuals e[i][j] at [j][i]
  float sb[WT][OP];  // right operand, [k][col]; the tile's input R[i][j] at [j][i]
  float sl[WT][WT];  // scaled in-tile La: La[j][j'] alpha_j' / alpha_j
  float su[WT][WT];  // scaled column updates u'[j][i]
};

// s[k][o] = P[o * ld + k]: operand contiguous along k
__device__ __forceinline__ void stage_kmaj(float (*s)[OP], const float* __restrict__ P, int64_t ld,
                                           int tid) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int idx = tid + 256 * q;
    const int o = idx >> 4, k = (idx & 15) * 4;
    const f32x4 v = *reinterpret_cast<const f32x4*>(P + (int64_t)o * ld + k);
    s[k][o] = v[0];
    s[k + 1][o] = v[1];
    s[k + 2][o] = v[2];
    s[k + 3][o] = v[3];
  }
}

// s[k][o] = P[k * ld + o]: operand contiguous along o
__device__ __forceinline__ void stage_omaj(float (*s)[OP], const float* __restrict__ P, int64_t ld,
                                           int tid) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int idx = tid + 256 * q;
    const int k = idx >> 4, o = (idx & 15) * 4;
    *reinterpret_cast<f32x4*>(&s[k][o]) = *reinterpret_cast<const f32x4*>(P + (int64_t)k * ld + o);
  }
}

// acc += sa^T sb over k < 64 for this wave's 32 x 32 quadrant (wm, wn).
__device__ __forceinline__ void mac64(const float (*sa)[OP], const float (*sb)[OP], f32x16& acc,
                                      int wm, int wn, int lane) {
#pragma unroll
  for (int s = 0; s < WT / 2; ++s) {
    const int kr = 2 * s + (lane >> 5);
    const float a = sa[kr][wm * 32 + (lane & 31)];
    const float b = sb[kr][wn * 32 + (lane & 31)];
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc, 0, 0, 0);
  }
}

// Row and column of accumulator element r of this lane in the 64 x 64 tile.
__device__ __forceinline__ int acc_row(int wm, int lane, int r) {
  return wm * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
}
__device__ __forceinline__ int acc_col(int wn, int lane) { return wn * 32 + (lane & 31); }

__device__ __forceinline__ void load_tile(f32x16& acc, const float* __restrict__ P, int wm, int wn,
                                          int lane) {
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = P[acc_row(wm, lane, r) * WT + acc_col(wn, lane)];
}

__device__ __forceinline__ void store_tile(const f32x16& acc, float* __restrict__ P, int wm, int wn,
                                           int lane) {
#pragma unroll
  for (int r = 0; r < 16; ++r) P[acc_row(wm, lane, r) * WT + acc_col(wn, lane)] = acc[r];
}

// The wave-0 recurrence of one tile.  R (at sb[j][i]) holds every
// contribution from outside the tile; writes codes, residuals (sa[j][i] and
// the transposed residual tile Et[j * 64 + i]) and returns this lane's share
// of sum (L^B_ii e_ij L^A_jj)^2.
__device__ __forceinline__ double tile_recurrence(const WkParams& p, WkLDS& sm, int I, int J,
                                                  float* __restrict__ Et, int lane) {
  const int i = lane;
  const int64_t r0 = (int64_t)I * WT, c0 = (int64_t)J * WT;
  const int64_t gi = r0 + i;
  const float bi = p.beta[gi];
  // row i of the in-tile Lb, scaled by beta_k / beta_i, strictly below the diagonal
  float lbs[WT];
  const float* lrow = p.Lb + gi * p.mq + r0;
#pragma unroll
  for (int k4 = 0; k4 < WT; k4 += 4) {
    const f32x4 v = *reinterpret_cast<const f32x4*>(lrow + k4);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int k = k4 + e;
      lbs[k] = k < i ? v[e] * (p.beta[r0 + k] / bi) : 0.0f;
    }
  }
  const bool row_live = gi < p.m;
  const double dbi = (double)p.dB[gi];
  double dist = 0.0;
  for (int j = 0; j < WT; ++j) {
    const int64_t gj = c0 + j;
    const float step = p.alpha[gj] * bi;
    // column coupling: sum_{j' < j} La~[j][j'] u'[j'][i], four partial sums
    float b0 = 0.0f, b1 = 0.0f, b2 = 0.0f, b3 = 0.0f;
    int jp = 0;
    for (; jp + 4 <= j; jp += 4) {
      b0 = fmaf(sm.sl[j][jp], sm.su[jp][i], b0);
      b1 = fmaf(sm.sl[j][jp + 1], sm.su[jp + 1][i], b1);
      b2 = fmaf(sm.sl[j][jp + 2], sm.su[jp + 2][i], b2);
      b3 = fmaf(sm.sl[j][jp + 3], sm.su[jp + 3][i], b3);
    }
    for (; jp < j; ++jp) b0 = fmaf(sm.sl[j][jp], sm.su[jp][i], b0);
    float q = sm.sb[j][i] / step + ((b0 + b1) + (b2 + b3));
    const float qs = q;
    // row chain: at step k row k is final; its scaled residual updates the rows below
#pragma unroll
    for (int k = 0; k < WT; ++k) {
      const float dd = __builtin_rintf(q) - q;
      q = fmaf(lbs[k], bcastf(dd, k), q);
    }
    const float z = __builtin_rintf(q);
    const float e = (z - q) * step;
    sm.su[j][i] = z - qs;
    sm.sa[j][i] = e;
    Et[j * WT + i] = e;
    if (row_live && gj < p.n) {
      p.Z[gi * p.n + gj] = (int32_t)z;
      const double t = dbi * (double)e * (double)p.dA[gj];
      dist += t * t;
    }
  }
  return dist;
}

__global__ __launch_bounds__(256) void k_wk_diagonal(WkParams p, int d, int nrec, int ilo) {
  if (ff_halted(p.st)) return;
  __shared__ __align__(16) WkLDS sm;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int wm = wave >> 1, wn = wave & 1;
  const int bid = blockIdx.x;
  const int NT = p.NT, MT = p.MT;
  auto blk = [&](float* base, int I, int J) { return base + ((int64_t)I * NT + J) * WTT; };

  if (bid < nrec) {
    // ------------------------------------------------ tile (I, J) of diagonal d
    const int I = ilo + bid, J = d - I;
    const int64_t r0 = (int64_t)I * WT, c0 = (int64_t)J * WT;
    f32x16 pre;
    load_tile(pre, blk(p.Pre, I, J), wm, wn, lane);
    if (J > 0) {  // + E[I][J-1] La[J][J-1]^T
      stage_omaj(sm.sa, blk(p.E, I, J - 1), WT, tid);
      stage_kmaj(sm.sb, p.La + c0 * p.nq + (c0 - WT), p.nq, tid);
      __syncthreads();
      mac64(sm.sa, sm.sb, pre, wm, wn, lane);
      __syncthreads();
    }
    f32x16 racc;
    load_tile(racc, blk(p.Racc, I, J), wm, wn, lane);
    if (I > 0) {  // + Lb[I][I-1] X[I-1][J]
      stage_kmaj(sm.sa, p.Lb + r0 * p.mq + (r0 - WT), p.mq, tid);
      stage_omaj(sm.sb, blk(p.X, I - 1, J), WT, tid);
      __syncthreads();
      mac64(sm.sa, sm.sb, racc, wm, wn, lane);
      __syncthreads();
    }
    // + Lb[I][I] Pre
    stage_kmaj(sm.sa, p.Lb + r0 * p.mq + r0, p.mq, tid);
#pragma unroll
    for (int r = 0; r < 16; ++r) sm.sb[acc_row(wm, lane, r)][acc_col(wn, lane)] = pre[r];
    __syncthreads();
    mac64(sm.sa, sm.sb, racc, wm, wn, lane);
    __syncthreads();
    // R = W + racc, transposed into sb; scaled in-tile La into sl
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int i = acc_row(wm, lane, r), j = acc_col(wn, lane);
      const int64_t gi = r0 + i, gj = c0 + j;
      const float w = (gi < p.m && gj < p.n) ? p.W[gi * p.n + gj] : 0.0f;
      sm.sb[j][i] = racc[r] + w;
    }
    for (int idx = tid; idx < WTT; idx += 256) {
      const int j = idx >> 6, jq = idx & 63;
      sm.sl[j][jq] = jq < j ? p.La[(c0 + j) * p.nq + c0 + jq] * (p.alpha[c0 + jq] / p.alpha[c0 + j])
                            : 0.0f;
    }
    __syncthreads();
    float* Et = blk(p.E, I, J);
    if (wave == 0) {
      double dist = tile_recurrence(p, sm, I, J, Et, lane);
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) dist += __shfl_xor(dist, o);
      if (lane == 0) p.dpart[(int64_t)I * NT + J] = dist;
    }
    __syncthreads();
    // X[I][J] = Pre + E La[J][J]^T  (residuals already at sa[j][i])
    stage_kmaj(sm.sb, p.La + c0 * p.nq + c0, p.nq, tid);
    __syncthreads();
    mac64(sm.sa, sm.sb, pre, wm, wn, lane);
    store_tile(pre, blk(p.X, I, J), wm, wn, lane);
    return;
  }

  // ------------------------------------------ push of a tile of diagonal d - 1
  int u = bid - nrec;
  const int sd = d - 1;
  const int slo = sd - (NT - 1) > 0 ? sd - (NT - 1) : 0;
  const int shi = sd < MT - 1 ? sd : MT - 1;
  for (int Is = slo; Is <= shi; ++Is) {
    const int Js = sd - Is;
    const int nR = MT - Is - 2 > 0 ? MT - Is - 2 : 0;
    if (u < nR) {  // Racc[I][Js] += Lb[I][Is] X[Is][Js]
      const int I = Is + 2 + u;
      f32x16 acc;
      load_tile(acc, blk(p.Racc, I, Js), wm, wn, lane);
      stage_kmaj(sm.sa, p.Lb + (int64_t)I * WT * p.mq + (int64_t)Is * WT, p.mq, tid);
      stage_omaj(sm.sb, blk(p.X, Is, Js), WT, tid);
      __syncthreads();
      mac64(sm.sa, sm.sb, acc, wm, wn, lane);
      store_tile(acc, blk(p.Racc, I, Js), wm, wn, lane);
      return;
    }
    u -= nR;
    const int nP = NT - Js - 2 > 0 ? NT - Js - 2 : 0;
    if (u < nP) {  // Pre[Is][J2] += E[Is][Js] La[J2][Js]^T
      const int J2 = Js + 2 + u;
      f32x16 acc;
      load_tile(acc, blk(p.Pre, Is, J2), wm, wn, lane);
      stage_omaj(sm.sa, blk(p.E, Is, Js), WT, tid);
      stage_kmaj(sm.sb, p.La + (int64_t)J2 * WT * p.nq + (int64_t)Js * WT, p.nq, tid);
      __syncthreads();
      mac64(sm.sa, sm.sb, acc, wm, wn, lane);
      store_tile(acc, blk(p.Pre, Is, J2), wm, wn, lane);
      return;
    }
    u -= nP;
  }
}

// V[i][j] = alpha[j] beta[i] Z[i][j]
__global__ __launch_bounds__(256) void k_wk_dequant(const int32_t* __restrict__ Z, int64_t m,
                                                    int64_t n, const float* __restrict__ alpha,
                                                    const float* __restrict__ beta,
                                                    float* __restrict__ V, const int* st) {
  if (ff_halted(st)) return;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= m * n) return;
  const int64_t i = idx / n, j = idx % n;
  V[idx] = (alpha[j] * beta[i]) * (float)Z[idx];
}

// out = scale * sum of part[0..count) in a fixed order (one workgroup).
__global__ __launch_bounds__(256) void k_wk_sum(const double* __restrict__ part, int64_t count,
                                                double scale, double* __restrict__ out,
                                                const int* st) {
  if (ff_halted(st)) return;
  __shared__ double red[256];
  double s = 0.0;
  for (int64_t k = threadIdx.x; k < count; k += 256) s += part[k];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int o = 128; o >= 1; o >>= 1) {
    if ((int)threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) *out = red[0] * scale;
}

uint32_t blocks_for(int64_t count) { return (uint32_t)((count + 255) / 256); }

}  // namespace

int64_t wk_push_units(int d, int MT, int NT) {
  if (d < 1) return 0;
  const int sd = d - 1;
  const int slo = sd - (NT - 1) > 0 ? sd - (NT - 1) : 0;
  const int shi = sd < MT - 1 ? sd : MT - 1;
  int64_t units = 0;
  for (int Is = slo; Is <= shi; ++Is) {
    const int Js = sd - Is;
    units += (MT - Is - 2 > 0 ? MT - Is - 2 : 0) + (NT - Js - 2 > 0 ? NT - Js - 2 : 0);
  }
  return units;
}

hipError_t launch_wk_reverse(const float* M, int64_t d, float* out, const int* st, hipStream_t s) {
  if (d < 1 || d > (1 << 20)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_wk_reverse, dim3(blocks_for(d * d)), dim3(256), 0, s, M, d, out, st);
  return hipGetLastError();
}

hipError_t launch_wk_normalise(const float* Ci, int64_t d, int64_t dq, float* Lt, float* diag,
                               const int* st, hipStream_t s) {
  if (d < 1 || dq < d || dq % WT != 0 || dq > (1 << 20)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_wk_normalise, dim3(blocks_for(dq * dq)), dim3(256), 0, s, Ci, d, dq, Lt,
                     diag, st);
  return hipGetLastError();
}

hipError_t launch_wk_scales(const float* diag, int64_t d, int64_t dq, const double* slots,
                            int nslots, double gamma, int given, float* user, float* scale,
                            const int* st, hipStream_t s) {
  if (d < 1 || dq < d || nslots < 1 || (!given && !(gamma > 0.0))) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_wk_scales, dim3(1), dim3(256), 0, s, diag, d, dq, slots, nslots, gamma,
                     given, user, scale, st);
  return hipGetLastError();
}

hipError_t launch_wk_diagonal(const WkParams& p, int d, hipStream_t s) {
  if (p.MT < 1 || p.NT < 1 || d < 0 || d > p.MT + p.NT - 2) return hipErrorInvalidValue;
  if (p.mq != (int64_t)p.MT * WT || p.nq != (int64_t)p.NT * WT) return hipErrorInvalidValue;
  const int ilo = d - (p.NT - 1) > 0 ? d - (p.NT - 1) : 0;
  const int ihi = d < p.MT - 1 ? d : p.MT - 1;
  const int nrec = ihi - ilo + 1;
  const int64_t grid = nrec + wk_push_units(d, p.MT, p.NT);
  if (grid > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_wk_diagonal, dim3((uint32_t)grid), dim3(256), 0, s, p, d, nrec, ilo);
  return hipGetLastError();
}

hipError_t launch_wk_dequant(const int32_t* Z, int64_t m, int64_t n, const float* alpha,
                             const float* beta, float* V, const int* st, hipStream_t s) {
  if (m < 1 || n < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_wk_dequant, dim3(blocks_for(m * n)), dim3(256), 0, s, Z, m, n, alpha, beta, V,
                     st);
  return hipGetLastError();
}

hipError_t launch_wk_sum(const double* part, int64_t count, double scale, double* out,
                         const int* st, hipStream_t s) {
  if (count < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_wk_sum, dim3(1), dim3(256), 0, s, part, count, scale, out, st);
  return hipGetLastError();
}

}  // namespace ff
