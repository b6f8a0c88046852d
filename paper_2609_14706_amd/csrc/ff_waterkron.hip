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
constexpr int ST = 16;   // sub-tile edge
constexpr int CP = 68;   // pitch of the in-tile contributions and residuals
constexpr int PP = 17;   // pitch of a sub-tile product scratch
constexpr int DP = 272;  // stride of the diagonal La blocks (16 x 16 + a bank offset)

// LDS of a workgroup, in floats.  Tile workgroups: phase 1 (products from
// outside the tile) stages operands in SA / SB; phase 2 (the in-tile sweep)
// keeps Lb[I][I] and La[J][J] (row r rotated by 4 (r mod 16) to spread the
// banks), the contributions C^T of the tile (a 16 x 16 block is replaced by
// the row-block prefix Xs^T of its sub-tile once that sub-tile is done), the
// residuals E^T, per-wave product scratch, the diagonal 16 x 16 blocks of
// La[J][J] transposed, and the tile's scales.  Push workgroups use SA / SB.
constexpr int L_LB = 0, L_LA = WTT, L_SA = 2 * WTT, L_SB = L_SA + WT * OP, L_TOTAL = L_SB + WT * OP;
constexpr int L_CT = 2 * WTT, L_ET = L_CT + WT * CP, L_PS = L_ET + WT * CP;
constexpr int L_LAD = L_PS + 4 * ST * PP, L_AL = L_LAD + 4 * DP;
constexpr int L_BE = L_AL + WT, L_DA = L_BE + WT, L_DB = L_DA + WT;
static_assert(L_DB + WT <= L_TOTAL, "tile LDS map");

__device__ __forceinline__ int rot(int r, int c) { return r * WT + ((c + 4 * (r & 15)) & 63); }

typedef __attribute__((ext_vector_type(4))) float f32x4v;

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

// acc += A B over k < 64 for this wave's 32 x 32 quadrant (wm, wn) of a
// 64 x 64 product; fa(i, k) and fb(k, j) read the operands.
template <class FA, class FB>
__device__ __forceinline__ void mac64f(FA fa, FB fb, f32x16& acc, int wm, int wn, int lane) {
#pragma unroll
  for (int s = 0; s < WT / 2; ++s) {
    const int kr = 2 * s + (lane >> 5);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(fa(wm * 32 + (lane & 31), kr),
                                               fb(kr, wn * 32 + (lane & 31)), acc, 0, 0, 0);
  }
}

__device__ __forceinline__ void mac64(const float (*sa)[OP], const float (*sb)[OP], f32x16& acc,
                                      int wm, int wn, int lane) {
  mac64f([&](int i, int k) { return sa[k][i]; }, [&](int k, int j) { return sb[k][j]; }, acc, wm,
         wn, lane);
}

// acc += A B over k < 16 for one 16 x 16 block on the 16 x 16 x 4 fp32
// matrix cores: fa(m, k), fb(k, n); this lane holds D[4 (lane / 16) + r][lane % 16].
template <class FA, class FB>
__device__ __forceinline__ void mac16(FA fa, FB fb, f32x4v& acc, int lane) {
  const int n = lane & 15, g = lane >> 4;
#pragma unroll
  for (int q = 0; q < 4; ++q)
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(fa(n, 4 * q + g), fb(4 * q + g, n), acc, 0, 0, 0);
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

// State of wave 0's lanes over the 16 columns of a sub-diagonal (lane row
// = one sub-tile, lane = one of its rows i).
struct ChainCtx {
  float lbs[ST];    // row i of the diagonal Lb block scaled by beta_k / beta_i, below the diagonal
  float step[ST];   // alpha_j beta_i of the 16 columns
  float rstep[ST];  // 1 / step
  float bq[ST];     // column coupling inside the sub-tile (unscaled)
  float cv[ST];     // contributions C^T[j][i] from outside the sub-tile
  float da[ST];     // RevCholesky diagonal of A at the 16 columns
  f32x4 cn[4];      // this column's coupling coefficients La[j'][j], j' = 16 b + 0..15
  f32x4 cp[4];      // the previous column's
  float u, e, z;    // the previous column's update, residual and code
  float dist;
  const float* ladT;  // La[J][J] block (b, b) transposed: ladT[c * 16 + c2] = La[16 b + c2][16 b + c]
  float* et;          // E^T in LDS at (16 b, i)
  float* erow;        // the transposed residual tile in memory at (16 b, i)
  int32_t* zrow;      // padded codes at (i, 16 b)
};

__device__ __forceinline__ float cf(const f32x4 (&v)[4], int k) { return v[k >> 2][k & 3]; }

// Work of the previous column C - 1 spread over the row steps K of column C:
// loads of column C's coefficients (K < 4), the coupling updates of the
// columns after C (one per step), and the previous column's stores.
template <int C, int K>
__device__ __forceinline__ void side(ChainCtx& x) {
  if constexpr (K < 4)
    x.cn[K] = *reinterpret_cast<const f32x4*>(x.ladT + C * ST + 4 * K);
  if constexpr (C > 0) {
    constexpr int c2 = C + 1 + K;  // updates of bq[c2] with the previous column's u
    if constexpr (c2 < ST) x.bq[c2] = fmaf(cf(x.cp, c2), x.u, x.bq[c2]);
    if constexpr (K == 12) x.et[(C - 1) * CP] = x.e;
    if constexpr (K == 13) x.erow[(C - 1) * WT] = x.e;
    if constexpr (K == 14) x.zrow[C - 1] = (int32_t)x.z;
    if constexpr (K == 15) {
      const float t = x.e * x.da[C - 1];
      x.dist = fmaf(t, t, x.dist);
    }
  }
}

// Row step K of column C: row K is final; its scaled residual is broadcast
// within the lane row (DPP row_newbcast) and updates the rows below it.
template <int C, int K>
__device__ __forceinline__ void rowstep(ChainCtx& x, float& q) {
  const float dd = __builtin_rintf(q) - q;
  __builtin_amdgcn_sched_barrier(0);
  side<C, K>(x);
  __builtin_amdgcn_sched_barrier(0);
  const float D =
      __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(dd), 0x150 + K, 0xF, 0xF, true));
  q = fmaf(x.lbs[K], D, q);
  if constexpr (K + 1 < ST) rowstep<C, K + 1>(x, q);
}

template <int C>
__device__ __forceinline__ void column(ChainCtx& x) {
  float q = (x.cv[C] + x.bq[C]) * x.rstep[C];
  const float qs = q;
  rowstep<C, 0>(x, q);
  const float z = __builtin_rintf(q);
  x.e = (z - q) * x.step[C];
  x.u = (z - qs) * x.step[C];
  x.z = z;
#pragma unroll
  for (int k = 0; k < 4; ++k) x.cp[k] = x.cn[k];
  if constexpr (C + 1 < ST) {
    x.bq[C + 1] = fmaf(cf(x.cp, C + 1), x.u, x.bq[C + 1]);  // the next column needs it now
    column<C + 1>(x);
  }
}

// Wave 0: the sub-tiles (a, s - a) of in-tile sub-diagonal s, one per row of
// 16 lanes (slot = lane / 16, a = alo + slot; rows of lanes beyond the nv
// sub-tiles repeat slot 0 and store the same values).  Reads the
// contributions C^T, writes residuals (LDS and the transposed residual tile
// Et) and the padded codes; returns this lane's share of
// sum (L^B_ii e_ij L^A_jj)^2 (the diagonals are 0 in the padding).
__device__ __forceinline__ double subdiag_chain(const WkParams& p, float* lds, int s, int alo,
                                                int nv, int64_t r0, int64_t c0,
                                                float* __restrict__ Et, int lane) {
  const int slot = lane >> 4, rr = lane & 15;
  const bool live = slot < nv;
  const int a = alo + (live ? slot : 0), b = s - a;
  const int i = ST * a + rr;
  const float bi = lds[L_BE + i];
  ChainCtx x;
#pragma unroll
  for (int k = 0; k < ST; ++k)
    x.lbs[k] = k < rr ? lds[L_LB + rot(i, ST * a + k)] * (lds[L_BE + ST * a + k] / bi) : 0.0f;
  const float* ct = lds + L_CT + (ST * b) * CP + i;
#pragma unroll
  for (int c = 0; c < ST; ++c) {
    x.step[c] = lds[L_AL + ST * b + c] * bi;
    x.rstep[c] = 1.0f / x.step[c];
    x.bq[c] = 0.0f;
    x.cv[c] = ct[c * CP];
    x.da[c] = lds[L_DA + ST * b + c];
  }
  x.ladT = lds + L_LAD + b * DP;
  x.et = lds + L_ET + (ST * b) * CP + i;
  x.erow = Et + (ST * b) * WT + i;
  x.zrow = p.Z + (r0 + i) * p.nq + c0 + ST * b;
  x.dist = 0.0f;
  column<0>(x);
  // the last column's stores
  x.et[(ST - 1) * CP] = x.e;
  x.erow[(ST - 1) * WT] = x.e;
  x.zrow[ST - 1] = (int32_t)x.z;
  const float t = x.e * x.da[ST - 1];
  x.dist = fmaf(t, t, x.dist);
  const double db = live ? (double)lds[L_DB + i] : 0.0;
  return db * db * (double)x.dist;
}

// Wave w = slot: the contributions a sub-tile (a, b) of sub-diagonal s still
// lacks, from the sub-tiles above it and to its left inside the tile:
//   P^T[j][i]  = sum_{b' < b} sum_{j' in b'} La[j][j'] e[i][j']
//   C^T[j][i] += sum_{a' < a} sum_{i' in a'} Xs^T[j][i'] Lb[i][i'] + sum_{i' in a} P^T[j][i'] Lb[i][i']
// (transposed 16 x 16 blocks; Xs^T of the finished sub-tiles sits in their
// blocks of C^T).  P is returned for the row-block prefix of (a, b).
__device__ __forceinline__ void subtile_pull(float* lds, int a, int b, int wave, int lane,
                                             f32x4v& P) {
  const int n = lane & 15, g = lane >> 4;
  P = f32x4v{0.0f, 0.0f, 0.0f, 0.0f};
  for (int bp = 0; bp < b; ++bp)
    mac16([&](int m, int k) { return lds[L_LA + rot(ST * b + m, ST * bp + k)]; },
          [&](int k, int nn) { return lds[L_ET + (ST * bp + k) * CP + ST * a + nn]; }, P, lane);
  float* ps = lds + L_PS + wave * ST * PP;
#pragma unroll
  for (int r = 0; r < 4; ++r) ps[(4 * g + r) * PP + n] = P[r];
  float* cblk = lds + L_CT + (ST * b) * CP + ST * a;
  f32x4v acc;
#pragma unroll
  for (int r = 0; r < 4; ++r) acc[r] = cblk[(4 * g + r) * CP + n];
  for (int ap = 0; ap < a; ++ap)
    mac16([&](int m, int k) { return lds[L_CT + (ST * b + m) * CP + ST * ap + k]; },
          [&](int k, int nn) { return lds[L_LB + rot(ST * a + nn, ST * ap + k)]; }, acc, lane);
  mac16([&](int m, int k) { return ps[m * PP + k]; },
        [&](int k, int nn) { return lds[L_LB + rot(ST * a + nn, ST * a + k)]; }, acc, lane);
#pragma unroll
  for (int r = 0; r < 4; ++r) cblk[(4 * g + r) * CP + n] = acc[r];
}

// After its chain: Xs^T = P^T + (La[b][b] e_ab^T), stored over the consumed
// contribution block (a, b).
__device__ __forceinline__ void subtile_prefix(float* lds, int a, int b, int lane, f32x4v P) {
  const int n = lane & 15, g = lane >> 4;
  mac16([&](int m, int k) { return lds[L_LA + rot(ST * b + m, ST * b + k)]; },
        [&](int k, int nn) { return lds[L_ET + (ST * b + k) * CP + ST * a + nn]; }, P, lane);
  float* cblk = lds + L_CT + (ST * b) * CP + ST * a;
#pragma unroll
  for (int r = 0; r < 4; ++r) cblk[(4 * g + r) * CP + n] = P[r];
}

__global__ __launch_bounds__(256, 2) void k_wk_diagonal(WkParams p, int d, int nrec, int ilo) {
  if (ff_halted(p.st)) return;
  __shared__ __align__(16) float lds[L_TOTAL];
  float(*SA)[OP] = reinterpret_cast<float(*)[OP]>(lds + L_SA);
  float(*SB)[OP] = reinterpret_cast<float(*)[OP]>(lds + L_SB);
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int wm = wave >> 1, wn = wave & 1;
  const int bid = blockIdx.x;
  const int NT = p.NT, MT = p.MT;
  auto blk = [&](float* base, int I, int J) { return base + ((int64_t)I * NT + J) * WTT; };

  if (bid < nrec) {
    // ------------------------------------------------ tile (I, J) of diagonal d
    const int I = ilo + bid, J = d - I;
    const int64_t r0 = (int64_t)I * WT, c0 = (int64_t)J * WT;
    // the tile's diagonal factor blocks, rows rotated
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int idx = tid + 256 * q;
      const int r = idx >> 4, c = (idx & 15) * 4;
      *reinterpret_cast<f32x4*>(&lds[L_LB + rot(r, c)]) =
          *reinterpret_cast<const f32x4*>(p.Lb + (r0 + r) * p.mq + r0 + c);
      *reinterpret_cast<f32x4*>(&lds[L_LA + rot(r, c)]) =
          *reinterpret_cast<const f32x4*>(p.La + (c0 + r) * p.nq + c0 + c);
    }
    f32x16 pre;
    load_tile(pre, blk(p.Pre, I, J), wm, wn, lane);
    if (J > 0) {  // + E[I][J-1] La[J][J-1]^T
      stage_omaj(SA, blk(p.E, I, J - 1), WT, tid);
      stage_kmaj(SB, p.La + c0 * p.nq + (c0 - WT), p.nq, tid);
      __syncthreads();
      mac64(SA, SB, pre, wm, wn, lane);
      __syncthreads();
    }
    f32x16 racc;
    load_tile(racc, blk(p.Racc, I, J), wm, wn, lane);
    if (I > 0) {  // + Lb[I][I-1] X[I-1][J]
      stage_kmaj(SA, p.Lb + r0 * p.mq + (r0 - WT), p.mq, tid);
      stage_omaj(SB, blk(p.X, I - 1, J), WT, tid);
      __syncthreads();
      mac64(SA, SB, racc, wm, wn, lane);
      __syncthreads();
    }
    // + Lb[I][I] Pre
#pragma unroll
    for (int r = 0; r < 16; ++r) SB[acc_row(wm, lane, r)][acc_col(wn, lane)] = pre[r];
    __syncthreads();
    mac64f([&](int i, int k) { return lds[L_LB + rot(i, k)]; },
           [&](int k, int j) { return SB[k][j]; }, racc, wm, wn, lane);
    __syncthreads();
    // C^T = (W + racc)^T; the tile's scales and RevCholesky diagonals
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int i = acc_row(wm, lane, r), j = acc_col(wn, lane);
      const int64_t gi = r0 + i, gj = c0 + j;
      const float w = (gi < p.m && gj < p.n) ? p.W[gi * p.n + gj] : 0.0f;
      lds[L_CT + j * CP + i] = racc[r] + w;
    }
    if (tid < WT) {
      lds[L_AL + tid] = p.alpha[c0 + tid];
      lds[L_BE + tid] = p.beta[r0 + tid];
      lds[L_DA + tid] = p.dA[c0 + tid];
      lds[L_DB + tid] = p.dB[r0 + tid];
    }
    for (int idx = tid; idx < 4 * ST * ST; idx += 256) {  // diagonal La blocks, transposed
      const int bb = idx >> 8, c2 = (idx >> 4) & 15, c = idx & 15;
      lds[L_LAD + bb * DP + c * ST + c2] = p.La[(c0 + ST * bb + c2) * p.nq + c0 + ST * bb + c];
    }
    __syncthreads();
    float* Et = blk(p.E, I, J);
    double dist = 0.0;
    for (int s = 0; s < 7; ++s) {
      const int alo = s > 3 ? s - 3 : 0;
      const int nv = (s < 3 ? s : 3) - alo + 1;
      const bool src = wave < nv;
      const int a = alo + (src ? wave : 0), b = s - a;
      f32x4v P;
      if (src) subtile_pull(lds, a, b, wave, lane, P);
      __syncthreads();
      if (wave == 0) dist += subdiag_chain(p, lds, s, alo, nv, r0, c0, Et, lane);
      __syncthreads();
      if (src) subtile_prefix(lds, a, b, lane, P);
      __syncthreads();
    }
    if (wave == 0) {
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) dist += __shfl_xor(dist, o);
      if (lane == 0) p.dpart[(int64_t)I * NT + J] = dist;
    }
    // X[I][J] = Pre + E La[J][J]^T
    mac64f([&](int i, int k) { return lds[L_ET + k * CP + i]; },
           [&](int k, int j) { return lds[L_LA + rot(j, k)]; }, pre, wm, wn, lane);
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
      stage_kmaj(SA, p.Lb + (int64_t)I * WT * p.mq + (int64_t)Is * WT, p.mq, tid);
      stage_omaj(SB, blk(p.X, Is, Js), WT, tid);
      __syncthreads();
      mac64(SA, SB, acc, wm, wn, lane);
      store_tile(acc, blk(p.Racc, I, Js), wm, wn, lane);
      return;
    }
    u -= nR;
    const int nP = NT - Js - 2 > 0 ? NT - Js - 2 : 0;
    if (u < nP) {  // Pre[Is][J2] += E[Is][Js] La[J2][Js]^T
      const int J2 = Js + 2 + u;
      f32x16 acc;
      load_tile(acc, blk(p.Pre, Is, J2), wm, wn, lane);
      stage_omaj(SA, blk(p.E, Is, Js), WT, tid);
      stage_kmaj(SB, p.La + (int64_t)J2 * WT * p.nq + (int64_t)Js * WT, p.nq, tid);
      __syncthreads();
      mac64(SA, SB, acc, wm, wn, lane);
      store_tile(acc, blk(p.Pre, Is, J2), wm, wn, lane);
      return;
    }
    u -= nP;
  }
}

// Z[i][j] = Zp[i][j] (padded codes, leading dimension nq) and, when V is
// non-null, V[i][j] = alpha[j] beta[i] Z[i][j].
__global__ __launch_bounds__(256) void k_wk_finish(const int32_t* __restrict__ Zp, int64_t nq,
                                                   int64_t m, int64_t n,
                                                   const float* __restrict__ alpha,
                                                   const float* __restrict__ beta,
                                                   int32_t* __restrict__ Z, float* __restrict__ V,
                                                   const int* st) {
  if (ff_halted(st)) return;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= m * n) return;
  const int64_t i = idx / n, j = idx % n;
  const int32_t z = Zp[i * nq + j];
  Z[idx] = z;
  if (V != nullptr) V[idx] = (alpha[j] * beta[i]) * (float)z;
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

hipError_t launch_wk_finish(const int32_t* Zp, int64_t nq, int64_t m, int64_t n,
                           const float* alpha, const float* beta, int32_t* Z, float* V,
                           const int* st, hipStream_t s) {
  if (m < 1 || n < 1 || nq < n) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_wk_finish, dim3(blocks_for(m * n)), dim3(256), 0, s, Zp, nq, m, n, alpha,
                     beta, Z, V, st);
  return hipGetLastError();
}

hipError_t launch_wk_sum(const double* part, int64_t count, double scale, double* out,
                         const int* st, hipStream_t s) {
  if (count < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_wk_sum, dim3(1), dim3(256), 0, s, part, count, scale, out, st);
  return hipGetLastError();
}

}  // namespace ff
