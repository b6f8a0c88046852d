// Kernels of the blocked Cholesky factorisation and inverse (fp32).
//
// The factors' inverses enter every flip-flop update (Section 5: A^-1 and
// B^-1 in the two half steps); the iteration whitens with the inverse of the
// lower Cholesky factor, L^-1 (Section 2 notation: Cholesky(M) is the lower
// L with positive diagonal and L L^T = M).  The host factors right-looking
// over 128-column panels with two kernels per panel: k_panel_solve (the
// panel L_ik = A_ik L_kk^-T) and k_chol_step, in which one workgroup factors
// and inverts the next 128 x 128 diagonal block while the others apply the
// panel's update to the trailing lower triangle.
//
// Inside the block a recursion runs in LDS: for a block [[A11, .],
// [A21, A22]] of size s (halves h = s/2)
//     (L11, X11) = cholinv(A11);  L21 = A21 X11^T;  A22 -= L21 L21^T;
//     (L22, X22) = cholinv(A22);  X21 = -X22 (L21 X11)
// with X = L^-1.  32 x 32 base blocks are factored and inverted by one wave
// in registers (half the lanes hold rows of L, half columns of L^-1; each new
// column of L is broadcast through LDS); the products run on the fp32 matrix
// cores, one output tile per wave.  While wave 0 factors a base block, the
// other three waves do work off the pivot chain: the rest of the panel's
// update of the block (first two base blocks) and the stores of the parts of
// L and L^-1 already final (third).  A ragged block (b < 128) is padded with
// the identity.
#include <math.h>

#include <algorithm>
#include <type_traits>

#include "ff_common.hpp"
#include "ff_kernels.hpp"

namespace ff {
namespace {

constexpr int NB = 128;     // block size
constexpr int BS = 32;      // base block
constexpr int SP = NB + 1;  // LDS row pitch (conflict-free column reads)

struct LeafLDS {
  float C[BS][BS];  // column j of the base block's L at pivot step j (first, so
                    // its addresses fit the LDS instructions' immediate offset)
  float S[NB][SP];  // A, overwritten by L (lower triangle)
  float X[NB][SP];  // L^-1
  float T[64][65];  // product scratch
  float dg[NB];  // diagonal of L (log-determinant)
  int bad;
};

__device__ __forceinline__ float bcast(float v, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

// Factor and invert the 32 x 32 block at (o, o) with one wave.  Lane r < 32
// holds row r of the block, which becomes row r of L; lane 32 + r holds
// column r of X = L^-1 (starting from the unit vector).  Pivot step j
// scales entry j of every lane by 1 / L[j][j] (lane j keeps L[j][j]) and
// subtracts v[j] times column j of L from entries j+1.. of every lane: for
// the row lanes this is the Cholesky update, for the column lanes the
// forward substitution of L X = I.  Only entry j+1 of that update lies on
// the path to the next pivot: its multiplier L[j+1][j] is broadcast with
// v_readlane and applied at the start of the next step.  The rest of the
// column goes through LDS (sm.C[j][.], read back as uniform vectors) and is
// applied one step later, off that path.  Row-lane entries above the
// diagonal are never read for the lower triangle and are cleared at the end.
// base_factor leaves the lane's row of L or column of X in v (and L[r][r]
// in diag) and returns the block-relative failing column or -1;
// base_store writes them to S and X and L[r][r] to dg.
__device__ __forceinline__ int base_factor(LeafLDS& sm, int o, int lane, float (&v)[BS], float& diag) {
  float col[BS], nxt[BS];
  const int r = lane & 31;
  const bool rowlane = lane < BS;
#pragma unroll
  for (int c = 0; c < BS; ++c) {
    v[c] = rowlane ? (c <= r ? sm.S[o + r][o + c] : 0.0f) : (c == r ? 1.0f : 0.0f);
    col[c] = 0.0f;
    nxt[c] = 0.0f;
  }
  int bad = -1;
  diag = 1.0f;                 // L[r][r] (row lanes)
  float vp = 0.0f, lp = 0.0f;  // previous step's multiplier v[j-1] and L[j][j-1]
#pragma unroll
  for (int j = 0; j < BS; ++j) {
    if (j > 0) v[j] -= vp * lp;  // last update of entry j (from step j-1)
    const float d = bcast(v[j], j);
    if (!(d > 0.0f) || !(d < INFINITY)) {
      if (bad < 0) bad = j;
    }
    const float rs = __builtin_amdgcn_rsqf(d), s = d * rs;  // 1 / L[j][j], L[j][j]
    if (lane == j) diag = s;
    const float vj = lane == j ? s : v[j] * rs;
    v[j] = vj;
    const float ln = j + 1 < BS ? bcast(vj, j + 1) : 0.0f;  // L[j+1][j]
    if (j + 2 < BS) {
      if (rowlane) sm.C[j][r] = vj;
#pragma unroll
      for (int c = j + 2; c < BS; ++c) nxt[c] = sm.C[j][c];  // L[c][j], uniform
    }
    // the rest of step j-1's update
    if (j > 0) {
#pragma unroll
      for (int c = j + 1; c < BS; ++c) v[c] -= vp * col[c];
    }
    // bounded register lifetimes: step j-1 is complete here
#pragma unroll
    for (int c = j + 1; c < BS; ++c) asm volatile("" : "+v"(v[c]));
#pragma unroll
    for (int c = j + 2; c < BS; ++c) col[c] = nxt[c];
    if (j + 1 < BS) col[j + 1] = 0.0f;  // entry j+1 is updated through lp instead
    vp = vj;
    lp = ln;
  }
  return bad;
}

__device__ __forceinline__ void base_store(LeafLDS& sm, int o, int lane, const float (&v)[BS], float diag) {
  const int r = lane & 31;
  const bool rowlane = lane < BS;
  // one store per entry for all lanes: row r of S (row lanes) or column r
  // of X (column lanes)
  float* dst = rowlane ? &sm.S[o + r][o] : &sm.X[o][o + r];
  const int step = rowlane ? 1 : SP;
#pragma unroll
  for (int c = 0; c < BS; ++c) dst[c * step] = (rowlane && c > r) ? 0.0f : v[c];
  if (rowlane) sm.dg[o + r] = diag;
}

// The products of a recursion level are h x h (h = 64 or 32) with k running
// over h; each of the four waves owns one output tile: a 32 x 32 tile
// (v_mfma_f32_32x32x2_f32) when h = 64, a 16 x 16 tile
// (v_mfma_f32_16x16x4_f32) when h = 32.  geta(i, k) / getb(k, j) read LDS
// with i, j relative to the h x h output.
template <int H>
struct LevelTile {
  static constexpr int T = H / 2;  // tile edge
  typedef typename std::conditional<H == 64, f32x16, f32x4>::type Acc;
  static constexpr int NACC = H == 64 ? 16 : 4;

  template <class GA, class GB>
  __device__ __forceinline__ static Acc product(int wave, int lane, const GA& geta, const GB& getb) {
    const int ti = wave >> 1, tj = wave & 1;
    Acc acc;
#pragma unroll
    for (int r = 0; r < NACC; ++r) acc[r] = 0.0f;
    // the operands of eight k steps are read before their products are issued
    if constexpr (H == 64) {
      const int li = lane & 31, lk = lane >> 5;
#pragma unroll
      for (int k = 0; k < H; k += 16) {
        float a[8], b[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          a[e] = geta(ti * T + li, k + 2 * e + lk);
          b[e] = getb(k + 2 * e + lk, tj * T + li);
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[e], b[e], acc, 0, 0, 0);
      }
    } else {
      const int li = lane & 15, lk = lane >> 4;
      float a[H / 4], b[H / 4];
#pragma unroll
      for (int e = 0; e < H / 4; ++e) {
        a[e] = geta(ti * T + li, 4 * e + lk);
        b[e] = getb(4 * e + lk, tj * T + li);
      }
#pragma unroll
      for (int e = 0; e < H / 4; ++e) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[e], b[e], acc, 0, 0, 0);
    }
    return acc;
  }
  // Output coordinates of accumulator element r of this lane.
  __device__ __forceinline__ static int row(int wave, int r, int lane) {
    return (wave >> 1) * T + (H == 64 ? 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3) : 4 * (lane >> 4) + r);
  }
  __device__ __forceinline__ static int col(int wave, int lane) {
    return (wave & 1) * T + (H == 64 ? (lane & 31) : (lane & 15));
  }
};

template <int NT>
__device__ __forceinline__ void pre_update(LeafLDS& sm, int lane, const int (&ts)[NT]);

// Base block at (o, o) by wave 0; everyone waits.  Records the first failure.
// A leaf whose update A -= P P^T (P staged in X) has been applied to the
// lower 32 x 32 tile (0, 0) only gives the rest to waves 1..3 during its
// first two base blocks: pre = 1 (the block at 0) the six tiles of block
// rows 1..3 that read rows 0..63 of P, after which the block's own writes to
// X (over P's first rows) may go ahead; pre = 2 (the block at 32) the three
// tiles (2,2) (3,2) (3,3), which read only rows 64.. of P and are needed
// from the second half on.  Otherwise waves 1..3 run side (thread index
// 0..191 among them) meanwhile.
struct NoSide {
  __device__ void operator()(int) const {}
};
template <class Side = NoSide>
__device__ __forceinline__ void base_step(LeafLDS& sm, int o, int wave, int lane, int pre,
                                          const Side& side = Side()) {
  float v[BS], diag = 1.0f;
  int b = -1;
  if (wave == 0) {
    b = base_factor(sm, o, lane, v, diag);
  } else if (pre == 1) {
    const int ts[2] = {wave, wave == 1 ? 4 : wave + 4};  // (1,0) (2,1) | (1,1) (3,0) | (2,0) (3,1)
    pre_update<2>(sm, lane, ts);
  } else if (pre == 2) {
    const int ts[1] = {wave == 1 ? 5 : wave + 6};  // (2,2) | (3,2) | (3,3)
    pre_update<1>(sm, lane, ts);
  } else {
    side((int)threadIdx.x - 64);
  }
  if (pre == 1) {
    __syncthreads();
    // the recursion reads X only where it has written it, except the block
    // above the diagonal inside X11 (and X22, see leaf_body) of the top
    // level: zero X[0:32][32:64]
    const int r = threadIdx.x >> 3, c = 4 * (threadIdx.x & 7);
#pragma unroll
    for (int e = 0; e < 4; ++e) sm.X[r][32 + c + e] = 0.0f;
  }
  if (wave == 0) {
    base_store(sm, o, lane, v, diag);
    if (lane == 0 && b >= 0 && sm.bad < 0) sm.bad = o + b;
  }
  __syncthreads();
}

// Recursive cholinv of the block at (o, o) of size S (64 or 128, unrolled at
// compile time); every wave takes every barrier.  Returns the failing column
// or -1.  pre, side: see base_step (pre = 1 goes to the first base block,
// pre = 2 to the second); side2, side3: side work for the first and second
// base blocks of the second half.  A side3 other than NoSide computes this
// level's Y = L21 X11 into T (the level then skips that product).
template <int S, class Side = NoSide, class Side2 = NoSide, class Side3 = NoSide>
__device__ __forceinline__ int cholinv_lds(LeafLDS& sm, int o, int wave, int lane, int pre = 0,
                                           const Side& side = Side(), const Side2& side2 = Side2(),
                                           const Side3& side3 = Side3()) {
  constexpr int h = S / 2;
  typedef LevelTile<h> LT;
  if constexpr (h == BS) base_step(sm, o, wave, lane, pre, side);
  else cholinv_lds<h>(sm, o, wave, lane, pre, side);
  if (sm.bad >= 0) return sm.bad;
  const int o2 = o + h;
  const int oc = LT::col(wave, lane);
  // L21 = A21 X11^T, kept in registers until every wave has read A21
  const typename LT::Acc l21 = LT::product(wave, lane, [&](int i, int k) { return sm.S[o2 + i][o + k]; },
                                           [&](int k, int j) { return sm.X[o + j][o + k]; });
  __syncthreads();
#pragma unroll
  for (int r = 0; r < LT::NACC; ++r) sm.S[o2 + LT::row(wave, r, lane)][o + oc] = l21[r];
  __syncthreads();
  // A22 -= L21 L21^T
  {
    const typename LT::Acc u = LT::product(wave, lane, [&](int i, int k) { return sm.S[o2 + i][o + k]; },
                                           [&](int k, int j) { return sm.S[o2 + j][o + k]; });
#pragma unroll
    for (int r = 0; r < LT::NACC; ++r) sm.S[o2 + LT::row(wave, r, lane)][o2 + oc] -= u[r];
  }
  __syncthreads();
  if constexpr (h == BS) base_step(sm, o2, wave, lane, pre == 1 ? 2 : 0, side2);
  else cholinv_lds<h>(sm, o2, wave, lane, 0, side2, side3);
  if (sm.bad >= 0) return sm.bad;
  // Y = L21 X11 (into C at h = 32, T at h = 64: the second half's Y may be
  // in T already, made by side3);  X21 = -X22 Y
  auto ybuf = [&](int k, int j) -> float& {
    if constexpr (h == BS) return sm.C[k][j];
    else return sm.T[k][j];
  };
  if constexpr (std::is_same<Side3, NoSide>::value) {
    const typename LT::Acc y = LT::product(wave, lane, [&](int i, int k) { return sm.S[o2 + i][o + k]; },
                                           [&](int k, int j) { return sm.X[o + k][o + j]; });
#pragma unroll
    for (int r = 0; r < LT::NACC; ++r) ybuf(LT::row(wave, r, lane), oc) = y[r];
    __syncthreads();
  }
  {
    const typename LT::Acc x21 = LT::product(wave, lane, [&](int i, int k) { return sm.X[o2 + i][o2 + k]; },
                                             [&](int k, int j) { return ybuf(k, j); });
#pragma unroll
    for (int r = 0; r < LT::NACC; ++r) sm.X[o2 + LT::row(wave, r, lane)][o + oc] = -x21[r];
  }
  __syncthreads();
  return -1;
}

// 128 x 128 x 128 product of two LDS operands held as rows (pitch SP):
// acc[a][b] = P[rows of tile a] Q[rows of tile b]^T over all 128 k, for the
// 64 x 64 quadrant (wm, wn) of this wave (2 x 2 tiles of 32 x 32).  The
// operands of eight k steps are read before their products are issued.
__device__ __forceinline__ void quad_product(const float (*P)[SP], const float (*Q)[SP], int wave,
                                             int lane, f32x16 (&acc)[2][2]) {
  const int wm = wave >> 1, wn = wave & 1, li = lane & 31, lk = lane >> 5;
  const float* pp[2] = {&P[wm * 64 + li][lk], &P[wm * 64 + 32 + li][lk]};
  const float* qq[2] = {&Q[wn * 64 + li][lk], &Q[wn * 64 + 32 + li][lk]};
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][c][r] = 0.0f;
#pragma unroll
  for (int k = 0; k < NB; k += 16) {
    float pv[2][8], qv[2][8];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        pv[t][e] = pp[t][k + 2 * e];
        qv[t][e] = qq[t][k + 2 * e];
      }
#pragma unroll
    for (int e = 0; e < 8; ++e)
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int c = 0; c < 2; ++c)
          acc[a][c] = __builtin_amdgcn_mfma_f32_32x32x2f32(pv[a][e], qv[c][e], acc[a][c], 0, 0, 0);
  }
}
// Quadrant-relative row / column of element r of this lane in tile (a, c).
__device__ __forceinline__ int quad_row(int wave, int a, int r, int lane) {
  return (wave >> 1) * 64 + a * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
}
__device__ __forceinline__ int quad_col(int wave, int c, int lane) {
  return (wave & 1) * 64 + c * 32 + (lane & 31);
}

// rows [0, 128) x 128 columns of M (ld) from row r0 / column c0 into T
// (pitch SP); rows at or beyond rlim are zero.  16-byte loads when aligned.
__device__ __forceinline__ void load_rows(float (*T)[SP], const float* M, int64_t ld, int64_t r0,
                                          int64_t c0, int64_t rlim, int tid) {
  if ((ld & 3) == 0 && ((reinterpret_cast<uintptr_t>(M + c0) & 15) == 0)) {
    const int q = tid & 31, r = tid >> 5;
    float4 v[NB / 8];
#pragma unroll
    for (int t = 0; t < NB / 8; ++t) {
      const int64_t i = r0 + r + 8 * t;
      v[t] = i < rlim ? *reinterpret_cast<const float4*>(M + i * ld + c0 + 4 * q)
                      : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int t = 0; t < NB / 8; ++t) {
      float* d = &T[r + 8 * t][4 * q];
      d[0] = v[t].x;
      d[1] = v[t].y;
      d[2] = v[t].z;
      d[3] = v[t].w;
    }
  } else {
    const int j = tid & (NB - 1), i0 = tid >> 7;
    for (int i = i0; i < NB; i += 2) T[i][j] = r0 + i < rlim ? M[(r0 + i) * ld + c0 + j] : 0.0f;
  }
}

// A -= P P^T on the lower triangle of the block in S, with P (128 x 128)
// staged in X, for NT of the ten lower 32 x 32 tiles (ti >= tj), numbered in
// the order (0,0) (1,0) (1,1) (2,0) (2,1) (2,2) (3,0) (3,1) (3,2) (3,3): the
// tiles ts.  The operands of eight k steps are read before their products
// are issued.
template <int NT>
__device__ __forceinline__ void pre_update(LeafLDS& sm, int lane, const int (&ts)[NT]) {
  const int li = lane & 31, lk = lane >> 5;
  const float* pa[NT];
  const float* pb[NT];
  int ti[NT], tj[NT];
#pragma unroll
  for (int q = 0; q < NT; ++q) {
    const int t = ts[q];
    ti[q] = t < 1 ? 0 : t < 3 ? 1 : t < 6 ? 2 : 3;
    tj[q] = t - ti[q] * (ti[q] + 1) / 2;
    pa[q] = &sm.X[ti[q] * 32 + li][lk];
    pb[q] = &sm.X[tj[q] * 32 + li][lk];
  }
  f32x16 u[NT];
#pragma unroll
  for (int q = 0; q < NT; ++q)
#pragma unroll
    for (int r = 0; r < 16; ++r) u[q][r] = 0.0f;
#pragma unroll
  for (int k = 0; k < NB; k += 16) {
    float a[NT][8], b[NT][8];
#pragma unroll
    for (int q = 0; q < NT; ++q)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        a[q][e] = pa[q][k + 2 * e];
        b[q][e] = pb[q][k + 2 * e];
      }
#pragma unroll
    for (int e = 0; e < 8; ++e)
#pragma unroll
      for (int q = 0; q < NT; ++q) u[q] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[q][e], b[q][e], u[q], 0, 0, 0);
  }
  // all reads before the first write (entries above the diagonal of a
  // diagonal tile are written back unchanged; no other wave touches the tile)
  float sv[NT][16];
#pragma unroll
  for (int q = 0; q < NT; ++q)
#pragma unroll
    for (int r = 0; r < 16; ++r) sv[q][r] = sm.S[ti[q] * 32 + 8 * (r >> 2) + 4 * lk + (r & 3)][tj[q] * 32 + li];
#pragma unroll
  for (int q = 0; q < NT; ++q)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int i = ti[q] * 32 + 8 * (r >> 2) + 4 * lk + (r & 3), j = tj[q] * 32 + li;
      sm.S[i][j] = j <= i ? sv[q][r] - u[q][r] : sv[q][r];
    }
}

// Thread tid's share of a 128 x 128 block moved as float4: rows
// row0 + 8 t (t < 16), columns col..col+3.  The 32 lanes of a half wave
// cover 4 rows x 32 columns, so that with the odd LDS pitch their entries
// fall in distinct banks, and each row's 128 bytes form one global segment.
__device__ __forceinline__ void quad4_map(int tid, int& row0, int& col) {
  row0 = ((tid >> 7) << 2) + ((tid >> 3) & 3);
  col = 32 * ((tid >> 5) & 3) + 4 * (tid & 7);
}

// 64 x 64 block of an LDS operand (from row r0, column c0) to dst (leading
// dimension ld) as float4 moves; mode 0: as is, 1: lower triangle (zeros
// above the block's diagonal), 2: zeros.  Thread t of STRIDE; the 32 lanes of
// a half wave cover 4 rows x 32 columns (distinct banks, 128-byte segments).
template <int STRIDE>
__device__ __forceinline__ void store64(const float (*src)[SP], int r0, int c0, float* dst, int64_t ld,
                                        int mode, int t) {
#pragma unroll
  for (int k = 0; k < (1024 + STRIDE - 1) / STRIDE; ++k) {
    const int f = t + k * STRIDE;
    if (f < 1024) {
      const int r = 4 * (f >> 6) + ((f >> 3) & 3), c = 32 * ((f >> 5) & 1) + 4 * (f & 7);
      float e[4];
#pragma unroll
      for (int q = 0; q < 4; ++q)
        e[q] = (mode == 2 || (mode == 1 && c + q > r)) ? 0.0f : src[r0 + r][c0 + c + q];
      *reinterpret_cast<float4*>(dst + (int64_t)r * ld + c) = make_float4(e[0], e[1], e[2], e[3]);
    }
  }
}

// Cholesky + inverse of one diagonal block of size b <= 128 by one
// workgroup: reads the lower triangle of Lblk (ld), writes the block of L^-1
// (lower, zeros above) to Liblk and, when Lout is not null, L itself over the
// block; sum(log diag L) into logdet[slot]; on a non-positive or NaN pivot
// sets st = {iteration, side, pivot_base + j} and returns (the outputs then
// hold partial results, at most the first half's).  Lpre (optional): the
// block row of the last panel to the left (b rows x 128, leading dimension
// ld), whose update A -= Lpre Lpre^T is applied to the block first.
__device__ __forceinline__ void leaf_body(LeafLDS& sm, const float* Lblk, float* __restrict__ Liblk,
                                          int64_t ld, int b, int64_t pivot_base, double* logdet,
                                          int slot, int iteration, int side, int* st, float* Lout,
                                          const float* Lpre) {
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int j = tid & (NB - 1), i0 = tid >> 7;
  bool pre_loaded = false;  // Lpre already staged in X
  if (b == NB && (ld & 3) == 0 && (reinterpret_cast<uintptr_t>(Lblk) & 15) == 0) {
    // full block, float4 moves (quad4_map); all sixteen loads (thirty-two
    // with the panel's block row) are in flight before the first is used
    int r, c;
    quad4_map(tid, r, c);
    const bool pre = Lpre != nullptr && (reinterpret_cast<uintptr_t>(Lpre) & 15) == 0;
    float4 v[NB / 8], u[NB / 8];
#pragma unroll
    for (int t = 0; t < NB / 8; ++t)
      v[t] = *reinterpret_cast<const float4*>(Lblk + (int64_t)(r + 8 * t) * ld + c);
    if (pre) {
#pragma unroll
      for (int t = 0; t < NB / 8; ++t)
        u[t] = *reinterpret_cast<const float4*>(Lpre + (int64_t)(r + 8 * t) * ld + c);
    }
#pragma unroll
    for (int t = 0; t < NB / 8; ++t) {
      const int i = r + 8 * t;
      sm.S[i][c + 0] = c + 0 <= i ? v[t].x : 0.0f;
      sm.S[i][c + 1] = c + 1 <= i ? v[t].y : 0.0f;
      sm.S[i][c + 2] = c + 2 <= i ? v[t].z : 0.0f;
      sm.S[i][c + 3] = c + 3 <= i ? v[t].w : 0.0f;
      if (pre) {
        sm.X[i][c + 0] = u[t].x;
        sm.X[i][c + 1] = u[t].y;
        sm.X[i][c + 2] = u[t].z;
        sm.X[i][c + 3] = u[t].w;
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) sm.X[i][c + e] = 0.0f;
      }
    }
    pre_loaded = pre;
  } else {
    // ragged block (b < 128), padded with the identity: thread (i0, j) moves
    // rows i0, i0 + 2, ... of column j, from clamped (always valid) addresses
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      float v[NB / 4];
#pragma unroll
      for (int t = 0; t < NB / 4; ++t) {
        const int i = i0 + 2 * (half * (NB / 4) + t);
        const float x = Lblk[(int64_t)min(i, b - 1) * ld + min(j, b - 1)];
        v[t] = (i < b && j <= i) ? x : (i == j ? 1.0f : 0.0f);
      }
#pragma unroll
      for (int t = 0; t < NB / 4; ++t) {
        const int i = i0 + 2 * (half * (NB / 4) + t);
        sm.S[i][j] = v[t];
        sm.X[i][j] = 0.0f;
      }
    }
  }
  if (tid == 0) sm.bad = -1;
  __syncthreads();
  if (Lpre != nullptr) {
    // A -= Lpre Lpre^T (Lpre staged in X)
    if (!pre_loaded) {
      load_rows(sm.X, Lpre, ld, 0, 0, b, tid);
      __syncthreads();
    }
    // tile (0, 0) now, the other nine during the first two base blocks.
    // Tile (0, 0) splits k over the four waves (k in [32 w, 32 w + 32) on
    // wave w), whose partial products meet in T and are summed in a fixed
    // order.
    {
      const int li = lane & 31, lk = lane >> 5;
      const float* pa = &sm.X[li][32 * wave + lk];
      float a[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) a[e] = pa[2 * e];
      f32x16 u;
#pragma unroll
      for (int r = 0; r < 16; ++r) u[r] = 0.0f;
#pragma unroll
      for (int e = 0; e < 16; ++e) u = __builtin_amdgcn_mfma_f32_32x32x2f32(a[e], a[e], u, 0, 0, 0);
#pragma unroll
      for (int r = 0; r < 16; ++r)
        sm.T[32 * (wave >> 1) + 8 * (r >> 2) + 4 * lk + (r & 3)][32 * (wave & 1) + li] = u[r];
    }
    __syncthreads();
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int f = tid + 256 * e, i = f >> 5, jj = f & 31;
      if (jj <= i) sm.S[i][jj] -= (sm.T[i][jj] + sm.T[i][32 + jj]) + (sm.T[32 + i][jj] + sm.T[32 + i][32 + jj]);
    }
    __syncthreads();
  }
  const bool vec_out = b == NB && (ld & 3) == 0 && (reinterpret_cast<uintptr_t>(Liblk) & 15) == 0 &&
                       (reinterpret_cast<uintptr_t>(Lout) & 15) == 0;
  // While wave 0 factors the first base block of the second half, waves
  // 1..3 store what is final by then: L11, L^-1 11, the zeros above them and
  // L21.  (Without P, X was zeroed when the block was read.)
  auto early = [&](int t) {
    // the block above the diagonal inside X22 is read before it is written:
    // zero X[64:96][96:128] (P no longer needed)
#pragma unroll
    for (int f = t; f < 1024; f += 192) sm.X[64 + (f >> 5)][96 + (f & 31)] = 0.0f;
    if (!vec_out) return;
    store64<192>(sm.X, 0, 0, Liblk, ld, 1, t);
    store64<192>(sm.X, 0, 0, Liblk + 64, ld, 2, t);
    if (Lout != nullptr) {
      store64<192>(sm.S, 0, 0, Lout, ld, 1, t);
      store64<192>(sm.S, 0, 0, Lout + 64, ld, 2, t);
      store64<192>(sm.S, 64, 0, Lout + 64 * ld, ld, 0, t);
    }
  };
  // While it factors the second: the top level's Y = L21 X11 (64 x 64 x 64)
  // into T, the four 32 x 32 tiles on waves 1..3 (1: tiles 0 and 3).
  auto top_y = [&](int) {
    typedef LevelTile<64> LT;
    const int w = (int)threadIdx.x >> 6;
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int tw = q == 0 ? w - 1 : 3;
      if (q == 1 && w != 1) break;
      const LT::Acc y = LT::product(tw, lane, [&](int i, int k) { return sm.S[64 + i][k]; },
                                    [&](int k, int j) { return sm.X[k][j]; });
#pragma unroll
      for (int r = 0; r < LT::NACC; ++r) sm.T[LT::row(tw, r, lane)][LT::col(tw, lane)] = y[r];
    }
  };
  const int bad = cholinv_lds<NB>(sm, 0, wave, lane, Lpre != nullptr ? 1 : 0, NoSide(), early, top_y);
  if (bad >= 0) {
    if (tid == 0) {
      st[1] = side;
      st[2] = (int)(pivot_base + bad);
      __threadfence();
      st[0] = iteration;
    }
    return;
  }
  if (vec_out) {
    // the rest: L22, L^-1 22 and L^-1 21
    store64<256>(sm.X, 64, 64, Liblk + 64 * ld + 64, ld, 1, tid);
    store64<256>(sm.X, 64, 0, Liblk + 64 * ld, ld, 0, tid);
    if (Lout != nullptr) store64<256>(sm.S, 64, 64, Lout + 64 * ld + 64, ld, 1, tid);
  } else if (j < b) {
#pragma unroll 8
    for (int i = i0; i < b; i += 2) Liblk[(int64_t)i * ld + j] = j <= i ? sm.X[i][j] : 0.0f;
    if (Lout != nullptr) {  // the factor itself, over the block it was read from
#pragma unroll 8
      for (int i = i0; i < b; i += 2) Lout[(int64_t)i * ld + j] = j <= i ? sm.S[i][j] : 0.0f;
    }
  }
  // log-determinant share, sum of log L_jj over the block (kept off the
  // pivots' path; ragged blocks are padded with unit pivots)
  if (wave == 0) {
    double ls = log((double)sm.dg[lane]) + log((double)sm.dg[lane + 64]);
#pragma unroll
    for (int w = 32; w >= 1; w >>= 1) ls += __shfl_xor(ls, w, 64);
    if (lane == 0) logdet[slot] = ls;
  }
}

// Trailing-update tile of a right-looking step: the two 128-row blocks of
// the panel (columns ok.., rows i0.. and j0..) in LDS.
struct TrailLDS {
  float a[NB][SP];
  float b[NB][SP];
};
union StepLDS {
  LeafLDS leaf;
  TrailLDS trail;
};

// One step of the blocked factorisation: workgroup 0 factors and inverts
// the diagonal block at d0, after applying to it the update of the panel in
// columns ok..ok+127 (already holding L) when ok >= 0; workgroups
// 1..gridDim.x-1 apply that panel's update A_ij -= L_i,ok L_j,ok^T to every
// other 128 x 128 block of the trailing lower triangle at or below d0 whose
// block column starts before jend (the diagonal block excluded), round robin
// over block columns then rows.
__global__ __launch_bounds__(256) void k_chol_step(float* __restrict__ L, float* __restrict__ Li,
                                                   int64_t dim, int64_t d0, int64_t ok, int64_t jend,
                                                   double* logdet, int iteration, int side, int* st) {
  if (ff_halted(st)) return;
  __shared__ StepLDS sm;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  if (blockIdx.x == 0) {
    const int b = (int)min<int64_t>(NB, dim - d0);
    float* Akk = L + d0 * dim + d0;
    leaf_body(sm.leaf, Akk, Li + d0 * dim + d0, dim, b, d0, logdet, (int)(d0 / NB), iteration, side,
              st, Akk, ok >= 0 ? L + d0 * dim + ok : nullptr);
    return;
  }
  const int64_t R = (dim - d0 + NB - 1) / NB;   // block rows at or below d0
  const int64_t T = (jend - d0 + NB - 1) / NB;  // block columns updated
  // tiles: block column bj < T holds block rows bj..R-1; skip (0, 0)
  const int64_t ntiles = T * R - T * (T - 1) / 2 - 1;
  for (int64_t t = blockIdx.x - 1; t < ntiles; t += gridDim.x - 1) {
    int64_t u = t + 1, bj = 0;
    while (u >= R - bj) {
      u -= R - bj;
      ++bj;
    }
    const int64_t bi = bj + u;
    const int64_t i0 = d0 + bi * NB, j0 = d0 + bj * NB;
    load_rows(sm.trail.a, L, dim, i0, ok, dim, tid);
    if (bi != bj) load_rows(sm.trail.b, L, dim, j0, ok, dim, tid);
    __syncthreads();
    // this lane's 64 entries of the block, read (from clamped addresses)
    // before the product so that their latency overlaps it
    float cv[2][2][16];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int64_t i = min<int64_t>(i0 + quad_row(wave, a, r, lane), dim - 1);
          const int64_t j = min<int64_t>(j0 + quad_col(wave, c, lane), dim - 1);
          cv[a][c][r] = L[i * dim + j];
        }
    f32x16 u4[2][2];
    quad_product(sm.trail.a, bi != bj ? sm.trail.b : sm.trail.a, wave, lane, u4);
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int64_t i = i0 + quad_row(wave, a, r, lane), j = j0 + quad_col(wave, c, lane);
          if (i < dim && j < dim && (bi != bj || j <= i)) L[i * dim + j] = cv[a][c][r] - u4[a][c][r];
        }
    __syncthreads();  // before the next tile's rows overwrite LDS
  }
}

// Panel of the blocked factorisation: L_ik = A_ik L_kk^-T for the rows
// below a diagonal block, in place.  One workgroup per 64 rows holds its rows
// (64 x 128) and the block's inverse (128 x 128, zero above the diagonal) in
// LDS; wave w computes output columns 32 w .. 32 w + 31 (two 32 x 32 tiles).
struct PanelLDS {
  float a[64][SP];
  float x[NB][SP];
};

// Column blocks CA and CB (CB < CA) of row half h of the panel product:
// acc0 over k < 32 (CA + 1), acc1 over k < 32 (CB + 1), with the operands of
// eight k steps read before their products are issued.
template <int CA, int CB>
__device__ __forceinline__ void panel_tiles(const PanelLDS& sm, int h, int li, int lk, f32x16& acc0,
                                            f32x16& acc1) {
  const float* pa = &sm.a[h * 32 + li][lk];
  const float* px = &sm.x[CA * 32 + li][lk];
  const float* py = &sm.x[CB * 32 + li][lk];
#pragma unroll
  for (int r = 0; r < 16; ++r) acc0[r] = acc1[r] = 0.0f;
#pragma unroll
  for (int k = 0; k < 32 * (CA + 1); k += 16) {
    float av[8], xv[8], yv[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      av[e] = pa[k + 2 * e];
      xv[e] = px[k + 2 * e];
      if (k < 32 * (CB + 1)) yv[e] = py[k + 2 * e];
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      acc0 = __builtin_amdgcn_mfma_f32_32x32x2f32(av[e], xv[e], acc0, 0, 0, 0);
      if (k < 32 * (CB + 1)) acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(av[e], yv[e], acc1, 0, 0, 0);
    }
  }
}

__global__ __launch_bounds__(256) void k_panel_solve(float* __restrict__ P, const float* __restrict__ Xkk,
                                                     int64_t ld, int64_t rows, const int* st) {
  if (ff_halted(st)) return;
  __shared__ PanelLDS sm;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int64_t r0 = (int64_t)blockIdx.x * 64;
  const bool vec = (ld & 3) == 0 && (reinterpret_cast<uintptr_t>(P) & 15) == 0 &&
                   (reinterpret_cast<uintptr_t>(Xkk) & 15) == 0;
  if (vec) {
    const int q = tid & 31, r = tid >> 5;
    float4 va[8], vx[16];
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const int64_t i = r0 + r + 8 * t;
      va[t] = i < rows ? *reinterpret_cast<const float4*>(P + i * ld + 4 * q) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int t = 0; t < 16; ++t) vx[t] = *reinterpret_cast<const float4*>(Xkk + (int64_t)(r + 8 * t) * ld + 4 * q);
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      float* d = &sm.a[r + 8 * t][4 * q];
      d[0] = va[t].x; d[1] = va[t].y; d[2] = va[t].z; d[3] = va[t].w;
    }
#pragma unroll
    for (int t = 0; t < 16; ++t) {
      float* d = &sm.x[r + 8 * t][4 * q];
      d[0] = vx[t].x; d[1] = vx[t].y; d[2] = vx[t].z; d[3] = vx[t].w;
    }
  } else {
    const int j = tid & (NB - 1), i0 = tid >> 7;
    for (int i = i0; i < 64; i += 2) sm.a[i][j] = r0 + i < rows ? P[(r0 + i) * ld + j] : 0.0f;
    for (int i = i0; i < NB; i += 2) sm.x[i][j] = Xkk[(int64_t)i * ld + j];
  }
  __syncthreads();
  // out(i, j) = sum_k a[i][k] x[j][k], k <= j (x lower triangular): column
  // block c needs k < 32 (c + 1).  Wave w takes row half w % 2 and column
  // blocks 3 and 0 (waves 0, 1) or 2 and 1 (waves 2, 3): 160 k each.
  const int li = lane & 31, lk = lane >> 5;
  const int h = wave & 1, cA = wave < 2 ? 3 : 2, cB = 3 - cA;
  f32x16 acc0, acc1;
  if (wave < 2) panel_tiles<3, 0>(sm, h, li, lk, acc0, acc1);
  else panel_tiles<2, 1>(sm, h, li, lk, acc0, acc1);
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int64_t g = r0 + h * 32 + 8 * (r >> 2) + 4 * lk + (r & 3);
    if (g < rows) {
      P[g * ld + cA * 32 + li] = acc0[r];
      P[g * ld + cB * 32 + li] = acc1[r];
    }
  }
}

}  // namespace

hipError_t launch_chol_step(float* L, float* Li, int64_t dim, int64_t d0, int64_t ok, int64_t jend,
                            double* logdet, int iteration, int side, int* st, hipStream_t s) {
  if (dim < 1 || d0 < 0 || d0 >= dim || d0 % kLeaf != 0) return hipErrorInvalidValue;
  if (ok >= 0 && (ok % kLeaf != 0 || ok + kLeaf > d0 || jend <= d0 || jend > dim))
    return hipErrorInvalidValue;
  int64_t ntiles = 0;
  if (ok >= 0) {
    const int64_t R = (dim - d0 + kLeaf - 1) / kLeaf, T = (jend - d0 + kLeaf - 1) / kLeaf;
    ntiles = T * R - T * (T - 1) / 2 - 1;
  }
  const int64_t grid = 1 + std::min<int64_t>(ntiles, kStepWorkers);
  hipLaunchKernelGGL(k_chol_step, dim3((uint32_t)grid), dim3(256), 0, s, L, Li, dim, d0,
                     ok >= 0 ? ok : (int64_t)-1, jend, logdet, iteration, side, st);
  return hipGetLastError();
}

hipError_t launch_panel_solve(float* P, const float* Xkk, int64_t ld, int64_t rows, const int* st,
                              hipStream_t s) {
  if (rows < 0 || ld < kLeaf) return hipErrorInvalidValue;
  if (rows == 0) return hipSuccess;
  const int64_t grid = (rows + 63) / 64;
  if (grid > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_panel_solve, dim3((uint32_t)grid), dim3(256), 0, s, P, Xkk, ld, rows, st);
  return hipGetLastError();
}

}  // namespace ff
