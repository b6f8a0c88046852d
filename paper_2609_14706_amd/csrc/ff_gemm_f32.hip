// General fp32 product on the fp32 matrix cores (v_mfma_f32_32x32x2_f32).
//
// Used wherever the iteration needs fp32 products: the blocked Cholesky and
// triangular inverse of the factors, the whole fp32 sample path (whitening
// and symmetric product), and the Kronecker application.  128 x 128 output
// tiles, four waves of 64 x 64 (2 x 2 matrix-core tiles), 32-wide k slices
// staged through double-buffered LDS; when fewer than 256 such tiles would be
// launched, 64 x 64 tiles (one 32 x 32 matrix-core tile per wave) with 64-wide
// k slices.  Any shape and either operand
// transpose; k ranges can be clipped to the non-zero triangle of a
// triangular operand, k can run over segments (the stacked samples), and k
// can be split over the grid into partial outputs.  When every operand is
// 16-byte aligned with leading dimensions divisible by 4, global loads are
// 16-byte vectors (edge vectors fall back to element loads).
#include "ff_common.hpp"
#include "ff_kernels.hpp"

namespace ff {
namespace {

constexpr int LDPMAX = 128 + 4;
// k range per workgroup above which products use two-level accumulation
constexpr int64_t kDeepK = 16384;

// k per LDS slice: 32 for 128 x 128 tiles, 64 for 64 x 64 tiles (the small
// products of the factorisation are latency bound: fewer, larger slices).
template <int BT>
constexpr int slice_k() { return BT == 128 ? 32 : 64; }

// Offset of k in a k axis made of segments of kseg, seg apart (kseg == 0:
// one contiguous axis, no division).
__device__ __forceinline__ int64_t seg_off(int64_t k, int64_t kseg, int64_t seg) {
  return kseg ? (k / kseg) * seg + (k % kseg) : k;
}

// One operand slice: 128 "outer" indices (rows of op(A) or columns of op(B))
// x 16 k.  KMAJ: the operand is contiguous along k (element (o, k) at
// P[o * ld + koff(k)]); otherwise contiguous along o (at P[koff(k) * ld + o]).
// Each thread fetches NQ 4-element groups; slice[k][o] is written to LDS.
// FAST: the whole slice is in bounds and 16-byte vectors can be used.
template <int BT, bool KMAJ, bool FAST>
struct SliceLoader {
  static constexpr int BK = slice_k<BT>();
  static constexpr int NQ = BT * BK / 4 / 256;  // 4-element groups per thread
  static constexpr int OQ = BT / 4;             // 4-element groups per k row (non-k-major)
  f32x4 v[NQ];
  __device__ __forceinline__ void load(const float* P, int64_t ld, int64_t o0, int64_t olim,
                                       int64_t k0, int64_t khi, int64_t kseg, int64_t seg,
                                       int tid) {
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int idx = tid + 256 * q;
      const int o = KMAJ ? idx / (BK / 4) : (idx % OQ) * 4;
      const int k = KMAJ ? (idx % (BK / 4)) * 4 : idx / OQ;
      const int64_t go = o0 + o, gk = k0 + k;
      if (FAST) {
        const int64_t ko = seg_off(gk, kseg, seg);
        v[q] = KMAJ ? *reinterpret_cast<const f32x4*>(P + go * ld + ko)
                    : *reinterpret_cast<const f32x4*>(P + ko * ld + go);
      } else {
        f32x4 r = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int64_t eo = KMAJ ? go : go + e, ek = KMAJ ? gk + e : gk;
          if (eo < olim && ek < khi) {
            const int64_t ko = seg_off(ek, kseg, seg);
            r[e] = KMAJ ? P[eo * ld + ko] : P[ko * ld + eo];
          }
        }
        v[q] = r;
      }
    }
  }
  __device__ __forceinline__ void store(float (*S)[BT + 4], int tid) const {
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int idx = tid + 256 * q;
      if (KMAJ) {
        const int o = idx / (BK / 4), k = (idx % (BK / 4)) * 4;
#pragma unroll
        for (int e = 0; e < 4; ++e) S[k + e][o] = v[q][e];
      } else {
        const int k = idx / OQ, o = (idx % OQ) * 4;
        *reinterpret_cast<f32x4*>(&S[k][o]) = v[q];
      }
    }
  }
};

template <int BT>
struct TileLDS {
  float a[2][slice_k<BT>()][BT + 4];
  float b[2][slice_k<BT>()][BT + 4];
};

// acc += op(A)[i0.., klo..khi) op(B)[klo..khi), j0..) for one BT x BT tile
// (each wave a (BT/2) x (BT/2) quadrant of MT x MT 32 x 32 matrix-core tiles).
// DEEP: two-level accumulation (see below), for long k ranges only: its
// second set of accumulators halves the waves a CU can hold.
template <int BT, bool AK, bool BKM, bool FAST, bool DEEP>
__device__ __forceinline__ void tile_product(const GemmF32& p, const float* A, const float* B,
                                             int64_t i0, int64_t j0, int64_t klo, int64_t khi,
                                             TileLDS<BT>& sm, f32x16 (&acc)[BT / 64][BT / 64]) {
  constexpr int MT = BT / 64, BK = slice_k<BT>();
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int wm = wave >> 1, wn = wave & 1;
  SliceLoader<BT, AK, FAST> la;
  SliceLoader<BT, BKM, FAST> lb;
  la.load(A, p.lda, i0, p.M, klo, khi, p.kseg, p.segA, tid);
  lb.load(B, p.ldb, j0, p.N, klo, khi, p.kseg, p.segB, tid);
  la.store(sm.a[0], tid);
  lb.store(sm.b[0], tid);
  __syncthreads();
  // Two-level accumulation: the products of up to CHUNK slices go into a
  // fresh accumulator that is then added to acc.  Long k ranges (the
  // stacked samples, hundreds of thousands deep) thus round each output
  // element about CHUNK * BK / 2 + K / (CHUNK * BK) times instead of K / 2.
  constexpr int CHUNK = 8;
  f32x16 loc[MT][MT];
#pragma unroll
  for (int a = 0; a < MT; ++a)
#pragma unroll
    for (int b = 0; b < MT; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) loc[a][b][r] = 0.0f;
  int cnt = 0;
  int cur = 0;
  for (int64_t k0 = klo; k0 < khi; k0 += BK) {
    const bool more = k0 + BK < khi;
    if (more) {
      la.load(A, p.lda, i0, p.M, k0 + BK, khi, p.kseg, p.segA, tid);
      lb.load(B, p.ldb, j0, p.N, k0 + BK, khi, p.kseg, p.segB, tid);
    }
    __builtin_amdgcn_sched_barrier(0);
    // operands of k-step s + 1 are read while the products of step s run
    float fa[2][MT], fb[2][MT];
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      fa[0][t] = sm.a[cur][lane >> 5][wm * (BT / 2) + t * 32 + (lane & 31)];
      fb[0][t] = sm.b[cur][lane >> 5][wn * (BT / 2) + t * 32 + (lane & 31)];
    }
#pragma unroll
    for (int s = 0; s < BK / 2; ++s) {
      if (s + 1 < BK / 2) {
        const int kr = 2 * (s + 1) + (lane >> 5);
#pragma unroll
        for (int t = 0; t < MT; ++t) {
          fa[(s + 1) & 1][t] = sm.a[cur][kr][wm * (BT / 2) + t * 32 + (lane & 31)];
          fb[(s + 1) & 1][t] = sm.b[cur][kr][wn * (BT / 2) + t * 32 + (lane & 31)];
        }
      }
      __builtin_amdgcn_sched_barrier(0);  // keep the reads ahead of the products
#pragma unroll
      for (int a = 0; a < MT; ++a)
#pragma unroll
        for (int b = 0; b < MT; ++b) {
          if constexpr (DEEP)
            loc[a][b] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[s & 1][a], fb[s & 1][b], loc[a][b], 0, 0, 0);
          else
            acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[s & 1][a], fb[s & 1][b], acc[a][b], 0, 0, 0);
        }
    }
    if (DEEP && (++cnt == CHUNK || !more)) {
#pragma unroll
      for (int a = 0; a < MT; ++a)
#pragma unroll
        for (int b = 0; b < MT; ++b) {
          acc[a][b] += loc[a][b];
#pragma unroll
          for (int r = 0; r < 16; ++r) loc[a][b][r] = 0.0f;
        }
      cnt = 0;
    }
    __builtin_amdgcn_sched_barrier(0);
    if (more) {
      la.store(sm.a[cur ^ 1], tid);
      lb.store(sm.b[cur ^ 1], tid);
    }
    __syncthreads();
    cur ^= 1;
  }
}

template <int BT, int TA, int TBT, bool VEC, bool DEEP>
__global__ __launch_bounds__(256) void k_gemm_f32(GemmF32 p) {
  constexpr int MT = BT / 64, BK = slice_k<BT>();
  if (ff_halted(p.st)) return;
  // With a triangular operand the k range, hence the work, of a tile grows
  // along one tile index: walk the tiles with that index slowest and from the
  // long end, so that the longest workgroups start first.
  int64_t bx = blockIdx.x, by = blockIdx.y;
  if (p.flags & (kKHiRow | kKLoRow)) {
    const int64_t lin = bx + (int64_t)gridDim.x * by;
    bx = lin / gridDim.y;
    by = lin % gridDim.y;
    if (p.flags & kKHiRow) bx = gridDim.x - 1 - bx;
  } else if (p.flags & (kKHiCol | kKLoCol)) {
    if (p.flags & kKHiCol) by = gridDim.y - 1 - by;
  }
  const int64_t i0 = bx * BT, j0 = by * BT;
  if ((p.flags & kCLower) && j0 > i0 + BT - 1) return;
  const float* A = p.A;
  const float* B = p.B;
  float* C = p.C;
  int64_t klo = 0, khi = p.K;
  if (p.flags & kKHiRow) khi = min(khi, i0 + BT);
  if (p.flags & kKLoRow) klo = max(klo, i0);
  if (p.flags & kKHiCol) khi = min(khi, j0 + BT);
  if (p.flags & kKLoCol) klo = max(klo, j0);
  if (p.ksplit > 1) {
    const int64_t span = khi > klo ? khi - klo : 0;
    const int64_t chunk = ((span + p.ksplit - 1) / p.ksplit + BK - 1) / BK * BK;
    klo = klo + (int64_t)blockIdx.z * chunk;
    khi = min(khi, klo + chunk);
    C += (int64_t)blockIdx.z * p.sC;
  } else {
    A += (int64_t)blockIdx.z * p.sA;
    B += (int64_t)blockIdx.z * p.sB;
    C += (int64_t)blockIdx.z * p.sC;
  }
  __shared__ __align__(16) TileLDS<BT> sm;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  f32x16 acc[MT][MT];
#pragma unroll
  for (int a = 0; a < MT; ++a)
#pragma unroll
    for (int b = 0; b < MT; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.0f;
  if (klo < khi) {
    const bool fast = VEC && i0 + BT <= p.M && j0 + BT <= p.N && (khi - klo) % BK == 0;
    if (fast) tile_product<BT, TA == 0, TBT != 0, VEC, DEEP>(p, A, B, i0, j0, klo, khi, sm, acc);
    else tile_product<BT, TA == 0, TBT != 0, false, DEEP>(p, A, B, i0, j0, klo, khi, sm, acc);
  }
  const bool lower = (p.flags & kCLower) != 0;
  const bool use_beta = p.ksplit <= 1 && p.beta != 0.0f;
#pragma unroll
  for (int a = 0; a < MT; ++a)
#pragma unroll
    for (int b = 0; b < MT; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t i = i0 + wm * (BT / 2) + a * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        const int64_t j = j0 + wn * (BT / 2) + b * 32 + (lane & 31);
        if (i < p.M && j < p.N && (!lower || i >= j)) {
          float v = p.alpha * acc[a][b][r];
          if (use_beta) v += p.beta * C[i * p.ldc + j];
          C[i * p.ldc + j] = v;
        }
      }
}

__global__ __launch_bounds__(256) void k_reduce_rowmajor(const float* __restrict__ P, int splits,
                                                         int64_t dim_p, float* __restrict__ F,
                                                         int64_t dim, float scale, const int* st) {
  if (ff_halted(st)) return;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= dim * dim) return;
  const int64_t i = idx / dim, j = idx % dim;
  if (j > i) return;
  float s = 0.0f;
  for (int z = 0; z < splits; ++z) s += P[(int64_t)z * dim_p * dim_p + i * dim_p + j];
  s *= scale;
  F[i * dim + j] = s;
  F[j * dim + i] = s;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

}  // namespace

template <int BT>
hipError_t launch_tiles(const GemmF32& p, int batch, bool vec, hipStream_t s) {
  const int64_t gx = (p.M + BT - 1) / BT, gy = (p.N + BT - 1) / BT;
  const int gz = p.ksplit > 1 ? p.ksplit : batch;
  if (gx > 0x7fffffff || gy > 65535 || gz > 65535) return hipErrorInvalidValue;
  const dim3 grid((uint32_t)gx, (uint32_t)gy, (uint32_t)gz);
  // two-level accumulation when a workgroup's k range is long (the stacked samples)
  const int64_t kwg = p.ksplit > 1 ? (p.K + p.ksplit - 1) / p.ksplit : p.K;
  const bool deep = kwg > kDeepK;
  const int sel = (p.transA ? 1 : 0) | (p.transB ? 2 : 0) | (vec ? 4 : 0) | (deep ? 8 : 0);
  switch (sel) {
#define FF_GEMM_CASE(c, ta, tb, v, dp) \
    case c: hipLaunchKernelGGL((k_gemm_f32<BT, ta, tb, v, dp>), grid, dim3(256), 0, s, p); break;
    FF_GEMM_CASE(0, 0, 0, false, false)
    FF_GEMM_CASE(1, 1, 0, false, false)
    FF_GEMM_CASE(2, 0, 1, false, false)
    FF_GEMM_CASE(3, 1, 1, false, false)
    FF_GEMM_CASE(4, 0, 0, true, false)
    FF_GEMM_CASE(5, 1, 0, true, false)
    FF_GEMM_CASE(6, 0, 1, true, false)
    FF_GEMM_CASE(7, 1, 1, true, false)
    FF_GEMM_CASE(8, 0, 0, false, true)
    FF_GEMM_CASE(9, 1, 0, false, true)
    FF_GEMM_CASE(10, 0, 1, false, true)
    FF_GEMM_CASE(11, 1, 1, false, true)
    FF_GEMM_CASE(12, 0, 0, true, true)
    FF_GEMM_CASE(13, 1, 0, true, true)
    FF_GEMM_CASE(14, 0, 1, true, true)
    default: hipLaunchKernelGGL((k_gemm_f32<BT, 1, 1, true, true>), grid, dim3(256), 0, s, p); break;
#undef FF_GEMM_CASE
  }
  return hipGetLastError();
}

hipError_t launch_gemm_f32(const GemmF32& p, int batch, hipStream_t s) {
  if (p.M < 0 || p.N < 0 || p.K < 0 || batch < 1 || p.kseg < 1) return hipErrorInvalidValue;
  if (p.ksplit > 1 && batch != 1) return hipErrorInvalidValue;
  if (p.M == 0 || p.N == 0) return hipSuccess;
  const bool segmented = p.kseg < p.K;
  const bool vec = aligned16(p.A) && aligned16(p.B) && p.lda % 4 == 0 && p.ldb % 4 == 0 &&
                   (batch == 1 || (p.sA % 4 == 0 && p.sB % 4 == 0)) &&
                   (!segmented || (p.kseg % 4 == 0 && p.segA % 4 == 0 && p.segB % 4 == 0));
  // 128 x 128 tiles when they fill the GPU, 64 x 64 (four times the workgroups) otherwise.
  const int64_t big_tiles = ((p.M + 127) / 128) * ((p.N + 127) / 128) *
                            (p.ksplit > 1 ? p.ksplit : batch);
  GemmF32 q = p;
  if (!segmented) q.kseg = 0;  // plain k axis: the kernels skip the segment arithmetic
  if (p.tile == 64) return launch_tiles<64>(q, batch, vec, s);
  if (p.tile == 128 || big_tiles >= 256) return launch_tiles<128>(q, batch, vec, s);
  return launch_tiles<64>(q, batch, vec, s);
}

hipError_t launch_reduce_rowmajor(const float* P, int splits, int64_t dim_p, float* F,
                                  int64_t dim, double scale, const int* st, hipStream_t s) {
  if (dim <= 0 || dim > dim_p || splits < 1) return hipErrorInvalidValue;
  const int64_t blocks = (dim * dim + 255) / 256;
  hipLaunchKernelGGL(k_reduce_rowmajor, dim3((uint32_t)blocks), dim3(256), 0, s, P, splits, dim_p,
                     F, dim, (float)scale, st);
  return hipGetLastError();
}

}  // namespace ff
