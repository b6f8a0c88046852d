// bf16 matrix-core kernels of the flip-flop iteration (gfx950).
//
// Both hot products of an iteration are "NT" contractions with both operands
// contiguous along k, computed as 256 x 256 output tiles by one workgroup of
// four waves (each wave a 128 x 128 quadrant = 4 x 4 tiles of the
// v_mfma_f32_32x32x16_bf16 instruction, fp32 accumulation):
//
//  * whitening  C = X Y^T with Y = L^-1 lower triangular (Section 5: the
//    factor inverse enters every update as G A^-1 G^T = (G L^-T)(G L^-T)^T),
//    k restricted to the non-zero triangle of Y;
//  * symmetric product X X^T over the stacked whitened samples (the sum over
//    i of the Section 5 updates), upper tiles only, split over k into
//    deterministic partial sums that a second kernel adds in fixed order.
//
// Operands are staged through LDS in 64-wide k slices, double buffered, with
// an XOR swizzle of the 16-byte chunks of each 128-byte row so that the
// matrix-core fragment reads of 32 consecutive rows hit distinct banks.
#include "ff_common.hpp"
#include "ff_kernels.hpp"

namespace ff {
namespace {

constexpr int TM = 256;       // tile rows (and columns)
constexpr int TK = 64;        // k per LDS stage
constexpr int CH = TK / 8;    // 16-byte chunks per tile row
constexpr int NTHR = 256;     // four waves
constexpr int TILE_FLOATS = TM * TM;

typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;

struct __align__(16) Stage {
  u32x4 a[TM * CH];
  u32x4 b[TM * CH];
};

__device__ __forceinline__ int swz(int row, int chunk) { return row * CH + (chunk ^ (row & 7)); }

// Per-thread share of one operand slice: chunk (tid & 7) of rows
// (tid >> 3) + 32 q, q = 0..7.
struct Loader {
  uint32_t off[8];
  __device__ __forceinline__ void init(int tid, uint32_t ld) {
#pragma unroll
    for (int q = 0; q < 8; ++q) off[q] = (uint32_t)((tid >> 3) + 32 * q) * ld + (uint32_t)(tid & 7) * 8u;
  }
  __device__ __forceinline__ void load(const bf16_t* base, u32x4 (&r)[8]) const {
#pragma unroll
    for (int q = 0; q < 8; ++q) r[q] = *reinterpret_cast<const u32x4*>(base + off[q]);
  }
};

__device__ __forceinline__ void stage_store(u32x4* dst, int tid, const u32x4 (&r)[8]) {
#pragma unroll
  for (int q = 0; q < 8; ++q) dst[swz((tid >> 3) + 32 * q, tid & 7)] = r[q];
}

__device__ __forceinline__ void stage_compute(const Stage& sm, int wave, int lane,
                                              f32x16 (&acc)[4][4]) {
  const int wm = wave >> 1, wn = wave & 1;
  const int lrow = lane & 31, kh = lane >> 5;
#pragma unroll
  for (int kk = 0; kk < TK / 16; ++kk) {
    bf16x8 fa[4], fb[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      fa[t] = __builtin_bit_cast(bf16x8, sm.a[swz(wm * 128 + t * 32 + lrow, kk * 2 + kh)]);
      fb[t] = __builtin_bit_cast(bf16x8, sm.b[swz(wn * 128 + t * 32 + lrow, kk * 2 + kh)]);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
  }
}

// acc += sum over k slices [kt0, kt1) of Aslice(kt) Bslice(kt)^T, where
// addr(kt, pa, pb) yields the slice base pointers (row 0, k = 64 kt).
template <class Addr>
__device__ __forceinline__ void mainloop(Stage* sm, int kt0, int kt1, uint32_t lda, uint32_t ldb,
                                         const Addr& addr, f32x16 (&acc)[4][4]) {
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  if (kt0 >= kt1) return;
  Loader la, lb;
  la.init(tid, lda);
  lb.init(tid, ldb);
  u32x4 ra[8], rb[8];
  const bf16_t *pa, *pb;
  addr(kt0, pa, pb);
  la.load(pa, ra);
  lb.load(pb, rb);
  stage_store(sm[0].a, tid, ra);
  stage_store(sm[0].b, tid, rb);
  __syncthreads();
  int cur = 0;
  for (int kt = kt0; kt + 1 < kt1; ++kt) {
    addr(kt + 1, pa, pb);
    la.load(pa, ra);
    lb.load(pb, rb);
    stage_compute(sm[cur], wave, lane, acc);
    stage_store(sm[cur ^ 1].a, tid, ra);
    stage_store(sm[cur ^ 1].b, tid, rb);
    __syncthreads();
    cur ^= 1;
  }
  stage_compute(sm[cur], wave, lane, acc);
  __syncthreads();
}

__device__ __forceinline__ void zero_acc(f32x16 (&acc)[4][4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;
}

__global__ __launch_bounds__(NTHR, 1) void k_whiten_bf16(const bf16_t* __restrict__ X,
                                                         const bf16_t* __restrict__ Y,
                                                         const bf16_t* __restrict__ Y2,
                                                         bf16_t* __restrict__ C, uint32_t Kp,
                                                         const int* st) {
  if (ff_halted(st)) return;
  __shared__ Stage sm[2];
  const uint32_t ncol = Kp / TM;
  const uint32_t t = xcd_remap(blockIdx.x, gridDim.x);
  const uint32_t rb = t / ncol;
  const uint32_t cj = ncol - 1 - t % ncol;  // heaviest column tiles first
  const int kt1 = (int)((cj + 1) * (TM / TK));
  const bf16_t* xa = X + (size_t)rb * TM * Kp;
  f32x16 acc[4][4];
  zero_acc(acc);
  {
    const bf16_t* yb = Y + (size_t)cj * TM * Kp;
    auto addr = [&](int kt, const bf16_t*& pa, const bf16_t*& pb) {
      pa = xa + kt * TK;
      pb = yb + kt * TK;
    };
    mainloop(sm, 0, kt1, Kp, Kp, addr, acc);
  }
  if (Y2 != nullptr) {
    const bf16_t* yb = Y2 + (size_t)cj * TM * Kp;
    auto addr = [&](int kt, const bf16_t*& pa, const bf16_t*& pb) {
      pa = xa + kt * TK;
      pb = yb + kt * TK;
    };
    mainloop(sm, 0, kt1, Kp, Kp, addr, acc);
  }
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int wm = wave >> 1, wn = wave & 1;
  bf16_t* cb = C + (size_t)rb * TM * Kp + (size_t)cj * TM;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = wm * 128 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        const int col = wn * 128 + j * 32 + (lane & 31);
        cb[(size_t)row * Kp + col] = f32_to_bf16(acc[i][j][r]);
      }
}

// Upper-triangle tile index -> (ti, tj), ti <= tj, row-major over the triangle.
__device__ __forceinline__ void upper_tile(uint32_t idx, uint32_t T, uint32_t& ti, uint32_t& tj) {
  uint32_t i = 0, rowlen = T;
  while (idx >= rowlen) {
    idx -= rowlen;
    ++i;
    --rowlen;
  }
  ti = i;
  tj = i + idx;
}

__global__ __launch_bounds__(NTHR, 1) void k_syrk_bf16(const bf16_t* __restrict__ X, uint32_t ld,
                                                       uint64_t seg_stride, uint32_t nseg,
                                                       uint32_t T, uint32_t ntiles, uint32_t splits,
                                                       float* __restrict__ P, const int* st) {
  if (ff_halted(st)) return;
  __shared__ Stage sm[2];
  const uint32_t t = xcd_remap(blockIdx.x, gridDim.x);
  const uint32_t z = t / ntiles, tile = t % ntiles;
  uint32_t ti, tj;
  upper_tile(tile, T, ti, tj);
  const uint32_t kps = ld / TK;  // k slices per segment
  const uint64_t ktot = (uint64_t)kps * nseg;
  const int kt0 = (int)(ktot * z / splits), kt1 = (int)(ktot * (z + 1) / splits);
  const bf16_t* xa = X + (size_t)ti * TM * ld;
  const bf16_t* xb = X + (size_t)tj * TM * ld;
  f32x16 acc[4][4];
  zero_acc(acc);
  auto addr = [&](int kt, const bf16_t*& pa, const bf16_t*& pb) {
    const uint32_t s = (uint32_t)kt / kps, o = (uint32_t)kt % kps;
    const size_t base = (size_t)s * seg_stride + (size_t)o * TK;
    pa = xa + base;
    pb = xb + base;
  };
  mainloop(sm, kt0, kt1, ld, ld, addr, acc);
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  float* pt = P + ((size_t)z * ntiles + tile) * TILE_FLOATS;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      f32x4* dst = reinterpret_cast<f32x4*>(pt + ((size_t)((wave * 16 + i * 4 + j) * 64 + lane)) * 16);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        f32x4 v = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
        dst[q] = v;
      }
    }
}

// One thread per 4 consecutive fragment floats (4 rows, one column) of a tile.
__global__ __launch_bounds__(256) void k_reduce_frag(const float* __restrict__ P, uint32_t splits,
                                                     uint32_t ntiles, uint32_t T, float* __restrict__ F,
                                                     uint32_t dim, float scale, const int* st) {
  if (ff_halted(st)) return;
  const uint32_t tile = blockIdx.x;
  const uint32_t f = blockIdx.y * 256 + threadIdx.x;  // float4 index in the tile
  uint32_t ti, tj;
  upper_tile(tile, T, ti, tj);
  f32x4 s = {0.f, 0.f, 0.f, 0.f};
  for (uint32_t z = 0; z < splits; ++z) {
    const f32x4 v = reinterpret_cast<const f32x4*>(P + ((size_t)z * ntiles + tile) * TILE_FLOATS)[f];
    s += v;
  }
  const uint32_t q = f & 3, lane = (f >> 2) & 63, rest = f >> 8;
  const uint32_t wave = rest >> 4, mt = (rest >> 2) & 3, nt = rest & 3;
  const uint32_t i0 = ti * TM + (wave >> 1) * 128 + mt * 32 + 8 * q + 4 * (lane >> 5);
  const uint32_t j = tj * TM + (wave & 1) * 128 + nt * 32 + (lane & 31);
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint32_t i = i0 + e;
    if (i < dim && j < dim && (ti < tj || i <= j)) {
      const float v = s[e] * scale;
      F[(size_t)i * dim + j] = v;
      F[(size_t)j * dim + i] = v;
    }
  }
}

}  // namespace

hipError_t launch_whiten_bf16(const bf16_t* X, const bf16_t* Y, const bf16_t* Y2, bf16_t* C,
                              int64_t rows, int64_t Kp, const int* st, hipStream_t s) {
  if (rows <= 0 || Kp <= 0 || rows % TM || Kp % TM || Kp > (1 << 20)) return hipErrorInvalidValue;
  const int64_t tiles = (rows / TM) * (Kp / TM);
  if (tiles > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_whiten_bf16, dim3((uint32_t)tiles), dim3(NTHR), 0, s, X, Y, Y2, C,
                     (uint32_t)Kp, st);
  return hipGetLastError();
}

hipError_t launch_syrk_bf16(const bf16_t* X, int64_t dim_p, int64_t ld, int64_t seg_stride,
                            int64_t nseg, int splits, float* P, const int* st, hipStream_t s) {
  if (dim_p <= 0 || dim_p % TM || ld <= 0 || ld % TK || nseg <= 0 || splits <= 0)
    return hipErrorInvalidValue;
  const int64_t T = dim_p / TM, ntiles = T * (T + 1) / 2;
  if ((int64_t)splits > (ld / TK) * nseg) return hipErrorInvalidValue;
  if (ntiles * splits > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_syrk_bf16, dim3((uint32_t)(ntiles * splits)), dim3(NTHR), 0, s, X,
                     (uint32_t)ld, (uint64_t)seg_stride, (uint32_t)nseg, (uint32_t)T,
                     (uint32_t)ntiles, (uint32_t)splits, P, st);
  return hipGetLastError();
}

hipError_t launch_reduce_frag(const float* P, int splits, int64_t dim_p, float* F, int64_t dim,
                              double scale, const int* st, hipStream_t s) {
  if (dim_p <= 0 || dim_p % TM || dim > dim_p || splits <= 0) return hipErrorInvalidValue;
  const int64_t T = dim_p / TM, ntiles = T * (T + 1) / 2;
  hipLaunchKernelGGL(k_reduce_frag, dim3((uint32_t)ntiles, TILE_FLOATS / 4 / 256), dim3(256), 0, s,
                     P, (uint32_t)splits, (uint32_t)ntiles, (uint32_t)T, F, (uint32_t)dim,
                     (float)scale, st);
  return hipGetLastError();
}

}  // namespace ff
