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
// Operands move global -> LDS with the direct-to-LDS loads of gfx950
// (global_load_lds_dwordx4, no register staging) in 32-wide k slices through
// a 5-slot ring (160 KB), four slices in flight ahead of the matrix cores, which
// covers the memory latency with one workgroup of four waves per CU.  The
// 16-byte chunks of each 64-byte row are XOR-swizzled so that fragment
// reads of consecutive rows hit distinct banks.
#include "ff_common.hpp"
#include "ff_kernels.hpp"

namespace ff {
namespace {

constexpr int TM = 256;       // tile rows (and columns)
constexpr int TK = 32;        // k per LDS stage
constexpr int NSTAGE = 5;     // LDS ring depth (four slices in flight, 160 KB)
constexpr int NTHR = 256;     // four waves
constexpr int TILE_FLOATS = TM * TM;
constexpr int CHUNKS = TM * TK / 8;  // 16-byte chunks per operand per stage (1024)

typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((address_space(3))) void lds_void;

// Stage layout: chunk position P = 4 row + slot; slot s of row r holds the
// 16-byte k chunk c = s ^ swz(r).  A fragment read moves one chunk of each
// of 32 consecutive rows; the LDS serves it 16 lanes (16 rows, 256 bytes) at
// a time across its 64 banks, so the 16 chunks must cover all 16 positions
// modulo 16, i.e. (r mod 4, slot) must differ across 16 consecutive rows.
// swz(r) = ((r >> 1) & 3) ^ ((r >> 3) & 1) gives that, and also keeps any 8
// consecutive rows on distinct 128-byte bank groups.
struct __align__(16) Ring {
  u32x4 a[NSTAGE][CHUNKS];
  u32x4 b[NSTAGE][CHUNKS];
};

__device__ __forceinline__ int swz(int row) { return ((row >> 1) & 3) ^ ((row >> 3) & 1); }
__device__ __forceinline__ int chunk_pos(int row, int c) { return row * 4 + (c ^ swz(row)); }

// vmcnt(N) with the other counters left alone (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmem() {
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// lgkmcnt(0) with the other counters left alone.
__device__ __forceinline__ void wait_lds() { __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4)); }

// Per-lane element offsets of the four chunks this lane moves per operand and
// stage: instruction q of wave w fills positions (4 q + w) 64 + lane.
__device__ __forceinline__ void chunk_offsets(int wave, int lane, uint32_t ld, uint32_t (&off)[4]) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int P = (q * 4 + wave) * 64 + lane;
    const int row = P >> 2, slot = P & 3;
    const int c = slot ^ swz(row);
    off[q] = (uint32_t)row * ld + (uint32_t)c * 8u;
  }
}

// Asynchronous global -> LDS copy of one k slice of both operands.
__device__ __forceinline__ void issue_stage(Ring& sm, int buf, const bf16_t* pa, const bf16_t* pb,
                                            const uint32_t (&oa)[4], const uint32_t (&ob)[4],
                                            int wave) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    __builtin_amdgcn_global_load_lds((const void*)(pa + oa[q]),
                                     (lds_void*)&sm.a[buf][(q * 4 + wave) * 64], 16, 0, 0);
    __builtin_amdgcn_global_load_lds((const void*)(pb + ob[q]),
                                     (lds_void*)&sm.b[buf][(q * 4 + wave) * 64], 16, 0, 0);
  }
}

// Matrix-core fragments of one LDS slot: for each of the two 16-wide k
// steps, the rows (A side) and columns (B side) of this wave's 128 x 128
// quadrant, 8 consecutive k per lane.  f[kk][0..3] = A, f[kk][4..7] = B.
typedef bf16x8 Frags[2][8];

__device__ __forceinline__ void read_frags(const Ring& sm, int buf, int wave, int lane, Frags& f) {
  const int wm = wave >> 1, wn = wave & 1;
  const int lrow = lane & 31;
#pragma unroll
  for (int kk = 0; kk < 2; ++kk) {
    const int c = kk * 2 + (lane >> 5);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      f[kk][t] = __builtin_bit_cast(bf16x8, sm.a[buf][chunk_pos(wm * 128 + t * 32 + lrow, c)]);
      f[kk][4 + t] = __builtin_bit_cast(bf16x8, sm.b[buf][chunk_pos(wn * 128 + t * 32 + lrow, c)]);
    }
  }
}

// SW = false: acc[i][j] = A rows of tile i x B rows of tile j (element r of
// lane l: row 8 (r/4) + 4 (l/32) + r%4, column l%32).  SW = true: the
// operands swapped, acc[i][j] holds the transposed tile (row l%32, column
// 8 (r/4) + 4 (l/32) + r%4), so each lane holds 16 values of one row.
template <bool SW = false>
__device__ __forceinline__ void mfma_slot(const Frags& f, f32x16 (&acc)[4][4]) {
#pragma unroll
  for (int kk = 0; kk < 2; ++kk)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = SW ? __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[kk][4 + j], f[kk][i], acc[i][j], 0, 0, 0)
                       : __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[kk][i], f[kk][4 + j], acc[i][j], 0, 0, 0);
}

// Single pieces of a step, for the explicitly interleaved steady state:
// product m (k half m / 16, tile pair ((m / 4) % 4, m % 4)), fragment read q
// (k half q / 8; A tiles for q % 8 < 4, B tiles above) and copy q (operand
// q % 2, chunk group q / 2) of one stage.
template <bool SW>
__device__ __forceinline__ void mfma_one(const Frags& f, f32x16 (&acc)[4][4], int m) {
  const int kk = m >> 4, i = (m >> 2) & 3, j = m & 3;
  acc[i][j] = SW ? __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[kk][4 + j], f[kk][i], acc[i][j], 0, 0, 0)
                 : __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[kk][i], f[kk][4 + j], acc[i][j], 0, 0, 0);
}

__device__ __forceinline__ void read_frag_one(const Ring& sm, int buf, int wave, int lane, Frags& f,
                                              int q) {
  const int kk = q >> 3, t = q & 7;
  const int c = kk * 2 + (lane >> 5);
  const int row = (t < 4 ? (wave >> 1) : (wave & 1)) * 128 + (t & 3) * 32 + (lane & 31);
  f[kk][t] = __builtin_bit_cast(bf16x8, t < 4 ? sm.a[buf][chunk_pos(row, c)] : sm.b[buf][chunk_pos(row, c)]);
}

__device__ __forceinline__ void issue_one(Ring& sm, int buf, const bf16_t* pa, const bf16_t* pb,
                                          const uint32_t (&oa)[4], const uint32_t (&ob)[4], int wave,
                                          int q) {
  const int g = q >> 1;
  if (q & 1)
    __builtin_amdgcn_global_load_lds((const void*)(pb + ob[g]), (lds_void*)&sm.b[buf][(g * 4 + wave) * 64],
                                     16, 0, 0);
  else
    __builtin_amdgcn_global_load_lds((const void*)(pa + oa[g]), (lds_void*)&sm.a[buf][(g * 4 + wave) * 64],
                                     16, 0, 0);
}

// Slices requested but not yet known to have landed may number at most
// `pending` (0..4) when this returns (eight copies per slice and lane).
__device__ __forceinline__ void wait_pending(int pending) {
  if (pending >= 4) wait_vmem<32>();
  else if (pending == 3) wait_vmem<24>();
  else if (pending == 2) wait_vmem<16>();
  else if (pending == 1) wait_vmem<8>();
  else wait_vmem<0>();
}

// One k slice i (not the last) of the main loop, register set CUR holding
// its fragments: wait for slice i + 1, barrier (every wave has slice i in
// registers, so its slot is free), request slice i + 5 into that slot, then
// read slice i + 1 into the other register set interleaved with the 32
// products of slice i.  STEADY steps (i + 5 < n, so slice i + 5 exists and
// exactly three slices besides i + 1 are in flight) are branch-free, and
// their eight copies are spread over the first half of the products instead
// of being issued in one burst behind the barrier, where they would hold up
// the first product while the four waves' copies queue at the address unit.
template <bool SW, int CUR, bool STEADY, class Addr>
__device__ __forceinline__ void loop_step(Ring& sm, int i, int n, int kt0, const Addr& addr,
                                          const uint32_t (&oa)[4], const uint32_t (&ob)[4],
                                          int wave, int lane, Frags (&F)[2],
                                          f32x16 (&acc)[4][4]) {
  if constexpr (STEADY) wait_vmem<(NSTAGE - 2) * 8>();
  else wait_pending(min(n, i + NSTAGE) - (i + 2));
  wait_lds();  // this wave's reads of slice i (issued one step ago) are complete
  __builtin_amdgcn_s_barrier();
  if constexpr (STEADY) {
    const bf16_t *pa, *pb;
    addr(kt0 + i + NSTAGE, pa, pb);
    const int wbuf = (i + NSTAGE) % NSTAGE, rbuf = (i + 1) % NSTAGE;
    // products in program order, fenced; the 16 LDS reads of the next slice
    // follow products 0, 1, 3, 4, ..., 22 (read q after product 3q/2), so
    // the last one has nine products to land before the next step's wait,
    // and the eight copies follow products 2, 5, ..., 23
#pragma unroll
    for (int m = 0; m < 32; ++m) {
      mfma_one<SW>(F[CUR], acc, m);
      if (m < 24) {
        if (m % 3 == 2) issue_one(sm, wbuf, pa, pb, oa, ob, wave, m / 3);
        else read_frag_one(sm, rbuf, wave, lane, F[CUR ^ 1], (2 * m + (m % 3)) / 3);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  } else {
    if (i + NSTAGE < n) {
      const bf16_t *pa, *pb;
      addr(kt0 + i + NSTAGE, pa, pb);
      issue_stage(sm, (i + NSTAGE) % NSTAGE, pa, pb, oa, ob, wave);
    }
    read_frags(sm, (i + 1) % NSTAGE, wave, lane, F[CUR ^ 1]);
    mfma_slot<SW>(F[CUR], acc);
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);  // two matrix-core products
    }
  }
}

// acc += sum over k slices [kt0, kt1) of Aslice(kt) Bslice(kt)^T, where
// addr(kt, pa, pb) yields the slice base pointers (row 0, k = 32 kt).
// Slices are copied global -> LDS five slots ahead; fragments are read one
// slice ahead into a second register set.
template <bool SW = false, class Addr>
__device__ __forceinline__ void mainloop(Ring& sm, int kt0, int kt1, uint32_t lda, uint32_t ldb,
                                         const Addr& addr, f32x16 (&acc)[4][4]) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: LDS bases in SGPRs
  const int n = kt1 - kt0;
  if (n <= 0) return;
  uint32_t oa[4], ob[4];
  chunk_offsets(wave, lane, lda, oa);
  chunk_offsets(wave, lane, ldb, ob);
  for (int s = 0; s < NSTAGE && s < n; ++s) {
    const bf16_t *pa, *pb;
    addr(kt0 + s, pa, pb);
    issue_stage(sm, s, pa, pb, oa, ob, wave);
  }
  wait_pending(min(n, NSTAGE) - 1);
  __builtin_amdgcn_s_barrier();
  Frags F[2];
  read_frags(sm, 0, wave, lane, F[0]);
  int i = 0;
  for (; i + NSTAGE + 1 < n; i += 2) {  // both steps of the pair request a slice
    loop_step<SW, 0, true>(sm, i, n, kt0, addr, oa, ob, wave, lane, F, acc);
    loop_step<SW, 1, true>(sm, i + 1, n, kt0, addr, oa, ob, wave, lane, F, acc);
  }
  for (; i + 2 < n; i += 2) {
    loop_step<SW, 0, false>(sm, i, n, kt0, addr, oa, ob, wave, lane, F, acc);
    loop_step<SW, 1, false>(sm, i + 1, n, kt0, addr, oa, ob, wave, lane, F, acc);
  }
  if (n - i == 2) {
    loop_step<SW, 0, false>(sm, i, n, kt0, addr, oa, ob, wave, lane, F, acc);
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int t = 0; t < 8; ++t) F[0][kk][t] = F[1][kk][t];
  }
  mfma_slot<SW>(F[0], acc);
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

// Tiles of the whitening products.  Output tile (rb, cj) needs k in
// [0, 256 (cj + 1)) (Y is lower triangular), so tile lengths range from 8 to
// 8 ncol slices.  One workgroup takes the pair cj = c and cj = ncol - 1 - c
// of one row block: c with k ascending, then its partner with k descending.
// Every workgroup then runs 8 (ncol + 1) slices, and at slice step t of the
// workgroup all pairs of a row block sit at k slice t or 8 (ncol + 1) - 1 - t,
// so the workgroups that run together on an XCD (consecutive pairs of a few
// row blocks) stay in step and share their operand slices in its L2.
template <bool SW, bool REV>
__device__ __forceinline__ void whiten_tile(Ring& sm, const bf16_t* xa, const bf16_t* Y, const bf16_t* Y2,
                                            uint32_t cj, uint32_t Kp, f32x16 (&acc)[4][4]) {
  const int kt1 = (int)((cj + 1) * (TM / TK));
  zero_acc(acc);
  {
    const bf16_t* yb = Y + (size_t)cj * TM * Kp;
    auto addr = [&](int kt, const bf16_t*& pa, const bf16_t*& pb) {
      const int k = REV ? kt1 - 1 - kt : kt;
      pa = xa + k * TK;
      pb = yb + k * TK;
    };
    mainloop<SW>(sm, 0, kt1, Kp, Kp, addr, acc);
  }
  if (Y2 != nullptr) {
    const bf16_t* yb = Y2 + (size_t)cj * TM * Kp;
    auto addr = [&](int kt, const bf16_t*& pa, const bf16_t*& pb) {
      const int k = REV ? kt1 - 1 - kt : kt;
      pa = xa + k * TK;
      pb = yb + k * TK;
    };
    mainloop<SW>(sm, 0, kt1, Kp, Kp, addr, acc);
  }
}

__device__ __forceinline__ void store_whitened(const f32x16 (&acc)[4][4], bf16_t* C, uint32_t rb,
                                               uint32_t cj, uint32_t Kp) {
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

__global__ __launch_bounds__(NTHR, 1) void k_whiten_bf16(const bf16_t* __restrict__ X,
                                                         const bf16_t* __restrict__ Y,
                                                         const bf16_t* __restrict__ Y2,
                                                         bf16_t* __restrict__ C, uint32_t Kp,
                                                         const int* st) {
  if (ff_halted(st)) return;
  __shared__ Ring sm;
  const uint32_t ncol = Kp / TM, npair = (ncol + 1) / 2;
  const uint32_t t = xcd_remap(blockIdx.x, gridDim.x);
  const uint32_t rb = t / npair, c = t % npair;
  const bf16_t* xa = X + (size_t)rb * TM * Kp;
  f32x16 acc[4][4];
  whiten_tile<false, false>(sm, xa, Y, Y2, c, Kp, acc);
  store_whitened(acc, C, rb, c, Kp);
  if (ncol - 1 - c != c) {
    whiten_tile<false, true>(sm, xa, Y, Y2, ncol - 1 - c, Kp, acc);
    store_whitened(acc, C, rb, ncol - 1 - c, Kp);
  }
}

// Row norms of the whitened rows, for the rank-one (per-token) form of the
// updates (Section 5: the weight of token t in one half step is x_t^T A^-1 x_t
// = ||L^-1 x_t||^2).  Same tiles, pairs and k ranges as k_whiten_bf16, with
// the operands swapped so that every lane holds values of one row; the
// whitened values are never stored.  part[row][2 cj + wn] receives the sum of
// squares over the 128 columns of wave column wn of tile column cj.
__device__ __forceinline__ void store_norms(const f32x16 (&acc)[4][4], float* part, uint32_t rb,
                                            uint32_t cj, uint32_t ncol) {
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int wm = wave >> 1, wn = wave & 1;
  const uint32_t npart = 2 * ncol;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float s = 0.0f;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) s += acc[i][j][r] * acc[i][j][r];
    s += __shfl_xor(s, 32);  // lanes l and l + 32 hold the two column halves of row l % 32
    if (lane < 32) {
      const size_t row = (size_t)rb * TM + wm * 128 + i * 32 + lane;
      part[row * npart + 2 * cj + wn] = s;
    }
  }
}

__global__ __launch_bounds__(NTHR, 1) void k_whiten_norm_bf16(const bf16_t* __restrict__ X,
                                                              const bf16_t* __restrict__ Y,
                                                              const bf16_t* __restrict__ Y2,
                                                              float* __restrict__ part, uint32_t Kp,
                                                              const int* st) {
  if (ff_halted(st)) return;
  __shared__ Ring sm;
  const uint32_t ncol = Kp / TM, npair = (ncol + 1) / 2;
  const uint32_t t = xcd_remap(blockIdx.x, gridDim.x);
  const uint32_t rb = t / npair, c = t % npair;
  const bf16_t* xa = X + (size_t)rb * TM * Kp;
  f32x16 acc[4][4];
  whiten_tile<true, false>(sm, xa, Y, Y2, c, Kp, acc);
  store_norms(acc, part, rb, c, ncol);
  if (ncol - 1 - c != c) {
    whiten_tile<true, true>(sm, xa, Y, Y2, ncol - 1 - c, Kp, acc);
    store_norms(acc, part, rb, ncol - 1 - c, ncol);
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
  __shared__ Ring sm;
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
  const int64_t tiles = (rows / TM) * ((Kp / TM + 1) / 2);  // one workgroup per tile pair
  if (tiles > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_whiten_bf16, dim3((uint32_t)tiles), dim3(NTHR), 0, s, X, Y, Y2, C,
                     (uint32_t)Kp, st);
  return hipGetLastError();
}

hipError_t launch_whiten_norm_bf16(const bf16_t* X, const bf16_t* Y, const bf16_t* Y2, float* part,
                                   int64_t rows, int64_t Kp, const int* st, hipStream_t s) {
  if (rows <= 0 || Kp <= 0 || rows % TM || Kp % TM || Kp > (1 << 20)) return hipErrorInvalidValue;
  const int64_t tiles = (rows / TM) * ((Kp / TM + 1) / 2);  // one workgroup per tile pair
  if (tiles > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_whiten_norm_bf16, dim3((uint32_t)tiles), dim3(NTHR), 0, s, X, Y, Y2, part,
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
