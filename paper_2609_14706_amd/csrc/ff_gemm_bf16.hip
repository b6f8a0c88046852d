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
// Operands move global -> LDS with the direct-to-LDS buffer loads of gfx950
// (buffer_load_dwordx4 ... lds, no register staging) in 64-wide k pairs, so
// that every copy request is a whole 128-byte line (half-line requests cost
// about 15% of the symmetric product's time in L2 traffic), through two pair
// slots (128 KB), one pair in flight ahead of the matrix cores.  The 16-byte
// chunks of each 128-byte row are XOR-swizzled so that fragment reads of
// consecutive rows hit distinct banks.  Copy and fragment-read addresses are
// fixed per lane and set up once: inside the loop only scalar bases and
// instruction offsets change (about 7 vector instructions per 64 products
// instead of 30-50; worth about 1% under sustained load, where the clock is
// power limited).
#include "ff_common.hpp"
#include "ff_kernels.hpp"

namespace ff {
namespace {

constexpr int TM = 256;       // tile rows (and columns)
constexpr int TK = 32;        // k per matrix-core step (two 16-wide products)
constexpr int PK = 64;        // k per copied pair of steps: 128-byte row segments
constexpr int NPAIR = 2;      // LDS pair slots (128 KB)
constexpr int NTHR = 256;     // four waves
constexpr int TILE_FLOATS = TM * TM;
constexpr int PCH = TM * PK / 8;  // 16-byte chunks per operand per pair (2048)

typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((address_space(3))) void lds_void;

// Pair layout: each operand row holds the 8 chunks (16 bytes, 8 k) of a 64-k
// pair, chunk c at position 8 row + (c ^ swz(row)).  A fragment read moves
// one chunk of each of 32 consecutive rows; the LDS serves it 16 lanes (16
// rows, 256 bytes) at a time across its 64 four-byte banks.  With 128-byte
// rows, position p of row r starts at bank 32 (r & 1) + 4 p, so the read is
// conflict-free when its 16 rows cover all 16 pairs (r & 1, p); swz(row) =
// (row >> 1) & 7 gives that.  A copy instruction fills 1 KB of consecutive
// positions, i.e. eight whole rows: eight complete 128-byte lines.
struct __align__(16) Ring {
  u32x4 a[NPAIR][PCH];
  u32x4 b[NPAIR][PCH];
};

__device__ __forceinline__ int swz(int row) { return (row >> 1) & 7; }

// vmcnt(N) with the other counters left alone (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmem() {
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// lgkmcnt(0) with the other counters left alone.
__device__ __forceinline__ void wait_lds() { __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4)); }

// Byte offset of the chunk this lane copies with instruction 0 of a pair;
// instruction q (0..7) of wave w fills positions (4 q + w) 64 + lane, which
// lie 32 q rows further down with the same swizzle, so its offset is
// off + 64 q ld bytes (a scalar offset of the instruction).
__device__ __forceinline__ uint32_t chunk_offset(int wave, int lane, uint32_t ld) {
  const int P = wave * 64 + lane;
  const int row = P >> 3, c = (P & 7) ^ swz(row);
  return ((uint32_t)row * ld + (uint32_t)c * 8u) * 2u;  // bytes
}

// Buffer resource of a pair's operand (gfx9 descriptor: base, stride 0, no
// effective range limit, raw dword data format).  The copies then address
// base (scalar) + the lane's fixed byte offset (vector) + the instruction's
// row-group offset (scalar): no per-lane address arithmetic in the loop.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t pair_rsrc(const bf16_t* p) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(p), (short)0, (int)0x7fffffff, 0x00020000);
}

// Copy q (0..15) of a pair: operand q % 2, instruction q / 2.
__device__ __forceinline__ void issue_one(Ring& sm, int slot, const bf16_t* pa, const bf16_t* pb,
                                          uint32_t oa, uint32_t ob, uint32_t lda, uint32_t ldb,
                                          int wave, int q) {
  const int g = q >> 1;
  if (q & 1)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(pair_rsrc(pb), (lds_void*)&sm.b[slot][(g * 4 + wave) * 64],
                                             16, (int)ob, (int)((uint32_t)g * 64u * ldb), 0, 0);
  else
    __builtin_amdgcn_raw_ptr_buffer_load_lds(pair_rsrc(pa), (lds_void*)&sm.a[slot][(g * 4 + wave) * 64],
                                             16, (int)oa, (int)((uint32_t)g * 64u * lda), 0, 0);
}

__device__ __forceinline__ void issue_pair(Ring& sm, int slot, const bf16_t* pa, const bf16_t* pb,
                                           uint32_t oa, uint32_t ob, uint32_t lda, uint32_t ldb,
                                           int wave) {
#pragma unroll
  for (int q = 0; q < 16; ++q) issue_one(sm, slot, pa, pb, oa, ob, lda, ldb, wave, q);
}

// Matrix-core fragments of one 32-k step: for each of its two 16-wide k
// halves, the rows (A side) and columns (B side) of this wave's 128 x 128
// quadrant, 8 consecutive k per lane.  f[kk][0..3] = A, f[kk][4..7] = B.
typedef bf16x8 Frags[2][8];

// Byte offsets (from the start of the Ring) of this lane's fragment chunks
// in slot 0 for tile 0 of each operand, k half and 16-wide k step.  The
// swizzle of a fragment row depends on the lane only (the tile's first row
// is a multiple of 32), so every read is one of these eight registers plus
// a constant: the slot (32 KB) and the tile (4 KB).
struct FragBase {
  uint32_t v[2][2][2];  // [operand B][half][kk]
};

__device__ __forceinline__ FragBase frag_base(int wave, int lane) {
  FragBase fb;
  const uint32_t s = (uint32_t)swz(lane & 31), hl = (uint32_t)(lane >> 5);
#pragma unroll
  for (int o = 0; o < 2; ++o)
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        const uint32_t c = (uint32_t)(h * 4 + kk * 2) + hl;
        const uint32_t row = (uint32_t)(o ? (wave & 1) : (wave >> 1)) * 128u + (uint32_t)(lane & 31);
        fb.v[o][h][kk] = (o ? (uint32_t)sizeof(Ring::a) : 0u) + row * 128u + 16u * (c ^ s);
      }
  return fb;
}

// Fragment read q (0..15) of step `half` (0, 1) of the pair in `slot`:
// k half q / 8, A tiles for q % 8 < 4, B tiles above.
__device__ __forceinline__ void read_frag_one(const Ring& sm, int slot, int half, const FragBase& fb,
                                              Frags& f, int q) {
  const int kk = q >> 3, t = q & 7;
  const uint32_t off = fb.v[t >= 4][half][kk] + (uint32_t)slot * (uint32_t)(PCH * 16) + (uint32_t)(t & 3) * 4096u;
  f[kk][t] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(reinterpret_cast<const char*>(&sm) + off));
}

// Product m (0..31) of a step: k half m / 16, tile pair ((m / 4) % 4, m % 4).
// SW = false: acc[i][j] = A rows of tile i x B rows of tile j (element r of
// lane l: row 8 (r/4) + 4 (l/32) + r%4, column l%32).  SW = true: the
// operands swapped, acc[i][j] holds the transposed tile (row l%32, column
// 8 (r/4) + 4 (l/32) + r%4), so each lane holds 16 values of one row.
template <bool SW>
__device__ __forceinline__ void mfma_one(const Frags& f, f32x16 (&acc)[4][4], int m) {
  const int kk = m >> 4, i = (m >> 2) & 3, j = m & 3;
  acc[i][j] = SW ? __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[kk][4 + j], f[kk][i], acc[i][j], 0, 0, 0)
                 : __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[kk][i], f[kk][4 + j], acc[i][j], 0, 0, 0);
}

// One step: the 32 products of `cur` in program order, fenced one by one.
// If READ, the 16 fragment reads of step `rhalf` of the pair in `rslot` go
// into `nxt` after products 0, 1, 3, 4, ..., 22 (read q after product 3q/2),
// so the last one has nine products to land; if LOADS, the 16 copies of the
// pair at (pa, pb) into `lslot` follow the even products.
template <bool SW, bool READ, bool LOADS>
__device__ __forceinline__ void step(Ring& sm, const Frags& cur, Frags& nxt, int rslot, int rhalf,
                                     int lslot, const bf16_t* pa, const bf16_t* pb, uint32_t oa,
                                     uint32_t ob, uint32_t lda, uint32_t ldb, int wave, const FragBase& fb,
                                     f32x16 (&acc)[4][4]) {
#pragma unroll
  for (int m = 0; m < 32; ++m) {
    mfma_one<SW>(cur, acc, m);
    if (READ && m < 24 && m % 3 != 2)
      read_frag_one(sm, rslot, rhalf, fb, nxt, (2 * m + (m % 3)) / 3);
    if (LOADS && m % 2 == 0) issue_one(sm, lslot, pa, pb, oa, ob, lda, ldb, wave, m / 2);
    __builtin_amdgcn_sched_barrier(0);
  }
}

// acc += sum over k pairs [p0, p1) of Apair(p) Bpair(p)^T, where
// addr(p, pa, pb) yields the pair's base pointers (row 0, k = 64 p).  Pairs
// are copied global -> LDS one ahead, into two slots.  Per pair, step A
// multiplies the pair's first 32 k from registers while reading its second
// half; step B waits for the next pair, takes the pair's one barrier (every
// wave has finished reading this pair's slot and sees the next pair), then
// multiplies the second half while reading the next pair's first half and
// copying the pair after next into the slot just freed.
// The first two pairs' copies of mainloop (p0 and p0 + 1 into slots 0, 1).
template <class Addr>
__device__ __forceinline__ void issue_prologue(Ring& sm, int p0, int p1, uint32_t lda, uint32_t ldb,
                                               const Addr& addr) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint32_t oa = chunk_offset(wave, lane, lda), ob = chunk_offset(wave, lane, ldb);
  const bf16_t *pa, *pb;
  addr(p0, pa, pb);
  issue_pair(sm, 0, pa, pb, oa, ob, lda, ldb, wave);
  if (p1 - p0 > 1) {
    addr(p0 + 1, pa, pb);
    issue_pair(sm, 1, pa, pb, oa, ob, lda, ldb, wave);
  }
}

// PRE: the caller has issued the prologue's copies (issue_prologue) after
// its last other vector-memory instruction.
template <bool SW = false, bool PRE = false, class Addr>
__device__ __forceinline__ void mainloop(Ring& sm, int p0, int p1, uint32_t lda, uint32_t ldb,
                                         const Addr& addr, f32x16 (&acc)[4][4]) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: LDS bases in SGPRs
  const int n = p1 - p0;
  if (n <= 0) return;
  const uint32_t oa = chunk_offset(wave, lane, lda), ob = chunk_offset(wave, lane, ldb);
  const FragBase fb = frag_base(wave, lane);
  const bf16_t *pa, *pb;
  if (!PRE) issue_prologue(sm, p0, p1, lda, ldb, addr);
  if (n > 1) {
    wait_vmem<16>();
  } else {
    wait_vmem<0>();
  }
  __builtin_amdgcn_s_barrier();
  Frags F[2];
#pragma unroll
  for (int q = 0; q < 16; ++q) read_frag_one(sm, 0, 0, fb, F[0], q);
  int j = 0;
  for (; j + 2 < n; ++j) {  // steady: step B also copies pair j + 2
    const int slot = j & 1;
    step<SW, true, false>(sm, F[0], F[1], slot, 1, 0, nullptr, nullptr, 0, 0, lda, ldb, wave, fb, acc);
    wait_vmem<0>();  // pair j + 1 (the only pair in flight)
    wait_lds();      // this wave's reads of pair j are complete
    __builtin_amdgcn_s_barrier();
    addr(p0 + j + 2, pa, pb);
    step<SW, true, true>(sm, F[1], F[0], slot ^ 1, 0, slot, pa, pb, oa, ob, lda, ldb, wave, fb, acc);
  }
  if (j + 1 < n) {
    const int slot = j & 1;
    step<SW, true, false>(sm, F[0], F[1], slot, 1, 0, nullptr, nullptr, 0, 0, lda, ldb, wave, fb, acc);
    wait_vmem<0>();
    wait_lds();
    __builtin_amdgcn_s_barrier();
    step<SW, true, false>(sm, F[1], F[0], slot ^ 1, 0, 0, nullptr, nullptr, 0, 0, lda, ldb, wave, fb, acc);
    ++j;
  }
  step<SW, true, false>(sm, F[0], F[1], j & 1, 1, 0, nullptr, nullptr, 0, 0, lda, ldb, wave, fb, acc);
  step<SW, false, false>(sm, F[1], F[0], 0, 0, 0, nullptr, nullptr, 0, 0, lda, ldb, wave, fb, acc);
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
// Operand addresses of pair p of tile column cj (pass 0: Y, pass 1: Y2).
struct WhitenAddr {
  const bf16_t* xa;
  const bf16_t* yb;
  int np;
  bool rev;
  __device__ __forceinline__ void operator()(int p, const bf16_t*& pa, const bf16_t*& pb) const {
    const int k = rev ? np - 1 - p : p;
    pa = xa + k * PK;
    pb = yb + k * PK;
  }
};

__device__ __forceinline__ WhitenAddr whiten_addr(const bf16_t* xa, const bf16_t* Y, uint32_t cj,
                                                  bool rev, uint32_t Kp, bool full) {
  const int np = (int)((full ? Kp / TM : cj + 1) * (TM / PK));
  return WhitenAddr{xa, Y + (size_t)cj * TM * Kp, np, rev};
}

// acc = X Y^T (+ X Y2^T) over tile column cj; PRE: the first pass's prologue
// copies are issued and acc is zero already.
template <bool SW, bool PRE>
__device__ __forceinline__ void whiten_tile(Ring& sm, const bf16_t* xa, const bf16_t* Y, const bf16_t* Y2,
                                            uint32_t cj, bool rev, uint32_t Kp, bool full,
                                            f32x16 (&acc)[4][4]) {
  if (!PRE) zero_acc(acc);
  const WhitenAddr a0 = whiten_addr(xa, Y, cj, rev, Kp, full);
  mainloop<SW, PRE>(sm, 0, a0.np, Kp, Kp, a0, acc);
  if (Y2 != nullptr) {
    const WhitenAddr a1 = whiten_addr(xa, Y2, cj, rev, Kp, full);
    mainloop<SW>(sm, 0, a1.np, Kp, Kp, a1, acc);
  }
}

__device__ __forceinline__ void store_whitened(const f32x16 (&acc)[4][4], bf16_t* C, uint32_t rb,
                                               uint32_t cj, uint32_t Kp) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  // per-lane base (row 4 (l / 32), column l % 32 of the wave's quadrant);
  // the offsets of the accumulator elements below are wave-uniform.  The
  // opaque copy of the row pitch keeps the compiler from computing those
  // offsets once ahead of the tile loop and holding them across the main loop.
  uint32_t ldc = Kp;
  asm volatile("" : "+s"(ldc));
  bf16_t* lp = C + ((size_t)rb * TM + wm * 128 + 4 * (lane >> 5)) * ldc + (size_t)cj * TM + wn * 128 +
               (lane & 31);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const uint32_t row = i * 32 + 8 * (r >> 2) + (r & 3);
        lp[row * ldc + j * 32] = f32_to_bf16(acc[i][j][r]);
      }
}

__global__ __launch_bounds__(NTHR, 1) void k_whiten_bf16(const bf16_t* __restrict__ X,
                                                         const bf16_t* __restrict__ Y,
                                                         const bf16_t* __restrict__ Y2,
                                                         const int* __restrict__ use2, const int* __restrict__ use2b,
                                                         bf16_t* __restrict__ C, uint32_t Kp,
                                                         uint32_t full, const int* st) {
  if (ff_halted(st)) return;
  if (use2 != nullptr && *use2 == 0 && (use2b == nullptr || *use2b == 0)) Y2 = nullptr;  // one pass
  __shared__ Ring sm;
  const uint32_t ncol = Kp / TM, npair = (ncol + 1) / 2;
  const uint32_t t = xcd_remap(blockIdx.x, gridDim.x);
  const uint32_t rb = t / npair, c = t % npair;
  const bf16_t* xa = X + (size_t)rb * TM * Kp;
  f32x16 acc[4][4];
  // the second tile's first copies go out right behind the first tile's
  // stores, so that their latency overlaps the stores' drain
  whiten_tile<false, false>(sm, xa, Y, Y2, c, false, Kp, full != 0, acc);
  store_whitened(acc, C, rb, c, Kp);
  if (ncol - 1 - c != c) {
    const uint32_t cj = ncol - 1 - c;
    const WhitenAddr a0 = whiten_addr(xa, Y, cj, true, Kp, full != 0);
    issue_prologue(sm, 0, a0.np, Kp, Kp, a0);
    zero_acc(acc);
    whiten_tile<false, true>(sm, xa, Y, Y2, cj, true, Kp, full != 0, acc);
    store_whitened(acc, C, rb, cj, Kp);
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
                                                              const int* __restrict__ use2, const int* __restrict__ use2b,
                                                              float* __restrict__ part, uint32_t Kp,
                                                              const int* st) {
  if (ff_halted(st)) return;
  if (use2 != nullptr && *use2 == 0 && (use2b == nullptr || *use2b == 0)) Y2 = nullptr;  // one pass
  __shared__ Ring sm;
  const uint32_t ncol = Kp / TM, npair = (ncol + 1) / 2;
  const uint32_t t = xcd_remap(blockIdx.x, gridDim.x);
  const uint32_t rb = t / npair, c = t % npair;
  const bf16_t* xa = X + (size_t)rb * TM * Kp;
  f32x16 acc[4][4];
  for (uint32_t h = 0; h < (ncol - 1 - c != c ? 2u : 1u); ++h) {
    const uint32_t cj = h ? ncol - 1 - c : c;
    whiten_tile<true, false>(sm, xa, Y, Y2, cj, h != 0, Kp, false, acc);
    store_norms(acc, part, rb, cj, ncol);
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

// Order in which the workgroups of one k split visit the upper tiles: tile
// rows and columns are grouped in fours; the 4 x 4 groups are visited
// column by column (group Q = 0, 1, ..., and in group column Q the groups
// P = 0..Q), the tiles of an off-diagonal group column-major and those of a
// diagonal group row-major over its upper triangle.  Consecutive workgroups
// share an XCD (and its L2); in this order a window of them reads fewer
// distinct tile rows than in the row-major order (12% fewer L2 misses and
// 3% less time on the 4096-wide symmetric product).
constexpr uint32_t TGRP = 4;
__device__ __forceinline__ void grouped_tile(uint32_t idx, uint32_t T, uint32_t& ti, uint32_t& tj) {
  for (uint32_t Q = 0, q0 = 0; q0 < T; ++Q, q0 += TGRP) {
    const uint32_t sq = min(TGRP, T - q0);          // tiles in this group column
    const uint32_t off = Q * TGRP * sq;             // its off-diagonal groups (all full height)
    const uint32_t cnt = off + sq * (sq + 1) / 2;
    if (idx < cnt) {
      if (idx < off) {
        const uint32_t P = idx / (TGRP * sq), r = idx % (TGRP * sq);
        ti = P * TGRP + r % TGRP;
        tj = q0 + r / TGRP;
      } else {
        uint32_t a, b;
        upper_tile(idx - off, sq, a, b);
        ti = q0 + a;
        tj = q0 + b;
      }
      return;
    }
    idx -= cnt;
  }
  ti = tj = 0;
}

// Work item of workgroup b when the dispatcher places b on XCD b % 8 and
// each XCD runs its workgroups in order, 32 at a time: round r of XCD x
// takes items 256 r + 32 x .. + 31, so that the eight XCDs work on
// neighbouring items (the same k split) at the same time and each XCD's
// 32 co-resident workgroups take consecutive items (a compact group of
// tiles).  The workgroups past the last full round take the remaining
// items XCD by XCD.  A bijection of [0, total).
__device__ __forceinline__ uint32_t round_item(uint32_t b, uint32_t total) {
  const uint32_t q = total >> 3, rem = total & 7u;
  const uint32_t x = b & 7u, li = b >> 3;
  const uint32_t full = (q / 32u) * 32u;  // local indices in full rounds (every XCD has them)
  if (li < full) return (li / 32u) * 256u + x * 32u + (li % 32u);
  // tail: XCD x holds wx - full items, wx = q + (x < rem)
  const uint32_t tail = q - full;
  const uint32_t before = x * tail + min(x, rem);
  return full * 8u + before + (li - full);
}

__global__ __launch_bounds__(NTHR, 1) void k_syrk_bf16(const bf16_t* __restrict__ X,
                                                       const bf16_t* __restrict__ Xb, uint32_t ld,
                                                       uint64_t seg_stride, uint32_t nseg,
                                                       uint32_t T, uint32_t ntiles, uint32_t splits,
                                                       float* __restrict__ P, const int* st) {
  if (ff_halted(st)) return;
  __shared__ Ring sm;
  const uint32_t t = round_item(blockIdx.x, gridDim.x);
  const uint32_t z = t / ntiles, tile = t % ntiles;
  uint32_t ti, tj;
  grouped_tile(tile, T, ti, tj);
  const uint32_t pps = ld / PK;  // k pairs per segment
  const uint64_t ptot = (uint64_t)pps * nseg;
  const int p0 = (int)(ptot * z / splits), p1 = (int)(ptot * (z + 1) / splits);
  const bf16_t* xa = X + (size_t)ti * TM * ld;
  const bf16_t* xb = (Xb != nullptr ? Xb : X) + (size_t)tj * TM * ld;
  f32x16 acc[4][4];
  zero_acc(acc);
  auto addr = [&](int p, const bf16_t*& pa, const bf16_t*& pb) {
    const uint32_t s = (uint32_t)p / pps, o = (uint32_t)p % pps;
    const size_t base = (size_t)s * seg_stride + (size_t)o * PK;
    pa = xa + base;
    pb = xb + base;
  };
  mainloop(sm, p0, p1, ld, ld, addr, acc);
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
  grouped_tile(tile, T, ti, tj);
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

hipError_t launch_whiten_bf16(const bf16_t* X, const bf16_t* Y, const bf16_t* Y2, const int* use2,
                              const int* use2b, bf16_t* C, int64_t rows, int64_t Kp, const int* st,
                              hipStream_t s, bool full) {
  // Kp <= 2^20 keeps every copy's byte offset from its pair base below 2^31
  if (rows <= 0 || Kp <= 0 || rows % TM || Kp % TM || Kp > (1 << 20)) return hipErrorInvalidValue;
  const int64_t tiles = (rows / TM) * ((Kp / TM + 1) / 2);  // one workgroup per tile pair
  if (tiles > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_whiten_bf16, dim3((uint32_t)tiles), dim3(NTHR), 0, s, X, Y, Y2, use2, use2b, C,
                     (uint32_t)Kp, (uint32_t)full, st);
  return hipGetLastError();
}

hipError_t launch_whiten_norm_bf16(const bf16_t* X, const bf16_t* Y, const bf16_t* Y2,
                                   const int* use2, const int* use2b, float* part, int64_t rows,
                                   int64_t Kp, const int* st, hipStream_t s) {
  if (rows <= 0 || Kp <= 0 || rows % TM || Kp % TM || Kp > (1 << 20)) return hipErrorInvalidValue;
  const int64_t tiles = (rows / TM) * ((Kp / TM + 1) / 2);  // one workgroup per tile pair
  if (tiles > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_whiten_norm_bf16, dim3((uint32_t)tiles), dim3(NTHR), 0, s, X, Y, Y2, use2,
                     use2b, part,
                     (uint32_t)Kp, st);
  return hipGetLastError();
}

hipError_t launch_syrk_bf16(const bf16_t* X, int64_t dim_p, int64_t ld, int64_t seg_stride,
                            int64_t nseg, int splits, float* P, const int* st, hipStream_t s,
                            const bf16_t* Xb) {
  // ld <= 2^20 keeps every copy's byte offset from its pair base below 2^31
  if (dim_p <= 0 || dim_p % TM || ld <= 0 || ld % PK || ld > (1 << 20) || nseg <= 0 || splits <= 0)
    return hipErrorInvalidValue;
  const int64_t T = dim_p / TM, ntiles = T * (T + 1) / 2;
  if ((int64_t)splits > (ld / PK) * nseg) return hipErrorInvalidValue;
  if (ntiles * splits > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_syrk_bf16, dim3((uint32_t)(ntiles * splits)), dim3(NTHR), 0, s, X, Xb,
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
