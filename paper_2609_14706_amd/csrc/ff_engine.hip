// Host runtime of the FlipFlop engine: workspace layout, the stream-ordered
// iteration pipeline and the C ABI declared in ff.h.
//
// One flip-flop iteration (Section 5; Appendix B order: B first, from A = I):
//   whiten   W_i = G_i L_A^-T            (L_A^-1 from the previous step)
//   symmetric product, reduce            B = (1/(N n)) sum_i W_i W_i^T   [+ damping]
//   Cholesky + inverse of B              L_B^-1
//   whiten   V_i = G_i^T L_B^-T          (on the transposed sample copy)
//   symmetric product, reduce            A = (1/(N m)) sum_i V_i V_i^T   [+ damping]
//   normalise                            c = tr(A)/n, A /= c, B *= c
//   Cholesky + inverse of A              L_A^-1 for the next iteration, log|A|
// All of it is enqueued on the caller's stream without host round trips; the
// stream is synchronised once at the end of ff_iterate.
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "ff.h"
#include "ff_kernels.hpp"

using namespace ff;

namespace {

thread_local std::string g_last_error;

ff_status fail(ff_status s, const std::string& msg) {
  g_last_error = msg;
  return s;
}

#define FF_HIP(call)                                                                     \
  do {                                                                                   \
    hipError_t e_ = (call);                                                              \
    if (e_ != hipSuccess)                                                                \
      return fail(FF_ERR_HIP, std::string(#call) + ": " + hipGetErrorString(e_));        \
  } while (0)

constexpr size_t kAlign = 256;
constexpr int64_t kTokenSeg = 256;  // tokens per segment of the weighted, transposed tokens
constexpr int kLLCap = 1024;      // log-likelihood values per device ring
constexpr int kTimedKernels = 5;  // whiten, symmetric product, reduction, factorisation,
                                  // quantiser anti-diagonal

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
int64_t round_up(int64_t x, int64_t g) { return (x + g - 1) / g * g; }

struct Side {
  int64_t dim = 0, dim_p = 0;
  float* F[2] = {nullptr, nullptr};  // the factor, double buffered by iteration parity
  float* L = nullptr;                // Cholesky work copy
  float* Li = nullptr;               // L^-1 (fp32, lower)
  void* Lw = nullptr;                // whitening operand (elem, dim_p x dim_p)
  void* Lw2 = nullptr;               // its low bf16 part (whiten_split = 2 or automatic)
  int* split_flag = nullptr;         // automatic split: 1 = whiten with hi + lo parts
  double* split_stat = nullptr;      // automatic split: the rounding sensitivity s of Lw
  double* spart = nullptr;           // automatic split: partial sums of its statistic
  bool stat_known = false;           // automatic split: split_stat has been written
  double* slots = nullptr;           // per-leaf sum log L_jj
  int nslots = 0;
  double* tr = nullptr;              // trace after the last update
  int splits = 1;                    // k-splits of the symmetric product producing this side
  size_t partial_floats = 0;
  bool lw_valid = false;             // Lw holds the inverse factor of F[cur]
  bool start_identity = false;       // the starting factor is I (no A0 / B0 given)
  int code = 0;                      // 1 = A, 2 = B
  // second stream of the blocked factorisation (created on first use): it
  // builds the off-diagonal blocks of the inverse
  hipStream_t istream = nullptr;
  hipEvent_t ev_leaf = nullptr, ev_inv = nullptr;
};

struct Layout {
  int64_t m_p, n_p;
  bool own_gx;
  bool rank1;
  int64_t T_p;  // rank-one form: padded token count
  // dense: gx = padded G, gt = padded transposed G, w = whitened samples;
  // rank-one: gx = padded x (T_p x n_p), gt = padded g (T_p x m_p),
  // w = row-norm partials (bf16) or whitened tokens (fp32), s = weighted
  // transposed tokens, wv = token weights (2 T_p floats)
  size_t off_small, off_ll, off_diag, off_slotsA, off_slotsB, off_gx, off_gt, off_w, off_p, off_s,
      off_wv, off_split;
  size_t w_bytes;  // capacity of the w region
  size_t off_A[6], off_B[6];  // F0, F1, L, Li, Lw, Lw2
  size_t total;
  int splitsA, splitsB;
  size_t partialA, partialB;
};

bool is_bf16(const ff_config* c) { return c->dtype == FF_BF16; }
int elem_bytes(const ff_config* c) { return is_bf16(c) ? 2 : 4; }
int granule(const ff_config* c) { return is_bf16(c) ? kTileBF16 : 64; }

// Splits of the bf16 symmetric product: minimise (rounds of 256 workgroups) x
// (k slices per workgroup) plus the cost of writing and re-reading partials.
int choose_splits_bf16(int64_t dim_p, int64_t kslices) {
  const int64_t T = dim_p / kTileBF16, tiles = T * (T + 1) / 2;
  double best = 1e300;
  int bestS = 1;
  const int64_t maxS = std::min<int64_t>(128, kslices);
  for (int64_t S = 1; S <= maxS; ++S) {
    const double rounds = (double)((tiles * S + 255) / 256);
    const double t = rounds * (double)((kslices + S - 1) / S) * 1.7e-6 +
                     (double)(tiles * S) * 0.5e6 / 4.0e12;
    if (t < best * (1.0 - 1e-9)) {
      best = t;
      bestS = (int)S;
    }
  }
  return bestS;
}

int choose_splits_f32(int64_t dim_p, int64_t K) {
  const int64_t T = (dim_p + 127) / 128, tiles = T * (T + 1) / 2;
  int64_t S = std::max<int64_t>(1, 512 / tiles);
  S = std::min<int64_t>(S, std::max<int64_t>(1, K / 256));
  return (int)std::min<int64_t>(S, 256);
}

ff_status validate_shape(const ff_config* c) {
  if (c == nullptr) return fail(FF_ERR_INVALID_ARG, "config is NULL");
  if (c->m < 1 || c->n < 1 || c->N < 1)
    return fail(FF_ERR_INVALID_ARG, "m, n and N must be >= 1");
  if (c->dtype != FF_F32 && c->dtype != FF_BF16) return fail(FF_ERR_INVALID_ARG, "unknown dtype");
  if (c->form != FF_SAMPLES_DENSE && c->form != FF_SAMPLES_RANK1)
    return fail(FF_ERR_INVALID_ARG, "unknown sample form");
  if (c->form == FF_SAMPLES_DENSE && c->N > 65535)
    return fail(FF_ERR_INVALID_ARG, "N must be <= 65535");
  if (c->form == FF_SAMPLES_RANK1 && c->N > (1 << 22))
    return fail(FF_ERR_INVALID_ARG, "N (tokens) must be <= 4194304");
  if (c->estimator < FF_EST_FLIPFLOP || c->estimator > FF_EST_INPUT)
    return fail(FF_ERR_INVALID_ARG, "unknown estimator");
  if (c->estimator == FF_EST_FROBENIUS && c->order != FF_ORDER_B_FIRST)
    return fail(FF_ERR_INVALID_ARG,
                "the Frobenius iteration runs B first (with A first its scale diverges)");
  if ((c->estimator == FF_EST_MARGINAL || c->estimator == FF_EST_INPUT) &&
      c->form != FF_SAMPLES_RANK1)
    return fail(FF_ERR_INVALID_ARG, "the Marginal and Input estimators need the rank-one form");
  if (c->m > (1 << 20) || c->n > (1 << 20))
    return fail(FF_ERR_INVALID_ARG, "m and n must be <= 1048576");
  if (is_bf16(c) && c->whiten_split != 0 && c->whiten_split != 1 && c->whiten_split != 2)
    return fail(FF_ERR_INVALID_ARG, "whiten_split must be 0 (automatic), 1 or 2");
  return FF_OK;
}

Layout make_layout(const ff_config* c) {
  Layout L{};
  const int g = granule(c), e = elem_bytes(c);
  const int64_t m = c->m, n = c->n, N = c->N;
  L.m_p = round_up(m, g);
  L.n_p = round_up(n, g);
  L.rank1 = c->form == FF_SAMPLES_RANK1;
  L.own_gx = L.rank1 || !(L.m_p == m && L.n_p == n);
  L.T_p = L.rank1 ? round_up(N, 256) : 0;  // a multiple of the token segment (and of g)
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes);
    return o;
  };
  L.off_small = take(kAlign);  // status[4] @0, c @64, trA @128, trB @192
  L.off_ll = take(sizeof(double) * kLLCap);
  // relative changes (kLLCap), their partial sums (8 per workgroup) and the
  // damped trace term's partial sums (2 per workgroup)
  L.off_diag = take(sizeof(double) * (kLLCap + 10 * kDiagBlocks));
  L.off_slotsA = take(sizeof(double) * ((n + kLeaf - 1) / kLeaf));
  L.off_slotsB = take(sizeof(double) * ((m + kLeaf - 1) / kLeaf));
  const int64_t dmax = std::max(L.m_p, L.n_p);
  if (L.rank1) {
    L.off_gx = take((size_t)L.T_p * L.n_p * e);
    L.off_gt = take((size_t)L.T_p * L.m_p * e);
    L.w_bytes = std::max(is_bf16(c) ? (size_t)L.T_p * 2 * (dmax / kTileBF16) * sizeof(float)
                                    : (size_t)L.T_p * dmax * sizeof(float),
                         (size_t)m * n * sizeof(float));
    L.off_w = take(L.w_bytes);
    L.off_s = take((size_t)dmax * L.T_p * e);
    L.off_wv = take(2 * (size_t)L.T_p * sizeof(float));
  } else {
    const size_t gbytes = (size_t)N * L.m_p * L.n_p * e;
    L.off_gx = L.own_gx ? take(gbytes) : 0;
    L.off_gt = take(gbytes);
    L.w_bytes = std::max(gbytes, (size_t)m * n * sizeof(float));
    L.off_w = take(L.w_bytes);
  }
  // k depth of the symmetric products: the stacked samples, or the tokens
  const int64_t kB = L.rank1 ? L.T_p : N * L.n_p, kA = L.rank1 ? L.T_p : N * L.m_p;
  if (is_bf16(c)) {
    L.splitsB = choose_splits_bf16(L.m_p, kB / 64);
    L.splitsA = choose_splits_bf16(L.n_p, kA / 64);
    const int64_t TB = L.m_p / kTileBF16, TA = L.n_p / kTileBF16;
    L.partialB = (size_t)L.splitsB * (TB * (TB + 1) / 2) * kTileBF16 * kTileBF16;
    L.partialA = (size_t)L.splitsA * (TA * (TA + 1) / 2) * kTileBF16 * kTileBF16;
  } else {
    L.splitsB = choose_splits_f32(L.m_p, kB);
    L.splitsA = choose_splits_f32(L.n_p, kA);
    L.partialB = (size_t)L.splitsB * L.m_p * L.m_p;
    L.partialA = (size_t)L.splitsA * L.n_p * L.n_p;
  }
  L.off_p = take(sizeof(float) * std::max(L.partialA, L.partialB));
  const bool split2 = is_bf16(c) && c->whiten_split != 1;  // 2, or automatic
  // automatic split: per side a flag and its statistic (256 bytes) and the
  // statistic's partial sums
  L.off_split = split2 && c->whiten_split == 0
                    ? take(2 * (kAlign + align_up(sizeof(double) * convert_parts(dmax))))
                    : 0;
  auto side = [&](size_t* o, int64_t dim, int64_t dim_p) {
    const size_t fb = (size_t)dim * dim * sizeof(float);
    o[0] = take(fb);
    o[1] = take(fb);
    o[2] = take(fb);
    o[3] = take(fb);
    o[4] = take((size_t)dim_p * dim_p * e);
    o[5] = split2 ? take((size_t)dim_p * dim_p * 2) : 0;
  };
  side(L.off_A, n, L.n_p);
  side(L.off_B, m, L.m_p);
  L.total = off;
  return L;
}

}  // namespace

struct ff_handle_s {
  ff_config cfg{};
  hipStream_t stream = nullptr;
  hipStream_t aux = nullptr;            // second stream of ff_quantize (created on first use)
  hipEvent_t fork = nullptr, join = nullptr;
  int device = 0;
  int64_t m = 0, n = 0, N = 0;
  bool bf16 = false;
  int elem = 4;
  Layout lay{};
  const void* Gx = nullptr;
  void* Gt = nullptr;
  void* W = nullptr;
  float* P = nullptr;
  void* S = nullptr;      // rank-one form: weighted transposed tokens
  float* wv = nullptr;    // rank-one form: token weights (2 x T_p)
  Side A, B;
  int* st = nullptr;
  double* c = nullptr;
  double* ll = nullptr;
  double* delta = nullptr;   // relative change of A (x) B per iteration (ring of kLLCap)
  double* dpart = nullptr;   // its partial sums
  double* spart = nullptr;   // partial sums of the damped log-likelihood's trace term
  bool single_stream = false;  // no second stream: the inverse tree runs on the main stream
  int64_t iters_total = 0;
  int cur = 0;
  // measurement hook
  bool timing = false;
  std::vector<hipEvent_t> events;
  size_t ev_used = 0;
  struct Pending { int kernel; size_t ev; double flop; };
  std::vector<Pending> pending;
  int64_t t_launches[kTimedKernels] = {};
  double t_ms[kTimedKernels] = {};
  double t_flop[kTimedKernels] = {};
};

namespace {

// ------------------------------------------------------------------ timing
struct Timed {
  ff_handle_s* h;
  int kernel;
  double flop;
  size_t ev = SIZE_MAX;
  Timed(ff_handle_s* hh, int k, double f) : h(hh), kernel(k), flop(f) {
    if (h->timing && h->ev_used + 2 <= h->events.size()) {
      ev = h->ev_used;
      h->ev_used += 2;
      // a failed record only loses this measurement; a broken stream shows
      // at the call's next checked launch
      (void)hipEventRecord(h->events[ev], h->stream);
    }
  }
  ~Timed() {
    if (ev != SIZE_MAX) {
      (void)hipEventRecord(h->events[ev + 1], h->stream);
      h->pending.push_back({kernel, ev, flop});
    }
  }
};

void collect_timing(ff_handle_s* h) {
  for (const auto& p : h->pending) {
    float ms = 0.0f;
    if (hipEventElapsedTime(&ms, h->events[p.ev], h->events[p.ev + 1]) == hipSuccess) {
      h->t_launches[p.kernel] += 1;
      h->t_ms[p.kernel] += ms;
      h->t_flop[p.kernel] += p.flop;
    }
  }
  h->pending.clear();
  h->ev_used = 0;
}

// ------------------------------------------------------- factorisation
ff_status side_streams(Side& s) {
  if (s.istream == nullptr) {
    FF_HIP(hipStreamCreateWithFlags(&s.istream, hipStreamNonBlocking));
    FF_HIP(hipEventCreateWithFlags(&s.ev_leaf, hipEventDisableTiming));
    FF_HIP(hipEventCreateWithFlags(&s.ev_inv, hipEventDisableTiming));
  }
  return FF_OK;
}

// Off-diagonal blocks of L^-1 for the node [o, o + sz) of the leaf tree, on
// stream st, in two products: P1, T^T = (L21 Li11)^T, parked in the node's
// block above the diagonal of s.L, needs the left half done (its inverse and
// the panels below it); P2, Li21 = -Li22 T, needs the right half's inverse
// too.  64 x 64 tiles below 2048 rows: with one operand triangular, 128 x 128
// tiles leave a few long workgroups to finish alone.
struct TreeNode {
  int64_t hh, r;
  float *L21, *Li11, *Li21, *Li22, *Tt;
};

TreeNode tree_node(Side& s, int64_t o, int64_t sz) {
  const int64_t d = s.dim;
  const int64_t nl = (sz + kLeaf - 1) / kLeaf;
  TreeNode t;
  t.hh = (nl + 1) / 2 * kLeaf;
  t.r = sz - t.hh;
  t.L21 = s.L + (o + t.hh) * d + o;
  t.Li11 = s.Li + o * d + o;
  t.Li21 = s.Li + (o + t.hh) * d + o;
  t.Li22 = s.Li + (o + t.hh) * d + (o + t.hh);
  t.Tt = s.L + o * d + (o + t.hh);
  return t;
}

GemmF32 tree_gemm(ff_handle_s* h, Side& s, const TreeNode& t) {
  GemmF32 g{};
  g.tile = t.hh < 2048 ? 64 : 0;
  g.lda = g.ldb = g.ldc = s.dim;
  g.kseg = INT64_MAX / 4;
  g.ksplit = 1;
  g.st = h->st;
  return g;
}

ff_status inverse_p1(ff_handle_s* h, Side& s, int64_t o, int64_t sz, hipStream_t st) {
  const TreeNode t = tree_node(s, o, sz);
  GemmF32 g = tree_gemm(h, s, t);
  // T^T = (L21 Li11)^T = Li11^T L21^T  (hh x r)
  g.A = t.Li11; g.B = t.L21; g.C = t.Tt; g.M = t.hh; g.N = t.r; g.K = t.hh;
  g.transA = 1; g.transB = 1; g.alpha = 1.f; g.beta = 0.f; g.flags = kKLoRow;
  FF_HIP(launch_gemm_f32(g, 1, st));
  return FF_OK;
}

ff_status inverse_p2(ff_handle_s* h, Side& s, int64_t o, int64_t sz, hipStream_t st) {
  const TreeNode t = tree_node(s, o, sz);
  GemmF32 g = tree_gemm(h, s, t);
  // Li21 = -Li22 T
  g.A = t.Li22; g.B = t.Tt; g.C = t.Li21; g.M = t.r; g.N = t.hh; g.K = t.r;
  // up to 2048 columns 64 x 64 tiles here too: the root's second product of
  // a 4096 factor runs alone after the last leaf, and with 128 x 128 tiles
  // its workgroups of the last row block (k = 2048) finish long after the rest
  if (t.hh <= 2048) g.tile = 64;
  g.transA = 0; g.transB = 1; g.alpha = -1.f; g.beta = 0.f; g.flags = kKHiRow;
  FF_HIP(launch_gemm_f32(g, 1, st));
  return FF_OK;
}

// Enqueue, in post order, P2 of every node of [o, o + sz) whose last leaf is
// leaf `last` (children first).
ff_status inverse_p2_ending(ff_handle_s* h, Side& s, int64_t o, int64_t sz, int64_t last,
                            hipStream_t st) {
  if (sz <= kLeaf) return FF_OK;
  const int64_t nl = (sz + kLeaf - 1) / kLeaf;
  const int64_t hh = (nl + 1) / 2 * kLeaf;
  const int64_t end_leaf = (o + sz - 1) / kLeaf;
  ff_status rc;
  if (last < (o + hh) / kLeaf) return inverse_p2_ending(h, s, o, hh, last, st);
  if ((rc = inverse_p2_ending(h, s, o + hh, sz - hh, last, st)) != FF_OK) return rc;
  if (end_leaf == last) return inverse_p2(h, s, o, sz, st);
  return FF_OK;
}

// Enqueue P1 of the node of [o, o + sz) whose left half ends with leaf k
// (every leaf but the last ends the left half of exactly one node).
ff_status inverse_p1_split(ff_handle_s* h, Side& s, int64_t o, int64_t sz, int64_t k,
                           hipStream_t st) {
  if (sz <= kLeaf) return FF_OK;
  const int64_t nl = (sz + kLeaf - 1) / kLeaf;
  const int64_t hh = (nl + 1) / 2 * kLeaf;
  const int64_t split = (o + hh) / kLeaf - 1;
  if (k == split) return inverse_p1(h, s, o, sz, st);
  if (k < split) return inverse_p1_split(h, s, o, hh, k, st);
  return inverse_p1_split(h, s, o + hh, sz - hh, k, st);
}

// Cholesky factor L (lower, in place in s.L) and its inverse (s.Li) of the
// matrix in s.L: right-looking over 128-column panels, two launches per
// panel k on the main stream: the panel L_ik = A_ik L_kk^-T (in place), then
// one step kernel in which one workgroup factors and inverts diagonal block
// k + 1 (after applying the panel's update to it) while the others apply the
// panel's update to the rest of the trailing lower triangle.  (Trailing
// updates on a second stream, overlapping the diagonal blocks, delayed the
// small kernels on the critical path instead: concurrent kernels share the
// CUs.)  Factors wider than kTwoLevel go in outer panels of kOuter columns:
// the steps update only the outer panel's columns, and one large product
// applies the outer panel's rank-kOuter update to the rest (rank-128 updates
// of a large matrix are bound by its reads and writes).  The off-diagonal
// blocks of L^-1 are built on a second stream from the binary tree of
// leaves, each node's first product as soon as its left half and its panels
// are done, its second when its last leaf is; the work is handed over every
// kInvEvery panels (an event on the main stream costs a few microseconds
// there), and every second panel near the end, where what is still undone
// after the last leaf is the factorisation's tail.  The upper triangle of
// s.L is scratch.
constexpr int64_t kInvEvery = 8;
constexpr int64_t kTwoLevel = 6144;
constexpr int64_t kOuter = 2048;

ff_status chol_blocked(ff_handle_s* h, Side& s, int iteration) {
  // One stream (h->single_stream): the inverse products go on the main
  // stream in the same order, after the panels they need.
  const bool two = !h->single_stream;
  ff_status rc = two ? side_streams(s) : FF_OK;
  if (rc != FF_OK) return rc;
  const int64_t d = s.dim;
  const int64_t nb = (d + kLeaf - 1) / kLeaf;
  const int64_t outer = d > kTwoLevel ? kOuter : nb * kLeaf;
  hipStream_t ms = h->stream;
  hipStream_t is = two ? s.istream : ms;
  // the inverse stream starts after the work already on the main stream
  if (two) {
    FF_HIP(hipEventRecord(s.ev_leaf, ms));
    FF_HIP(hipStreamWaitEvent(is, s.ev_leaf, 0));
  }
  int64_t handed = 0;  // leaves whose inverse products are enqueued
  // Leaves [handed, upto] are done, and the panel below leaf upto too when
  // panel_done (all earlier panels are).
  auto hand_over = [&](int64_t upto, bool panel_done) -> ff_status {
    if (two) {
      FF_HIP(hipEventRecord(s.ev_leaf, ms));
      FF_HIP(hipStreamWaitEvent(is, s.ev_leaf, 0));
    }
    for (int64_t j = handed; j <= upto; ++j) {
      ff_status r2 = inverse_p2_ending(h, s, 0, d, j, is);
      if (r2 != FF_OK) return r2;
      if (j + 1 < nb && (panel_done || j < upto)) {
        r2 = inverse_p1_split(h, s, 0, d, j, is);
        if (r2 != FF_OK) return r2;
      }
    }
    handed = upto + 1;
    return FF_OK;
  };
  for (int64_t p = 0; p < d; p += outer) {
    const int64_t pe = std::min(p + outer, d);
    // the outer panel's first diagonal block has every earlier update
    FF_HIP(launch_chol_step(s.L, s.Li, d, p, -1, 0, s.slots, iteration, s.code, h->st, ms));
    for (int64_t o = p; o + kLeaf < pe || (o + kLeaf < d && o + kLeaf == pe); o += kLeaf) {
      const int64_t k = o / kLeaf, rest = d - o - kLeaf;
      // the panel L_ik = A_ik Li_kk^T, in place
      FF_HIP(launch_panel_solve(s.L + (o + kLeaf) * d + o, s.Li + o * d + o, d, rest, h->st, ms));
      // every kInvEvery panels, and every second one among the last
      // kInvEvery and the one before the last leaf (the last steps leave most
      // CUs idle for the tree's products)
      const bool tail = k + 1 + kInvEvery >= nb && ((k + 1) % 2 == 0 || k + 2 == nb);
      if (((k + 1) % kInvEvery == 0 || tail) && (rc = hand_over(k, true)) != FF_OK) return rc;
      if (o + kLeaf == pe) break;  // the last panel of the outer panel
      // diagonal block k + 1 and the panel's update of the outer panel's columns
      FF_HIP(launch_chol_step(s.L, s.Li, d, o + kLeaf, o, pe, s.slots, iteration, s.code, h->st, ms));
    }
    if (pe < d) {
      // A_22 -= L_21 L_21^T over the outer panel's columns
      GemmF32 g{};
      g.lda = g.ldb = g.ldc = d;
      g.kseg = INT64_MAX / 4;
      g.ksplit = 1;
      g.st = h->st;
      g.A = s.L + pe * d + p; g.B = g.A; g.C = s.L + pe * d + pe;
      g.M = d - pe; g.N = d - pe; g.K = pe - p;
      g.transA = 0; g.transB = 1; g.alpha = -1.f; g.beta = 1.f; g.flags = kCLower;
      FF_HIP(launch_gemm_f32(g, 1, ms));
    }
  }
  if ((rc = hand_over(nb - 1, false)) != FF_OK) return rc;
  if (two) {
    FF_HIP(hipEventRecord(s.ev_inv, is));
    FF_HIP(hipStreamWaitEvent(ms, s.ev_inv, 0));
  }
  return FF_OK;
}

// Automatic split (whiten_split = 0): whiten with the hi + lo bf16 parts of
// L^-1 while s = (1/dim) sum_j F_jj (F^-1)_jj of either factor exceeds this,
// i.e. when the rms distortion 2^-9 sqrt(s/3) of the whitened metric by the
// bf16 rounding of that factor's L^-1 would exceed about 4.5e-3.  Measured
// (bf16 against fp32 / split 2 after the workloads' iteration counts): the
// 4096 x 4096 layer (s(A) = 6.1) 2.5e-4, 11008 x 4096 (7.4) 4.2e-4,
// 4096 x 11008 (13) 3.5e-4 with one pass; the 8192 x 28672 layer
// (s(A) = 21) 2.4e-3 and a 512 x 1280 layer from 4 samples (s(A) up to 26)
// 7.9e-3 with one pass, which the second pass removes.
constexpr double kSplitThreshold = 16.0;
// Automatic split, shape rule: the whitening's rounding perturbs every
// sample's term alike, and the iteration amplifies that perturbation the
// more, the fewer samples determine each factor.  Across the measured cases
// the one-pass error follows r = min(N m / n, N n / m) (rank-one form:
// T / max(m, n)), samples per dimension of the less determined factor,
// rather than s: r = 128, 48, 24 (the three widest-sampled layers) gave
// 2.4e-4 to 4.2e-4, while r = 11 (768 x 512, 16 samples; s <= 4.6) gave
// 1.1e-3, r = 6 (11008 x 4096, 16 samples; s <= 15.5) 3.4e-3 against 2.8e-4
// with two passes, r = 1.6 (512 x 1280, 4 samples) 7.9e-3.  Below this r
// both whitenings always use two passes.
constexpr double kMinSamplesPerDim = 16.0;

// Samples per dimension of the less determined factor (see above).
double samples_per_dim(const ff_handle_s* h) {
  const double m = (double)h->m, n = (double)h->n, N = (double)h->N;
  if (h->lay.rank1) return N / std::max(m, n);
  return N * std::min(m, n) / std::max(m, n);
}

// L^-1 of the dim x dim factor at src into s.Li and the whitening operand
// s.Lw; sum log L_jj per leaf into s.slots.
ff_status cholinv_from(ff_handle_s* h, Side& s, const float* src, int iteration) {
  Timed t(h, 3, (double)s.dim * s.dim * s.dim / 3.0);
  FF_HIP(launch_copy_f32(src, s.L, s.dim * s.dim, h->st, h->stream));
  ff_status rc = chol_blocked(h, s, iteration);
  if (rc != FF_OK) return rc;
  FF_HIP(launch_convert_inverse(s.Li, s.dim, s.Lw, s.Lw2, s.dim_p, h->elem, src, s.spart, h->st,
                                h->stream));
  if (s.split_flag != nullptr) {
    FF_HIP(launch_split_decide(s.spart, s.dim, s.dim_p, kSplitThreshold, s.split_flag,
                               s.split_stat, h->st, h->stream));
    s.stat_known = true;
  }
  return FF_OK;
}

ff_status cholinv(ff_handle_s* h, Side& s, int slot, int iteration) {
  return cholinv_from(h, s, s.F[slot], iteration);
}

// Frobenius estimator: the half steps B = (1/(N n)) sum_i G_i A G_i^T and
// A = (1/(N m)) sum_i G_i^T B G_i use the factor itself, so the operand is F
// rounded to the samples' type (dense, both triangles; hi + lo parts with
// whiten_split = 2): the products P_i = G_i F and then the symmetric
// sum_i P_i G_i^T need no factorisation, so a factor of any condition
// number (the undamped power iteration's estimates lose rank quickly) is
// handled as the oracle handles it.
ff_status frob_operand(ff_handle_s* h, Side& s, const float* src) {
  Timed t(h, 3, 0.0);
  FF_HIP(launch_convert_inverse(src, s.dim, s.Lw, s.Lw2, s.dim_p, h->elem, nullptr, nullptr, h->st,
                                h->stream, 1));
  return FF_OK;
}

// The whitening operand of the estimator for factor s.F[slot].
ff_status operand(ff_handle_s* h, Side& s, int slot, int iteration) {
  if (h->cfg.estimator == FF_EST_FROBENIUS) return frob_operand(h, s, s.F[slot]);
  return cholinv(h, s, slot, iteration);
}

// The low bf16 part of side p's whitening operand for the whitening kernels
// (nullptr: one pass) and, with the automatic split, the two device flags
// (one per factor) that decide between one and two passes: two when either
// factor's latest statistic is above the threshold.  The distortion of the
// whitening by p's operand goes into the update of the other factor, whose
// own conditioning then amplifies it in its small eigenvalues (an
// 8192 x 28672 layer with s(A) = 21 and s(B) = 2.3 keeps a flat likelihood
// only with both whitenings split); and always two when few samples
// determine the factors (kMinSamplesPerDim).  The Frobenius operand is not
// an inverse, so the statistic does not apply to it: one pass.
const bf16_t* second_part(const ff_handle_s* h, const Side& p, const int** use2,
                          const int** use2b) {
  *use2 = *use2b = nullptr;
  if (p.Lw2 == nullptr) return nullptr;
  if (h->cfg.whiten_split == 2) return (const bf16_t*)p.Lw2;
  if (h->cfg.estimator == FF_EST_FROBENIUS) return nullptr;
  if (samples_per_dim(h) < kMinSamplesPerDim) return (const bf16_t*)p.Lw2;
  *use2 = h->A.split_flag;
  *use2b = h->B.split_flag;
  return (const bf16_t*)p.Lw2;
}

// Rank-one form: token weights wbuf[t] = ||L_p^-1 v_t||^2 for the token
// vectors v_t of side p's dimension (x_t when p = A, g_t when p = B); for
// the Frobenius estimator v_t^T F_p v_t, from P = V F_p and a row-wise dot
// product with V.
ff_status token_weights(ff_handle_s* h, Side& p, float* wbuf) {
  const void* V = (&p == &h->A) ? h->Gx : h->Gt;
  const int64_t T_p = h->lay.T_p, Kp = p.dim_p;
  const bool frob = h->cfg.estimator == FF_EST_FROBENIUS;
  const double wflop = (frob ? 2.0 : 1.0) * (double)h->N * p.dim * p.dim;
  Timed t(h, 0, wflop);
  if (frob) {
    // P goes into the weighted-token buffer, which is free until the weights exist
    void* P = h->bf16 ? h->S : h->W;
    if (h->bf16) {
      const bf16_t* Y2 = h->cfg.whiten_split == 2 ? (const bf16_t*)p.Lw2 : nullptr;
      FF_HIP(launch_whiten_bf16((const bf16_t*)V, (const bf16_t*)p.Lw, Y2, nullptr, nullptr,
                                (bf16_t*)P, T_p, Kp, h->st, h->stream, true));
    } else {
      GemmF32 g{};
      g.st = h->st;
      g.ksplit = 1;
      g.kseg = Kp;
      g.A = (const float*)V; g.lda = Kp; g.transA = 0;
      g.B = (const float*)p.Lw; g.ldb = Kp; g.transB = 1;
      g.C = (float*)P; g.ldc = Kp;
      g.M = T_p; g.N = Kp; g.K = Kp;
      g.alpha = 1.f; g.beta = 0.f; g.flags = 0;
      FF_HIP(launch_gemm_f32(g, 1, h->stream));
    }
    FF_HIP(launch_row_dot(P, V, T_p, Kp, h->elem, wbuf, h->st, h->stream));
    return FF_OK;
  }
  if (h->bf16) {
    const int *use2 = nullptr, *use2b = nullptr;
    const bf16_t* Y2 = second_part(h, p, &use2, &use2b);
    FF_HIP(launch_whiten_norm_bf16((const bf16_t*)V, (const bf16_t*)p.Lw, Y2, use2, use2b,
                                   (float*)h->W, T_p, Kp, h->st, h->stream));
    FF_HIP(launch_row_sums((const float*)h->W, T_p, 2 * (Kp / kTileBF16), 0, wbuf, h->st,
                           h->stream));
  } else {
    GemmF32 g{};
    g.st = h->st;
    g.ksplit = 1;
    g.kseg = Kp;
    g.A = (const float*)V; g.lda = Kp; g.transA = 0;
    g.B = (const float*)p.Lw; g.ldb = Kp; g.transB = 1;
    g.C = (float*)h->W; g.ldc = Kp;
    g.M = T_p; g.N = Kp; g.K = Kp;
    g.alpha = 1.f; g.beta = 0.f; g.flags = kKHiCol;
    FF_HIP(launch_gemm_f32(g, 1, h->stream));
    FF_HIP(launch_row_sums((const float*)h->W, T_p, Kp, 1, wbuf, h->st, h->stream));
  }
  return FF_OK;
}

// Rank-one form of the half step (Section 5): s.F[slot] =
// (1/(N p.dim)) sum_t ||L_p^-1 v_t||^2 u_t u_t^T with u_t the token vector of
// side s, as a symmetric product over tokens of the weighted, transposed u.
// unit: all weights 1 and scale 1/N (the token mean E[u u^T] of the Marginal
// and Input estimators, Table 1).
ff_status update_rank1(ff_handle_s* h, Side& s, Side& p, int slot, bool finish,
                       bool unit = false, float* dst = nullptr) {
  float* F = dst != nullptr ? dst : s.F[slot];
  float* wbuf = h->wv;
  const int64_t T_p = h->lay.T_p;
  if (unit) {
    FF_HIP(launch_fill_f32(wbuf, T_p, 1.0f, h->stream));
  } else {
    ff_status rc = token_weights(h, p, wbuf);
    if (rc != FF_OK) return rc;
  }
  const void* U = (&s == &h->B) ? h->Gt : h->Gx;
  const double scale = unit ? 1.0 / (double)h->N : 1.0 / ((double)h->N * (double)p.dim);
  const double sflop = (double)h->N * s.dim * s.dim;
  // tokens in segments of kTokenSeg: the product streams short rows
  const int64_t seg = kTokenSeg, nseg = T_p / kTokenSeg;
  {
    Timed t(h, 2, 0.0);
    FF_HIP(launch_scale_transpose(U, wbuf, T_p, s.dim_p, seg, h->S, h->elem, h->st, h->stream));
  }
  if (h->bf16) {
    {
      Timed t(h, 1, sflop);
      FF_HIP(launch_syrk_bf16((const bf16_t*)h->S, s.dim_p, seg, s.dim_p * seg, nseg, s.splits,
                              h->P, h->st, h->stream));
    }
    Timed t(h, 2, 0.0);
    FF_HIP(launch_reduce_frag(h->P, s.splits, s.dim_p, F, s.dim, scale, h->st, h->stream));
  } else {
    {
      Timed t(h, 1, sflop);
      GemmF32 q{};
      q.st = h->st;
      q.A = (const float*)h->S; q.lda = seg; q.transA = 0;
      q.B = (const float*)h->S; q.ldb = seg; q.transB = 1;
      q.C = h->P; q.ldc = s.dim_p; q.sC = s.dim_p * s.dim_p;
      q.M = s.dim_p; q.N = s.dim_p; q.K = T_p;
      q.kseg = seg; q.segA = q.segB = s.dim_p * seg;
      q.alpha = 1.f; q.beta = 0.f; q.flags = kCLower; q.ksplit = s.splits;
      FF_HIP(launch_gemm_f32(q, 1, h->stream));
    }
    Timed t(h, 2, 0.0);
    FF_HIP(launch_reduce_rowmajor(h->P, s.splits, s.dim_p, F, s.dim, scale, h->st, h->stream));
  }
  if (finish) FF_HIP(launch_trace_damp(F, s.dim, h->cfg.damping, s.tr, h->st, h->stream));
  return FF_OK;
}

// s.F[slot] (or dst) = (1/(N p.dim)) sum_i X_i Li_p^T Li_p X_i^T  (+ damping), trace into
// s.tr; with finish = false, without damping and trace.  p_identity: p's
// factor is exactly I (the default start), so Li_p = I and the whitened
// samples are the samples themselves (bitwise: a product with I is exact);
// the symmetric product then reads X directly.  Frobenius estimator:
// (1/(N p.dim)) sum_i (X_i F_p) X_i^T, the dense product P = X F_p first
// (twice the whitening's work), then the upper tiles of P X^T.
ff_status update(ff_handle_s* h, Side& s, Side& p, int slot, bool finish = true,
                 bool p_identity = false, float* dst = nullptr) {
  if (h->lay.rank1) return update_rank1(h, s, p, slot, finish, false, dst);
  float* F = dst != nullptr ? dst : s.F[slot];
  const void* X = (&s == &h->B) ? h->Gx : h->Gt;
  const int64_t N = h->N, rows = N * s.dim_p, Kp = p.dim_p;
  const double scale = 1.0 / ((double)N * (double)p.dim);
  const bool frob = h->cfg.estimator == FF_EST_FROBENIUS && !p_identity;
  const double wflop = (frob ? 2.0 : 1.0) * (double)N * s.dim * p.dim * p.dim;
  const double sflop = (double)N * p.dim * s.dim * s.dim;
  const void* Wsrc = p_identity ? X : (const void*)h->W;
  if (h->bf16) {
    if (!p_identity) {
      Timed t(h, 0, wflop);
      const int *use2 = nullptr, *use2b = nullptr;
      const bf16_t* Y2 = second_part(h, p, &use2, &use2b);
      FF_HIP(launch_whiten_bf16((const bf16_t*)X, (const bf16_t*)p.Lw, Y2, use2, use2b,
                                (bf16_t*)h->W, rows, Kp, h->st, h->stream, frob));
    }
    {
      Timed t(h, 1, sflop);
      FF_HIP(launch_syrk_bf16((const bf16_t*)Wsrc, s.dim_p, Kp, s.dim_p * Kp, N, s.splits, h->P,
                              h->st, h->stream, frob ? (const bf16_t*)X : nullptr));
    }
    {
      Timed t(h, 2, 0.0);
      FF_HIP(launch_reduce_frag(h->P, s.splits, s.dim_p, F, s.dim, scale, h->st, h->stream));
    }
  } else {
    GemmF32 g{};
    g.st = h->st;
    g.ksplit = 1;
    if (!p_identity) {
      Timed t(h, 0, wflop);
      g.A = (const float*)X; g.lda = Kp; g.transA = 0;
      g.B = (const float*)p.Lw; g.ldb = Kp; g.transB = 1;
      g.C = (float*)h->W; g.ldc = Kp;
      g.M = rows; g.N = Kp; g.K = Kp; g.kseg = Kp;
      g.alpha = 1.f; g.beta = 0.f; g.flags = frob ? 0 : kKHiCol;
      FF_HIP(launch_gemm_f32(g, 1, h->stream));
    }
    {
      Timed t(h, 1, sflop);
      GemmF32 q{};
      q.st = h->st;
      q.A = (const float*)Wsrc; q.lda = Kp; q.transA = 0;
      q.B = (const float*)(frob ? X : Wsrc); q.ldb = Kp; q.transB = 1;
      q.C = h->P; q.ldc = s.dim_p; q.sC = s.dim_p * s.dim_p;
      q.M = s.dim_p; q.N = s.dim_p; q.K = N * Kp;
      q.kseg = Kp; q.segA = q.segB = s.dim_p * Kp;
      q.alpha = 1.f; q.beta = 0.f; q.flags = kCLower; q.ksplit = s.splits;
      FF_HIP(launch_gemm_f32(q, 1, h->stream));
    }
    {
      Timed t(h, 2, 0.0);
      FF_HIP(launch_reduce_rowmajor(h->P, s.splits, s.dim_p, F, s.dim, scale, h->st, h->stream));
    }
  }
  if (finish) FF_HIP(launch_trace_damp(F, s.dim, h->cfg.damping, s.tr, h->st, h->stream));
  return FF_OK;
}

ff_status read_status(ff_handle_s* h, int st[4]) {
  FF_HIP(hipMemcpyAsync(st, h->st, 4 * sizeof(int), hipMemcpyDeviceToHost, h->stream));
  FF_HIP(hipStreamSynchronize(h->stream));
  return FF_OK;
}

ff_status clear_status(ff_handle_s* h) {
  FF_HIP(launch_set_int(h->st, 4, 0, h->stream));
  return FF_OK;
}

// Relative change of A (x) B between the iterate in `slot` and the one
// before it (fp64 on the device, into h->delta[k]); with tol > 0 a change
// <= tol sets st[3] = g and the rest of the enqueued pipeline halts.
ff_status enqueue_delta(ff_handle_s* h, int slot, int k, int64_t g, double tol) {
  FF_HIP(launch_delta(h->A.F[slot], h->A.F[slot ^ 1], h->n * h->n, h->B.F[slot], h->B.F[slot ^ 1],
                      h->m * h->m, h->dpart, h->delta + k, tol, (int)g, h->st, h->stream));
  return FF_OK;
}

// After the chunk's single synchronisation: the number of iterations that
// completed (a failing factorisation, st[0], or the tolerance, st[3]), the
// host copies of the per-iteration outputs, and the handle's counters.
// Returns the status to report; *converged is set when the tolerance stopped
// the chunk, *failed when a factorisation failed (both cached whitening
// operands are then stale).
ff_status finish_chunk(ff_handle_s* h, int64_t base, int iters, int* done, double* loglik,
                       double* delta, bool has_loglik, bool* converged, bool* failed) {
  int st[4];
  ff_status rc = read_status(h, st);
  if (rc != FF_OK) return rc;
  if (h->timing) collect_timing(h);
  int completed = iters;
  *converged = false;
  *failed = st[0] != 0;
  if (st[0] != 0) {
    completed = (int)std::max<int64_t>(0, std::min<int64_t>(iters, st[0] - 1 - base));
  } else if (st[3] != 0) {
    completed = (int)std::max<int64_t>(0, std::min<int64_t>(iters, st[3] - base));
    *converged = true;
  }
  if (completed > 0) {
    if (loglik != nullptr) {
      if (has_loglik)
        FF_HIP(hipMemcpy(loglik, h->ll, sizeof(double) * completed, hipMemcpyDeviceToHost));
      else
        for (int k = 0; k < completed; ++k) loglik[k] = NAN;
    }
    if (delta != nullptr)
      FF_HIP(hipMemcpy(delta, h->delta, sizeof(double) * completed, hipMemcpyDeviceToHost));
    if (st[0] != 0) {  // the closing factorisation of the last one failed
      if (loglik != nullptr) loglik[completed - 1] = NAN;
      if (delta != nullptr) delta[completed - 1] = NAN;
    }
  }
  h->iters_total = base + completed;
  h->cur = (int)(h->iters_total & 1);
  *done = completed;
  if (st[0] != 0 || st[3] != 0) {
    if ((rc = clear_status(h)) != FF_OK) return rc;
    FF_HIP(hipStreamSynchronize(h->stream));
  }
  if (st[0] != 0) {
    h->A.lw_valid = h->B.lw_valid = false;
    if (st[0] == base + iters + 1) return FF_OK;  // only the look-ahead failed
    char msg[160];
    snprintf(msg, sizeof msg, "factor %s not positive definite at iteration %d (pivot %d)",
             st[1] == 1 ? "A" : "B", st[0], st[2]);
    return fail(FF_ERR_NOT_SPD, msg);
  }
  return FF_OK;
}

// Up to kLLCap iterations; synchronises once.
//
// The factorisation of the second-updated factor that closes iteration g is
// the one iteration g + 1 needs, so its failure is attributed to g + 1:
// iteration g is complete (the oracle also returns such a singular factor),
// and only a later iteration that would invert it fails.
// Marginal / Input estimators (Table 1): token means, no factorisation.
ff_status iterate_means(ff_handle_s* h, int iters, int* done, double* loglik, double tol,
                        double* delta, bool* converged) {
  *done = 0;
  const int64_t base = h->iters_total;
  const bool want_delta = delta != nullptr || tol > 0.0;
  ff_status rc;
  for (int k = 1; k <= iters; ++k) {
    const int slot = (int)((base + k) & 1);
    if ((rc = update_rank1(h, h->A, h->B, slot, true, true)) != FF_OK) return rc;
    if (h->cfg.estimator == FF_EST_MARGINAL) {
      if ((rc = update_rank1(h, h->B, h->A, slot, true, true)) != FF_OK) return rc;
    } else {
      FF_HIP(launch_identity_f32(h->B.F[slot], h->m, h->stream));
      FF_HIP(launch_trace_damp(h->B.F[slot], h->m, h->cfg.damping, h->B.tr, h->st, h->stream));
    }
    FF_HIP(launch_normalise(h->A.F[slot], h->n, h->B.F[slot], h->m, h->A.tr, h->c, h->st,
                            h->stream));
    if (want_delta && (rc = enqueue_delta(h, slot, k - 1, base + k, tol)) != FF_OK) return rc;
  }
  bool failed = false;
  rc = finish_chunk(h, base, iters, done, loglik, delta, false, converged, &failed);
  h->A.lw_valid = h->B.lw_valid = false;
  return rc;
}

ff_status iterate_chunk(ff_handle_s* h, int iters, int* done, double* loglik, double tol,
                        double* delta, bool* converged) {
  if (h->cfg.estimator == FF_EST_MARGINAL || h->cfg.estimator == FF_EST_INPUT)
    return iterate_means(h, iters, done, loglik, tol, delta, converged);
  *done = 0;
  *converged = false;
  const bool bfirst = h->cfg.order == FF_ORDER_B_FIRST;
  const bool flipflop = h->cfg.estimator == FF_EST_FLIPFLOP;
  const bool want_delta = delta != nullptr || tol > 0.0;
  const double kappa = h->cfg.damping;
  Side& first = bfirst ? h->B : h->A;
  Side& second = bfirst ? h->A : h->B;
  const int64_t base = h->iters_total;
  ff_status rc;
  // Before the first iteration the factor updated second may still be the
  // default start I: its whitening operand is I, nothing to factorise or apply.
  const bool start_id = base == 0 && second.start_identity && !h->lay.rank1;
  if (!second.lw_valid && !start_id) {
    rc = operand(h, second, h->cur, (int)(base + 1));
    if (rc != FF_OK) return rc;
  }
  for (int k = 1; k <= iters; ++k) {
    const int64_t g = base + k;
    const int slot = (int)(g & 1);
    if ((rc = update(h, first, second, slot, true, start_id && k == 1)) != FF_OK) return rc;
    if ((rc = operand(h, first, slot, (int)g)) != FF_OK) return rc;
    if ((rc = update(h, second, first, slot)) != FF_OK) return rc;
    FF_HIP(launch_normalise(h->A.F[slot], h->n, h->B.F[slot], h->m, h->A.tr, h->c, h->st,
                            h->stream));
    if ((rc = operand(h, second, slot, (int)(g + 1))) != FF_OK) return rc;
    if (flipflop) {
      // with damping the trace term needs ||L^-1||_F^2 of the factor just factorised
      if (kappa > 0.0)
        FF_HIP(launch_sumsq_trace(second.Li, second.F[slot], second.dim, h->spart, h->st,
                                  h->stream));
      FF_HIP(launch_loglik(h->A.slots, h->A.nslots, h->B.slots, h->B.nslots, h->c, bfirst ? 1 : 0,
                           (double)h->m, (double)h->n, (double)h->N, kappa,
                           kappa > 0.0 ? h->spart : nullptr, h->ll + (k - 1), h->st, h->stream));
    }
    if (want_delta && (rc = enqueue_delta(h, slot, k - 1, g, tol)) != FF_OK) return rc;
  }
  bool failed = false;
  rc = finish_chunk(h, base, iters, done, loglik, delta, flipflop, converged, &failed);
  if (rc != FF_OK) return rc;
  // the look-ahead factorisation of the last completed iteration ran unless
  // a factorisation failed (then both cached operands are stale)
  if (!failed) second.lw_valid = true;
  return FF_OK;
}

// Chunks of at most kLLCap iterations (32 when timing, to bound the events
// in flight), each synchronised once; stops early when a chunk converged.
ff_status run_iterations(ff_handle_s* h, int iters, double tol, int* iters_done, double* loglik,
                         double* delta) {
  if (iters_done != nullptr) *iters_done = 0;
  if (h == nullptr) return fail(FF_ERR_INVALID_ARG, "handle is NULL");
  if (iters < 0) return fail(FF_ERR_INVALID_ARG, "iters must be >= 0");
  if (h->iters_total + (int64_t)iters > 0x7fffffffLL)
    return fail(FF_ERR_STATE, "iteration counter overflow");
  int total = 0;
  const int cap = h->timing ? 32 : kLLCap;
  while (total < iters) {
    const int chunk = std::min(cap, iters - total);
    int done = 0;
    bool converged = false;
    ff_status rc = iterate_chunk(h, chunk, &done, loglik ? loglik + total : nullptr, tol,
                                 delta ? delta + total : nullptr, &converged);
    total += done;
    if (iters_done != nullptr) *iters_done = total;
    if (rc != FF_OK || converged) return rc;
  }
  return FF_OK;
}

// Everything ff_init checks besides the workspace.
ff_status validate_config(const ff_config* cfg) {
  ff_status rc = validate_shape(cfg);
  if (rc != FF_OK) return rc;
  if (cfg->form == FF_SAMPLES_RANK1) {
    if (cfg->x == nullptr || cfg->g == nullptr || ((uintptr_t)cfg->x % 16) != 0 ||
        ((uintptr_t)cfg->g % 16) != 0)
      return fail(FF_ERR_INVALID_ARG, "x and g must be non-NULL 16-byte aligned device pointers");
  } else if (cfg->G == nullptr || ((uintptr_t)cfg->G % 16) != 0) {
    return fail(FF_ERR_INVALID_ARG, "G must be a non-NULL 16-byte aligned device pointer");
  }
  if (cfg->order != FF_ORDER_B_FIRST && cfg->order != FF_ORDER_A_FIRST)
    return fail(FF_ERR_INVALID_ARG, "unknown order");
  if (!(cfg->damping >= 0.0) || !isfinite(cfg->damping))
    return fail(FF_ERR_INVALID_ARG, "damping must be finite and >= 0");
  if (((uintptr_t)cfg->A0 % 16) != 0 || ((uintptr_t)cfg->B0 % 16) != 0)
    return fail(FF_ERR_INVALID_ARG, "A0/B0 must be 16-byte aligned");
  return FF_OK;
}

// Fill the handle for cfg over the workspace and enqueue the set-up.
ff_status init_handle(const ff_config* cfg, const Layout& lay, ff_handle_s* h) {
  h->cfg = *cfg;
  if (!is_bf16(cfg)) h->cfg.whiten_split = 1;
  h->stream = (hipStream_t)cfg->stream;
  h->m = cfg->m;
  h->n = cfg->n;
  h->N = cfg->N;
  h->bf16 = is_bf16(cfg);
  h->elem = elem_bytes(cfg);
  h->lay = lay;
  if (hipGetDevice(&h->device) != hipSuccess) return fail(FF_ERR_HIP, "hipGetDevice failed");
  char* ws = (char*)cfg->workspace;
  h->st = (int*)(ws + lay.off_small);
  h->c = (double*)(ws + lay.off_small + 64);
  h->A.tr = (double*)(ws + lay.off_small + 128);
  h->B.tr = (double*)(ws + lay.off_small + 192);
  h->ll = (double*)(ws + lay.off_ll);
  h->delta = (double*)(ws + lay.off_diag);
  h->dpart = h->delta + kLLCap;
  h->spart = h->dpart + 8 * kDiagBlocks;
  h->A.slots = (double*)(ws + lay.off_slotsA);
  h->B.slots = (double*)(ws + lay.off_slotsB);
  h->A.nslots = (int)((h->n + kLeaf - 1) / kLeaf);
  h->B.nslots = (int)((h->m + kLeaf - 1) / kLeaf);
  h->Gx = lay.own_gx ? (const void*)(ws + lay.off_gx) : cfg->G;
  h->Gt = ws + lay.off_gt;
  h->W = ws + lay.off_w;
  h->P = (float*)(ws + lay.off_p);
  if (lay.rank1) {
    h->S = ws + lay.off_s;
    h->wv = (float*)(ws + lay.off_wv);
  }
  auto side = [&](Side& s, const size_t* o, int64_t dim, int64_t dim_p, int splits, int code) {
    s.dim = dim;
    s.dim_p = dim_p;
    s.F[0] = (float*)(ws + o[0]);
    s.F[1] = (float*)(ws + o[1]);
    s.L = (float*)(ws + o[2]);
    s.Li = (float*)(ws + o[3]);
    s.Lw = ws + o[4];
    s.Lw2 = h->bf16 && h->cfg.whiten_split != 1 ? (void*)(ws + o[5]) : nullptr;
    if (h->bf16 && h->cfg.whiten_split == 0) {
      const int64_t dmax = std::max(lay.m_p, lay.n_p);
      char* b = ws + lay.off_split + (code - 1) * (kAlign + align_up(sizeof(double) * convert_parts(dmax)));
      s.split_flag = (int*)b;
      s.split_stat = (double*)(b + 64);
      s.spart = (double*)(b + kAlign);
    }
    s.splits = splits;
    s.code = code;
  };
  side(h->A, lay.off_A, h->n, lay.n_p, lay.splitsA, 1);
  side(h->B, lay.off_B, h->m, lay.m_p, lay.splitsB, 2);
  h->A.start_identity = cfg->A0 == nullptr;
  h->B.start_identity = cfg->B0 == nullptr;

  auto setup = [&]() -> ff_status {
    FF_HIP(launch_set_int(h->st, 4, 0, h->stream));
    const int64_t N = h->N, m = h->m, n = h->n;
    if (lay.rank1) {
      // tokens as one padded matrix each: x -> T_p x n_p, g -> T_p x m_p
      FF_HIP(launch_pack(cfg->x, (void*)h->Gx, 1, N, n, lay.T_p, lay.n_p, 0, h->elem, h->stream));
      FF_HIP(launch_pack(cfg->g, h->Gt, 1, N, m, lay.T_p, lay.m_p, 0, h->elem, h->stream));
    } else {
      if (lay.own_gx)
        FF_HIP(launch_pack(cfg->G, (void*)h->Gx, N, m, n, lay.m_p, lay.n_p, 0, h->elem, h->stream));
      FF_HIP(launch_pack(cfg->G, h->Gt, N, m, n, lay.n_p, lay.m_p, 1, h->elem, h->stream));
    }
    // automatic split: no factor is known to need the second pass yet
    if (h->A.split_flag != nullptr) {
      FF_HIP(launch_set_int(h->A.split_flag, 1, 0, h->stream));
      FF_HIP(launch_set_int(h->B.split_flag, 1, 0, h->stream));
    }
    // Upper blocks of L^-1 are never written by the factorisation: zero once.
    FF_HIP(launch_fill_f32(h->A.Li, n * n, 0.0f, h->stream));
    FF_HIP(launch_fill_f32(h->B.Li, m * m, 0.0f, h->stream));
    if (cfg->A0 != nullptr)
      FF_HIP(hipMemcpyAsync(h->A.F[0], cfg->A0, n * n * sizeof(float), hipMemcpyDeviceToDevice,
                            h->stream));
    else
      FF_HIP(launch_identity_f32(h->A.F[0], n, h->stream));
    if (cfg->B0 != nullptr)
      FF_HIP(hipMemcpyAsync(h->B.F[0], cfg->B0, m * m * sizeof(float), hipMemcpyDeviceToDevice,
                            h->stream));
    else
      FF_HIP(launch_identity_f32(h->B.F[0], m, h->stream));
    return FF_OK;
  };
  return setup();
}


// ------------------------------------------------------------ quantiser
struct QuantLayout {
  int MT, NT;
  int64_t mq, nq;
  size_t off_La, off_Lb, off_al, off_be, off_dA, off_dB, off_racc, off_pre, off_x, off_e, off_z,
      off_dpart, off_dist, total;
};

QuantLayout quant_layout(int64_t m, int64_t n) {
  QuantLayout q{};
  q.MT = (int)((m + kTileWK - 1) / kTileWK);
  q.NT = (int)((n + kTileWK - 1) / kTileWK);
  q.mq = (int64_t)q.MT * kTileWK;
  q.nq = (int64_t)q.NT * kTileWK;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes);
    return o;
  };
  const size_t tiles = (size_t)q.MT * q.NT * kTileWK * kTileWK * sizeof(float);
  q.off_La = take((size_t)q.nq * q.nq * sizeof(float));
  q.off_Lb = take((size_t)q.mq * q.mq * sizeof(float));
  q.off_al = take((size_t)q.nq * sizeof(float));
  q.off_be = take((size_t)q.mq * sizeof(float));
  q.off_dA = take((size_t)q.nq * sizeof(float));
  q.off_dB = take((size_t)q.mq * sizeof(float));
  q.off_racc = take(tiles);
  q.off_pre = take(tiles);
  q.off_x = take(tiles);
  q.off_e = take(tiles);
  q.off_z = take((size_t)q.mq * q.nq * sizeof(int32_t));
  q.off_dpart = take((size_t)q.MT * q.NT * sizeof(double));
  q.off_dist = take(sizeof(double));
  q.total = off;
  return q;
}

// Normalised inverse of RevCholesky(M) (padded), its diagonal and the padded
// scales of one side: J M J is factorised in s.L / s.Li.
ff_status quant_side(ff_handle_s* h, Side& s, const float* M, int64_t dq, float* Lt, float* diag,
                     double gamma, int given, float* user, float* scale) {
  FF_HIP(launch_wk_reverse(M, s.dim, s.L, h->st, h->stream));
  {
    Timed t(h, 3, (double)s.dim * s.dim * s.dim / 3.0);
    ff_status rc = chol_blocked(h, s, -1);
    if (rc != FF_OK) return rc;
  }
  FF_HIP(launch_wk_normalise(s.Li, s.dim, dq, Lt, diag, h->st, h->stream));
  FF_HIP(launch_wk_scales(diag, s.dim, dq, s.slots, s.nslots, gamma, given, user, scale, h->st,
                          h->stream));
  return FF_OK;
}

bool finite_positive(const float* dev, int64_t count, hipStream_t stream, std::string* why) {
  std::vector<float> host((size_t)count);
  if (hipMemcpyAsync(host.data(), dev, (size_t)count * sizeof(float), hipMemcpyDeviceToHost,
                     stream) != hipSuccess ||
      hipStreamSynchronize(stream) != hipSuccess) {
    *why = "copying the given scales failed";
    return false;
  }
  for (int64_t k = 0; k < count; ++k)
    if (!(host[(size_t)k] > 0.0f) || !isfinite(host[(size_t)k])) {
      *why = "given scales must be finite and > 0 (index " + std::to_string(k) + ")";
      return false;
    }
  return true;
}

}  // namespace

// ================================================= allocation-free scratch
// Device scratch of ff_fit_noalloc, for callers that cannot allocate device
// memory.  Each device the library runs on holds its own copy until the
// process ends.  In host code `scratch` is only a stand-in for the symbol:
// its device address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) unsigned char scratch[FF_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Address of the current device's copy of `scratch`.
ff_status scratch_on_current_device(void** out) {
  int dev = 0;
  FF_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(FF_ERR_INVALID_ARG, "device index out of range");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    FF_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (p == nullptr || ((uintptr_t)p % kAlign) != 0)
      return fail(FF_ERR_HIP, "device scratch has no usable address");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return FF_OK;
}
}  // namespace

// ====================================================================== ABI
extern "C" {

const char* ff_status_string(ff_status s) {
  switch (s) {
    case FF_OK: return "ok";
    case FF_ERR_INVALID_ARG: return "invalid argument";
    case FF_ERR_NOT_SPD: return "factor not positive definite";
    case FF_ERR_WORKSPACE: return "workspace missing, too small or misaligned";
    case FF_ERR_HIP: return "HIP runtime error";
    case FF_ERR_STATE: return "invalid handle state";
  }
  return "unknown status";
}

const char* ff_last_error(void) { return g_last_error.c_str(); }

ff_status ff_workspace_size(const ff_config* cfg, size_t* bytes) {
  ff_status rc = validate_shape(cfg);
  if (rc != FF_OK) return rc;
  if (bytes == nullptr) return fail(FF_ERR_INVALID_ARG, "bytes is NULL");
  *bytes = make_layout(cfg).total;
  return FF_OK;
}

ff_status ff_init(const ff_config* cfg, ff_handle* out) {
  ff_status rc = validate_config(cfg);
  if (rc != FF_OK) return rc;
  if (out == nullptr) return fail(FF_ERR_INVALID_ARG, "out is NULL");
  const Layout lay = make_layout(cfg);
  if (cfg->workspace == nullptr || ((uintptr_t)cfg->workspace % kAlign) != 0)
    return fail(FF_ERR_WORKSPACE, "workspace must be a non-NULL 256-byte aligned device pointer");
  if (cfg->workspace_bytes < lay.total) {
    char msg[128];
    snprintf(msg, sizeof msg, "workspace too small: %zu < %zu bytes", cfg->workspace_bytes,
             lay.total);
    return fail(FF_ERR_WORKSPACE, msg);
  }
  ff_handle_s* h = new (std::nothrow) ff_handle_s();
  if (h == nullptr) return fail(FF_ERR_INVALID_ARG, "host allocation of the handle failed");
  rc = init_handle(cfg, lay, h);
  if (rc != FF_OK) {
    delete h;
    return rc;
  }
  *out = h;
  return FF_OK;
}

ff_status ff_iterate(ff_handle h, int iters, int* iters_done, double* loglik) {
  return run_iterations(h, iters, 0.0, iters_done, loglik, nullptr);
}

ff_status ff_fit_noalloc(const ff_config* cfg, int iters, int* iters_done, double* loglik,
                         float* A, float* B) {
  if (iters_done != nullptr) *iters_done = 0;
  ff_status rc = validate_config(cfg);
  if (rc != FF_OK) return rc;
  if (iters < 0) return fail(FF_ERR_INVALID_ARG, "iters must be >= 0");
  if (A == nullptr || B == nullptr || ((uintptr_t)A % 16) != 0 || ((uintptr_t)B % 16) != 0)
    return fail(FF_ERR_INVALID_ARG, "A and B must be non-NULL 16-byte aligned device pointers");
  const Layout lay = make_layout(cfg);
  if (lay.total > (size_t)FF_NOALLOC_SCRATCH_BYTES) {
    char msg[192];
    snprintf(msg, sizeof msg,
             "problem needs %zu bytes of scratch; the allocation-free entry point holds %zu "
             "(use ff_init with a workspace)", lay.total, (size_t)FF_NOALLOC_SCRATCH_BYTES);
    return fail(FF_ERR_WORKSPACE, msg);
  }
  void* ws = nullptr;
  if ((rc = scratch_on_current_device(&ws)) != FF_OK) return rc;
  ff_config c = *cfg;
  c.workspace = ws;
  c.workspace_bytes = FF_NOALLOC_SCRATCH_BYTES;
  // The handle lives on this stack frame; with one stream and no timing it
  // creates no streams or events, so there is nothing to release.
  ff_handle_s h;
  h.single_stream = true;
  if ((rc = init_handle(&c, lay, &h)) != FF_OK) return rc;
  rc = run_iterations(&h, iters, 0.0, iters_done, loglik, nullptr);
  if (rc == FF_OK) {
    FF_HIP(hipMemcpyAsync(A, h.A.F[h.cur], h.n * h.n * sizeof(float), hipMemcpyDeviceToDevice,
                          h.stream));
    FF_HIP(hipMemcpyAsync(B, h.B.F[h.cur], h.m * h.m * sizeof(float), hipMemcpyDeviceToDevice,
                          h.stream));
  }
  FF_HIP(hipStreamSynchronize(h.stream));
  return rc;
}

ff_status ff_iterate_tol(ff_handle h, int max_iters, double tol, int* iters_done, double* loglik,
                         double* delta) {
  if (!(tol >= 0.0) || !isfinite(tol)) {
    if (iters_done != nullptr) *iters_done = 0;
    return fail(FF_ERR_INVALID_ARG, "tol must be finite and >= 0");
  }
  return run_iterations(h, max_iters, tol, iters_done, loglik, delta);
}

ff_status ff_half_step(ff_handle h, ff_half which, const float* F, float* out) {
  if (h == nullptr) return fail(FF_ERR_INVALID_ARG, "handle is NULL");
  if (which != FF_HALF_B && which != FF_HALF_A) return fail(FF_ERR_INVALID_ARG, "unknown half step");
  if (h->cfg.estimator != FF_EST_FLIPFLOP && h->cfg.estimator != FF_EST_FROBENIUS)
    return fail(FF_ERR_INVALID_ARG, "half steps exist for the FlipFlop and Frobenius estimators");
  if (out == nullptr || ((uintptr_t)out % 16) != 0 || ((uintptr_t)F % 16) != 0)
    return fail(FF_ERR_INVALID_ARG, "out (and F if given) must be 16-byte aligned device pointers");
  Side& s = which == FF_HALF_B ? h->B : h->A;  // the factor computed
  Side& p = which == FF_HALF_B ? h->A : h->B;  // the factor held fixed
  const float* src = F != nullptr ? F : p.F[h->cur];
  // the whitening operands no longer belong to the current factors
  h->A.lw_valid = h->B.lw_valid = false;
  ff_status rc = h->cfg.estimator == FF_EST_FROBENIUS ? frob_operand(h, p, src)
                                                      : cholinv_from(h, p, src, -1);
  if (rc != FF_OK) return rc;
  if ((rc = update(h, s, p, 0, false, false, out)) != FF_OK) return rc;
  int st[4];
  if ((rc = read_status(h, st)) != FF_OK) return rc;
  if (st[0] != 0) {
    if ((rc = clear_status(h)) != FF_OK) return rc;
    FF_HIP(hipStreamSynchronize(h->stream));
    return fail(FF_ERR_NOT_SPD, std::string("the fixed factor (") + (st[1] == 1 ? "A" : "B") +
                                    ") is not positive definite in ff_half_step");
  }
  return FF_OK;
}

ff_status ff_factors(ff_handle h, float* A, float* B, int on_host) {
  if (h == nullptr) return fail(FF_ERR_INVALID_ARG, "handle is NULL");
  const hipMemcpyKind kind = on_host ? hipMemcpyDeviceToHost : hipMemcpyDeviceToDevice;
  if (A != nullptr)
    FF_HIP(hipMemcpyAsync(A, h->A.F[h->cur], h->n * h->n * sizeof(float), kind, h->stream));
  if (B != nullptr)
    FF_HIP(hipMemcpyAsync(B, h->B.F[h->cur], h->m * h->m * sizeof(float), kind, h->stream));
  if (on_host) FF_HIP(hipStreamSynchronize(h->stream));
  return FF_OK;
}

ff_status ff_kron_apply(ff_handle h, const float* X, float* Y, int64_t batch, ff_apply_mode mode) {
  if (h == nullptr) return fail(FF_ERR_INVALID_ARG, "handle is NULL");
  if (batch < 0) return fail(FF_ERR_INVALID_ARG, "batch must be >= 0");
  if (mode != FF_APPLY && mode != FF_APPLY_INV) return fail(FF_ERR_INVALID_ARG, "unknown mode");
  if (batch == 0) return FF_OK;
  if (X == nullptr || Y == nullptr || ((uintptr_t)X % 16) || ((uintptr_t)Y % 16))
    return fail(FF_ERR_INVALID_ARG, "X and Y must be non-NULL 16-byte aligned device pointers");
  const int64_t m = h->m, n = h->n, mn = m * n;
  const char* xb = (const char*)X;
  const char* yb = (const char*)Y;
  if (xb < yb + batch * mn * 4 && yb < xb + batch * mn * 4)
    return fail(FF_ERR_INVALID_ARG, "X and Y overlap");
  const int cur = h->cur;
  ff_status rc;
  if (mode == FF_APPLY_INV) {
    // Fresh factorisations of the current factors (label 0 marks them).
    if ((rc = cholinv(h, h->A, cur, -1)) != FF_OK) return rc;
    if ((rc = cholinv(h, h->B, cur, -1)) != FF_OK) return rc;
    // the cached whitening operands of the other estimators are now stale
    if (h->cfg.estimator != FF_EST_FLIPFLOP) h->A.lw_valid = h->B.lw_valid = false;
  }
  float* T = (float*)h->W;
  const size_t tcap = h->lay.w_bytes / sizeof(float);  // >= m n floats
  const int64_t chunk = std::max<int64_t>(1, (int64_t)(tcap / (size_t)mn));
  for (int64_t b0 = 0; b0 < batch; b0 += chunk) {
    const int bc = (int)std::min<int64_t>(chunk, batch - b0);
    const float* Xc = X + b0 * mn;
    float* Yc = Y + b0 * mn;
    GemmF32 g{};
    g.st = h->st;
    g.kseg = INT64_MAX / 4;
    g.ksplit = 1;
    g.alpha = 1.f;
    g.beta = 0.f;
    auto gemm = [&](const float* Aop, int64_t lda, int64_t sA, int tA, const float* Bop,
                    int64_t ldb, int64_t sB, int tB, float* C, int64_t M, int64_t Nn, int64_t K,
                    int flags) -> ff_status {
      g.A = Aop; g.lda = lda; g.sA = sA; g.transA = tA;
      g.B = Bop; g.ldb = ldb; g.sB = sB; g.transB = tB;
      g.C = C; g.ldc = Nn; g.sC = mn;
      g.M = M; g.N = Nn; g.K = K; g.flags = flags;
      FF_HIP(launch_gemm_f32(g, bc, h->stream));
      return FF_OK;
    };
    if (mode == FF_APPLY) {
      // T = B X ; Y = T A
      if ((rc = gemm(h->B.F[cur], m, 0, 0, Xc, n, mn, 0, T, m, n, m, 0)) != FF_OK) return rc;
      if ((rc = gemm(T, n, mn, 0, h->A.F[cur], n, 0, 0, Yc, m, n, n, 0)) != FF_OK) return rc;
    } else {
      // B^-1 X A^-1 = Li_B^T Li_B X Li_A^T Li_A
      if ((rc = gemm(h->B.Li, m, 0, 0, Xc, n, mn, 0, T, m, n, m, kKHiRow)) != FF_OK) return rc;
      if ((rc = gemm(h->B.Li, m, 0, 1, T, n, mn, 0, Yc, m, n, m, kKLoRow)) != FF_OK) return rc;
      if ((rc = gemm(Yc, n, mn, 0, h->A.Li, n, 0, 1, T, m, n, n, kKHiCol)) != FF_OK) return rc;
      if ((rc = gemm(T, n, mn, 0, h->A.Li, n, 0, 0, Yc, m, n, n, kKLoCol)) != FF_OK) return rc;
    }
  }
  int st[4];
  if ((rc = read_status(h, st)) != FF_OK) return rc;
  if (st[0] != 0) {
    if ((rc = clear_status(h)) != FF_OK) return rc;
    FF_HIP(hipStreamSynchronize(h->stream));
    h->A.lw_valid = h->B.lw_valid = false;
    return fail(FF_ERR_NOT_SPD, std::string("factor ") + (st[1] == 1 ? "A" : "B") +
                                    " not positive definite in ff_kron_apply");
  }
  return FF_OK;
}

ff_status ff_objective(ff_handle h, const float* A, const float* B, double* psi) {
  if (h == nullptr) return fail(FF_ERR_INVALID_ARG, "handle is NULL");
  if (psi == nullptr) return fail(FF_ERR_INVALID_ARG, "psi is NULL");
  const int cur = h->cur, spare = cur ^ 1;
  const float* Af = A != nullptr ? A : h->A.F[cur];
  const float* Bf = B != nullptr ? B : h->B.F[cur];
  // The whitening operands no longer belong to the current factors.
  h->A.lw_valid = h->B.lw_valid = false;
  ff_status rc;
  if ((rc = cholinv_from(h, h->A, Af, -1)) != FF_OK) return rc;
  if ((rc = cholinv_from(h, h->B, Bf, -1)) != FF_OK) return rc;
  if (h->lay.rank1) {
    // tr(B^-1 g x^T A^-1 x g^T) = (x^T A^-1 x)(g^T B^-1 g): a dot of token weights
    float* w = h->wv;
    float* v = h->wv + h->lay.T_p;
    if ((rc = token_weights(h, h->A, w)) != FF_OK) return rc;
    if ((rc = token_weights(h, h->B, v)) != FF_OK) return rc;
    double* scratch = reinterpret_cast<double*>(h->P);
    double* out = scratch + 512;
    FF_HIP(launch_objective_terms(w, v, h->lay.T_p, h->A.slots, h->A.nslots, h->B.slots,
                                  h->B.nslots, scratch, out, h->st, h->stream));
    double terms[3];
    FF_HIP(hipMemcpyAsync(terms, out, sizeof terms, hipMemcpyDeviceToHost, h->stream));
    int st[4];
    if ((rc = read_status(h, st)) != FF_OK) return rc;
    if (st[0] != 0) {
      if ((rc = clear_status(h)) != FF_OK) return rc;
      FF_HIP(hipStreamSynchronize(h->stream));
      return fail(FF_ERR_NOT_SPD, std::string("factor ") + (st[1] == 1 ? "A" : "B") +
                                      " not positive definite in ff_objective");
    }
    const double mn = (double)h->m * (double)h->n;
    *psi = log(terms[0] / ((double)h->N * mn)) + terms[1] / (double)h->n + terms[2] / (double)h->m;
    return FF_OK;
  }
  // M = (1/(N n)) sum_i G_i A^-1 G_i^T into the spare B buffer (no damping)
  if ((rc = update(h, h->B, h->A, spare, false)) != FF_OK) return rc;
  // Y = L_B^-1 M; tr(B^-1 M) = sum_jk Y_jk (L_B^-1)_jk
  const int64_t m = h->m;
  GemmF32 g{};
  g.st = h->st;
  g.kseg = INT64_MAX / 4;
  g.ksplit = 1;
  g.A = h->B.Li; g.lda = m; g.transA = 0;
  g.B = h->B.F[spare]; g.ldb = m; g.transB = 0;
  g.C = h->B.L; g.ldc = m;
  g.M = m; g.N = m; g.K = m;
  g.alpha = 1.f; g.beta = 0.f; g.flags = kKHiRow;
  FF_HIP(launch_gemm_f32(g, 1, h->stream));
  double* scratch = reinterpret_cast<double*>(h->P);
  double* out = scratch + 512;
  FF_HIP(launch_objective_terms(h->B.L, h->B.Li, m * m, h->A.slots, h->A.nslots, h->B.slots,
                                h->B.nslots, scratch, out, h->st, h->stream));
  double terms[3];
  FF_HIP(hipMemcpyAsync(terms, out, sizeof terms, hipMemcpyDeviceToHost, h->stream));
  int st[4];
  if ((rc = read_status(h, st)) != FF_OK) return rc;
  if (st[0] != 0) {
    if ((rc = clear_status(h)) != FF_OK) return rc;
    FF_HIP(hipStreamSynchronize(h->stream));
    return fail(FF_ERR_NOT_SPD, std::string("factor ") + (st[1] == 1 ? "A" : "B") +
                                    " not positive definite in ff_objective");
  }
  // (1/(N m n)) sum_i tr(B^-1 G_i A^-1 G_i^T) = tr(B^-1 M) / m
  *psi = log(terms[0] / (double)m) + terms[1] / (double)h->n + terms[2] / (double)m;
  return FF_OK;
}

ff_status ff_quantize_workspace_size(int64_t m, int64_t n, size_t* bytes) {
  if (m < 1 || n < 1 || m > (1 << 20) || n > (1 << 20))
    return fail(FF_ERR_INVALID_ARG, "m and n must be in [1, 1048576]");
  if (bytes == nullptr) return fail(FF_ERR_INVALID_ARG, "bytes is NULL");
  *bytes = quant_layout(m, n).total;
  return FF_OK;
}

ff_status ff_quantize(ff_handle h, const float* W, const float* A, const float* B, double gamma,
                      ff_scale_mode mode, float* alpha, float* beta, int32_t* Z, float* V,
                      double* distortion, void* workspace, size_t workspace_bytes) {
  if (h == nullptr) return fail(FF_ERR_INVALID_ARG, "handle is NULL");
  if (mode != FF_SCALES_WATERFILL && mode != FF_SCALES_GIVEN)
    return fail(FF_ERR_INVALID_ARG, "unknown scale mode");
  const int given = mode == FF_SCALES_GIVEN ? 1 : 0;
  if (!given && !(gamma > 0.0 && isfinite(gamma)))
    return fail(FF_ERR_INVALID_ARG, "gamma must be finite and > 0");
  if (W == nullptr || Z == nullptr || alpha == nullptr || beta == nullptr)
    return fail(FF_ERR_INVALID_ARG, "W, Z, alpha and beta must be non-NULL device pointers");
  auto misaligned = [](const void* p) { return ((uintptr_t)p % 4) != 0; };
  if (misaligned(W) || misaligned(Z) || misaligned(alpha) || misaligned(beta) ||
      misaligned(V) || misaligned(A) || misaligned(B))
    return fail(FF_ERR_INVALID_ARG, "device arrays must be 4-byte aligned");
  const int64_t m = h->m, n = h->n;
  const QuantLayout q = quant_layout(m, n);
  if (workspace == nullptr || ((uintptr_t)workspace % kAlign) != 0)
    return fail(FF_ERR_WORKSPACE, "workspace must be a non-NULL 256-byte aligned device pointer");
  if (workspace_bytes < q.total) {
    char msg[128];
    snprintf(msg, sizeof msg, "workspace too small: %zu < %zu bytes", workspace_bytes, q.total);
    return fail(FF_ERR_WORKSPACE, msg);
  }
  if (given) {
    std::string why;
    if (!finite_positive(alpha, n, h->stream, &why) || !finite_positive(beta, m, h->stream, &why))
      return fail(FF_ERR_INVALID_ARG, why);
  }
  char* ws = (char*)workspace;
  float* La = (float*)(ws + q.off_La);
  float* Lb = (float*)(ws + q.off_Lb);
  float* al = (float*)(ws + q.off_al);
  float* be = (float*)(ws + q.off_be);
  float* dA = (float*)(ws + q.off_dA);
  float* dB = (float*)(ws + q.off_dB);
  double* dpart = (double*)(ws + q.off_dpart);
  double* dist = (double*)(ws + q.off_dist);
  // The factorisation buffers are reused: the whitening operands are stale.
  h->A.lw_valid = h->B.lw_valid = false;
  const int cur = h->cur;
  ff_status rc;
  // The two factorisations are independent and latency bound: B's runs on a
  // second stream, forked from and joined back into the handle's stream.
  if (h->aux == nullptr) {
    FF_HIP(hipStreamCreateWithFlags(&h->aux, hipStreamNonBlocking));
    FF_HIP(hipEventCreateWithFlags(&h->fork, hipEventDisableTiming));
    FF_HIP(hipEventCreateWithFlags(&h->join, hipEventDisableTiming));
  }
  FF_HIP(hipEventRecord(h->fork, h->stream));
  FF_HIP(hipStreamWaitEvent(h->aux, h->fork, 0));
  if ((rc = quant_side(h, h->A, A != nullptr ? A : h->A.F[cur], q.nq, La, dA, gamma, given, alpha,
                       al)) != FF_OK)
    return rc;
  {
    const hipStream_t main = h->stream;
    h->stream = h->aux;
    rc = quant_side(h, h->B, B != nullptr ? B : h->B.F[cur], q.mq, Lb, dB, gamma, given, beta, be);
    h->stream = main;
    if (rc != FF_OK) return rc;
  }
  FF_HIP(hipEventRecord(h->join, h->aux));
  FF_HIP(hipStreamWaitEvent(h->stream, h->join, 0));
  int st[4];
  if ((rc = read_status(h, st)) != FF_OK) return rc;
  if (st[0] != 0) {
    if ((rc = clear_status(h)) != FF_OK) return rc;
    FF_HIP(hipStreamSynchronize(h->stream));
    if (h->timing) collect_timing(h);
    return fail(FF_ERR_NOT_SPD, std::string("factor ") + (st[1] == 1 ? "A" : "B") +
                                    " not positive definite in ff_quantize");
  }
  const int64_t tile_floats = (int64_t)q.MT * q.NT * kTileWK * kTileWK;
  FF_HIP(launch_fill_f32((float*)(ws + q.off_racc), tile_floats, 0.0f, h->stream));
  FF_HIP(launch_fill_f32((float*)(ws + q.off_pre), tile_floats, 0.0f, h->stream));
  WkParams p{};
  p.W = W;
  p.m = m;
  p.n = n;
  p.La = La;
  p.Lb = Lb;
  p.alpha = al;
  p.beta = be;
  p.dA = dA;
  p.dB = dB;
  p.Racc = (float*)(ws + q.off_racc);
  p.Pre = (float*)(ws + q.off_pre);
  p.X = (float*)(ws + q.off_x);
  p.E = (float*)(ws + q.off_e);
  p.Z = (int32_t*)(ws + q.off_z);
  p.dpart = dpart;
  p.mq = q.mq;
  p.nq = q.nq;
  p.MT = q.MT;
  p.NT = q.NT;
  p.st = h->st;
  const int ndiag = q.MT + q.NT - 1;
  const double dflop = ((double)m * m * n + (double)m * n * n) / ndiag;
  for (int d = 0; d < ndiag; ++d) {
    Timed t(h, 4, dflop);
    FF_HIP(launch_wk_diagonal(p, d, h->stream));
  }
  FF_HIP(launch_wk_finish(p.Z, q.nq, m, n, al, be, Z, V, h->st, h->stream));
  FF_HIP(launch_wk_sum(dpart, (int64_t)q.MT * q.NT, 1.0 / ((double)m * (double)n), dist, h->st,
                       h->stream));
  double dh = 0.0;
  FF_HIP(hipMemcpyAsync(&dh, dist, sizeof dh, hipMemcpyDeviceToHost, h->stream));
  if ((rc = read_status(h, st)) != FF_OK) return rc;
  if (h->timing) collect_timing(h);
  if (st[0] != 0) {
    if ((rc = clear_status(h)) != FF_OK) return rc;
    FF_HIP(hipStreamSynchronize(h->stream));
    return fail(FF_ERR_STATE, "device status set during the quantiser sweep");
  }
  if (distortion != nullptr) *distortion = dh;
  return FF_OK;
}

ff_status ff_destroy(ff_handle h) {
  if (h == nullptr) return FF_OK;
  // best-effort teardown: every object is released even if an earlier
  // release reports an error (there is nothing left to report it to)
  (void)hipStreamSynchronize(h->stream);
  if (h->aux != nullptr) {
    (void)hipStreamSynchronize(h->aux);
    (void)hipStreamDestroy(h->aux);
    (void)hipEventDestroy(h->fork);
    (void)hipEventDestroy(h->join);
  }
  for (Side* sd : {&h->A, &h->B}) {
    if (sd->istream != nullptr) {
      (void)hipStreamSynchronize(sd->istream);
      (void)hipStreamDestroy(sd->istream);
      (void)hipEventDestroy(sd->ev_leaf);
      (void)hipEventDestroy(sd->ev_inv);
    }
  }
  for (hipEvent_t e : h->events) (void)hipEventDestroy(e);
  delete h;
  return FF_OK;
}

ff_status ff_set_timing(ff_handle h, int enable) {
  if (h == nullptr) return fail(FF_ERR_INVALID_ARG, "handle is NULL");
  if (enable && h->events.empty()) {
    h->events.resize(2 * 1024 + 16);  // enough for one quantiser sweep up to m + n = 65000
    for (auto& e : h->events) FF_HIP(hipEventCreate(&e));
  }
  h->timing = enable != 0;
  for (int k = 0; k < kTimedKernels; ++k) {
    h->t_launches[k] = 0;
    h->t_ms[k] = 0;
    h->t_flop[k] = 0;
  }
  return FF_OK;
}

ff_status ff_whiten_split_state(ff_handle h, double* s_A, double* s_B, int* passes_A,
                                int* passes_B) {
  if (h == nullptr) return fail(FF_ERR_INVALID_ARG, "handle is NULL");
  double sv[2] = {NAN, NAN};
  int passes = 1;
  if (h->bf16 && h->A.Lw2 != nullptr) {
    if (h->cfg.whiten_split == 2) {
      passes = 2;
    } else if (h->cfg.estimator != FF_EST_FROBENIUS && h->A.split_flag != nullptr) {
      if (samples_per_dim(h) < kMinSamplesPerDim) passes = 2;
      int flag[2] = {0, 0};
      const Side* sides[2] = {&h->A, &h->B};
      for (int k = 0; k < 2; ++k) {
        FF_HIP(hipMemcpyAsync(&flag[k], sides[k]->split_flag, sizeof(int), hipMemcpyDeviceToHost,
                              h->stream));
        if (sides[k]->stat_known)
          FF_HIP(hipMemcpyAsync(&sv[k], sides[k]->split_stat, sizeof(double),
                                hipMemcpyDeviceToHost, h->stream));
      }
      FF_HIP(hipStreamSynchronize(h->stream));
      if (flag[0] || flag[1]) passes = 2;
    }
  }
  if (s_A) *s_A = sv[0];
  if (s_B) *s_B = sv[1];
  if (passes_A) *passes_A = passes;
  if (passes_B) *passes_B = passes;
  return FF_OK;
}

ff_status ff_kernel_timing(ff_handle h, int kernel, int64_t* launches, double* total_ms,
                           double* alg_flop) {
  if (h == nullptr) return fail(FF_ERR_INVALID_ARG, "handle is NULL");
  if (kernel < 0 || kernel >= kTimedKernels) return fail(FF_ERR_INVALID_ARG, "unknown kernel id");
  if (launches) *launches = h->t_launches[kernel];
  if (total_ms) *total_ms = h->t_ms[kernel];
  if (alg_flop) *alg_flop = h->t_flop[kernel];
  return FF_OK;
}

}  // extern "C"
