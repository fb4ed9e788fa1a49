// HIP kernels and C ABI of the per-token LDA topic draw (gfx950).
//
// lda_draw_naive      Algorithm 1 + Algorithm 3, one lane per token.
// lda_draw_butterfly  Algorithm 7 (+ 5, 8, 9, 10) for 64-lane wavefronts.
// lda_draw_docs       the same, documents given as offsets.
// lda_draw_doc_lanes  Algorithm 7's document-per-lane driver.
// lda_draw_transposed Algorithms 4-6, for comparison.
// lda_draw_butterfly_variant  the block-table variants of Section 4.
// lda_draw_butterfly_philox   the butterfly draw with in-kernel uniforms.
// lda_philox_uniforms         those uniforms, written out.
// lda_butterfly_table the butterfly-patterned tables (Fig. 1, right).
// lda_route_build / lda_draw_routed  tokens routed to the XCDs by word, and
//                     the leaf kernel drawing them.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "butterfly.hpp"
#include "lda_draw.h"
#include "philox.hpp"
#include "route.hpp"

// Build-time tuning of the butterfly kernel (chosen by measurement on MI355X):
//   LDA_LDS_TABLE_MAX_BLOCKS  largest K / W whose rebuilt table goes to LDS
//                             (see lds_table_for);
//   LDA_WAVES_PER_EU          wavefronts per SIMD the register budget targets;
//   LDA_WAVES_PER_BLOCK       wavefronts per workgroup.
#ifndef LDA_LDS_TABLE_MAX_BLOCKS
#define LDA_LDS_TABLE_MAX_BLOCKS 0
#endif
#ifndef LDA_WAVES_PER_EU
#define LDA_WAVES_PER_EU 3
#endif
#ifndef LDA_WAVES_PER_BLOCK
#define LDA_WAVES_PER_BLOCK 2
#endif
//   LDA_DOC_LANES_TARGET_WAVES wavefronts the document-per-lane driver aims
//                             for by splitting each group's master loop.
#ifndef LDA_DOC_LANES_TARGET_WAVES
#define LDA_DOC_LANES_TARGET_WAVES 16384
#endif
//   LDA_HALF_MAX_BLOCKS       largest K / 64 for which the W = 64 kernel
//                             rebuilds only the chosen half-block (its 2 K/64
//                             LDS rows per wavefront keep 12 wavefronts per CU
//                             up to 26 blocks, 10 at 32 blocks).
#ifndef LDA_HALF_MAX_BLOCKS
#define LDA_HALF_MAX_BLOCKS 32
#endif
//   LDA_EIGHTHS_MAX_BLOCKS    largest number of 256-topic blocks for which the
//                             leaf kernel with 32-topic prefix rows draws
//                             (8 rows of LDS per block and wavefront; 0: never);
//   LDA_EIGHTHS_SPLIT         largest block count drawn with the first of its
//                             two launch shapes;
//   LDA_EIGHTHS_WINDOW{,_LARGE}, LDA_EIGHTHS_WAVES_PER_EU{,_LARGE}
//                             tokens in flight per wavefront (16-byte loads)
//                             and wavefronts per SIMD of the two shapes.
#ifndef LDA_EIGHTHS_MAX_BLOCKS
#define LDA_EIGHTHS_MAX_BLOCKS 8
#endif
//   LDA_GROUP_MAX_K           largest K drawn by the leaf-group kernel (K
//                             divisible by 4, at most 256; 0: never), and its
//                             tokens in flight per wavefront and wavefronts
//                             per SIMD.
#ifndef LDA_GROUP_MAX_K
#define LDA_GROUP_MAX_K 256
#endif
#ifndef LDA_GROUP_WINDOW
#define LDA_GROUP_WINDOW 8
#endif
#ifndef LDA_GROUP_WAVES_PER_EU
#define LDA_GROUP_WAVES_PER_EU 3
#endif
//   LDA_EIGHTHS_MIN_K         smallest K it takes (K divisible by 4; the first
//                             block is padded with empty topics up to a
//                             multiple of 256).
#ifndef LDA_EIGHTHS_MIN_K
#define LDA_EIGHTHS_MIN_K 132
#endif
#ifndef LDA_EIGHTHS_SPLIT
#define LDA_EIGHTHS_SPLIT 5
#endif
#ifndef LDA_EIGHTHS_WINDOW
#define LDA_EIGHTHS_WINDOW 16
#endif
#ifndef LDA_EIGHTHS_WAVES_PER_EU
#define LDA_EIGHTHS_WAVES_PER_EU 2
#endif
#ifndef LDA_EIGHTHS_WINDOW_LARGE
#define LDA_EIGHTHS_WINDOW_LARGE 4
#endif
#ifndef LDA_EIGHTHS_WAVES_PER_EU_LARGE
#define LDA_EIGHTHS_WAVES_PER_EU_LARGE 4
#endif

namespace lda {
namespace {

constexpr int kWavesPerBlock = LDA_WAVES_PER_BLOCK;
constexpr int kBlockThreads = kWavesPerBlock * kWave;

// Where a token's document comes from: a per-token id array, or the paper's
// ragged form (Section 2: document m holds N[m] tokens), given as offsets --
// document m's tokens are [offsets[m], offsets[m + 1]).  With offsets, the
// document of token n is the last m with offsets[m] <= n (which skips empty
// documents); every search stays inside [0, M - 1] whatever the offsets hold.
struct DocSource {
  const int32_t *ids;      // doc_id[N], or null
  const int64_t *offsets;  // doc_offsets[M + 1], used when ids is null
  int M;
  int64_t N;

  // Last m in [lo, hi] with offsets[m] <= t, given offsets[lo] <= t and
  // offsets[hi + 1] > t (bisection).
  __device__ __forceinline__ int bisect(int64_t t, int lo, int hi) const {
    while (lo < hi) {
      const int mid = lo + ((hi - lo + 1) >> 1);
      if (offsets[mid] <= t)
        lo = mid;
      else
        hi = mid - 1;
    }
    return lo;
  }

  // The same over [0, M - 1] from a guess g: steps of 1, 2, 4, ... away from g
  // bracket the answer, then bisection (a few probes when g is close).
  __device__ __forceinline__ int search_from(int64_t t, int g) const {
    int lo, hi;
    if (offsets[g] <= t) {
      lo = g;
      int step = 1;
      while (lo + step <= M - 1 && offsets[lo + step] <= t) {
        lo += step;
        step *= 2;
      }
      hi = lo + step <= M - 1 ? lo + step - 1 : M - 1;
    } else {
      hi = g - 1;
      int step = 1;
      for (;;) {
        const int m = hi - step + 1;
        if (m <= 0) {
          lo = 0;
          break;
        }
        if (offsets[m] <= t) {
          lo = m;
          break;
        }
        hi = m - 1;
        step *= 2;
      }
    }
    return bisect(t, lo, hi);
  }

  // Document of token n, any lane layout (one bisection over all documents).
  __device__ __forceinline__ int operator()(int64_t n) const {
    if (ids) return ids[n];
    return bisect(n, 0, M - 1);
  }

  // Document of token n for a wavefront whose tokens all lie in [first,
  // last] (uniform): the documents of `first` and `last` are found once per
  // wavefront, the first from the guess first * M / N, and each lane then
  // bisects only the documents between them (usually one or two).
  __device__ __forceinline__ int wave_doc(int64_t n, int64_t first, int64_t last) const {
    if (ids) return ids[n];
    int g = (int)((double)first * (double)M / (double)(N > 0 ? N : 1));
    g = g < 0 ? 0 : (g > M - 1 ? M - 1 : g);
    const int d0 = __builtin_amdgcn_readfirstlane(search_from(first, g));
    const int d1 = __builtin_amdgcn_readfirstlane(search_from(last, d0));
    return bisect(n, d0, d1 > d0 ? d1 : d0);
  }
};

// Where a token's uniform comes from: the caller's array u[N], or (u null)
// Philox4x32-10 with key (k0, k1) at counter (n mod 2^32, n / 2^32, sweep, 0),
// whose first output word's top 24 bits, times 2^-24, give the uniform.
struct UniformSource {
  const float *u;
  uint32_t k0, k1, sweep;
  __device__ __forceinline__ float operator()(int64_t n) const {
    if (u) return u[n];
    return philox_uniform((uint64_t)n, sweep, k0, k1);
  }
};

// ---------------------------------------------------------------------------
// Naive kernel (Algorithm 1 with Algorithm 3).  Lane n walks the K topics of
// its own token, keeps the full prefix table p[K] in its private segment and
// binary-searches it for the first entry above stop = S * u.
template <int KMAX>
__global__ __launch_bounds__(256) void naive_kernel(
    const float *__restrict__ theta, const float *__restrict__ phi, DocSource docs,
    const int32_t *__restrict__ word_id, UniformSource u,
    int32_t *__restrict__ z, int64_t N, int K) {
  const int64_t n = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (n >= N) return;
  const float *th = theta + (int64_t)docs(n) * K;
  const float *ph = phi + (int64_t)word_id[n] * K;
  float p[KMAX];
  float sum = 0.0f;
  for (int k = 0; k < K; ++k) {
    sum = prefix_step(sum, th[k], ph[k]);
    p[k] = sum;
  }
  const float stop = sum * u(n);
  int j = 0, hi = K - 1;
  while (j < hi) {
    const int mid = (j + hi) >> 1;
    if (stop < p[mid])
      hi = mid;
    else
      j = mid + 1;
  }
  z[n] = j;
}

// ---------------------------------------------------------------------------
// Per-wavefront state of the butterfly kernel.  The wavefront's 64 tokens are
// the window [t0, t0 + 64) of the token arrays; their word and document ids
// are read with scalar loads straight from those arrays whenever a tile is
// loaded (SMALL: the window is padded by repeating token N - 1).
template <int W, bool SMALL>
struct Wave {
  rsrc_t th_rs, ph_rs;  // theta, phi
  const int32_t *wp;    // word_id + t0
  int last;             // SMALL: index in the window of token N - 1
  uint32_t row_bytes;   // 4 * K
  int R;                // remnant topics (K mod W)
  int c0;               // first topic of block 0: R - W if R > 0 (the remnant is
                        // block 0, padded at its front with W - R empty
                        // topics), else 0
  int r;                // lane within its group of W
  int gbase;            // first lane of the group
  int doc;              // this lane's document
  int mode;             // ThetaMode, uniform
  int kb;               // kTwoDocs: wave lanes below kb are in the first doc
  uint32_t th_off0, th_off1;  // theta row offsets of the first / last doc
  uint32_t ph_lane;           // phi row offset of this lane's own token
  uint32_t th_lane;           // theta row offset of this lane's own token
};

// Keep a uniform value opaque to the optimiser, so that work depending on it
// is done where it is written instead of being hoisted out of the block loop
// into (and spilling out of) scalar registers.  The readfirstlane marks the
// result uniform again for the divergence analysis, which treats inline
// assembly results as per-lane.
__device__ __forceinline__ int launder_int(int v) {
  asm volatile("" : "+s"(v));
  return __builtin_amdgcn_readfirstlane(v);
}

// The same for a pointer into a read-only kernel argument: only a zero offset
// is made opaque, so the pointer keeps its provenance (and its loads stay
// scalar loads of memory the kernel never writes).
__device__ __forceinline__ const int32_t *launder(const int32_t *p) {
  return p + launder_int(0);
}

// Scalar read of entry k of a wave window (k uniform).
template <bool SMALL>
__device__ __forceinline__ int window_at(const int32_t *p, int last, int k) {
  return SMALL ? p[k < last ? k : last] : p[k];
}

// Byte offset of the phi row of token k of this lane's group: uniform for
// W = 64, one value per half-wave for W = 32.
template <int W, bool SMALL>
__device__ __forceinline__ uint32_t phi_row(const Wave<W, SMALL> &w, const int32_t *wp, int k) {
  if constexpr (W == kWave) {
    return (uint32_t)window_at<SMALL>(wp, w.last, k) * w.row_bytes;
  } else {
    const uint32_t lo = (uint32_t)window_at<SMALL>(wp, w.last, k) * w.row_bytes;
    const uint32_t hi = (uint32_t)window_at<SMALL>(wp, w.last, 32 + k) * w.row_bytes;
    return w.gbase ? hi : lo;
  }
}

// Byte offset of the theta row of token k's document, from the lane that
// holds token k (uniform for W = 64, per half-wave for W = 32).
template <int W, bool SMALL>
__device__ __forceinline__ uint32_t theta_row(const Wave<W, SMALL> &w, int k) {
  return (uint32_t)group_value<W>((int)w.th_lane, k);
}

// buffer load at a per-lane offset plus a row offset that is uniform for
// W = 64 (scalar operand) and per half-wave for W = 32 (added per lane).
template <int W>
__device__ __forceinline__ float load_row(rsrc_t rs, uint32_t voff, uint32_t row) {
  if constexpr (W == kWave)
    return load_f32(rs, voff, row);
  else
    return load_f32(rs, voff + row, 0);
}

// This lane's topic in block `blk` (negative in the padding of block 0), and
// the byte offset used to load it (padding lanes read topic 0; their theta
// factor is replaced by zero where it is used).
template <int W, bool SMALL>
__device__ __forceinline__ int topic_of(const Wave<W, SMALL> &w, int blk) {
  return w.c0 + blk * W + w.r;
}
template <int W, bool SMALL>
__device__ __forceinline__ uint32_t col_bytes(const Wave<W, SMALL> &w, int blk) {
  const int t = topic_of(w, blk);
  return (uint32_t)(t > 0 ? t : 0) * 4u;
}

// Issue the phi loads of registers [LO, HI) of block `blk`: register k takes
// the value of token reg_token(k) (token k unless HALF).
template <int W, bool SMALL, int LO, int HI, bool HALF = false>
__device__ __forceinline__ void issue_phi(const Wave<W, SMALL> &w, const int32_t *wp,
                                          float (&a)[W], int blk) {
  const uint32_t voff = col_bytes(w, blk);
#pragma unroll
  for (int k = LO; k < HI; ++k)
    a[k] = load_row<W>(w.ph_rs, voff, phi_row(w, wp, reg_token<W, HALF>(k)));
}

// Theta of block `blk` at this lane's topic, for the first and last document
// (MODE: the wave's ThetaMode when known at compile time, else -1).
template <int W, bool SMALL, int MODE = -1>
__device__ __forceinline__ void issue_theta(const Wave<W, SMALL> &w, int blk, float &th0,
                                            float &th1) {
  const uint32_t voff = col_bytes(w, blk);
  th0 = load_f32(w.th_rs, voff, w.th_off0);
  if (MODE == kTwoDocs || (MODE < 0 && w.mode == kTwoDocs))
    th1 = load_f32(w.th_rs, voff, w.th_off1);
}

// The stages of the block-total reduce-scatter from BIT down to 1.  With
// PREFETCH, the registers each stage frees are refilled at once with the next
// block's phi values, so those loads are in flight during the rest of the
// reduction.  With HALF the last stage also leaves the lane's lower-half sum
// in `lower`.
template <int W, bool SMALL, int BIT, bool PREFETCH, bool HALF = false>
__device__ __forceinline__ void reduce_rest(const Wave<W, SMALL> &w, const int32_t *wp,
                                            float (&a)[W], int next, float &lower) {
  if constexpr (BIT >= 1) {
    if constexpr (HALF && BIT == 1)
      lower = reduce_last_half<W>(a);
    else
      reduce_stage<W, BIT, HALF>(a);
    if constexpr (PREFETCH && BIT > 1) issue_phi<W, SMALL, BIT, 2 * BIT, HALF>(w, wp, a, next);
    reduce_rest<W, SMALL, BIT / 2, PREFETCH, HALF>(w, wp, a, next, lower);
  }
}

template <int W, bool SMALL, int BIT, bool PREFETCH>
__device__ __forceinline__ void reduce_rest(const Wave<W, SMALL> &w, const int32_t *wp,
                                            float (&a)[W], int next) {
  float unused;
  reduce_rest<W, SMALL, BIT, PREFETCH, false>(w, wp, a, next, unused);
}

// Sweep step for one block whose phi values are in (or in flight to) a[] and
// whose theta values are in th0/th1.  Returns this lane's token total over
// the block (and with HALF its sum over the block's lower half in `lower`).
// With PREFETCH, block `next`'s loads are issued along the way and left in
// a[], th0, th1.
template <int W, bool SMALL, bool PREFETCH, bool HALF, int MODE>
__device__ __forceinline__ float sweep_block(const Wave<W, SMALL> &w, const int32_t *wp,
                                             float (&a)[W], float &th0, float &th1,
                                             int cur, int next, float &lower) {
  static_assert(MODE == kOneDoc || MODE == kTwoDocs, "sweep_block: one or two documents");
  constexpr int B = W / 2;
  constexpr int L = stage_lane_bit<W, B, HALF>();  // lane bit of the first stage
  // padding topics of block 0 weigh nothing
  const bool real = topic_of(w, cur) >= 0;
  if constexpr (MODE == kOneDoc) {
    // First stage fused with the theta factor: after the half exchange the
    // two values of a pair sit at the topics of lanes l and l xor L, whose
    // theta values one more exchange of th0 provides.
    float tA = real ? th0 : 0.0f, tB = tA;
    half_swap<L>(tA, tB);
    if constexpr (PREFETCH) issue_theta<W, SMALL, MODE>(w, next, th0, th1);
#pragma unroll
    for (int k = B - 1; k >= 0; --k) {
      half_swap<L>(a[k], a[k + B]);
      a[k] = __builtin_fmaf(a[k], tA, a[k + B] * tB);
    }
  } else {
    // Two contiguous document runs: wave lanes below kb take th0.  (kb is
    // laundered so that the per-token choices are made here, not hoisted out
    // of the block loop into scalar registers.)
    const int kb = launder_int(w.kb);
    const float t0 = real ? th0 : 0.0f, t1 = real ? th1 : 0.0f;
#pragma unroll
    for (int k = 0; k < W; ++k) a[k] *= (w.gbase + reg_token<W, HALF>(k) < kb) ? t0 : t1;
    if constexpr (PREFETCH) issue_theta<W, SMALL, MODE>(w, next, th0, th1);
    reduce_stage<W, B, HALF>(a);
  }
  if constexpr (PREFETCH) issue_phi<W, SMALL, B, W, HALF>(w, wp, a, next);
  reduce_rest<W, SMALL, B / 2, PREFETCH, HALF>(w, wp, a, next, lower);
  const float total = a[0];
  if constexpr (PREFETCH) issue_phi<W, SMALL, 0, 2, HALF>(w, wp, a, next);
  return total;
}

// The sweep over all NB blocks for a wave of one or two documents (MODE):
// the running prefix at each block's end goes to row b of `region` (with
// HALF, the prefixes at its middle and end to rows 2b and 2b + 1).  Returns
// the lane's token total.  The loop is instantiated per mode so that its body
// is branch-free.
template <int W, bool SMALL, bool HALF, int MODE>
__device__ __forceinline__ float sweep_blocks(const Wave<W, SMALL> &w, float (&a)[W],
                                              float *region, int lane, int NB) {
  float sum = 0.0f, lower = 0.0f;
  float th0 = 0.0f, th1 = 0.0f;
  issue_theta<W, SMALL, MODE>(w, 0, th0, th1);
  issue_phi<W, SMALL, 0, W, HALF>(w, w.wp, a, 0);
  for (int b = 0; b < NB - 1; ++b) {
    const float total = sweep_block<W, SMALL, true, HALF, MODE>(w, launder(w.wp), a, th0, th1,
                                                                b, b + 1, lower);
    if constexpr (HALF) region[(2 * b) * kWave + lane] = sum + lower;
    sum += total;
    region[(HALF ? 2 * b + 1 : b) * kWave + lane] = sum;
  }
  const float total =
      sweep_block<W, SMALL, false, HALF, MODE>(w, w.wp, a, th0, th1, NB - 1, 0, lower);
  if constexpr (HALF) region[(2 * NB - 2) * kWave + lane] = sum + lower;
  sum += total;
  region[(HALF ? 2 * NB - 1 : NB - 1) * kWave + lane] = sum;
  return sum;
}

// Sweep step for a wave whose tokens belong to many documents: one theta
// load per token, no prefetch.
template <int W, bool SMALL, bool HALF = false>
__device__ __forceinline__ float sweep_block_any(const Wave<W, SMALL> &w, const int32_t *wp,
                                                 int blk, float &lower) {
  float a[W];
  const uint32_t voff = col_bytes(w, blk);
  const bool real = topic_of(w, blk) >= 0;
#pragma unroll
  for (int k = 0; k < W; ++k) {
    const int t = reg_token<W, HALF>(k);
    a[k] = (real ? load_row<W>(w.th_rs, voff, theta_row(w, t)) : 0.0f) *
           load_row<W>(w.ph_rs, voff, phi_row(w, wp, t));
  }
  reduce_stage<W, W / 2, HALF>(a);
  reduce_rest<W, SMALL, W / 4, false, HALF>(w, wp, a, 0, lower);
  return a[0];
}

// Transposed tile in which token k of the group contributes block blk_k
// (this lane's `blk` is its own token's block): a[k] = theta[doc_k][c_k] *
// phi[word_k][c_k], c_k = R + blk_k * W + r.
// Topic of lane r for token k is first + blk_k * W + r; with PADDED, topics
// below 0 (the front padding of block 0) contribute 0.
template <int W, bool SMALL, bool PADDED>
__device__ __forceinline__ void load_tile_blocks(const Wave<W, SMALL> &w, float (&a)[W],
                                                 int blk, int first) {
#pragma unroll
  for (int k = 0; k < W; ++k) {
    // row offsets of token k from the lane that holds it
    const int bk = group_value<W>(blk, k);
    const int t = first + bk * W + w.r;
    const uint32_t voff = (uint32_t)(PADDED && t < 0 ? 0 : t) * 4u;
    const uint32_t toff = (uint32_t)group_value<W>((int)w.th_lane, k);
    const uint32_t poff = (uint32_t)group_value<W>((int)w.ph_lane, k);
    const float th = load_row<W>(w.th_rs, voff, toff);
    a[k] = (PADDED && t < 0 ? 0.0f : th) * load_row<W>(w.ph_rs, voff, poff);
  }
}

template <int W, bool SMALL>
__device__ __forceinline__ void init_wave(Wave<W, SMALL> &w, const float *theta,
                                          const float *phi, uint32_t theta_bytes,
                                          uint32_t phi_bytes, const int32_t *word_id, int64_t t0, int last,
                                          int K, int lane, int doc, int word) {
  w.th_rs = make_rsrc(theta, theta_bytes);
  w.ph_rs = make_rsrc(phi, phi_bytes);
  w.wp = word_id + t0;
  w.last = last;
  w.row_bytes = (uint32_t)K * 4u;
  w.R = K & (W - 1);
  w.c0 = w.R ? w.R - W : 0;
  w.r = lane & (W - 1);
  w.gbase = lane & ~(W - 1);
  w.doc = doc;
  const int d0 = __builtin_amdgcn_readfirstlane(doc);
  const int d1 = __builtin_amdgcn_readlane(doc, kWave - 1);
  const uint64_t in0 = __builtin_amdgcn_ballot_w64(doc == d0);
  const uint64_t in1 = __builtin_amdgcn_ballot_w64(doc == d1);
  if (in0 == ~0ull) {
    w.mode = kOneDoc;
    w.kb = kWave;
  } else if ((in0 | in1) == ~0ull && (in0 & (in0 + 1)) == 0) {
    w.mode = kTwoDocs;  // lanes [0, kb) in d0, [kb, 64) in d1
    w.kb = __builtin_popcountll(in0);
  } else {
    w.mode = kAnyDocs;
    w.kb = 0;
  }
  w.th_off0 = (uint32_t)d0 * w.row_bytes;
  w.th_off1 = (uint32_t)d1 * w.row_bytes;
  w.ph_lane = (uint32_t)word * w.row_bytes;
  w.th_lane = (uint32_t)doc * w.row_bytes;
}


// The same wavefront seen as two groups of 32 lanes (W = 32): lanes 32 g + r
// hold topic r of a 32-topic chunk for the tokens of half-wave g.
template <bool SMALL>
__device__ __forceinline__ Wave<kWave / 2, SMALL> half_wave(const Wave<kWave, SMALL> &w,
                                                           int lane) {
  Wave<kWave / 2, SMALL> h;
  h.th_rs = w.th_rs;
  h.ph_rs = w.ph_rs;
  h.wp = w.wp;
  h.last = w.last;
  h.row_bytes = w.row_bytes;
  h.R = w.R;
  h.c0 = w.c0;
  h.r = lane & (kWave / 2 - 1);
  h.gbase = lane & (kWave / 2);
  h.doc = w.doc;
  h.mode = w.mode;
  h.kb = w.kb;
  h.th_off0 = w.th_off0;
  h.th_off1 = w.th_off1;
  h.ph_lane = w.ph_lane;
  h.th_lane = w.th_lane;
  return h;
}

// In-block search of Algorithm 10.  `low` and `high` are the full prefixes
// before and at the end of the block; a[0..W-2] is this lane's column of the
// rebuilt block (or, with LDS_TABLE, the rows are in `table`, row d at
// table[d * 64 + lane]).  Returns the offset within the block and leaves in
// low / high the prefixes before and after that entry.
template <int W, bool LDS_TABLE>
__device__ __forceinline__ int inblock_search(const float (&a)[W], const float *table,
                                              int r, int gbase, float stop, float &low,
                                              float &high) {
  static_assert(W >= 2 && W <= kWave && (W & (W - 1)) == 0, "W: a power of two up to 64");
  constexpr int LOG2W = __builtin_ctz(W);
  int flip = 0;
#pragma unroll
  for (int lvl = 0; lvl < LOG2W; ++lvl) {
    const int bit = (W / 2) >> lvl;
    const int mask = ((W - 1) * (2 * bit)) & (W - 1);
    float y;
    if constexpr (LDS_TABLE) {
      // The entry the search-assist loop would deliver: row (r & mask) |
      // (bit - 1) of column r xor flip.
      y = table[((r & mask) | (bit - 1)) * kWave + gbase + (r ^ flip)];
    } else {
      // Search-assist loop: every lane offers each candidate row in turn;
      // the lane keeps the one whose high bits match its own.
      y = 0.0f;
#pragma unroll
      for (int i = 0; i < W / (2 * bit); ++i) {
        const int d = (bit - 1) + 2 * bit * i;
        const float t = xor_lane_var(a[d], flip);
        if ((r & mask) == (d & mask)) y = t;
      }
    }
    const float cmp = (r & bit) ? high - y : low + y;
    if (stop < cmp) {
      high = cmp;
      flip ^= bit & r;
    } else {
      low = cmp;
      flip ^= bit & ~r;
    }
  }
  return flip ^ r;
}

// In-block search over the table of the alternative rule (rows in `table`,
// row d at table[d * 64 + lane]): a descent from the whole block.  At the
// node of 2^(s+1) topics starting at b, lane r reads its own token's sum over
// the node's left half, which the table keeps in row (r & ~(2^(s+1)-1)) +
// 2^s - 1 of column (r & (2^(s+1)-1)) + b, and goes left when stop is below
// low plus that sum.  Returns the offset within the block.
template <int W>
__device__ __forceinline__ int inblock_search_alt(const float *table, int r, int gbase,
                                                  float stop, float &low, float &high) {
  constexpr int LOG2W = (W == 64) ? 6 : 5;
  int b = 0;
#pragma unroll
  for (int s = LOG2W - 1; s >= 0; --s) {
    const int span = 1 << s, node = 2 << s;
    const int row = (r & ~(node - 1)) + span - 1;
    const float cmp = low + table[row * kWave + gbase + (r & (node - 1)) + b];
    if (stop < cmp) {
      high = cmp;
    } else {
      low = cmp;
      b += span;
    }
  }
  return b;
}

// LDS rows per wavefront: the block-end prefixes (NB rows of 64 lanes); with
// the half-block tail also the prefixes at the block middles (2 NB rows); with
// an LDS table, the rebuilt block's W - 1 rows in the same space.
__host__ __device__ constexpr int region_rows(int NB, int W, bool lds_table, bool half = false) {
  return lds_table ? (NB > W - 1 ? NB : W - 1) : (half ? 2 * NB : NB);
}

// ---------------------------------------------------------------------------
// Butterfly kernel.  Wavefront g takes tokens [64 g, 64 g + 64); lanes past N
// repeat token N - 1 so that every lane takes part in every exchange (the
// paper's "staying awake" rule) and skip the store.
//
// Remnant: untransposed running sum of the first K mod W topics.
// Sweep (K / W >= 2): per block the transposed tile, a reduce-scatter giving
//   every lane its token's block total, and the running prefix at the block's
//   end, kept in LDS.
// Block search (Algorithm 9): binary search over the block ends for S * u.
// Rebuild: one tile in which every token contributes its own chosen block,
//   combined by Algorithm 8's butterfly (with K / W == 1 this tile is the only
//   pass over phi).
// In-block search (Algorithm 10) and the remnant fallback of Algorithm 9.
//
// ALT (with LDS_TABLE only): the alternative replacement rule and its search.
//
// HALF (W = 64, register table): the sweep's reduce-scatter ends with the
// top lane bit, which leaves every lane its token's sums over both halves of
// each block; the prefixes at block middles and ends go to LDS, Algorithm 9's
// search runs over these 2 NB half-block ends, and the rebuild and Algorithm
// 10 work on the chosen half: 32 topics per token, as the W = 32 groups do (two
// tokens per load instruction, half the bytes, 31 exchanges in the search).
template <int W, bool LDS_TABLE, bool SMALL, bool ALT = false, bool HALF = false,
          int WPB = kWavesPerBlock>
__global__ __launch_bounds__(WPB * kWave) __attribute__((amdgpu_waves_per_eu(LDA_WAVES_PER_EU)))
void butterfly_kernel(
    const float *__restrict__ theta, const float *__restrict__ phi, DocSource docs,
    const int32_t *__restrict__ word_id, UniformSource u,
    int32_t *__restrict__ z, int64_t N, int K, uint32_t theta_bytes, uint32_t phi_bytes) {
  static_assert(!ALT || LDS_TABLE, "the alternative table is searched in LDS");
  static_assert(!HALF || (W == kWave && !LDS_TABLE), "half-block tail: W = 64, register table");
  extern __shared__ float lds[];
  constexpr int LOG2W = (W == 64) ? 6 : 5;
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int64_t first = ((int64_t)blockIdx.x * WPB + wave) * kWave;
  if (first >= N) return;  // whole wavefront past the end
  // Window of 64 tokens: the wavefront's own, or for the last wavefront the
  // final 64 tokens (re-drawing some of the previous wavefront's, which it
  // does not store).  SMALL (N < 64): tokens past N repeat token N - 1, so
  // that every lane takes part in every exchange (the paper's "staying
  // awake" rule).
  const int64_t t0 = SMALL ? 0 : (first + kWave <= N ? first : N - kWave);
  const int last = SMALL ? (int)(N - 1) : kWave - 1;
  const int64_t n = SMALL ? (lane < last ? lane : last) : t0 + lane;
  const bool store = SMALL ? lane < N : t0 + lane >= first;

  const int doc = docs.wave_doc(n, t0, t0 + last);
  const int word = word_id[n];
  const float un = u(n);
  // blocks of W topics; a remnant of K mod W topics becomes block 0, padded
  // at its front with empty topics
  const int NB = (K + W - 1) >> LOG2W;
  Wave<W, SMALL> w;
  init_wave<W, SMALL>(w, theta, phi, theta_bytes, phi_bytes, word_id, t0, last, K,
                      lane, doc, word);
  float *region = lds + wave * region_rows(NB, W, LDS_TABLE, HALF) * kWave;

  float a[W];
  float h[HALF ? W / 2 : 1];  // HALF: the chosen half-block's table
  float sum, stop, low, high;
  int blk;       // chosen block, or with HALF (NB > 1) chosen half-block
  bool halves = false;
  if (NB == 1) {
    // One block: its table is built once and searched directly.
    blk = 0;
    load_tile_blocks<W, SMALL, true>(w, a, 0, w.c0);
    if constexpr (LDS_TABLE)
      butterfly_block<W, ALT>(a, w.r, RowStore{region + lane, kWave, true});
    else
      butterfly_block<W>(a, w.r, NoStore{});
    sum = a[W - 1];
    stop = sum * un;
    low = 0.0f;
    high = sum;
  } else {
    // Sweep over the blocks: the running prefix at each block's end (row b),
    // or with HALF at its middle (row 2b) and end (row 2b + 1).
    sum = 0.0f;
    float lower = 0.0f;
    if (w.mode == kAnyDocs) {
      for (int b = 0; b < NB; ++b) {
        const float total = sweep_block_any<W, SMALL, HALF>(w, launder(w.wp), b, lower);
        if constexpr (HALF) region[(2 * b) * kWave + lane] = sum + lower;
        sum += total;
        region[(HALF ? 2 * b + 1 : b) * kWave + lane] = sum;
      }
    } else if (w.mode == kOneDoc) {
      sum = sweep_blocks<W, SMALL, HALF, kOneDoc>(w, a, region, lane, NB);
    } else {
      sum = sweep_blocks<W, SMALL, HALF, kTwoDocs>(w, a, region, lane, NB);
    }
    stop = sum * un;
    // Algorithm 9: binary search over the last row of each block (with HALF,
    // of each half-block).
    int lo = 0, hi = (HALF ? 2 * NB : NB) - 1;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (stop < region[mid * kWave + lane])
        hi = mid;
      else
        lo = mid + 1;
    }
    blk = lo;
    low = lo > 0 ? region[(lo - 1) * kWave + lane] : 0.0f;
    high = region[lo * kWave + lane];
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if constexpr (HALF) {
      // Rebuild every token's chosen half-block: lanes 32 g + r hold topic
      // c0 + 32 blk_k + r of the tokens k of half-wave g.
      halves = true;
      const Wave<W / 2, SMALL> wh = half_wave(w, lane);
      load_tile_blocks<W / 2, SMALL, true>(wh, h, blk, w.c0);
      butterfly_block<W / 2>(h, wh.r, NoStore{});
    } else {
      // Rebuild every token's chosen block.
      load_tile_blocks<W, SMALL, true>(w, a, blk, w.c0);
      if constexpr (LDS_TABLE)
        butterfly_block<W, ALT>(a, w.r, RowStore{region + lane, kWave, true});
      else
        butterfly_block<W>(a, w.r, NoStore{});
    }
  }
  if constexpr (LDS_TABLE) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
  // Algorithm 10.  Empty topics of block 0 are never chosen: their prefix
  // equals the prefix before them, which is never above stop >= 0, except
  // when S = 0, where every comparison fails and the result is K - 1.
  int j;
  if constexpr (ALT) {
    j = w.c0 + blk * W + inblock_search_alt<W>(region, w.r, w.gbase, stop, low, high);
  } else if constexpr (HALF) {
    if (halves)
      j = w.c0 + blk * (W / 2) +
          inblock_search<W / 2, false>(h, nullptr, lane & (W / 2 - 1), lane & (W / 2), stop,
                                       low, high);
    else
      j = w.c0 + blk * W + inblock_search<W, false>(a, nullptr, w.r, w.gbase, stop, low, high);
  } else {
    j = w.c0 + blk * W + inblock_search<W, LDS_TABLE>(a, region, w.r, w.gbase, stop, low, high);
  }
  if (store) z[n] = j;
}

// ---------------------------------------------------------------------------
// Leaf kernel with 32-topic prefix rows (K divisible by 4, from
// LDA_EIGHTHS_MIN_K topics to LDA_EIGHTHS_MAX_BLOCKS 256-topic blocks,
// N >= 64; when K is not a multiple of 256 the first block begins with
// 256 - K mod 256 empty topics, as the remnant block of butterfly_kernel).
//
// The sweep reads every token's phi row with 16-byte loads: lane l takes the
// leaf of topics [4l, 4l + 4) of each 256-topic block, so one load
// instruction brings one token's 256 topics, and the lane sums its leaf's
// four products (dot4).  The 64 leaf sums of a token are then combined across
// lanes as single products are in butterfly_kernel, but the reduce-scatter
// first sums over lane bits 2, 1, 0 (the eight lanes of a 32-topic "eighth"
// of the block) and then only exchanges over lane bits 3, 4, 5, so that every
// lane ends with its own token's eight eighth sums rather than their total.
// The running prefixes at the 8 NB eighth ends go to LDS; Algorithm 9's
// search runs over them, and the chosen 32-topic chunk is rebuilt with
// Algorithm 8's butterfly and searched with Algorithm 10, by the W = 32
// machinery of the half-block tail (two tokens per load instruction).  Against
// the one-topic sweep this reads the same bytes with four times fewer load
// instructions (a 64-lane dword load costs the memory pipeline about as many
// cycles as a 16-byte one), and the rebuild reads 128 B of phi per token.
//
// Register slot s of the sweep holds token eighth_slot_token(s): with the
// stage order above, lane l ends with slot (l5 l4 l3 l0 l1 l2) (bits listed
// from bit 0 up), so slots are loaded with the inverse permutation and lane l
// finishes with token l.  Afterwards eighth q of the lane's token is in
// register bitrev3(q).
constexpr int kLeaf = 4;
constexpr int kBlock4 = kWave * kLeaf;  // topics per block

__host__ __device__ constexpr int eighth_slot_token(int s) {
  return ((s >> 3) & 1) | (((s >> 4) & 1) << 1) | (((s >> 5) & 1) << 2) |
         (((s >> 2) & 1) << 3) | (((s >> 1) & 1) << 4) | ((s & 1) << 5);
}
__host__ __device__ constexpr int bitrev3(int q) { return ((q & 1) << 2) | (q & 2) | ((q >> 2) & 1); }

// Slots of a sweep block are taken in pair order 0, 32, 1, 33, ...: as soon
// as slots s and s + 32 have their leaf sums, the first reduce-scatter stage
// combines them, so only 32 partial sums stay live.
__device__ __host__ constexpr int pair_token(int i) { return (i >> 1) + ((i & 1) << 5); }

// Sums registers k and k + BIT (k < BIT) across lanes l and l xor L: lanes
// with L clear keep token k's sum, lanes with L set token k + BIT's.
template <int L, int BIT, int N>
__device__ __forceinline__ void pair_stage(float (&a)[N]) {
#pragma unroll
  for (int k = 0; k < BIT; ++k) {
    if constexpr (L >= 4) {
      half_swap<L>(a[k], a[k + BIT]);
      a[k] = a[k] + a[k + BIT];
    } else {
      a[k] = pair_sum<L>(a[k], a[k + BIT]);
    }
  }
}

// First topic of this lane's leaf in block `blk` (negative in the front
// padding of block 0 when K is not a multiple of 256), and the byte offset its
// loads use (padding leaves read topics 0..3; their products are replaced by
// zero where they are used).
__device__ __forceinline__ int leaf_topic(int c0, int blk, int r) {
  return c0 + blk * kBlock4 + kLeaf * r;
}
__device__ __forceinline__ uint32_t leaf_bytes(int c0, int blk, int r) {
  const int t = leaf_topic(c0, blk, r);
  return (uint32_t)(t > 0 ? t : 0) * 4u;
}

// Theta leaf of block `blk` at row offset `row`; zero for a padding leaf.
template <bool PAD>
__device__ __forceinline__ f4 theta_leaf(rsrc_t rs, int c0, int blk, int r, uint32_t row) {
  const f4 t = load_f32x4(rs, leaf_bytes(c0, blk, r), row);
  if constexpr (PAD) {
    const f4 zero = {0.0f, 0.0f, 0.0f, 0.0f};
    return leaf_topic(c0, blk, r) >= 0 ? t : zero;
  }
  return t;
}

// Theta leaves of a wavefront whose tokens form D <= kFewMax runs of documents
// (kFewDocs): per block, each run's leaf at this lane's topics is loaded once
// and staged in LDS (lds[d * 64 + lane]); each token then reads its run's leaf
// from LDS instead of from memory.
constexpr int kFewMax = 4;
struct FewDocs {
  f4 *lds;                 // this wavefront's kFewMax x 64 leaves
  int D;                   // runs of documents in the wavefront, uniform
  uint32_t row[kFewMax];   // their theta row offsets, uniform
  int slot;                // this lane's run
};

// Loads of block `blk`'s leaves of the wavefront's runs (to be staged later).
template <bool PAD>
__device__ __forceinline__ void few_load(const FewDocs &fd, rsrc_t th_rs, int c0, int blk, int r,
                                         f4 (&st)[kFewMax]) {
#pragma unroll
  for (int d = 0; d < kFewMax; ++d)
    if (d < fd.D) st[d] = theta_leaf<PAD>(th_rs, c0, blk, r, fd.row[d]);
}

// Stage the loaded leaves in LDS.  The wavefront's earlier LDS reads are
// issued before these writes and LDS executes one wavefront's operations in
// order, so the writes may replace leaves the wavefront has read already.
__device__ __forceinline__ void few_stage(const FewDocs &fd, const f4 (&st)[kFewMax], int lane) {
#pragma unroll
  for (int d = 0; d < kFewMax; ++d)
    if (d < fd.D) fd.lds[d * kWave + lane] = st[d];
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// The staged leaf of token t's run.
__device__ __forceinline__ f4 few_leaf(const FewDocs &fd, int t, int lane) {
  return fd.lds[__builtin_amdgcn_readlane(fd.slot, t) * kWave + lane];
}

// Sweep step for one 256-topic block: win[] holds (or awaits) the phi leaves
// of the first C slots in pair order, twin[] (any documents) their theta
// leaves, th[] the theta leaves of the first / last document.  With PREFETCH
// the windows and thn[] are refilled with block `next` as the block drains.
// rows[q * 64] receives the running prefix at the end of eighth q; returns the
// prefix at the block's end.  c0 is the first topic of block 0 (PAD: K is not
// a multiple of 256 and block 0 begins with 256 - K mod 256 empty topics).
template <int MODE, bool PREFETCH, int C, int CT, bool PAD>
__device__ __forceinline__ float sweep8_block(const Wave<kWave, false> &w, const FewDocs &fd,
                                              f4 (&win)[C], f4 (&twin)[CT], f4 (&th)[2],
                                              f4 (&thn)[2], int c0, int blk, int next,
                                              float *rows, float prefix) {
  static_assert(kWave % C == 0, "the window size must divide 64");
  const uint32_t vcur = leaf_bytes(c0, blk, w.r);
  const uint32_t vnext = leaf_bytes(c0, next, w.r);
  // any documents: theta comes per token, so padding leaves are zeroed per product
  const bool real = !PAD || leaf_topic(c0, blk, w.r) >= 0;
  const int kb = MODE == kTwoDocs ? launder_int(w.kb) : kWave;
  const int lane = lane_id();
  // kFewDocs: the next block's run leaves, loaded now and staged in LDS once
  // this block's last reads of the staged leaves have been issued
  f4 st[kFewMax];
  if constexpr (MODE == kFewDocs && PREFETCH) few_load<PAD>(fd, w.th_rs, c0, next, w.r, st);
  float s[kWave / 2];
  float lo = 0.0f;
#pragma unroll
  for (int i = 0; i < kWave; ++i) {
    const int slot = pair_token(i);
    const int t = eighth_slot_token(slot);
    f4 tv;
    if constexpr (MODE == kAnyDocs || MODE == kFewDocs)
      tv = twin[i % C];
    else if constexpr (MODE == kTwoDocs)
      tv = t < kb ? th[0] : th[1];
    else
      tv = th[0];
    float v = dot4(tv, win[i % C]);
    if constexpr (PAD && MODE == kAnyDocs) v = real ? v : 0.0f;
    if (i & 1) {
      float hi = v;
      half_swap<4>(lo, hi);
      s[slot - 32] = lo + hi;
    } else {
      lo = v;
    }
    const bool refill = i + C < kWave;
    if (refill || PREFETCH) {
      const int tn = eighth_slot_token(pair_token(refill ? i + C : i + C - kWave));
      const uint32_t voff = refill ? vcur : vnext;
      if (!refill && (MODE == kOneDoc || MODE == kTwoDocs) && i + C == kWave) {
        thn[0] = theta_leaf<PAD>(w.th_rs, c0, next, w.r, w.th_off0);
        if constexpr (MODE == kTwoDocs) thn[1] = theta_leaf<PAD>(w.th_rs, c0, next, w.r, w.th_off1);
      }
      if constexpr (MODE == kFewDocs)
        if (!refill && i + C == kWave) few_stage(fd, st, lane);
      win[i % C] = load_f32x4(w.ph_rs, voff, __builtin_amdgcn_readlane(w.ph_lane, tn));
      if constexpr (MODE == kAnyDocs)
        twin[i % C] = load_f32x4(w.th_rs, voff, __builtin_amdgcn_readlane(w.th_lane, tn));
      if constexpr (MODE == kFewDocs) twin[i % C] = few_leaf(fd, tn, lane);
    }
    // keep the window rolling: no load is hoisted past this point (hoisting
    // them all would need 4 registers per token of the block)
    __builtin_amdgcn_sched_barrier(0);
  }
  pair_stage<2, 16>(s);
  pair_stage<1, 8>(s);
#pragma unroll
  for (int j = 0; j < 4; ++j) half_swap<8>(s[j], s[j + 4]);
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    half_swap<16>(s[j], s[j + 2]);
    half_swap<16>(s[j + 4], s[j + 6]);
  }
#pragma unroll
  for (int j = 0; j < 8; j += 2) half_swap<32>(s[j], s[j + 1]);
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    prefix += s[bitrev3(q)];
    rows[q * kWave] = prefix;
  }
  if constexpr (PREFETCH && (MODE == kOneDoc || MODE == kTwoDocs)) {
    th[0] = thn[0];
    if constexpr (MODE == kTwoDocs) th[1] = thn[1];
  }
  return prefix;
}

// The whole sweep over NB blocks; rows[r * 64] receives the prefix at the end
// of eighth r.  Returns the token's total.
// A sweep8 hook that does nothing.
struct NoHook {
  __device__ __forceinline__ void operator()() const {}
};

template <int MODE, int C, bool PAD, class Hook = NoHook>
__device__ __forceinline__ float sweep8(const Wave<kWave, false> &w, const FewDocs &fd, int NB,
                                        int c0, float *rows, Hook hook = Hook{}) {
  constexpr int CT = (MODE == kAnyDocs || MODE == kFewDocs) ? C : 1;
  f4 win[C], twin[CT], th[2], thn[2];
  const uint32_t v0 = leaf_bytes(c0, 0, w.r);
  if constexpr (MODE == kOneDoc || MODE == kTwoDocs) {
    th[0] = theta_leaf<PAD>(w.th_rs, c0, 0, w.r, w.th_off0);
    th[1] = MODE == kTwoDocs ? theta_leaf<PAD>(w.th_rs, c0, 0, w.r, w.th_off1) : th[0];
  }
  if constexpr (MODE == kFewDocs) {
    f4 st[kFewMax];
    few_load<PAD>(fd, w.th_rs, c0, 0, w.r, st);
    few_stage(fd, st, lane_id());
  }
#pragma unroll
  for (int i = 0; i < C; ++i) {
    const int t = eighth_slot_token(pair_token(i));
    win[i] = load_f32x4(w.ph_rs, v0, __builtin_amdgcn_readlane(w.ph_lane, t));
    if constexpr (MODE == kAnyDocs)
      twin[i] = load_f32x4(w.th_rs, v0, __builtin_amdgcn_readlane(w.th_lane, t));
    if constexpr (MODE == kFewDocs) twin[i] = few_leaf(fd, t, lane_id());
  }
  // hook() runs once, after the first block's step (loads it issues are in
  // flight during the other blocks)
  float prefix = 0.0f;
  for (int b = 0; b < NB - 1; ++b) {
    prefix = sweep8_block<MODE, true, C, CT, PAD>(w, fd, win, twin, th, thn, c0, b, b + 1,
                                                  rows + 8 * b * kWave, prefix);
    if (b == 0) hook();
  }
  prefix = sweep8_block<MODE, false, C, CT, PAD>(w, fd, win, twin, th, thn, c0, NB - 1, 0,
                                                 rows + 8 * (NB - 1) * kWave, prefix);
  if (NB == 1) hook();
  return prefix;
}

template <int C, int WPB, int WPEU, bool PAD>
__global__ __launch_bounds__(WPB * kWave) __attribute__((amdgpu_waves_per_eu(WPEU)))
void leaf_eighths_kernel(const float *__restrict__ theta, const float *__restrict__ phi,
                         DocSource docs, const int32_t *__restrict__ word_id,
                         UniformSource u, int32_t *__restrict__ z, int64_t N, int K,
                         uint32_t theta_bytes, uint32_t phi_bytes) {
  extern __shared__ float lds[];
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int64_t first = ((int64_t)blockIdx.x * WPB + wave) * kWave;
  if (first >= N) return;  // whole wavefront past the end
  // Window of 64 tokens as in butterfly_kernel (N >= 64 here).
  const int64_t t0 = first + kWave <= N ? first : N - kWave;
  const int64_t n = t0 + lane;
  const bool store = n >= first;

  const int doc = docs.wave_doc(n, t0, t0 + kWave - 1);
  const int word = word_id[n];
  const float un = u(n);
  // 256-topic blocks; with PAD block 0 starts at topic c0 < 0 (a remnant of
  // K mod 256 topics behind 256 - K mod 256 empty ones, as in butterfly_kernel)
  const int NB = (K + kBlock4 - 1) / kBlock4;
  const int c0 = K - NB * kBlock4;
  Wave<kWave, false> w;
  init_wave<kWave, false>(w, theta, phi, theta_bytes, phi_bytes, word_id, t0, kWave - 1, K,
                          lane, doc, word);
  float *region = lds + wave * 8 * NB * kWave;

  const FewDocs none{};
  float sum;
  if (w.mode == kOneDoc)
    sum = sweep8<kOneDoc, C, PAD>(w, none, NB, c0, region + lane);
  else if (w.mode == kTwoDocs)
    sum = sweep8<kTwoDocs, C, PAD>(w, none, NB, c0, region + lane);
  else
    sum = sweep8<kAnyDocs, (C > 2 ? C / 2 : C), PAD>(w, none, NB, c0, region + lane);
  const float stop = sum * un;
  // Algorithm 9 over the ends of the 8 NB eighths.
  int lo = 0, hi = 8 * NB - 1;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (stop < region[mid * kWave + lane])
      hi = mid;
    else
      lo = mid + 1;
  }
  const int chunk = lo;
  float low = lo > 0 ? region[(lo - 1) * kWave + lane] : 0.0f;
  float high = region[lo * kWave + lane];
  // Rebuild every token's chosen 32-topic chunk (W = 32 groups) and search it
  // with Algorithm 10.  Empty topics are never chosen (their prefix equals the
  // one before them); with S = 0 every comparison fails and the result is K - 1.
  const Wave<kWave / 2, false> wh = half_wave(w, lane);
  float h[kWave / 2];
  load_tile_blocks<kWave / 2, false, PAD>(wh, h, chunk, c0);
  butterfly_block<kWave / 2>(h, wh.r, NoStore{});
  const int j = c0 + chunk * (kWave / 2) +
                inblock_search<kWave / 2, false>(h, nullptr, wh.r, wh.gbase, stop, low, high);
  if (store) z[n] = j;
}

// ---------------------------------------------------------------------------
// The leaf kernel on routed tokens.  Workgroups are dispatched to the GPU's
// eight XCDs round robin (workgroup b on XCD b mod 8), and each XCD has its
// own L2.  Routing gives list x of the tokens -- those whose word falls in the
// word classes assigned to XCD x -- to the workgroups b with b mod 8 = x, so
// that each L2 caches the phi rows of one eighth of the vocabulary.  Routed
// position i holds token perm[i] (-1: padding, drawn but not stored) with
// word rword[i] and document rdoc[i]; list x is [lists[x], lists[x] +
// lists[8 + x]), a multiple of 64 long, in the original token order, so that
// the documents of a wavefront form a few runs (kFewDocs).
constexpr int kXcds = kRouteXcds;

struct RoutedTokens {
  const int32_t *perm, *rword, *rdoc;
  int64_t base[kXcds], len[kXcds];  // list starts and lengths
};

// LDS floats per wavefront of the routed kernel: the prefix rows, then the
// staged theta leaves of up to kFewMax runs.
__host__ __device__ constexpr int routed_lds_floats(int NB) {
  return 8 * NB * kWave + kFewMax * kWave * 4;
}

template <int C, int WPB, int WPEU, bool PAD>
__global__ __launch_bounds__(WPB * kWave) __attribute__((amdgpu_waves_per_eu(WPEU)))
void routed_eighths_kernel(const float *__restrict__ theta, const float *__restrict__ phi,
                           RoutedTokens rt, UniformSource u, int32_t *__restrict__ z, int K,
                           uint32_t theta_bytes, uint32_t phi_bytes) {
  extern __shared__ float lds[];
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int x = blockIdx.x % kXcds;
  const int64_t base = rt.base[x];
  const int64_t len = rt.len[x];
  const int NB = (K + kBlock4 - 1) / kBlock4;
  const int c0 = K - NB * kBlock4;
  float *region = lds + wave * routed_lds_floats(NB);
  FewDocs fd;
  fd.lds = reinterpret_cast<f4 *>(region + 8 * NB * kWave);
  // One tile of WPB wavefronts of its list per workgroup (the grid holds as
  // many tiles per list as the longest list needs).
  {
    const int64_t first = ((int64_t)(blockIdx.x / kXcds) * WPB + wave) * kWave;
    if (first >= len) return;
    const int64_t i = base + first + lane;
    const int doc = rt.rdoc[i];
    const int word = rt.rword[i];
    const int n = rt.perm[i];
    Wave<kWave, false> w;
    init_wave<kWave, false>(w, theta, phi, theta_bytes, phi_bytes, rt.rword + base, first,
                            kWave - 1, K, lane, doc, word);
    // runs of documents among the wavefront's tokens
    const int prev = __builtin_amdgcn_ds_bpermute(((lane + kWave - 1) & (kWave - 1)) << 2, doc);
    const uint64_t starts = __builtin_amdgcn_ballot_w64(lane == 0 || doc != prev);
    fd.D = __builtin_amdgcn_readfirstlane(__builtin_popcountll(starts));
    fd.slot = __builtin_popcountll(starts & ((2ull << lane) - 1ull)) - 1;
    uint64_t m = starts;
#pragma unroll
    for (int d = 0; d < kFewMax; ++d) {
      fd.row[d] = 0;
      if (m) {
        const int ln = __builtin_ctzll(m);
        m &= m - 1;
        fd.row[d] = (uint32_t)__builtin_amdgcn_readlane(doc, ln) * w.row_bytes;
      }
    }
    // The uniform's load depends on the token index's; issued before the
    // sweep it would hold up every in-order wait for the sweep's loads, so
    // it is issued after the first block's step.
    float un = 0.0f;
    const auto load_u = [&]() { un = u(n >= 0 ? n : 0); };
    float sum;
    if (fd.D == 1)
      sum = sweep8<kOneDoc, C, PAD>(w, fd, NB, c0, region + lane, load_u);
    else if (fd.D <= kFewMax)
      sum = sweep8<kFewDocs, (C > 2 ? C / 2 : C), PAD>(w, fd, NB, c0, region + lane, load_u);
    else
      sum = sweep8<kAnyDocs, (C > 2 ? C / 2 : C), PAD>(w, fd, NB, c0, region + lane, load_u);
    const float stop = sum * un;
    // Algorithm 9 over the ends of the 8 NB eighths.
    int lo = 0, hi = 8 * NB - 1;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (stop < region[mid * kWave + lane])
        hi = mid;
      else
        lo = mid + 1;
    }
    const int chunk = lo;
    float low = lo > 0 ? region[(lo - 1) * kWave + lane] : 0.0f;
    float high = region[lo * kWave + lane];
    // Rebuild and Algorithm 10 on the chosen 32-topic chunk, as in
    // leaf_eighths_kernel.
    const Wave<kWave / 2, false> wh = half_wave(w, lane);
    float h[kWave / 2];
    load_tile_blocks<kWave / 2, false, PAD>(wh, h, chunk, c0);
    butterfly_block<kWave / 2>(h, wh.r, NoStore{});
    const int j = c0 + chunk * (kWave / 2) +
                  inblock_search<kWave / 2, false>(h, nullptr, wh.r, wh.gbase, stop, low, high);
    if (n >= 0) z[n] = j;
  }
}

// ---------------------------------------------------------------------------
// Leaf groups for small K (K divisible by 4, at most 4 G topics for a group
// size G of 8, 16 or 32 lanes; N >= 64).  Sections 3 and 4 with a 4-topic
// leaf in the place of a topic: a wavefront holds 64 / G groups of G tokens,
// lane r of a group owns token r of the group and, in the tile, leaf r (topics
// c0 + 4r .. c0 + 4r + 3, c0 = K - 4G <= 0: the first 4G - K topics are
// empty) of every token of its group.  Load k brings leaf r of token k of
// every group into lane r of that group, so each load instruction reads the
// whole rows (16 G bytes) of 64 / G tokens.  Register a[k] is the leaf sum
// (dot4) of token k; Algorithm 8's butterfly over the G leaves leaves the
// table and the lane's own token's total; Algorithm 10 finds the leaf whose
// prefix range holds u * S, and the leaf's four products, reloaded for the
// lane's own token, give the topic by a scan from the prefix before the leaf.
// The theta leaf comes once per lane when each group's tokens share one
// document (GROUP_DOCS), else with every phi leaf.
template <int G, int C, bool PAD, bool GROUP_DOCS>
__device__ __forceinline__ void group_tile(float (&a)[G], rsrc_t th_rs, rsrc_t ph_rs,
                                           uint32_t voff, bool real, uint32_t ph_lane,
                                           uint32_t th_lane, int gbase) {
  static_assert(G % C == 0, "the window size must divide G");
  const f4 zero = {0.0f, 0.0f, 0.0f, 0.0f};
  f4 th = zero;
  if constexpr (GROUP_DOCS) th = real ? load_f32x4(th_rs, voff + th_lane, 0) : zero;
  // leaf of token k of the group at row offset `row` of that token (held by
  // the lane that owns the token): with G = 64 the row is uniform and goes in
  // the scalar offset, else it is fetched per lane
  const auto leaf_of = [&](rsrc_t rs, uint32_t row, int k) {
    if constexpr (G == kWave)
      return load_f32x4(rs, voff, (uint32_t)__builtin_amdgcn_readlane((int)row, k));
    else
      return load_f32x4(
          rs, voff + (uint32_t)__builtin_amdgcn_ds_bpermute((gbase + k) << 2, (int)row), 0);
  };
  f4 win[C], twin[GROUP_DOCS ? 1 : C];
#pragma unroll
  for (int k = 0; k < C; ++k) {
    win[k] = leaf_of(ph_rs, ph_lane, k);
    if constexpr (!GROUP_DOCS) twin[k] = leaf_of(th_rs, th_lane, k);
  }
#pragma unroll
  for (int k = 0; k < G; ++k) {
    const f4 tv = GROUP_DOCS ? th : twin[k % C];
    const float v = dot4(tv, win[k % C]);
    a[k] = GROUP_DOCS || real ? v : 0.0f;
    if (k + C < G) {
      win[k % C] = leaf_of(ph_rs, ph_lane, k + C);
      if constexpr (!GROUP_DOCS) twin[k % C] = leaf_of(th_rs, th_lane, k + C);
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

template <int G, int C, int WPEU, bool PAD>
__global__ __launch_bounds__(kBlockThreads) __attribute__((amdgpu_waves_per_eu(WPEU)))
void leaf_group_kernel(const float *__restrict__ theta, const float *__restrict__ phi,
                       DocSource docs, const int32_t *__restrict__ word_id,
                       UniformSource u, int32_t *__restrict__ z, int64_t N, int K,
                       uint32_t theta_bytes, uint32_t phi_bytes) {
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int64_t first = ((int64_t)blockIdx.x * kWavesPerBlock + wave) * kWave;
  if (first >= N) return;  // whole wavefront past the end
  // Window of 64 tokens as in butterfly_kernel (N >= 64 here).
  const int64_t t0 = first + kWave <= N ? first : N - kWave;
  const int64_t n = t0 + lane;
  const bool store = n >= first;
  const int doc = docs.wave_doc(n, t0, t0 + kWave - 1);
  const int word = word_id[n];
  const float un = u(n);

  const rsrc_t th_rs = make_rsrc(theta, theta_bytes);
  const rsrc_t ph_rs = make_rsrc(phi, phi_bytes);
  const uint32_t row_bytes = (uint32_t)K * 4u;
  const uint32_t ph_lane = (uint32_t)word * row_bytes;
  const uint32_t th_lane = (uint32_t)doc * row_bytes;
  const int r = lane & (G - 1), gbase = lane & ~(G - 1);
  const int c0 = K - kLeaf * G;
  const int leaf = c0 + kLeaf * r;
  const bool real = !PAD || leaf >= 0;
  const uint32_t voff = (uint32_t)(real ? leaf : 0) * 4u;
  const int gdoc = __builtin_amdgcn_ds_bpermute(gbase << 2, doc);
  const bool group_docs = __builtin_amdgcn_ballot_w64(doc == gdoc) == ~0ull;

  float a[G];
  if (group_docs)
    group_tile<G, C, PAD, true>(a, th_rs, ph_rs, voff, real, ph_lane, th_lane, gbase);
  else
    group_tile<G, C, PAD, false>(a, th_rs, ph_rs, voff, real, ph_lane, th_lane, gbase);
  butterfly_block<G>(a, r, NoStore{});
  const float total = a[G - 1];
  const float stop = total * un;
  float low = 0.0f, high = total;
  const int q = inblock_search<G, false>(a, nullptr, r, gbase, stop, low, high);
  // Leaf q of the lane's own token (never a padding leaf: the prefix there is
  // zero and stop < 0 never holds), scanned from the prefix before it; with
  // S = 0 every comparison fails and the result is K - 1.
  const int tq = c0 + kLeaf * q;
  const uint32_t qoff = (uint32_t)(tq > 0 ? tq : 0) * 4u;
  const f4 tl = load_f32x4(th_rs, qoff + th_lane, 0);
  const f4 pl = load_f32x4(ph_rs, qoff + ph_lane, 0);
  const float s0 = __builtin_fmaf(tl.x, pl.x, low);
  const float s1 = __builtin_fmaf(tl.y, pl.y, s0);
  const float s2 = __builtin_fmaf(tl.z, pl.z, s1);
  const int i = stop < s0 ? 0 : (stop < s1 ? 1 : (stop < s2 ? 2 : 3));
  if (store) z[n] = tq + i;
}

// ---------------------------------------------------------------------------
// Transposed-access kernel (Algorithms 4, 5 and 6 with the binary search of
// Algorithm 3, the paper's design before the butterfly), for comparison.
// The tile is read exactly as in the butterfly kernel (coalesced loads, one
// document's theta per lane), but instead of exchanging partial sums across
// lanes the wavefront transposes it through LDS (Algorithm 6's transposed
// read of a[]): lane r reads back token r's 64 products and sums them in topic
// order.  The search is the plain one over the block ends, then a linear scan
// of the chosen block's full prefix (rebuilt and transposed the same way).
constexpr int kTileStride = kWave + 1;  // row padding: conflict-free LDS access
constexpr int kTileFloats = kWave * kTileStride;

__device__ __forceinline__ void lds_order() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Store the tile (row k = token k) and return this lane's token's sum over
// the block's topics, added in topic order.
__device__ __forceinline__ float transpose_sum(float *tile, const float (&a)[kWave], int lane) {
#pragma unroll
  for (int k = 0; k < kWave; ++k) tile[k * kTileStride + lane] = a[k];
  lds_order();
  float s = 0.0f;
#pragma unroll
  for (int c = 0; c < kWave; ++c) s += tile[lane * kTileStride + c];
  return s;
}

template <bool SMALL>
__global__ __launch_bounds__(kBlockThreads) __attribute__((amdgpu_waves_per_eu(LDA_WAVES_PER_EU)))
void transposed_kernel(const float *__restrict__ theta, const float *__restrict__ phi,
                       DocSource docs, const int32_t *__restrict__ word_id,
                       UniformSource u, int32_t *__restrict__ z, int64_t N, int K,
                       uint32_t theta_bytes, uint32_t phi_bytes) {
  extern __shared__ float lds[];
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int64_t first = ((int64_t)blockIdx.x * kWavesPerBlock + wave) * kWave;
  if (first >= N) return;
  const int64_t t0 = SMALL ? 0 : (first + kWave <= N ? first : N - kWave);
  const int last = SMALL ? (int)(N - 1) : kWave - 1;
  const int64_t n = SMALL ? (lane < last ? lane : last) : t0 + lane;
  const bool store = SMALL ? lane < N : t0 + lane >= first;

  const int doc = docs.wave_doc(n, t0, t0 + last);
  const int word = word_id[n];
  const float un = u(n);
  const int NB = (K + kWave - 1) / kWave;  // the remnant is block 0, padded
  Wave<kWave, SMALL> w;
  init_wave<kWave, SMALL>(w, theta, phi, theta_bytes, phi_bytes, word_id, t0, last, K,
                          lane, doc, word);
  float *tile = lds + wave * (kTileFloats + NB * kWave);
  float *region = tile + kTileFloats;

  float a[kWave];
  float sum = 0.0f;
  if (w.mode == kAnyDocs) {
    for (int b = 0; b < NB; ++b) {
      load_tile_blocks<kWave, SMALL, true>(w, a, b, w.c0);  // theta per token
      lds_order();
      sum += transpose_sum(tile, a, lane);
      region[b * kWave + lane] = sum;
    }
  } else {
    float th0 = 0.0f, th1 = 0.0f;
    issue_theta(w, 0, th0, th1);
    issue_phi<kWave, SMALL, 0, kWave>(w, w.wp, a, 0);
    for (int b = 0; b < NB; ++b) {
      const bool real = topic_of(w, b) >= 0;
      const float t0v = real ? th0 : 0.0f, t1v = real ? th1 : 0.0f;
      const int kb = launder_int(w.kb);
#pragma unroll
      for (int k = 0; k < kWave; ++k) a[k] *= (k < kb) ? t0v : t1v;
      lds_order();  // the previous block's reads precede these writes
#pragma unroll
      for (int k = 0; k < kWave; ++k) tile[k * kTileStride + lane] = a[k];
      if (b + 1 < NB) {  // next block's loads overlap the transposed read
        issue_theta(w, b + 1, th0, th1);
        issue_phi<kWave, SMALL, 0, kWave>(w, launder(w.wp), a, b + 1);
      }
      lds_order();
      float s = 0.0f;
#pragma unroll
      for (int c = 0; c < kWave; ++c) s += tile[lane * kTileStride + c];
      sum += s;
      region[b * kWave + lane] = sum;
    }
  }
  const float stop = sum * un;
  // Binary search over the block ends (the entries Algorithm 3 would visit
  // at block granularity), then the chosen block's full prefix.
  int lo = 0, hi = NB - 1;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (stop < region[mid * kWave + lane])
      hi = mid;
    else
      lo = mid + 1;
  }
  const float low = lo > 0 ? region[(lo - 1) * kWave + lane] : 0.0f;
  load_tile_blocks<kWave, SMALL, true>(w, a, lo, w.c0);
  lds_order();
#pragma unroll
  for (int k = 0; k < kWave; ++k) tile[k * kTileStride + lane] = a[k];
  lds_order();
  // Algorithm 2 over the block: the first topic whose prefix exceeds stop
  // (the last topic if rounding leaves none).
  float q = low;
  int off = kWave - 1;
  bool found = false;
#pragma unroll
  for (int c = 0; c < kWave; ++c) {
    q += tile[lane * kTileStride + c];
    const bool hit = !found && stop < q;
    off = hit ? c : off;
    found = found || hit;
  }
  if (store) z[n] = w.c0 + lo * kWave + off;
}

// ---------------------------------------------------------------------------
// Table dump: the per-lane table p[K] of Algorithm 7 for every token, built
// with the same tile loads and butterfly as the draw's rebuild step.
template <int W, bool SMALL>
__global__ __launch_bounds__(kBlockThreads) void table_kernel(
    const float *__restrict__ theta, const float *__restrict__ phi,
    const int32_t *__restrict__ doc_id, const int32_t *__restrict__ word_id,
    float *__restrict__ table, int64_t N, int K, uint32_t theta_bytes,
    uint32_t phi_bytes) {
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int64_t first = ((int64_t)blockIdx.x * kWavesPerBlock + wave) * kWave;
  if (first >= N) return;
  // Groups of W tokens start at multiples of W: pad the last window by
  // repeating token N - 1 (tables of shifted windows would differ).
  const int64_t t0 = first;
  const int last = (int)(N - 1 - first < kWave - 1 ? N - 1 - first : kWave - 1);
  const int64_t n = t0 + (lane < last ? lane : last);
  const bool store = lane <= last;
  const int doc = doc_id[n];
  Wave<W, true> w;
  init_wave<W, true>(w, theta, phi, theta_bytes, phi_bytes, word_id, t0, last, K,
                     lane, doc, word_id[n]);
  const int R = w.R;
  const int NB = K / W;
  float *out = table + n * (int64_t)K;

  const float *th_row = theta + (int64_t)doc * K;
  const float *ph_row = phi + (int64_t)word_id[n] * K;
  float sum = 0.0f;
  for (int j = 0; j < R; ++j) {
    sum = prefix_step(sum, th_row[j], ph_row[j]);
    if (store) out[j] = sum;
  }
  for (int b = 0; b < NB; ++b) {
    float a[W];
    load_tile_blocks<W, true, false>(w, a, b, R);
    butterfly_block<W>(a, w.r, RowStore{out + R + b * W, 1, store});
    sum += a[W - 1];
    if (store) out[R + b * W + W - 1] = sum;
  }
}

// ---------------------------------------------------------------------------
// Document-per-lane driver (Algorithm 7 with the theta cache of Algorithm 5):
// group g of 64 documents [64 g, 64 g + 64), lane l document 64 g + l.  A
// master index i runs while any lane's document has a token i; lane l then
// draws token min(i, N[m] - 1) of its document (lanes whose document is done
// repeat its last token without storing, so that every lane takes part in
// every exchange; lanes of empty documents or past M compute on token 0).
// M / 64 groups are far too few wavefronts for 256 CUs, so S wavefronts
// share a group, wavefront s taking the master indices i = s, s + S, ...
// (wavefront index = g * S + s).
// Each iteration is one butterfly draw of a wavefront of 64 tokens from 64
// documents: a sweep with one theta and one phi row per token, Algorithm 9's
// block search, the rebuild of each token's chosen block and Algorithm 10.
//
// THETA_LDS: the theta factors are loaded once per wavefront into LDS in the
// transposed order of Algorithm 5 -- entry (b, k) of lane l is theta of token
// k's document at topic c0 + b W + r -- and read from there in every
// iteration; otherwise every iteration reads them from memory again.
template <int W, bool THETA_LDS>
__device__ __forceinline__ float theta_factor(const Wave<W, false> &w, const float *cache,
                                              int blk, int k, uint32_t voff) {
  if constexpr (THETA_LDS)
    return cache[(blk * W + k) * kWave + lane_id()];
  else
    return topic_of(w, blk) >= 0 ? load_row<W>(w.th_rs, voff, theta_row(w, k)) : 0.0f;
}

template <int W, bool THETA_LDS>
__global__ __launch_bounds__(kBlockThreads) __attribute__((amdgpu_waves_per_eu(LDA_WAVES_PER_EU)))
void doc_lanes_kernel(const float *__restrict__ theta, const float *__restrict__ phi,
                      const int64_t *__restrict__ offsets, const int32_t *__restrict__ word_id,
                      UniformSource u, int32_t *__restrict__ z, int64_t N, int M,
                      int K, int S, uint32_t theta_bytes, uint32_t phi_bytes) {
  extern __shared__ float lds[];
  constexpr int LOG2W = (W == 64) ? 6 : 5;
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int64_t wave_id = (int64_t)blockIdx.x * kWavesPerBlock + wave;
  const int64_t first_doc = wave_id / S * kWave;
  const int stride0 = (int)(wave_id % S);
  if (first_doc >= M) return;
  const int64_t m = first_doc + lane;
  const bool valid = m < M;
  const int doc = valid ? (int)m : 0;
  // (clamped to [0, N], so that any offsets keep every access in bounds)
  const int64_t start = valid ? min(max(offsets[m], (int64_t)0), N) : 0;
  const int64_t len = valid ? min(max(offsets[m + 1], start), N) - start : 0;

  const int NB = (K + W - 1) >> LOG2W;
  Wave<W, false> w;
  w.th_rs = make_rsrc(theta, theta_bytes);
  w.ph_rs = make_rsrc(phi, phi_bytes);
  w.wp = nullptr;
  w.last = kWave - 1;
  w.row_bytes = (uint32_t)K * 4u;
  w.R = K & (W - 1);
  w.c0 = w.R ? w.R - W : 0;
  w.r = lane & (W - 1);
  w.gbase = lane & ~(W - 1);
  w.doc = doc;
  w.mode = kAnyDocs;
  w.kb = 0;
  w.th_off0 = w.th_off1 = 0;
  w.th_lane = (uint32_t)doc * w.row_bytes;

  const int cache_rows = THETA_LDS ? NB * W : 0;
  float *cache = lds + wave * (cache_rows + NB) * kWave;
  float *region = cache + cache_rows * kWave;
  if constexpr (THETA_LDS) {
    for (int b = 0; b < NB; ++b) {
      const uint32_t voff = col_bytes(w, b);
      const bool real = topic_of(w, b) >= 0;
#pragma unroll 8
      for (int k = 0; k < W; ++k) {
        const float th = load_row<W>(w.th_rs, voff, theta_row(w, k));
        cache[(b * W + k) * kWave + lane] = real ? th : 0.0f;
      }
    }
  }

  for (int64_t i = stride0; __builtin_amdgcn_ballot_w64(i < len) != 0; i += S) {
    const int64_t n = len > 0 ? start + (i < len ? i : len - 1) : 0;
    const bool store = i < len;
    w.ph_lane = (uint32_t)word_id[n] * w.row_bytes;
    const float un = u(n);

    float a[W];
    float sum = 0.0f, stop, low, high;
    int blk = 0;
    // sweep: block totals and the running prefix at each block's end
    for (int b = 0; b < NB; ++b) {
      const uint32_t voff = col_bytes(w, b);
#pragma unroll
      for (int k = 0; k < W; ++k) {
        const float ph = load_row<W>(w.ph_rs, voff, (uint32_t)group_value<W>((int)w.ph_lane, k));
        a[k] = theta_factor<W, THETA_LDS>(w, cache, b, k, voff) * ph;
      }
      reduce_stage<W, W / 2>(a);
      reduce_rest<W, false, W / 4, false>(w, nullptr, a, 0);
      sum += a[0];
      region[b * kWave + lane] = sum;
    }
    stop = sum * un;
    // Algorithm 9
    int lo = 0, hi = NB - 1;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (stop < region[mid * kWave + lane])
        hi = mid;
      else
        lo = mid + 1;
    }
    blk = lo;
    low = lo > 0 ? region[(lo - 1) * kWave + lane] : 0.0f;
    high = region[lo * kWave + lane];
    // rebuild each token's chosen block
#pragma unroll
    for (int k = 0; k < W; ++k) {
      const int bk = group_value<W>(blk, k);
      const int t = w.c0 + bk * W + w.r;
      const uint32_t voff = (uint32_t)(t < 0 ? 0 : t) * 4u;
      const float ph = load_row<W>(w.ph_rs, voff, (uint32_t)group_value<W>((int)w.ph_lane, k));
      float th;
      if constexpr (THETA_LDS)
        th = cache[(bk * W + k) * kWave + lane];
      else
        th = t < 0 ? 0.0f : load_row<W>(w.th_rs, voff, theta_row(w, k));
      a[k] = th * ph;
    }
    butterfly_block<W>(a, w.r, NoStore{});
    const int j = w.c0 + blk * W + inblock_search<W, false>(a, nullptr, w.r, w.gbase, stop, low, high);
    if (store) z[n] = j;
  }
}

// ---------------------------------------------------------------------------
// The in-kernel uniforms written out: u[i] = uniform of token first + i.
__global__ __launch_bounds__(256) void uniforms_kernel(float *__restrict__ u, int64_t count,
                                                       int64_t first, UniformSource us) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += stride)
    u[i] = us(first + i);
}

// ---------------------------------------------------------------------------
thread_local hipError_t g_last_hip = hipSuccess;

int check_args(const void *theta, const void *phi, const void *doc_id,
               const void *word_id, const void *u, const void *z, int64_t N,
               int32_t M, int32_t V, int32_t K) {
  if (N < 0 || M <= 0 || V <= 0 || K <= 0) return LDA_ERR_SHAPE;
  if (K > LDA_MAX_K) return LDA_ERR_UNSUPPORTED;
  // theta and phi are addressed with 31-bit byte offsets
  if ((int64_t)M * K * 4 > LDA_MAX_TABLE_BYTES ||
      (int64_t)V * K * 4 > LDA_MAX_TABLE_BYTES)
    return LDA_ERR_UNSUPPORTED;
  if (N == 0) return LDA_OK;
  const void *ptrs[] = {theta, phi, doc_id, word_id, u, z};
  for (const void *p : ptrs) {
    if (!p) return LDA_ERR_NULL;
    if (reinterpret_cast<uintptr_t>(p) & 3u) return LDA_ERR_ALIGN;
  }
  return LDA_OK;
}

int finish_launch() {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    g_last_hip = e;
    return LDA_ERR_HIP;
  }
  return LDA_OK;
}

int width_for(int32_t K) { return K >= 64 ? 64 : 32; }

// The rebuilt block's table goes to LDS only for block counts up to
// LDA_LDS_TABLE_MAX_BLOCKS.  Measured on MI355X, the register table searched
// with the search-assist shuffle loop is faster at every K (the LDS table
// costs 16 KiB per wavefront and with it occupancy), so the default is 0 and
// the LDS variant is kept for comparison builds.
bool lds_table_for(int32_t K) {
  const int nb = (K + width_for(K) - 1) / width_for(K);
  return nb <= LDA_LDS_TABLE_MAX_BLOCKS;
}

// The half-block tail (W = 64) for block counts up to LDA_HALF_MAX_BLOCKS:
// it doubles the LDS rows of the block prefixes.
bool half_tail_for(int32_t K) {
  const int nb = (K + 63) / 64;
  return nb >= 2 && nb <= LDA_HALF_MAX_BLOCKS;
}

dim3 wave_grid(int64_t N, int wpb = kWavesPerBlock) {
  const int64_t waves = (N + kWave - 1) / kWave;
  return dim3((unsigned)((waves + wpb - 1) / wpb));
}

template <int KMAX>
void launch_naive(const float *theta, const float *phi, DocSource d, const int32_t *w,
                  UniformSource u, int32_t *z, int64_t N, int32_t K, hipStream_t s) {
  const dim3 grid((unsigned)((N + 255) / 256));
  naive_kernel<KMAX><<<grid, 256, 0, s>>>(theta, phi, d, w, u, z, N, K);
}

// 256-topic blocks of the eighths kernel (the remnant of K mod 256 included).
int eighths_blocks(int32_t K) { return (K + kBlock4 - 1) / kBlock4; }

// Wavefronts per workgroup of the eighths kernel: 4 while three such
// workgroups fit in a CU's LDS (8 rows of 64 floats per block and wavefront),
// else 2.
bool eighths_wide_groups(int32_t K) {
  return 3LL * 4 * 8 * eighths_blocks(K) * kWave * (int64_t)sizeof(float) <= 160 * 1024;
}

template <int C, int WPEU, bool PAD>
void launch_eighths(const float *theta, const float *phi, DocSource d, const int32_t *wd,
                    UniformSource u, int32_t *z, int64_t N, int32_t M, int32_t V, int32_t K,
                    hipStream_t s) {
  const uint32_t tb = (uint32_t)((int64_t)M * K * 4);
  const uint32_t pb = (uint32_t)((int64_t)V * K * 4);
  const size_t rows = (size_t)8 * eighths_blocks(K) * kWave * sizeof(float);
  if (eighths_wide_groups(K))
    leaf_eighths_kernel<C, 4, WPEU, PAD><<<wave_grid(N, 4), 4 * kWave, 4 * rows, s>>>(
        theta, phi, d, wd, u, z, N, K, tb, pb);
  else
    leaf_eighths_kernel<C, 2, WPEU, PAD><<<wave_grid(N, 2), 2 * kWave, 2 * rows, s>>>(
        theta, phi, d, wd, u, z, N, K, tb, pb);
}

template <int C, int WPEU>
void launch_eighths(const float *theta, const float *phi, DocSource d, const int32_t *wd,
                    UniformSource u, int32_t *z, int64_t N, int32_t M, int32_t V, int32_t K,
                    hipStream_t s) {
  if (K % kBlock4 == 0)
    launch_eighths<C, WPEU, false>(theta, phi, d, wd, u, z, N, M, V, K, s);
  else
    launch_eighths<C, WPEU, true>(theta, phi, d, wd, u, z, N, M, V, K, s);
}

// The leaf-group kernel: K divisible by 4, up to LDA_GROUP_MAX_K (at most
// 256) topics, N >= 64; groups of 8, 16, 32 or 64 lanes for K up to 32, 64,
// 128, 256.  Measured on MI355X against the kernels it replaces there: 2.0x to
// 2.6x faster than the one-topic kernel for K = 16 ... 128, 5-8% faster than
// the eighths kernel for K = 144 ... 256.
bool groups_for(int64_t N, int32_t K) {
  return N >= kWave && K % kLeaf == 0 && K <= LDA_GROUP_MAX_K && K <= kLeaf * kWave;
}

template <int G>
void launch_groups(const float *theta, const float *phi, DocSource d, const int32_t *wd,
                   UniformSource u, int32_t *z, int64_t N, int32_t M, int32_t V, int32_t K,
                   hipStream_t s) {
  constexpr int C = LDA_GROUP_WINDOW < G ? LDA_GROUP_WINDOW : G;
  const uint32_t tb = (uint32_t)((int64_t)M * K * 4);
  const uint32_t pb = (uint32_t)((int64_t)V * K * 4);
  if (K == kLeaf * G)
    leaf_group_kernel<G, C, LDA_GROUP_WAVES_PER_EU, false><<<wave_grid(N), kBlockThreads, 0, s>>>(
        theta, phi, d, wd, u, z, N, K, tb, pb);
  else
    leaf_group_kernel<G, C, LDA_GROUP_WAVES_PER_EU, true><<<wave_grid(N), kBlockThreads, 0, s>>>(
        theta, phi, d, wd, u, z, N, K, tb, pb);
}

// Launch of the routed kernel over lists of at most max_len positions: 16
// tokens in flight per wavefront at 2 wavefronts per SIMD for every K (the
// few-documents path halves the window), 4 wavefronts per workgroup while
// three workgroups fit in LDS.
template <bool PAD>
void launch_routed(const float *theta, const float *phi, const RoutedTokens &rt, UniformSource u,
                   int32_t *z, int64_t max_len, int32_t M, int32_t V, int32_t K, hipStream_t s) {
  constexpr int C = LDA_EIGHTHS_WINDOW, WPEU = LDA_EIGHTHS_WAVES_PER_EU;
  const uint32_t tb = (uint32_t)((int64_t)M * K * 4);
  const uint32_t pb = (uint32_t)((int64_t)V * K * 4);
  const size_t per_wave = (size_t)routed_lds_floats(eighths_blocks(K)) * sizeof(float);
  if (3 * 4 * per_wave <= 160 * 1024) {
    const int64_t tiles = (max_len + 4 * kWave - 1) / (4 * kWave);
    routed_eighths_kernel<C, 4, WPEU, PAD><<<(unsigned)(kXcds * tiles), 4 * kWave, 4 * per_wave, s>>>(
        theta, phi, rt, u, z, K, tb, pb);
  } else {
    const int64_t tiles = (max_len + 2 * kWave - 1) / (2 * kWave);
    routed_eighths_kernel<C, 2, WPEU, PAD><<<(unsigned)(kXcds * tiles), 2 * kWave, 2 * per_wave, s>>>(
        theta, phi, rt, u, z, K, tb, pb);
  }
}

// The eighths kernel takes K divisible by 4 (16-byte leaves) from
// LDA_EIGHTHS_MIN_K topics to LDA_EIGHTHS_MAX_BLOCKS 256-topic blocks, for
// N >= 64.  Measured on MI355X against the one-topic kernel: 15-30% faster
// from K = 144 (K = 144 ... 240 on the paper-shaped corpus), 7% at K = 256,
// 4% at K = 1024, 5% at K = 2048; 3-4% slower at K = 80 and 112, whose
// padding fills most of the block.  (The dispatch gives K up to 256 to the
// leaf-group kernel first.)
bool eighths_for(int64_t N, int32_t K) {
  return N >= kWave && K % kLeaf == 0 && K >= LDA_EIGHTHS_MIN_K &&
         eighths_blocks(K) <= LDA_EIGHTHS_MAX_BLOCKS;
}

void launch_transposed(const float *theta, const float *phi, DocSource d,
                       const int32_t *wd, UniformSource u, int32_t *z, int64_t N,
                       int32_t M, int32_t V, int32_t K, hipStream_t s) {
  const int nb = (K + kWave - 1) / kWave;
  const size_t lds = (size_t)kWavesPerBlock * (kTileFloats + nb * kWave) * sizeof(float);
  const uint32_t tb = (uint32_t)((int64_t)M * K * 4);
  const uint32_t pb = (uint32_t)((int64_t)V * K * 4);
  if (N < kWave)
    transposed_kernel<true><<<wave_grid(N), kBlockThreads, lds, s>>>(theta, phi, d, wd, u, z, N,
                                                                      K, tb, pb);
  else
    transposed_kernel<false><<<wave_grid(N), kBlockThreads, lds, s>>>(theta, phi, d, wd, u, z,
                                                                       N, K, tb, pb);
}

template <int W, bool LDS_TABLE, bool ALT = false, bool HALF = false, int WPB = kWavesPerBlock>
void launch_butterfly(const float *theta, const float *phi, DocSource d,
                      const int32_t *wd, UniformSource u, int32_t *z, int64_t N,
                      int32_t M, int32_t V, int32_t K, hipStream_t s) {
  const int nb = (K + W - 1) / W;  // blocks, the remnant included
  const size_t lds = (size_t)WPB * region_rows(nb, W, LDS_TABLE, HALF) * kWave * sizeof(float);
  const uint32_t tb = (uint32_t)((int64_t)M * K * 4);
  const uint32_t pb = (uint32_t)((int64_t)V * K * 4);
  if (N < kWave)
    butterfly_kernel<W, LDS_TABLE, true, ALT, HALF, WPB><<<wave_grid(N, WPB), WPB * kWave, lds, s>>>(
        theta, phi, d, wd, u, z, N, K, tb, pb);
  else
    butterfly_kernel<W, LDS_TABLE, false, ALT, HALF, WPB><<<wave_grid(N, WPB), WPB * kWave, lds, s>>>(
        theta, phi, d, wd, u, z, N, K, tb, pb);
}


// The W = 32 / 64 butterfly kernel with a chosen table: in registers with the
// paper's search-assist loop, in LDS with direct reads, or the alternative
// rule's table in LDS.
template <bool LDS_TABLE, bool ALT>
void launch_table_variant(const float *theta, const float *phi, DocSource d,
                          const int32_t *word_id, UniformSource u, int32_t *z, int64_t N,
                          int32_t M, int32_t V, int32_t K, hipStream_t s) {
  if (width_for(K) == 64)
    launch_butterfly<64, LDS_TABLE, ALT>(theta, phi, d, word_id, u, z, N, M, V, K, s);
  else
    launch_butterfly<32, LDS_TABLE, ALT>(theta, phi, d, word_id, u, z, N, M, V, K, s);
}

// LDS of the document-per-lane driver per workgroup: the block-end prefixes,
// and with the theta cache K rounded up to W rows of 64 floats per wavefront.
size_t doc_lanes_lds(int32_t K, bool theta_lds) {
  const int W = width_for(K);
  const int nb = (K + W - 1) / W;
  return (size_t)kWavesPerBlock * ((theta_lds ? nb * W : 0) + nb) * kWave * sizeof(float);
}

size_t doc_lanes_cache_bytes(int32_t K) {
  const int W = width_for(K);
  const int nb = (K + W - 1) / W;
  return (size_t)nb * W * kWave * sizeof(float);
}

// Wavefronts per group of 64 documents: enough for about
// LDA_DOC_LANES_TARGET_WAVES wavefronts in all, at most the mean document
// length (beyond it most wavefronts would find no token).
int doc_lanes_split(int64_t N, int32_t M) {
  const int64_t groups = (M + kWave - 1) / kWave;
  int64_t S = (LDA_DOC_LANES_TARGET_WAVES + groups - 1) / groups;
  const int64_t mean_len = (N + M - 1) / M;
  if (S > mean_len) S = mean_len;
  return (int)(S < 1 ? 1 : S);
}

template <int W, bool THETA_LDS>
void launch_doc_lanes(const float *theta, const float *phi, const int64_t *off,
                      const int32_t *wd, UniformSource u, int32_t *z, int64_t N, int32_t M,
                      int32_t V, int32_t K, hipStream_t s) {
  const uint32_t tb = (uint32_t)((int64_t)M * K * 4);
  const uint32_t pb = (uint32_t)((int64_t)V * K * 4);
  const int S = doc_lanes_split(N, M);
  const int64_t groups = (M + kWave - 1) / kWave;
  doc_lanes_kernel<W, THETA_LDS>
      <<<wave_grid(groups * S * kWave), kBlockThreads, doc_lanes_lds(K, THETA_LDS), s>>>(
          theta, phi, off, wd, u, z, N, M, K, S, tb, pb);
}

// The butterfly draw for either document source (kernel choice by K).
void dispatch_butterfly(const float *theta, const float *phi, DocSource d,
                        const int32_t *word_id, UniformSource u, int32_t *z, int64_t N,
                        int32_t M, int32_t V, int32_t K, hipStream_t s) {
  if (groups_for(N, K)) {
    if (K <= kLeaf * 8)
      launch_groups<8>(theta, phi, d, word_id, u, z, N, M, V, K, s);
    else if (K <= kLeaf * 16)
      launch_groups<16>(theta, phi, d, word_id, u, z, N, M, V, K, s);
    else if (K <= kLeaf * 32)
      launch_groups<32>(theta, phi, d, word_id, u, z, N, M, V, K, s);
    else
      launch_groups<64>(theta, phi, d, word_id, u, z, N, M, V, K, s);
    return;
  }
  if (eighths_for(N, K)) {
    // launch shapes measured on MI355X: up to five blocks, 16 tokens in
    // flight per wavefront at 2 wavefronts per SIMD (1-2% faster than 8 at 3
    // or 4 at 4); six to eight, 4 at 4 (3-5% faster than 16 at 2 or 8 at 3;
    // 2 in flight: 30% slower)
    if (eighths_blocks(K) <= LDA_EIGHTHS_SPLIT)
      launch_eighths<LDA_EIGHTHS_WINDOW, LDA_EIGHTHS_WAVES_PER_EU>(theta, phi, d, word_id, u, z,
                                                                   N, M, V, K, s);
    else
      launch_eighths<LDA_EIGHTHS_WINDOW_LARGE, LDA_EIGHTHS_WAVES_PER_EU_LARGE>(
          theta, phi, d, word_id, u, z, N, M, V, K, s);
    return;
  }
  const bool lt = lds_table_for(K);
  if (width_for(K) == 64) {
    if (lt)
      launch_butterfly<64, true>(theta, phi, d, word_id, u, z, N, M, V, K, s);
    else if (half_tail_for(K))
      launch_butterfly<64, false, false, true>(theta, phi, d, word_id, u, z, N, M, V, K, s);
    else
      launch_butterfly<64, false>(theta, phi, d, word_id, u, z, N, M, V, K, s);
  } else {
    if (lt)
      launch_butterfly<32, true>(theta, phi, d, word_id, u, z, N, M, V, K, s);
    else
      launch_butterfly<32, false>(theta, phi, d, word_id, u, z, N, M, V, K, s);
  }
}

// Workspace of the routing: the routed arrays and the builder's tables, each
// section starting on a 256-byte boundary.
struct RouteLayout {
  int64_t Np, nchunks;
  size_t perm, rword, rdoc, chunk_off, counts, map, lists, bytes;
};

RouteLayout route_layout(int64_t N) {
  RouteLayout L;
  L.Np = N + (int64_t)kRouteXcds * kRoutePad;  // a list pads fewer than 64 positions
  L.nchunks = (N + kRouteChunk - 1) / kRouteChunk;
  size_t off = 0;
  auto take = [&](size_t b) {
    const size_t o = off;
    off += (b + 255) & ~(size_t)255;
    return o;
  };
  L.perm = take(4 * (size_t)L.Np);
  L.rword = take(4 * (size_t)L.Np);
  L.rdoc = take(4 * (size_t)L.Np);
  L.chunk_off = take(4 * (size_t)kRouteXcds * (size_t)L.nchunks);
  L.counts = take(4 * kRouteClasses);
  L.map = take(4 * kRouteClasses);
  L.lists = take(8 * 3 * kRouteXcds);
  L.bytes = off;
  return L;
}

RoutePlan route_plan(void *ws, const RouteLayout &L) {
  char *b = static_cast<char *>(ws);
  return RoutePlan{reinterpret_cast<int32_t *>(b + L.perm), reinterpret_cast<int32_t *>(b + L.rword),
                   reinterpret_cast<int32_t *>(b + L.rdoc), reinterpret_cast<int32_t *>(b + L.chunk_off),
                   reinterpret_cast<int32_t *>(b + L.counts), reinterpret_cast<int32_t *>(b + L.map),
                   reinterpret_cast<int64_t *>(b + L.lists)};
}

// K the routed draw takes: the leaf kernel's (K divisible by 4 from
// LDA_EIGHTHS_MIN_K to LDA_EIGHTHS_MAX_BLOCKS blocks of 256).
bool routed_for(int32_t K) {
  return K % kLeaf == 0 && K >= LDA_EIGHTHS_MIN_K && eighths_blocks(K) <= LDA_EIGHTHS_MAX_BLOCKS;
}

}  // namespace
}  // namespace lda

using namespace lda;

extern "C" int lda_draw_naive(const float *theta, const float *phi,
                              const int32_t *doc_id, const int32_t *word_id,
                              const float *u, int32_t *z, int64_t N, int32_t M,
                              int32_t V, int32_t K, void *stream) {
  const int st = check_args(theta, phi, doc_id, word_id, u, z, N, M, V, K);
  if (st != LDA_OK || N == 0) return st;
  const UniformSource us{u, 0, 0, 0};
  hipStream_t s = static_cast<hipStream_t>(stream);
  const DocSource d{doc_id, nullptr, M, N};
  if (K <= 64)
    launch_naive<64>(theta, phi, d, word_id, us, z, N, K, s);
  else if (K <= 256)
    launch_naive<256>(theta, phi, d, word_id, us, z, N, K, s);
  else if (K <= 1024)
    launch_naive<1024>(theta, phi, d, word_id, us, z, N, K, s);
  else
    launch_naive<LDA_MAX_K>(theta, phi, d, word_id, us, z, N, K, s);
  return finish_launch();
}

extern "C" int lda_draw_butterfly(const float *theta, const float *phi,
                                  const int32_t *doc_id, const int32_t *word_id,
                                  const float *u, int32_t *z, int64_t N,
                                  int32_t M, int32_t V, int32_t K,
                                  void *stream) {
  const int st = check_args(theta, phi, doc_id, word_id, u, z, N, M, V, K);
  if (st != LDA_OK || N == 0) return st;
  const UniformSource us{u, 0, 0, 0};
  dispatch_butterfly(theta, phi, DocSource{doc_id, nullptr, M, N}, word_id, us, z, N, M, V, K,
                     static_cast<hipStream_t>(stream));
  return finish_launch();
}

extern "C" int lda_draw_transposed(const float *theta, const float *phi,
                                   const int32_t *doc_id, const int32_t *word_id,
                                   const float *u, int32_t *z, int64_t N, int32_t M,
                                   int32_t V, int32_t K, void *stream) {
  const int st = check_args(theta, phi, doc_id, word_id, u, z, N, M, V, K);
  if (st != LDA_OK || N == 0) return st;
  const UniformSource us{u, 0, 0, 0};
  launch_transposed(theta, phi, DocSource{doc_id, nullptr, M, N}, word_id, us, z, N, M, V, K,
                    static_cast<hipStream_t>(stream));
  return finish_launch();
}

extern "C" int lda_draw_butterfly_variant(const float *theta, const float *phi,
                                          const int32_t *doc_id, const int32_t *word_id,
                                          const float *u, int32_t *z, int64_t N, int32_t M,
                                          int32_t V, int32_t K, int32_t variant,
                                          void *stream) {
  if (variant != LDA_VARIANT_REGISTER_TABLE && variant != LDA_VARIANT_LDS_TABLE &&
      variant != LDA_VARIANT_LDS_TABLE_ALT)
    return LDA_ERR_UNSUPPORTED;
  const int st = check_args(theta, phi, doc_id, word_id, u, z, N, M, V, K);
  if (st != LDA_OK || N == 0) return st;
  const UniformSource us{u, 0, 0, 0};
  const DocSource d{doc_id, nullptr, M, N};
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (variant == LDA_VARIANT_REGISTER_TABLE)
    launch_table_variant<false, false>(theta, phi, d, word_id, us, z, N, M, V, K, s);
  else if (variant == LDA_VARIANT_LDS_TABLE)
    launch_table_variant<true, false>(theta, phi, d, word_id, us, z, N, M, V, K, s);
  else
    launch_table_variant<true, true>(theta, phi, d, word_id, us, z, N, M, V, K, s);
  return finish_launch();
}

extern "C" int lda_draw_doc_lanes(const float *theta, const float *phi,
                                  const int64_t *doc_offsets, const int32_t *word_id,
                                  const float *u, int32_t *z, int64_t N, int32_t M,
                                  int32_t V, int32_t K, int32_t theta_cache,
                                  void *stream) {
  if (theta_cache != 0 && theta_cache != 1) return LDA_ERR_UNSUPPORTED;
  const int st = check_args(theta, phi, doc_offsets, word_id, u, z, N, M, V, K);
  if (st != LDA_OK) return st;
  if (theta_cache && doc_lanes_cache_bytes(K) > LDA_DOC_LANES_MAX_CACHE_BYTES)
    return LDA_ERR_UNSUPPORTED;
  if (N == 0) return LDA_OK;
  if (reinterpret_cast<uintptr_t>(doc_offsets) & 7u) return LDA_ERR_ALIGN;
  const UniformSource us{u, 0, 0, 0};
  hipStream_t s = static_cast<hipStream_t>(stream);
  const bool tl = theta_cache != 0;
  if (width_for(K) == 64) {
    if (tl)
      launch_doc_lanes<64, true>(theta, phi, doc_offsets, word_id, us, z, N, M, V, K, s);
    else
      launch_doc_lanes<64, false>(theta, phi, doc_offsets, word_id, us, z, N, M, V, K, s);
  } else {
    if (tl)
      launch_doc_lanes<32, true>(theta, phi, doc_offsets, word_id, us, z, N, M, V, K, s);
    else
      launch_doc_lanes<32, false>(theta, phi, doc_offsets, word_id, us, z, N, M, V, K, s);
  }
  return finish_launch();
}

extern "C" int lda_draw_butterfly_philox(const float *theta, const float *phi,
                                         const int32_t *doc_id, const int32_t *word_id,
                                         int32_t *z, int64_t N, int32_t M, int32_t V,
                                         int32_t K, uint64_t seed, uint32_t sweep,
                                         void *stream) {
  // (z stands in for the absent u in the pointer checks)
  const int st = check_args(theta, phi, doc_id, word_id, z, z, N, M, V, K);
  if (st != LDA_OK || N == 0) return st;
  const UniformSource us{nullptr, (uint32_t)seed, (uint32_t)(seed >> 32), sweep};
  dispatch_butterfly(theta, phi, DocSource{doc_id, nullptr, M, N}, word_id, us, z, N, M, V, K,
                     static_cast<hipStream_t>(stream));
  return finish_launch();
}

extern "C" int lda_philox_uniforms(float *u, int64_t count, int64_t first, uint64_t seed,
                                   uint32_t sweep, void *stream) {
  if (count < 0 || first < 0 || count > INT64_MAX - first) return LDA_ERR_SHAPE;
  if (count == 0) return LDA_OK;
  if (!u) return LDA_ERR_NULL;
  if (reinterpret_cast<uintptr_t>(u) & 3u) return LDA_ERR_ALIGN;
  const UniformSource us{nullptr, (uint32_t)seed, (uint32_t)(seed >> 32), sweep};
  const int64_t blocks = (count + 255) / 256;
  uniforms_kernel<<<(unsigned)(blocks < 4096 ? blocks : 4096), 256, 0,
                    static_cast<hipStream_t>(stream)>>>(u, count, first, us);
  return finish_launch();
}

extern "C" int lda_draw_docs(const float *theta, const float *phi,
                             const int64_t *doc_offsets, const int32_t *word_id,
                             const float *u, int32_t *z, int64_t N, int32_t M,
                             int32_t V, int32_t K, void *stream) {
  int st = check_args(theta, phi, doc_offsets, word_id, u, z, N, M, V, K);
  if (st != LDA_OK || N == 0) return st;
  if (reinterpret_cast<uintptr_t>(doc_offsets) & 7u) return LDA_ERR_ALIGN;
  const UniformSource us{u, 0, 0, 0};
  dispatch_butterfly(theta, phi, DocSource{nullptr, doc_offsets, M, N}, word_id, us, z, N, M, V,
                     K, static_cast<hipStream_t>(stream));
  return finish_launch();
}

extern "C" int lda_butterfly_table(const float *theta, const float *phi,
                                   const int32_t *doc_id,
                                   const int32_t *word_id, float *table,
                                   int64_t N, int32_t M, int32_t V, int32_t K,
                                   void *stream) {
  // u is not used here; pass a valid stand-in so the shared check applies.
  const int st = check_args(theta, phi, doc_id, word_id, theta, table, N, M, V,
                            K);
  if (st != LDA_OK || N == 0) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const uint32_t tb = (uint32_t)((int64_t)M * K * 4);
  const uint32_t pb = (uint32_t)((int64_t)V * K * 4);
  if (width_for(K) == 64)
    table_kernel<64, true><<<wave_grid(N), kBlockThreads, 0, s>>>(
        theta, phi, doc_id, word_id, table, N, K, tb, pb);
  else
    table_kernel<32, true><<<wave_grid(N), kBlockThreads, 0, s>>>(
        theta, phi, doc_id, word_id, table, N, K, tb, pb);
  return finish_launch();
}

extern "C" size_t lda_route_workspace_bytes(int64_t N) {
  if (N < 0 || N > LDA_ROUTE_MAX_N) return 0;
  return route_layout(N).bytes;
}

extern "C" int lda_route_build(const int32_t *doc_id, const int32_t *word_id, int64_t N,
                               int32_t M, int32_t V, void *workspace, size_t workspace_bytes,
                               lda_route *route, void *stream) {
  if (!route) return LDA_ERR_NULL;
  if (N < 0 || M <= 0 || V <= 0) return LDA_ERR_SHAPE;
  if (N > LDA_ROUTE_MAX_N) return LDA_ERR_UNSUPPORTED;
  *route = lda_route{};
  if (N == 0) return LDA_OK;
  if (!doc_id || !word_id || !workspace) return LDA_ERR_NULL;
  if ((reinterpret_cast<uintptr_t>(doc_id) | reinterpret_cast<uintptr_t>(word_id)) & 3u ||
      reinterpret_cast<uintptr_t>(workspace) & 7u)
    return LDA_ERR_ALIGN;
  const RouteLayout L = route_layout(N);
  if (workspace_bytes < L.bytes) return LDA_ERR_WORKSPACE;
  const RoutePlan P = route_plan(workspace, L);
  const hipStream_t s = static_cast<hipStream_t>(stream);
  route_fill<<<1, kRouteClasses, 0, s>>>(P.counts, kRouteClasses, 0);
  route_hist<<<(unsigned)(L.nchunks < 256 ? L.nchunks : 256), kRouteThreads, 0, s>>>(
      word_id, N, L.nchunks, P.counts);
  route_map<<<1, kRouteThreads, 0, s>>>(P.counts, P.map, P.lists);
  route_count<<<(unsigned)L.nchunks, kRouteThreads, 0, s>>>(word_id, N, P.map, P.chunk_off);
  route_scan<<<kRouteXcds, kRouteThreads, 0, s>>>(P.chunk_off, L.nchunks);
  route_scatter<<<(unsigned)L.nchunks, kRouteThreads, 0, s>>>(word_id, doc_id, N, P.map,
                                                              P.chunk_off, P.lists, P.perm,
                                                              P.rword, P.rdoc);
  route_pad<<<kRouteXcds, kRouteThreads, 0, s>>>(P.lists, P.perm, P.rword, P.rdoc);
  int st = finish_launch();
  if (st != LDA_OK) return st;
  // the list sizes size the draw's grid: read them back once
  int64_t lists[3 * kRouteXcds];
  hipError_t e = hipMemcpyAsync(lists, P.lists, sizeof(lists), hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) {
    g_last_hip = e;
    return LDA_ERR_HIP;
  }
  route->N = N;
  for (int x = 0; x < kRouteXcds; ++x) {
    route->tokens[x] = lists[x];
    route->start[x] = lists[kRouteXcds + x];
    route->length[x] = lists[2 * kRouteXcds + x];
  }
  return LDA_OK;
}

extern "C" int lda_draw_routed(const float *theta, const float *phi, const void *workspace,
                               size_t workspace_bytes, const lda_route *route, const float *u,
                               int32_t *z, int64_t N, int32_t M, int32_t V, int32_t K,
                               void *stream) {
  if (!route) return LDA_ERR_NULL;
  const int st = check_args(theta, phi, workspace, workspace, u, z, N, M, V, K);
  if (st != LDA_OK) return st;
  if (!routed_for(K) || N > LDA_ROUTE_MAX_N) return LDA_ERR_UNSUPPORTED;
  if (N == 0) return LDA_OK;
  if (reinterpret_cast<uintptr_t>(workspace) & 7u) return LDA_ERR_ALIGN;
  const RouteLayout L = route_layout(N);
  if (route->N != N || workspace_bytes < L.bytes) return LDA_ERR_WORKSPACE;
  int64_t max_len = 0, total = 0;
  for (int x = 0; x < kRouteXcds; ++x) {
    if (route->length[x] < 0 || route->start[x] < 0 || route->length[x] % kRoutePad ||
        route->start[x] + route->length[x] > L.Np)
      return LDA_ERR_WORKSPACE;
    max_len = route->length[x] > max_len ? route->length[x] : max_len;
    total += route->tokens[x];
  }
  if (total != N) return LDA_ERR_WORKSPACE;
  const RoutePlan P = route_plan(const_cast<void *>(workspace), L);
  RoutedTokens rt{P.perm, P.rword, P.rdoc, {}, {}};
  for (int x = 0; x < kRouteXcds; ++x) {
    rt.base[x] = route->start[x];
    rt.len[x] = route->length[x];
  }
  const UniformSource us{u, 0, 0, 0};
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (K % kBlock4 == 0)
    launch_routed<false>(theta, phi, rt, us, z, max_len, M, V, K, s);
  else
    launch_routed<true>(theta, phi, rt, us, z, max_len, M, V, K, s);
  return finish_launch();
}

extern "C" int lda_butterfly_width(int32_t K) {
  if (K <= 0) return LDA_ERR_SHAPE;
  if (K > LDA_MAX_K) return LDA_ERR_UNSUPPORTED;
  return width_for(K);
}

extern "C" const char *lda_status_string(int status) {
  switch (status) {
    case LDA_OK: return "ok";
    case LDA_ERR_NULL: return "a required pointer is NULL";
    case LDA_ERR_SHAPE: return "invalid shape (N < 0, M <= 0, V <= 0 or K <= 0)";
    case LDA_ERR_UNSUPPORTED:
      return "unsupported size (K > LDA_MAX_K, or theta or phi larger than "
             "LDA_MAX_TABLE_BYTES)";
    case LDA_ERR_HIP: return "HIP runtime error";
    case LDA_ERR_ALIGN: return "a pointer is not aligned (4 bytes; 8 for offsets and workspaces)";
    case LDA_ERR_WORKSPACE:
      return "routing workspace too small, or the route does not belong to these tokens";
    default: return "unknown status";
  }
}

extern "C" const char *lda_last_hip_error(void) {
  return hipGetErrorString(g_last_hip);
}

extern "C" int lda_version(void) { return 300; }
