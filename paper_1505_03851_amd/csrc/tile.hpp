// Wavefront state, tile loads and searches shared by the butterfly kernels (gfx950).
#pragma once

#include "sources.hpp"

namespace LDA_NS {
namespace {

// Order one wavefront's earlier LDS writes before its later LDS reads.
__device__ __forceinline__ void lds_order() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Per-wavefront state of the butterfly kernel.  The wavefront's 64 tokens are
// the window [t0, t0 + 64) of the token arrays; their word and document ids
// are read with scalar loads straight from those arrays whenever a tile is
// loaded (SMALL: the window is padded by repeating token N - 1).
template <int W, bool SMALL>
struct Wave {
  Table th, ph;         // theta, phi
  const int32_t *wp;    // word_id + t0
  int last;             // SMALL: index in the window of token N - 1
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

// Row offset of the phi row of token k of this lane's group: uniform for
// W = 64, one value per half-wave for W = 32.
template <int W, bool SMALL>
__device__ __forceinline__ uint32_t phi_row(const Wave<W, SMALL> &w, const int32_t *wp, int k) {
  if constexpr (W == kWave) {
    return w.ph.row((uint32_t)window_at<SMALL>(wp, w.last, k));
  } else {
    const uint32_t lo = w.ph.row((uint32_t)window_at<SMALL>(wp, w.last, k));
    const uint32_t hi = w.ph.row((uint32_t)window_at<SMALL>(wp, w.last, 32 + k));
    return w.gbase ? hi : lo;
  }
}

// Row offset of the theta row of token k's document, from the lane that
// holds token k (uniform for W = 64, per half-wave for W = 32).
template <int W, bool SMALL>
__device__ __forceinline__ uint32_t theta_row(const Wave<W, SMALL> &w, int k) {
  return (uint32_t)group_value<W>((int)w.th_lane, k);
}

// Load at a per-lane offset plus a row offset that is uniform for W = 64
// (scalar operand) and per half-wave for W = 32 (per lane).
template <int W>
__device__ __forceinline__ float load_row(const Table &t, uint32_t voff, uint32_t row) {
  if constexpr (W == kWave)
    return t.ld(voff, row);
  else
    return t.ldv(voff, row);
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
    a[k] = load_row<W>(w.ph, voff, phi_row(w, wp, reg_token<W, HALF>(k)));
}

// Theta of block `blk` at this lane's topic, for the first and last document
// (MODE: the wave's ThetaMode when known at compile time, else -1).
template <int W, bool SMALL, int MODE = -1>
__device__ __forceinline__ void issue_theta(const Wave<W, SMALL> &w, int blk, float &th0,
                                            float &th1) {
  const uint32_t voff = col_bytes(w, blk);
  th0 = w.th.ld(voff, w.th_off0);
  if (MODE == kTwoDocs || (MODE < 0 && w.mode == kTwoDocs))
    th1 = w.th.ld(voff, w.th_off1);
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
    a[k] = (real ? load_row<W>(w.th, voff, theta_row(w, t)) : 0.0f) *
           load_row<W>(w.ph, voff, phi_row(w, wp, t));
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
    const float th = load_row<W>(w.th, voff, toff);
    a[k] = (PADDED && t < 0 ? 0.0f : th) * load_row<W>(w.ph, voff, poff);
  }
}

template <int W, bool SMALL>
__device__ __forceinline__ void init_wave(Wave<W, SMALL> &w, const float *theta,
                                          const float *phi, uint32_t theta_extent,
                                          uint32_t phi_extent, const int32_t *word_id, int64_t t0, int last,
                                          int K, int lane, int doc, int word) {
  w.th = make_table(theta, theta_extent, K);
  w.ph = make_table(phi, phi_extent, K);
  w.wp = word_id + t0;
  w.last = last;
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
  w.th_off0 = w.th.row((uint32_t)d0);
  w.th_off1 = w.th.row((uint32_t)d1);
  w.ph_lane = w.ph.row((uint32_t)word);
  w.th_lane = w.th.row((uint32_t)doc);
}


// The same wavefront seen as two groups of 32 lanes (W = 32): lanes 32 g + r
// hold topic r of a 32-topic chunk for the tokens of half-wave g.
template <bool SMALL>
__device__ __forceinline__ Wave<kWave / 2, SMALL> half_wave(const Wave<kWave, SMALL> &w,
                                                           int lane) {
  Wave<kWave / 2, SMALL> h;
  h.th = w.th;
  h.ph = w.ph;
  h.wp = w.wp;
  h.last = w.last;
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

}  // namespace
}  // namespace LDA_NS
