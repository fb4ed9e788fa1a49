// One-topic-per-lane butterfly kernel (gfx950).
#pragma once

#include "tile.hpp"

namespace LDA_NS {
namespace {

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
    int32_t *__restrict__ z, int64_t N, int K, uint32_t theta_extent, uint32_t phi_extent) {
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
  init_wave<W, SMALL>(w, theta, phi, theta_extent, phi_extent, word_id, t0, last, K,
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
  // Algorithm 10.  Empty topics of block 0 have the prefix 0, which is never
  // above stop >= 0; but the search rebuilds prefixes as low + y or high - y,
  // and where the true prefix is 0 the rounding of high - y may leave a tiny
  // nonzero value, so that a stop of 0 (u = 0) or of a few ulps of S can end
  // the search among them: the draw is then topic 0 (a result inside the
  // rounding band).  With S = 0 every comparison fails and the result is
  // K - 1.
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
  if (store) z[n] = j < 0 ? 0 : j;
}

}  // namespace
}  // namespace LDA_NS
