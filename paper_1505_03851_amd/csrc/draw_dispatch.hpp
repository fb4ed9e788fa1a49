// Launches of the draw kernels and the choice among them by K (gfx950):
// lda_draw_butterfly, lda_draw_docs and lda_draw_butterfly_philox draw
// through dispatch_butterfly.  Included by each build of the kernels (the
// default one, and the one for tables past 4 GiB: see config.hpp).
#pragma once

#include <hip/hip_runtime.h>

#include <stdint.h>

#include "tuning.hpp"
#include "sources.hpp"
#include "tile.hpp"
#include "one_topic.hpp"
#include "leaf_eighths.hpp"
#include "leaf_group.hpp"

namespace LDA_NS {
namespace {

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

// 256-topic blocks of the eighths kernel (the remnant of K mod 256 included).
int eighths_blocks(int32_t K) { return (K + kBlock4 - 1) / kBlock4; }

// Wavefronts per workgroup of the eighths kernel: 4 while three such
// workgroups fit in a CU's LDS (8 rows of 64 floats per block and wavefront),
// else 2.
bool eighths_wide_groups(int32_t K) {
  return 3LL * 4 * 8 * eighths_blocks(K) * kWave * (int64_t)sizeof(float) <= 160 * 1024;
}
// Whether one-document wavefronts stage their theta row in LDS for the
// rebuild: while three 4-wavefront workgroups still fit with it.
bool eighths_stage_theta(int32_t K) {
  return 3LL * 4 * eighths_lds_floats(eighths_blocks(K), true) * (int64_t)sizeof(float) <=
         160 * 1024;
}

template <int C, int WPEU, bool PAD>
void launch_eighths(const float *theta, const float *phi, DocSource d, const int32_t *wd,
                    UniformSource u, int32_t *z, int64_t N, int32_t M, int32_t V, int32_t K,
                    hipStream_t s) {
  const uint32_t tb = table_extent(M, K);
  const uint32_t pb = table_extent(V, K);
  const int NB = eighths_blocks(K);
  const size_t rows = (size_t)eighths_lds_floats(NB, false) * sizeof(float);
  const size_t staged = (size_t)eighths_lds_floats(NB, true) * sizeof(float);
  if (eighths_stage_theta(K))
    leaf_eighths_kernel<C, 4, WPEU, PAD, true><<<wave_grid(N, 4), 4 * kWave, 4 * staged, s>>>(
        theta, phi, d, wd, u, z, N, K, tb, pb);
  else if (eighths_wide_groups(K))
    leaf_eighths_kernel<C, 4, WPEU, PAD, false><<<wave_grid(N, 4), 4 * kWave, 4 * rows, s>>>(
        theta, phi, d, wd, u, z, N, K, tb, pb);
  else
    leaf_eighths_kernel<C, 2, WPEU, PAD, false><<<wave_grid(N, 2), 2 * kWave, 2 * rows, s>>>(
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

// (8-topic leaves hold twice the registers: the 64-lane groups' setting)
template <int G, int H, int CW = (G == kWave ? LDA_GROUP64_WINDOW : LDA_GROUP_WINDOW),
          int WPEU = ((G == kWave || H > 1) ? LDA_GROUP64_WAVES_PER_EU : LDA_GROUP_WAVES_PER_EU)>
void launch_groups(const float *theta, const float *phi, DocSource d, const int32_t *wd,
                   UniformSource u, int32_t *z, int64_t N, int32_t M, int32_t V, int32_t K,
                   hipStream_t s) {
  constexpr int C = CW < G ? CW : G;
  const uint32_t tb = table_extent(M, K);
  const uint32_t pb = table_extent(V, K);
  const size_t lds = (size_t)kWavesPerBlock * group_lds_bytes<G, H>();
  if (K == kLeaf * H * G)
    leaf_group_kernel<G, H, C, WPEU, false><<<wave_grid(N), kBlockThreads, lds, s>>>(
        theta, phi, d, wd, u, z, N, K, tb, pb);
  else
    leaf_group_kernel<G, H, C, WPEU, true><<<wave_grid(N), kBlockThreads, lds, s>>>(
        theta, phi, d, wd, u, z, N, K, tb, pb);
}

// Groups of 64 lanes with 8-topic leaves for K from 260 to LDA_LEAF8_MAX_K
// (at most 512), multiples of 32 only up to LDA_LEAF8_ALIGNED_MAX_K: the
// whole row in one tile, as the leaf groups do up to 256.  Measured on MI355X
// against the eighths kernel, which pads such K to two 256-topic blocks:
// 17-21% faster at K = 260 ... 320, 7% at 384, 1-4% up to 508; 2-3% slower at
// K = 448, 480 and 512.
bool leaf8_for(int64_t N, int32_t K) {
  return N >= kWave && K % kLeaf == 0 && K > kLeaf * kWave && K <= LDA_LEAF8_MAX_K &&
         K <= 2 * kLeaf * kWave && (K % 32 != 0 || K <= LDA_LEAF8_ALIGNED_MAX_K);
}

// The eighths kernel takes K divisible by 4 (16-byte leaves) from
// LDA_EIGHTHS_MIN_K topics to LDA_EIGHTHS_MAX_BLOCKS 256-topic blocks, for
// N >= 64.  Measured on MI355X against the one-topic kernel: 15-30% faster
// from K = 144 (K = 144 ... 240 on the paper-shaped corpus), 7% at K = 256,
// 4% at K = 1024, 5% at K = 2048; 3-4% slower at K = 80 and 112, whose
// padding fills most of the block.  (The dispatch gives K up to 256, and
// most K up to 508, to the leaf-group kernel first.)
bool eighths_for(int64_t N, int32_t K) {
  return N >= kWave && K % kLeaf == 0 && K >= LDA_EIGHTHS_MIN_K &&
         eighths_blocks(K) <= LDA_EIGHTHS_MAX_BLOCKS;
}

template <int W, bool LDS_TABLE, bool ALT = false, bool HALF = false, int WPB = kWavesPerBlock>
void launch_butterfly(const float *theta, const float *phi, DocSource d,
                      const int32_t *wd, UniformSource u, int32_t *z, int64_t N,
                      int32_t M, int32_t V, int32_t K, hipStream_t s) {
  const int nb = (K + W - 1) / W;  // blocks, the remnant included
  const size_t lds = (size_t)WPB * region_rows(nb, W, LDS_TABLE, HALF) * kWave * sizeof(float);
  const uint32_t tb = table_extent(M, K);
  const uint32_t pb = table_extent(V, K);
  if (N < kWave)
    butterfly_kernel<W, LDS_TABLE, true, ALT, HALF, WPB><<<wave_grid(N, WPB), WPB * kWave, lds, s>>>(
        theta, phi, d, wd, u, z, N, K, tb, pb);
  else
    butterfly_kernel<W, LDS_TABLE, false, ALT, HALF, WPB><<<wave_grid(N, WPB), WPB * kWave, lds, s>>>(
        theta, phi, d, wd, u, z, N, K, tb, pb);
}

// The leaf-group kernel with groups just wide enough for K: K up to 32, 64,
// 128, 256 topics take 8, 16, 32, 64 lanes with 4-topic leaves (H = 1), half
// as many with 8-topic leaves (H = 2).
template <int H>
void dispatch_groups(const float *theta, const float *phi, DocSource d, const int32_t *word_id,
                     UniformSource u, int32_t *z, int64_t N, int32_t M, int32_t V, int32_t K,
                     hipStream_t s) {
  if (K <= kLeaf * 8)
    launch_groups<8 / H, H>(theta, phi, d, word_id, u, z, N, M, V, K, s);
  else if (K <= kLeaf * 16)
    launch_groups<16 / H, H>(theta, phi, d, word_id, u, z, N, M, V, K, s);
  else if (K <= kLeaf * 32)
    launch_groups<32 / H, H>(theta, phi, d, word_id, u, z, N, M, V, K, s);
  else
    launch_groups<64 / H, H>(theta, phi, d, word_id, u, z, N, M, V, K, s);
}

// The butterfly draw for either document source (kernel choice by K); with
// H = 2 the leaf groups take 8-topic leaves.
template <int H = LDA_GROUP_LEAF / kLeaf>
void dispatch_butterfly(const float *theta, const float *phi, DocSource d,
                        const int32_t *word_id, UniformSource u, int32_t *z, int64_t N,
                        int32_t M, int32_t V, int32_t K, hipStream_t s) {
  if (groups_for(N, K)) {
    dispatch_groups<H>(theta, phi, d, word_id, u, z, N, M, V, K, s);
    return;
  }
  if constexpr (LDA_LEAF8_MAX_K > 0) {
    if (leaf8_for(N, K)) {
      launch_groups<kWave, 2, LDA_LEAF8_WINDOW, LDA_LEAF8_WAVES_PER_EU>(theta, phi, d, word_id,
                                                                         u, z, N, M, V, K, s);
      return;
    }
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

}  // namespace
}  // namespace LDA_NS
