// Butterfly table dump kernel (gfx950).
#pragma once

#include "tile.hpp"

namespace LDA_NS {
namespace {

// Table dump: the per-lane table p[K] of Algorithm 7 for every token, built
// with the same tile loads and butterfly as the draw's rebuild step.
template <int W, bool SMALL>
__global__ __launch_bounds__(kBlockThreads) void table_kernel(
    const float *__restrict__ theta, const float *__restrict__ phi,
    const int32_t *__restrict__ doc_id, const int32_t *__restrict__ word_id,
    float *__restrict__ table, int64_t N, int K, uint32_t theta_extent,
    uint32_t phi_extent) {
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
  init_wave<W, true>(w, theta, phi, theta_extent, phi_extent, word_id, t0, last, K,
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

}  // namespace
}  // namespace LDA_NS
