// Transposed-access kernel, for comparison (gfx950).
#pragma once

#include "tile.hpp"

namespace LDA_NS {
namespace {

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
                       uint32_t theta_extent, uint32_t phi_extent) {
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
  init_wave<kWave, SMALL>(w, theta, phi, theta_extent, phi_extent, word_id, t0, last, K,
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

}  // namespace
}  // namespace LDA_NS
