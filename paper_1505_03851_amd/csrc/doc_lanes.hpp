// Document-per-lane driver kernel (gfx950).
#pragma once

#include "tile.hpp"

namespace LDA_NS {
namespace {

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
    return topic_of(w, blk) >= 0 ? load_row<W>(w.th, voff, theta_row(w, k)) : 0.0f;
}

template <int W, bool THETA_LDS>
__global__ __launch_bounds__(kBlockThreads) __attribute__((amdgpu_waves_per_eu(LDA_WAVES_PER_EU)))
void doc_lanes_kernel(const float *__restrict__ theta, const float *__restrict__ phi,
                      const int64_t *__restrict__ offsets, const int32_t *__restrict__ word_id,
                      UniformSource u, int32_t *__restrict__ z, int64_t N, int M,
                      int K, int S, uint32_t theta_extent, uint32_t phi_extent) {
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
  w.th = make_table(theta, theta_extent, K);
  w.ph = make_table(phi, phi_extent, K);
  w.wp = nullptr;
  w.last = kWave - 1;
  w.R = K & (W - 1);
  w.c0 = w.R ? w.R - W : 0;
  w.r = lane & (W - 1);
  w.gbase = lane & ~(W - 1);
  w.doc = doc;
  w.mode = kAnyDocs;
  w.kb = 0;
  w.th_off0 = w.th_off1 = 0;
  w.th_lane = w.th.row((uint32_t)doc);

  const int cache_rows = THETA_LDS ? NB * W : 0;
  float *cache = lds + wave * (cache_rows + NB) * kWave;
  float *region = cache + cache_rows * kWave;
  if constexpr (THETA_LDS) {
    for (int b = 0; b < NB; ++b) {
      const uint32_t voff = col_bytes(w, b);
      const bool real = topic_of(w, b) >= 0;
#pragma unroll 8
      for (int k = 0; k < W; ++k) {
        const float th = load_row<W>(w.th, voff, theta_row(w, k));
        cache[(b * W + k) * kWave + lane] = real ? th : 0.0f;
      }
    }
  }

  for (int64_t i = stride0; __builtin_amdgcn_ballot_w64(i < len) != 0; i += S) {
    const int64_t n = len > 0 ? start + (i < len ? i : len - 1) : 0;
    const bool store = i < len;
    w.ph_lane = w.ph.row((uint32_t)word_id[n]);
    const float un = u(n);

    float a[W];
    float sum = 0.0f, stop, low, high;
    int blk = 0;
    // sweep: block totals and the running prefix at each block's end
    for (int b = 0; b < NB; ++b) {
      const uint32_t voff = col_bytes(w, b);
#pragma unroll
      for (int k = 0; k < W; ++k) {
        const float ph = load_row<W>(w.ph, voff, (uint32_t)group_value<W>((int)w.ph_lane, k));
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
      const float ph = load_row<W>(w.ph, voff, (uint32_t)group_value<W>((int)w.ph_lane, k));
      float th;
      if constexpr (THETA_LDS)
        th = cache[(bk * W + k) * kWave + lane];
      else
        th = t < 0 ? 0.0f : load_row<W>(w.th, voff, theta_row(w, k));
      a[k] = th * ph;
    }
    butterfly_block<W>(a, w.r, NoStore{});
    const int j = w.c0 + blk * W + inblock_search<W, false>(a, nullptr, w.r, w.gbase, stop, low, high);
    // (a search ending among the empty topics of block 0, whose rebuilt
    // prefixes may round above a stop of a few ulps: topic 0)
    if (store) z[n] = j < 0 ? 0 : j;
  }
}

}  // namespace
}  // namespace LDA_NS
