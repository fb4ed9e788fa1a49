// Document and uniform sources of the draw kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "butterfly.hpp"
#include "philox.hpp"
#include "tuning.hpp"

namespace LDA_NS {
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

}  // namespace
}  // namespace LDA_NS
