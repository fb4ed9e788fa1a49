// Philox4x32-10 counter-based generator (Salmon, Moraes, Dror and Shaw,
// "Parallel random numbers: as easy as 1, 2, 3", SC 2011) for the draw with
// in-kernel uniforms.
//
// Ten rounds on a counter (x0, x1, x2, x3) and key (k0, k1) of 32-bit words;
// each round forms the 64-bit products M0 * x0 and M1 * x2 and replaces the
// counter by (hi(M1 x2) ^ x1 ^ k0, lo(M1 x2), hi(M0 x0) ^ x3 ^ k1, lo(M0 x0));
// the key advances by the Weyl increments (C0, C1) before every round but the
// first.  Only the first output word is used here.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "config.hpp"

namespace LDA_NS {

__device__ __forceinline__ uint32_t philox4x32_10_word0(uint32_t x0, uint32_t x1,
                                                        uint32_t x2, uint32_t x3,
                                                        uint32_t k0, uint32_t k1) {
  constexpr uint32_t kM0 = 0xD2511F53u, kM1 = 0xCD9E8D57u;
  constexpr uint32_t kC0 = 0x9E3779B9u, kC1 = 0xBB67AE85u;
#pragma unroll
  for (int round = 0; round < 10; ++round) {
    if (round > 0) {
      k0 += kC0;
      k1 += kC1;
    }
    const uint64_t p0 = (uint64_t)kM0 * x0;
    const uint64_t p1 = (uint64_t)kM1 * x2;
    const uint32_t y0 = (uint32_t)(p1 >> 32) ^ x1 ^ k0;
    const uint32_t y2 = (uint32_t)(p0 >> 32) ^ x3 ^ k1;
    x1 = (uint32_t)p1;
    x3 = (uint32_t)p0;
    x0 = y0;
    x2 = y2;
  }
  return x0;
}

// Uniform of token n in sweep `sweep`: counter (n mod 2^32, n / 2^32, sweep,
// 0), key (k0, k1); the top 24 bits of the first word times 2^-24 (exact in
// fp32, in [0, 1)).
__device__ __forceinline__ float philox_uniform(uint64_t n, uint32_t sweep, uint32_t k0,
                                                uint32_t k1) {
  const uint32_t y = philox4x32_10_word0((uint32_t)n, (uint32_t)(n >> 32), sweep, 0u, k0, k1);
  return (float)(y >> 8) * 0x1p-24f;
}

}  // namespace LDA_NS
