// Naive draw kernel (gfx950).
#pragma once

#include "sources.hpp"

namespace LDA_NS {
namespace {

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

}  // namespace
}  // namespace LDA_NS
