// Entry into the build of the draw kernels for tables past 4 GiB
// (lda_draw_wide.hip): theta and phi rows addressed by index with 64-bit
// loads, tables of any size (fewer than 2^31 rows).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lda_wide {

// lda_draw_butterfly's choice of kernel by K, launched on `s` over wide
// tables.  Documents from doc_id, or (doc_id null) from doc_offsets[M + 1];
// uniforms from u, or (u null) Philox4x32-10 under key (k0, k1) and `sweep`.
// The caller has checked every argument (N > 0).
void draw(const float *theta, const float *phi, const int32_t *doc_id,
          const int64_t *doc_offsets, const int32_t *word_id, const float *u, uint32_t k0,
          uint32_t k1, uint32_t sweep, int32_t *z, int64_t N, int32_t M, int32_t V, int32_t K,
          hipStream_t s);

}  // namespace lda_wide
