// The draw kernels built for tables past 4 GiB (gfx950).  The same kernels as
// lda_draw.hip, with theta and phi rows addressed by index and 64-bit loads
// (config.hpp), so that a table may be of any size (fewer than 2^31 rows).
// lda_draw_butterfly, lda_draw_docs and lda_draw_butterfly_philox come here
// when theta or phi is larger than LDA_MAX_TABLE_BYTES.
#define LDA_WIDE_TABLES 1

#include "draw_dispatch.hpp"
#include "wide.hpp"

namespace lda_wide {

void draw(const float *theta, const float *phi, const int32_t *doc_id,
          const int64_t *doc_offsets, const int32_t *word_id, const float *u, uint32_t k0,
          uint32_t k1, uint32_t sweep, int32_t *z, int64_t N, int32_t M, int32_t V, int32_t K,
          hipStream_t s) {
  const DocSource d{doc_id, doc_id ? nullptr : doc_offsets, M, N};
  const UniformSource us{u, k0, k1, sweep};
  dispatch_butterfly<1>(theta, phi, d, word_id, us, z, N, M, V, K, s);
}

}  // namespace lda_wide
