// Host side and C ABI of the per-token LDA topic draw (gfx950): argument
// checks, kernel choice and launches.
//
// lda_draw_naive      Algorithm 1 + Algorithm 3, one lane per token.
// lda_draw_butterfly  Algorithm 7 (+ 5, 8, 9, 10) for 64-lane wavefronts.
// lda_draw_docs       the same, documents given as offsets.
// lda_draw_doc_lanes  Algorithm 7's document-per-lane driver.
// lda_draw_transposed Algorithms 4-6, for comparison.
// lda_draw_butterfly_variant  the block-table variants of Section 4,
//                     8-topic leaves, and the build for tables past 4 GiB
//                     (lda_draw_wide.hip) at any size.
// lda_draw_butterfly_philox   the butterfly draw with in-kernel uniforms.
// lda_philox_uniforms         those uniforms, written out.
// lda_butterfly_table the butterfly-patterned tables (Fig. 1, right).
// lda_route_build / lda_draw_routed  tokens routed to the XCDs by word, and
//                     the leaf kernel drawing them (lda_draw_routed_philox:
//                     with in-kernel uniforms).
// lda_count_topics    the per-document and per-word topic counts of a set of
//                     draws (counts.hpp); lda_word_index_build and
//                     lda_count_topics_indexed: the same counts with the tokens
//                     grouped by word once per corpus (word_index.hpp).
//
// Device code: butterfly.hpp (lane exchanges, the butterfly, buffer loads),
// philox.hpp, sources.hpp (document and uniform sources), tile.hpp (the
// wavefront's tile loads and the in-block search), naive.hpp, one_topic.hpp
// (one topic per lane), leaf_group.hpp (K up to 256), leaf_eighths.hpp (K
// from 260 to 2048), route.hpp and routed_draw.hpp (routing to the XCDs),
// transposed.hpp, table.hpp and doc_lanes.hpp (comparisons and the table
// dump); tuning.hpp holds the build-time tuning.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include <mutex>

#include "lda_draw.h"
#include "tuning.hpp"
#include "sources.hpp"
#include "naive.hpp"
#include "tile.hpp"
#include "one_topic.hpp"
#include "leaf_eighths.hpp"
#include "draw_dispatch.hpp"
#include "wide.hpp"
#include "routed_draw.hpp"
#include "leaf_group.hpp"
#include "transposed.hpp"
#include "table.hpp"
#include "doc_lanes.hpp"
#include "counts.hpp"
#include "word_index.hpp"

namespace lda {
namespace {

thread_local hipError_t g_last_hip = hipSuccess;

// theta or phi larger than LDA_MAX_TABLE_BYTES: drawn by the wide build
bool wide_tables(int32_t M, int32_t V, int32_t K) {
  return (int64_t)M * K * 4 > LDA_MAX_TABLE_BYTES || (int64_t)V * K * 4 > LDA_MAX_TABLE_BYTES;
}

// WIDE_OK: the entry point draws tables of any size (the wide build past
// LDA_MAX_TABLE_BYTES, addressing rows by index; M and V are below 2^31);
// otherwise up to LDA_MAX_TABLE_BYTES (unsigned 32-bit byte offsets).
int check_args(const void *theta, const void *phi, const void *doc_id,
               const void *word_id, const void *u, const void *z, int64_t N,
               int32_t M, int32_t V, int32_t K, bool wide_ok = false) {
  if (N < 0 || M <= 0 || V <= 0 || K <= 0) return LDA_ERR_SHAPE;
  if (K > LDA_MAX_K || N > LDA_MAX_N) return LDA_ERR_UNSUPPORTED;
  if (!wide_ok && ((int64_t)M * K * 4 > LDA_MAX_TABLE_BYTES ||
                   (int64_t)V * K * 4 > LDA_MAX_TABLE_BYTES))
    return LDA_ERR_UNSUPPORTED;
  if (N == 0) return LDA_OK;
  const void *ptrs[] = {theta, phi, doc_id, word_id, u, z};
  for (const void *p : ptrs) {
    if (!p) return LDA_ERR_NULL;
    if (reinterpret_cast<uintptr_t>(p) & 3u) return LDA_ERR_ALIGN;
  }
  return LDA_OK;
}

int finish_launch() {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    g_last_hip = e;
    return LDA_ERR_HIP;
  }
  return LDA_OK;
}

template <int KMAX>
void launch_naive(const float *theta, const float *phi, DocSource d, const int32_t *w,
                  UniformSource u, int32_t *z, int64_t N, int32_t K, hipStream_t s) {
  const dim3 grid((unsigned)((N + 255) / 256));
  naive_kernel<KMAX><<<grid, 256, 0, s>>>(theta, phi, d, w, u, z, N, K);
}

// Launch of the routed kernel over lists of at most max_len positions: 16
// tokens in flight per wavefront at 2 wavefronts per SIMD for every K (in the
// few-documents path too, with theta leaves read 4 tokens ahead from LDS), 4
// wavefronts per workgroup while three workgroups fit in LDS.
template <bool PAD>
void launch_routed(const float *theta, const float *phi, const RoutedTokens &rt, UniformSource u,
                   int32_t *z, int64_t max_len, int32_t M, int32_t V, int32_t K, hipStream_t s) {
  constexpr int C = LDA_EIGHTHS_WINDOW, WPEU = LDA_EIGHTHS_WAVES_PER_EU;
  const uint32_t tb = table_extent(M, K);
  const uint32_t pb = table_extent(V, K);
  const int NB = eighths_blocks(K);
  const size_t per_wave = (size_t)routed_lds_floats(NB) * sizeof(float);
  // Measured on MI355X (16.8M tokens): 2 wavefronts per workgroup where the
  // runs' theta rows are staged (K <= 1024: 4 were 1-2% slower), 4 above,
  // two such workgroups fitting in LDS (0.5-2.6% faster than 2 from K = 1280
  // to 2048).
  if (NB > kRowsMaxBlocks && 2 * 4 * per_wave <= 160 * 1024) {
    const int64_t tiles = (max_len + 4 * kWave - 1) / (4 * kWave);
    routed_eighths_kernel<C, 4, WPEU, PAD><<<(unsigned)(kXcds * tiles), 4 * kWave, 4 * per_wave, s>>>(
        theta, phi, rt, u, z, K, tb, pb);
  } else {
    const int64_t tiles = (max_len + 2 * kWave - 1) / (2 * kWave);
    routed_eighths_kernel<C, 2, WPEU, PAD><<<(unsigned)(kXcds * tiles), 2 * kWave, 2 * per_wave, s>>>(
        theta, phi, rt, u, z, K, tb, pb);
  }
}

void launch_transposed(const float *theta, const float *phi, DocSource d,
                       const int32_t *wd, UniformSource u, int32_t *z, int64_t N,
                       int32_t M, int32_t V, int32_t K, hipStream_t s) {
  const int nb = (K + kWave - 1) / kWave;
  const size_t lds = (size_t)kWavesPerBlock * (kTileFloats + nb * kWave) * sizeof(float);
  const uint32_t tb = table_extent(M, K);
  const uint32_t pb = table_extent(V, K);
  if (N < kWave)
    transposed_kernel<true><<<wave_grid(N), kBlockThreads, lds, s>>>(theta, phi, d, wd, u, z, N,
                                                                      K, tb, pb);
  else
    transposed_kernel<false><<<wave_grid(N), kBlockThreads, lds, s>>>(theta, phi, d, wd, u, z,
                                                                       N, K, tb, pb);
}

// The W = 32 / 64 butterfly kernel with a chosen table: in registers with the
// paper's search-assist loop, in LDS with direct reads, or the alternative
// rule's table in LDS.
template <bool LDS_TABLE, bool ALT>
void launch_table_variant(const float *theta, const float *phi, DocSource d,
                          const int32_t *word_id, UniformSource u, int32_t *z, int64_t N,
                          int32_t M, int32_t V, int32_t K, hipStream_t s) {
  if (width_for(K) == 64)
    launch_butterfly<64, LDS_TABLE, ALT>(theta, phi, d, word_id, u, z, N, M, V, K, s);
  else
    launch_butterfly<32, LDS_TABLE, ALT>(theta, phi, d, word_id, u, z, N, M, V, K, s);
}

// LDS of the document-per-lane driver per workgroup: the block-end prefixes,
// and with the theta cache K rounded up to W rows of 64 floats per wavefront.
size_t doc_lanes_lds(int32_t K, bool theta_lds) {
  const int W = width_for(K);
  const int nb = (K + W - 1) / W;
  return (size_t)kWavesPerBlock * ((theta_lds ? nb * W : 0) + nb) * kWave * sizeof(float);
}

size_t doc_lanes_cache_bytes(int32_t K) {
  const int W = width_for(K);
  const int nb = (K + W - 1) / W;
  return (size_t)nb * W * kWave * sizeof(float);
}

// Wavefronts per group of 64 documents: enough for about
// LDA_DOC_LANES_TARGET_WAVES wavefronts in all, at most the mean document
// length (beyond it most wavefronts would find no token).
int doc_lanes_split(int64_t N, int32_t M) {
  const int64_t groups = (M + kWave - 1) / kWave;
  int64_t S = (LDA_DOC_LANES_TARGET_WAVES + groups - 1) / groups;
  const int64_t mean_len = (N + M - 1) / M;
  if (S > mean_len) S = mean_len;
  return (int)(S < 1 ? 1 : S);
}

template <int W, bool THETA_LDS>
void launch_doc_lanes(const float *theta, const float *phi, const int64_t *off,
                      const int32_t *wd, UniformSource u, int32_t *z, int64_t N, int32_t M,
                      int32_t V, int32_t K, hipStream_t s) {
  const uint32_t tb = table_extent(M, K);
  const uint32_t pb = table_extent(V, K);
  const int S = doc_lanes_split(N, M);
  const int64_t groups = (M + kWave - 1) / kWave;
  doc_lanes_kernel<W, THETA_LDS>
      <<<wave_grid(groups * S * kWave), kBlockThreads, doc_lanes_lds(K, THETA_LDS), s>>>(
          theta, phi, off, wd, u, z, N, M, K, S, tb, pb);
}

// Workspace of the routing: the routed arrays and the builder's tables, each
// section starting on a 256-byte boundary.
struct RouteLayout {
  int64_t Np, nchunks;
  size_t perm, rword, rdoc, chunk_off, counts, map, lists, chunk_hist, bytes;
};

RouteLayout route_layout(int64_t N) {
  RouteLayout L;
  L.Np = N + (int64_t)kRouteXcds * kRoutePad;  // a list pads fewer than 64 positions
  L.nchunks = (N + kRouteChunk - 1) / kRouteChunk;
  size_t off = 0;
  auto take = [&](size_t b) {
    const size_t o = off;
    off += (b + 255) & ~(size_t)255;
    return o;
  };
  L.perm = take(4 * (size_t)L.Np);
  L.rword = take(4 * (size_t)L.Np);
  L.rdoc = take(4 * (size_t)L.Np);
  L.chunk_off = take(4 * (size_t)kRouteXcds * (size_t)L.nchunks);
  L.counts = take(4 * kRouteClasses);
  L.map = take(4 * kRouteClasses);
  L.lists = take(8 * 3 * kRouteXcds);
  L.chunk_hist = take(4 * (size_t)kRouteClasses * (size_t)L.nchunks);
  L.bytes = off;
  return L;
}

RoutePlan route_plan(void *ws, const RouteLayout &L) {
  char *b = static_cast<char *>(ws);
  return RoutePlan{reinterpret_cast<int32_t *>(b + L.perm), reinterpret_cast<int32_t *>(b + L.rword),
                   reinterpret_cast<int32_t *>(b + L.rdoc), reinterpret_cast<int32_t *>(b + L.chunk_off),
                   reinterpret_cast<int32_t *>(b + L.counts), reinterpret_cast<int32_t *>(b + L.map),
                   reinterpret_cast<int64_t *>(b + L.lists),
                   reinterpret_cast<int32_t *>(b + L.chunk_hist)};
}

// K the routed draw takes: the eighths kernel's K from LDA_ROUTE_MIN_K up.
// Routing pays only where phi is far larger than the caches: measured on
// MI355X over 16.8M Zipf tokens with V = 100,000 words, the routed draw is
// 28% slower than the token-order draw at K = 256 and 3% at K = 512 (phi of
// 98 and 195 MiB: it fits the 256 MiB MALL, and the few-documents theta path
// costs more than routing saves), and 2-13% faster from K = 768 (293 MiB) to
// 2048 (28% on the Poisson corpus at K = 2048).  Smaller K are refused.
bool routed_for(int32_t K) {
  return K % kLeaf == 0 && K >= LDA_ROUTE_MIN_K && K >= LDA_EIGHTHS_MIN_K &&
         eighths_blocks(K) <= LDA_EIGHTHS_MAX_BLOCKS;
}

}  // namespace
}  // namespace lda

using namespace lda;

extern "C" int lda_draw_naive(const float *theta, const float *phi,
                              const int32_t *doc_id, const int32_t *word_id,
                              const float *u, int32_t *z, int64_t N, int32_t M,
                              int32_t V, int32_t K, void *stream) {
  const int st = check_args(theta, phi, doc_id, word_id, u, z, N, M, V, K);
  if (st != LDA_OK || N == 0) return st;
  const UniformSource us{u, 0, 0, 0};
  hipStream_t s = static_cast<hipStream_t>(stream);
  const DocSource d{doc_id, nullptr, M, N};
  if (K <= 64)
    launch_naive<64>(theta, phi, d, word_id, us, z, N, K, s);
  else if (K <= 256)
    launch_naive<256>(theta, phi, d, word_id, us, z, N, K, s);
  else if (K <= 1024)
    launch_naive<1024>(theta, phi, d, word_id, us, z, N, K, s);
  else
    launch_naive<LDA_MAX_K>(theta, phi, d, word_id, us, z, N, K, s);
  return finish_launch();
}

extern "C" int lda_draw_butterfly(const float *theta, const float *phi,
                                  const int32_t *doc_id, const int32_t *word_id,
                                  const float *u, int32_t *z, int64_t N,
                                  int32_t M, int32_t V, int32_t K,
                                  void *stream) {
  const int st = check_args(theta, phi, doc_id, word_id, u, z, N, M, V, K, true);
  if (st != LDA_OK || N == 0) return st;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (wide_tables(M, V, K))
    lda_wide::draw(theta, phi, doc_id, nullptr, word_id, u, 0, 0, 0, z, N, M, V, K, s);
  else
    dispatch_butterfly(theta, phi, DocSource{doc_id, nullptr, M, N}, word_id,
                       UniformSource{u, 0, 0, 0}, z, N, M, V, K, s);
  return finish_launch();
}

extern "C" int lda_draw_transposed(const float *theta, const float *phi,
                                   const int32_t *doc_id, const int32_t *word_id,
                                   const float *u, int32_t *z, int64_t N, int32_t M,
                                   int32_t V, int32_t K, void *stream) {
  const int st = check_args(theta, phi, doc_id, word_id, u, z, N, M, V, K);
  if (st != LDA_OK || N == 0) return st;
  const UniformSource us{u, 0, 0, 0};
  launch_transposed(theta, phi, DocSource{doc_id, nullptr, M, N}, word_id, us, z, N, M, V, K,
                    static_cast<hipStream_t>(stream));
  return finish_launch();
}

extern "C" int lda_draw_butterfly_variant(const float *theta, const float *phi,
                                          const int32_t *doc_id, const int32_t *word_id,
                                          const float *u, int32_t *z, int64_t N, int32_t M,
                                          int32_t V, int32_t K, int32_t variant,
                                          void *stream) {
  if (variant != LDA_VARIANT_REGISTER_TABLE && variant != LDA_VARIANT_LDS_TABLE &&
      variant != LDA_VARIANT_LDS_TABLE_ALT && variant != LDA_VARIANT_LEAF8 &&
      variant != LDA_VARIANT_WIDE_TABLES)
    return LDA_ERR_UNSUPPORTED;
  const bool wide = variant == LDA_VARIANT_WIDE_TABLES;
  const int st = check_args(theta, phi, doc_id, word_id, u, z, N, M, V, K, wide);
  if (st != LDA_OK || N == 0) return st;
  const UniformSource us{u, 0, 0, 0};
  const DocSource d{doc_id, nullptr, M, N};
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (wide)
    lda_wide::draw(theta, phi, doc_id, nullptr, word_id, u, 0, 0, 0, z, N, M, V, K, s);
  else if (variant == LDA_VARIANT_LEAF8)
    dispatch_butterfly<2>(theta, phi, d, word_id, us, z, N, M, V, K, s);
  else if (variant == LDA_VARIANT_REGISTER_TABLE)
    launch_table_variant<false, false>(theta, phi, d, word_id, us, z, N, M, V, K, s);
  else if (variant == LDA_VARIANT_LDS_TABLE)
    launch_table_variant<true, false>(theta, phi, d, word_id, us, z, N, M, V, K, s);
  else
    launch_table_variant<true, true>(theta, phi, d, word_id, us, z, N, M, V, K, s);
  return finish_launch();
}

extern "C" int lda_draw_doc_lanes(const float *theta, const float *phi,
                                  const int64_t *doc_offsets, const int32_t *word_id,
                                  const float *u, int32_t *z, int64_t N, int32_t M,
                                  int32_t V, int32_t K, int32_t theta_cache,
                                  void *stream) {
  if (theta_cache != 0 && theta_cache != 1) return LDA_ERR_UNSUPPORTED;
  const int st = check_args(theta, phi, doc_offsets, word_id, u, z, N, M, V, K);
  if (st != LDA_OK) return st;
  if (theta_cache && doc_lanes_cache_bytes(K) > LDA_DOC_LANES_MAX_CACHE_BYTES)
    return LDA_ERR_UNSUPPORTED;
  if (N == 0) return LDA_OK;
  if (reinterpret_cast<uintptr_t>(doc_offsets) & 7u) return LDA_ERR_ALIGN;
  const UniformSource us{u, 0, 0, 0};
  hipStream_t s = static_cast<hipStream_t>(stream);
  const bool tl = theta_cache != 0;
  if (width_for(K) == 64) {
    if (tl)
      launch_doc_lanes<64, true>(theta, phi, doc_offsets, word_id, us, z, N, M, V, K, s);
    else
      launch_doc_lanes<64, false>(theta, phi, doc_offsets, word_id, us, z, N, M, V, K, s);
  } else {
    if (tl)
      launch_doc_lanes<32, true>(theta, phi, doc_offsets, word_id, us, z, N, M, V, K, s);
    else
      launch_doc_lanes<32, false>(theta, phi, doc_offsets, word_id, us, z, N, M, V, K, s);
  }
  return finish_launch();
}

extern "C" int lda_draw_butterfly_philox(const float *theta, const float *phi,
                                         const int32_t *doc_id, const int32_t *word_id,
                                         int32_t *z, int64_t N, int32_t M, int32_t V,
                                         int32_t K, uint64_t seed, uint32_t sweep,
                                         void *stream) {
  // (z stands in for the absent u in the pointer checks)
  const int st = check_args(theta, phi, doc_id, word_id, z, z, N, M, V, K, true);
  if (st != LDA_OK || N == 0) return st;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
  if (wide_tables(M, V, K))
    lda_wide::draw(theta, phi, doc_id, nullptr, word_id, nullptr, k0, k1, sweep, z, N, M, V, K,
                   s);
  else
    dispatch_butterfly(theta, phi, DocSource{doc_id, nullptr, M, N}, word_id,
                       UniformSource{nullptr, k0, k1, sweep}, z, N, M, V, K, s);
  return finish_launch();
}

namespace lda {
namespace {

// The in-kernel uniforms written out: u[i] = uniform of token first + i.
__global__ __launch_bounds__(256) void uniforms_kernel(float *__restrict__ u, int64_t count,
                                                       int64_t first, UniformSource us) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += stride)
    u[i] = us(first + i);
}

}  // namespace
}  // namespace lda

extern "C" int lda_philox_uniforms(float *u, int64_t count, int64_t first, uint64_t seed,
                                   uint32_t sweep, void *stream) {
  if (count < 0 || first < 0 || count > INT64_MAX - first) return LDA_ERR_SHAPE;
  if (count == 0) return LDA_OK;
  if (!u) return LDA_ERR_NULL;
  if (reinterpret_cast<uintptr_t>(u) & 3u) return LDA_ERR_ALIGN;
  const UniformSource us{nullptr, (uint32_t)seed, (uint32_t)(seed >> 32), sweep};
  const int64_t blocks = (count + 255) / 256;
  uniforms_kernel<<<(unsigned)(blocks < 4096 ? blocks : 4096), 256, 0,
                    static_cast<hipStream_t>(stream)>>>(u, count, first, us);
  return finish_launch();
}

extern "C" int lda_draw_docs(const float *theta, const float *phi,
                             const int64_t *doc_offsets, const int32_t *word_id,
                             const float *u, int32_t *z, int64_t N, int32_t M,
                             int32_t V, int32_t K, void *stream) {
  int st = check_args(theta, phi, doc_offsets, word_id, u, z, N, M, V, K, true);
  if (st != LDA_OK || N == 0) return st;
  if (reinterpret_cast<uintptr_t>(doc_offsets) & 7u) return LDA_ERR_ALIGN;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (wide_tables(M, V, K))
    lda_wide::draw(theta, phi, nullptr, doc_offsets, word_id, u, 0, 0, 0, z, N, M, V, K, s);
  else
    dispatch_butterfly(theta, phi, DocSource{nullptr, doc_offsets, M, N}, word_id,
                       UniformSource{u, 0, 0, 0}, z, N, M, V, K, s);
  return finish_launch();
}

extern "C" int lda_butterfly_table(const float *theta, const float *phi,
                                   const int32_t *doc_id,
                                   const int32_t *word_id, float *table,
                                   int64_t N, int32_t M, int32_t V, int32_t K,
                                   void *stream) {
  // u is not used here; pass a valid stand-in so the shared check applies.
  const int st = check_args(theta, phi, doc_id, word_id, theta, table, N, M, V,
                            K);
  if (st != LDA_OK || N == 0) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const uint32_t tb = table_extent(M, K);
  const uint32_t pb = table_extent(V, K);
  if (width_for(K) == 64)
    table_kernel<64, true><<<wave_grid(N), kBlockThreads, 0, s>>>(
        theta, phi, doc_id, word_id, table, N, K, tb, pb);
  else
    table_kernel<32, true><<<wave_grid(N), kBlockThreads, 0, s>>>(
        theta, phi, doc_id, word_id, table, N, K, tb, pb);
  return finish_launch();
}

extern "C" size_t lda_route_workspace_bytes(int64_t N) {
  if (N < 0 || N > LDA_ROUTE_MAX_N) return 0;
  return route_layout(N).bytes;
}

namespace lda {
namespace {

// The routing's kernels and its one read-back, into a workspace already
// checked to hold route_layout(N).bytes (N > 0, arguments checked).
int route_build_into(const int32_t *doc_id, const int32_t *word_id, int64_t N, void *workspace,
                     lda_route *route, hipStream_t s) {
  const RouteLayout L = route_layout(N);
  const RoutePlan P = route_plan(workspace, L);
  route_fill<<<1, kRouteClasses, 0, s>>>(P.counts, kRouteClasses, 0);
  route_hist<<<(unsigned)(L.nchunks < 256 ? L.nchunks : 256), kRouteThreads, 0, s>>>(
      word_id, N, L.nchunks, P.chunk_hist, P.counts);
  int st = finish_launch();
  if (st != LDA_OK) return st;
  // the class counts, read back once: the host assigns the classes and lays
  // out the lists (whose sizes also size the draw's grid)
  int32_t counts[kRouteClasses];
  hipError_t e = hipMemcpyAsync(counts, P.counts, sizeof(counts), hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) {
    g_last_hip = e;
    return LDA_ERR_HIP;
  }
  const RouteAssignment a = route_assign(counts);
  route_set<<<1, kRouteThreads, 0, s>>>(a, P.map, P.lists);
  route_count<<<(unsigned)L.nchunks, kRouteThreads, 0, s>>>(P.chunk_hist, P.map, P.chunk_off);
  route_scan<<<kRouteXcds, kRouteThreads, 0, s>>>(P.chunk_off, L.nchunks);
  route_scatter<<<(unsigned)L.nchunks, kRouteThreads, 0, s>>>(word_id, doc_id, N, P.map,
                                                              P.chunk_off, P.lists, P.perm,
                                                              P.rword, P.rdoc);
  route_pad<<<kRouteXcds, kRouteThreads, 0, s>>>(P.lists, P.perm, P.rword, P.rdoc);
  st = finish_launch();
  if (st != LDA_OK) return st;
  const int64_t *lists = a.lists;
  route->N = N;
  for (int x = 0; x < kRouteXcds; ++x) {
    route->tokens[x] = lists[x];
    route->start[x] = lists[kRouteXcds + x];
    route->length[x] = lists[2 * kRouteXcds + x];
  }
  return LDA_OK;
}

}  // namespace
}  // namespace lda

extern "C" int lda_route_build(const int32_t *doc_id, const int32_t *word_id, int64_t N,
                               int32_t M, int32_t V, void *workspace, size_t workspace_bytes,
                               lda_route *route, void *stream) {
  if (!route) return LDA_ERR_NULL;
  if (N < 0 || M <= 0 || V <= 0) return LDA_ERR_SHAPE;
  if (N > LDA_ROUTE_MAX_N) return LDA_ERR_UNSUPPORTED;
  *route = lda_route{};
  if (N == 0) return LDA_OK;
  if (!doc_id || !word_id || !workspace) return LDA_ERR_NULL;
  if ((reinterpret_cast<uintptr_t>(doc_id) | reinterpret_cast<uintptr_t>(word_id)) & 3u ||
      reinterpret_cast<uintptr_t>(workspace) & 7u)
    return LDA_ERR_ALIGN;
  if (workspace_bytes < route_layout(N).bytes) return LDA_ERR_WORKSPACE;
  return route_build_into(doc_id, word_id, N, workspace, route, static_cast<hipStream_t>(stream));
}

namespace lda {
namespace {

// The routed draw for either uniform source.  `u_check` stands in for u in
// the pointer checks (z when the uniforms come from Philox).
int draw_routed(const float *theta, const float *phi, const void *workspace,
                size_t workspace_bytes, const lda_route *route, const void *u_check,
                const UniformSource &us, int32_t *z, int64_t N, int32_t M, int32_t V, int32_t K,
                void *stream) {
  if (!route) return LDA_ERR_NULL;
  const int st = check_args(theta, phi, workspace, workspace, u_check, z, N, M, V, K);
  if (st != LDA_OK) return st;
  if (!routed_for(K) || N > LDA_ROUTE_MAX_N) return LDA_ERR_UNSUPPORTED;
  if (N == 0) return LDA_OK;
  if (reinterpret_cast<uintptr_t>(workspace) & 7u) return LDA_ERR_ALIGN;
  const RouteLayout L = route_layout(N);
  if (route->N != N || workspace_bytes < L.bytes) return LDA_ERR_WORKSPACE;
  int64_t max_len = 0, total = 0;
  for (int x = 0; x < kRouteXcds; ++x) {
    if (route->length[x] < 0 || route->start[x] < 0 || route->length[x] % kRoutePad ||
        route->start[x] + route->length[x] > L.Np)
      return LDA_ERR_WORKSPACE;
    max_len = route->length[x] > max_len ? route->length[x] : max_len;
    total += route->tokens[x];
  }
  if (total != N) return LDA_ERR_WORKSPACE;
  const RoutePlan P = route_plan(const_cast<void *>(workspace), L);
  RoutedTokens rt{P.perm, P.rword, P.rdoc, {}, {}};
  for (int x = 0; x < kRouteXcds; ++x) {
    rt.base[x] = route->start[x];
    rt.len[x] = route->length[x];
  }
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (K % kBlock4 == 0)
    launch_routed<false>(theta, phi, rt, us, z, max_len, M, V, K, s);
  else
    launch_routed<true>(theta, phi, rt, us, z, max_len, M, V, K, s);
  return finish_launch();
}

}  // namespace
}  // namespace lda

extern "C" int lda_draw_routed(const float *theta, const float *phi, const void *workspace,
                               size_t workspace_bytes, const lda_route *route, const float *u,
                               int32_t *z, int64_t N, int32_t M, int32_t V, int32_t K,
                               void *stream) {
  return lda::draw_routed(theta, phi, workspace, workspace_bytes, route, u,
                          lda::UniformSource{u, 0, 0, 0}, z, N, M, V, K, stream);
}

extern "C" int lda_draw_routed_philox(const float *theta, const float *phi,
                                      const void *workspace, size_t workspace_bytes,
                                      const lda_route *route, int32_t *z, int64_t N, int32_t M,
                                      int32_t V, int32_t K, uint64_t seed, uint32_t sweep,
                                      void *stream) {
  const lda::UniformSource us{nullptr, (uint32_t)seed, (uint32_t)(seed >> 32), sweep};
  return lda::draw_routed(theta, phi, workspace, workspace_bytes, route, z, us, z, N, M, V, K,
                          stream);
}

// ---------------------------------------------------------------------------
// The routed draw for callers that cannot allocate: the routing lives in this
// file-scope array instead of a caller's workspace.  Each GPU the library
// runs on holds its own copy (LDA_ROUTED_SCRATCH_BYTES) until the process
// ends; its device address is looked up once per device (hipGetSymbolAddress,
// with the device current) and only that address is handed to kernels.
namespace lda {
namespace {

__device__ __align__(256) unsigned char scratch[LDA_ROUTED_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void *g_scratch_ptr[kMaxDevices] = {};

// The current device's address of `scratch` (looked up on the first call on
// that device), or nullptr with the HIP error recorded.
void *scratch_address() {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess && (dev < 0 || dev >= kMaxDevices)) e = hipErrorInvalidDevice;
  if (e != hipSuccess) {
    g_last_hip = e;
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void *ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) {
      g_last_hip = e != hipSuccess ? e : hipErrorInvalidSymbol;
      return nullptr;
    }
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}

}  // namespace
}  // namespace lda

extern "C" int lda_draw_routed_scratch(const float *theta, const float *phi,
                                       const int32_t *doc_id, const int32_t *word_id,
                                       const float *u, int32_t *z, int64_t N, int32_t M,
                                       int32_t V, int32_t K, void *stream) {
  // every check before any HIP call
  const int st = check_args(theta, phi, doc_id, word_id, u, z, N, M, V, K);
  if (st != LDA_OK) return st;
  if (!routed_for(K) || N > LDA_ROUTE_MAX_N) return LDA_ERR_UNSUPPORTED;
  if (N == 0) return LDA_OK;
  const size_t bytes = route_layout(N).bytes;
  if (bytes > LDA_ROUTED_SCRATCH_BYTES) return LDA_ERR_UNSUPPORTED;
  void *ws = scratch_address();
  if (!ws) return LDA_ERR_HIP;
  lda_route route{};
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const int b = route_build_into(doc_id, word_id, N, ws, &route, s);
  if (b != LDA_OK) return b;
  const UniformSource us{u, 0, 0, 0};
  return draw_routed(theta, phi, ws, bytes, &route, u, us, z, N, M, V, K, stream);
}

namespace lda {
namespace {

// Workgroups of count_docs_kernel for M documents: one per kDocWaves
// documents, at most kDocGridMax (the kernel strides over the rest).
unsigned doc_grid(int32_t M) {
  const int64_t b = ((int64_t)M + kDocWaves - 1) / kDocWaves;
  return (unsigned)(b < kDocGridMax ? b : kDocGridMax);
}

}  // namespace
}  // namespace lda

extern "C" int lda_count_topics(const int32_t *doc_id, const int32_t *word_id, const int32_t *z,
                                int64_t N, int32_t M, int32_t V, int32_t K, int32_t *ndk,
                                int32_t *nwk, void *stream) {
  if (N < 0 || M <= 0 || V <= 0 || K <= 0) return LDA_ERR_SHAPE;
  if (K > LDA_MAX_K || N > LDA_COUNT_MAX_N) return LDA_ERR_UNSUPPORTED;
  // cells are addressed by unsigned 32-bit indices (d K + k, w K + k)
  if ((int64_t)M * K * 4 > LDA_MAX_COUNT_TABLE_BYTES ||
      (int64_t)V * K * 4 > LDA_MAX_COUNT_TABLE_BYTES)
    return LDA_ERR_UNSUPPORTED;
  if (!ndk || !nwk) return LDA_ERR_NULL;
  if (N > 0 && (!doc_id || !word_id || !z)) return LDA_ERR_NULL;
  const void *ptrs[] = {ndk, nwk, doc_id, word_id, z};
  for (const void *p : ptrs)
    if (reinterpret_cast<uintptr_t>(p) & 3u) return LDA_ERR_ALIGN;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t cells[2] = {(int64_t)M * K, (int64_t)V * K};
  int32_t *tables[2] = {ndk, nwk};
  for (int t = 0; t < 2; ++t) {
    const int64_t blocks = (cells[t] / 4 + 255) / 256;
    count_clear<<<(unsigned)(blocks < 4096 ? (blocks > 0 ? blocks : 1) : 4096), 256, 0, s>>>(
        tables[t], cells[t]);
  }
  if (N > 0) {
    const int64_t chunks = (N + kCountChunk - 1) / kCountChunk;
    count_kernel<<<(unsigned)chunks, kCountThreads, 0, s>>>(doc_id, word_id, z, N, M, V, K, ndk,
                                                            nwk);
  }
  return finish_launch();
}

extern "C" int lda_count_topics_docs(const int64_t *doc_offsets, const int32_t *word_id,
                                     const int32_t *z, int64_t N, int32_t M, int32_t V,
                                     int32_t K, int32_t *ndk, int32_t *nwk, void *stream) {
  if (N < 0 || M <= 0 || V <= 0 || K <= 0) return LDA_ERR_SHAPE;
  if (K > LDA_MAX_K || N > LDA_COUNT_MAX_N) return LDA_ERR_UNSUPPORTED;
  // nwk's cells are keyed by unsigned 32-bit indices (w K + k); ndk's rows
  // are written whole at 64-bit addresses, of any size
  if ((int64_t)V * K * 4 > LDA_MAX_COUNT_TABLE_BYTES) return LDA_ERR_UNSUPPORTED;
  if (!ndk || !nwk || !doc_offsets) return LDA_ERR_NULL;
  if (N > 0 && (!word_id || !z)) return LDA_ERR_NULL;
  const void *ptrs[] = {ndk, nwk, word_id, z};
  for (const void *p : ptrs)
    if (reinterpret_cast<uintptr_t>(p) & 3u) return LDA_ERR_ALIGN;
  if (reinterpret_cast<uintptr_t>(doc_offsets) & 7u) return LDA_ERR_ALIGN;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t cells = (int64_t)V * K;
  const int64_t blocks = (cells / 4 + 255) / 256;
  count_clear<<<(unsigned)(blocks < 4096 ? (blocks > 0 ? blocks : 1) : 4096), 256, 0, s>>>(
      nwk, cells);
  const size_t lds = (size_t)kDocWaves * (size_t)K * sizeof(uint32_t);
  count_docs_kernel<<<doc_grid(M), kDocWaves * 64, lds, s>>>(doc_offsets, word_id, z, N, M, V,
                                                              K, ndk);
  if (N > 0) {
    const int64_t chunks = (N + kCountChunk - 1) / kCountChunk;
    count_words_kernel<<<(unsigned)chunks, kCountThreads, 0, s>>>(word_id, z, N, V, K, nwk);
  }
  return finish_launch();
}

// ---------------------------------------------------------------------------
// The word index: off [V + 1], the histogram / cursors [V kCounterStride],
// the scan's workgroup sums, perm [N] and wsorted [N], each section on a
// 256-byte boundary.
namespace lda {
namespace {

struct WordIndexLayout {
  size_t off, cursor, sums, perm, wsorted, bytes;
};

WordIndexLayout word_index_layout(int64_t N, int32_t V) {
  WordIndexLayout L;
  size_t at = 0;
  auto take = [&](size_t b) {
    const size_t o = at;
    at += (b + 255) & ~(size_t)255;
    return o;
  };
  L.off = take(4 * ((size_t)V + 1));
  L.cursor = take(4 * (size_t)V * kCounterStride);
  L.sums = take(4 * (size_t)kScanMaxBlocks);
  L.perm = take(4 * (size_t)(N > 0 ? N : 1));
  L.wsorted = take(4 * (size_t)(N > 0 ? N : 1));
  L.bytes = at;
  return L;
}

int check_word_index(int64_t N, int32_t V, const void *index, size_t index_bytes) {
  if (N < 0 || V <= 0) return LDA_ERR_SHAPE;
  if (N > LDA_COUNT_MAX_N || V > LDA_WORD_INDEX_MAX_V) return LDA_ERR_UNSUPPORTED;
  if (!index) return LDA_ERR_NULL;
  if (reinterpret_cast<uintptr_t>(index) & 7u) return LDA_ERR_ALIGN;
  if (index_bytes < word_index_layout(N, V).bytes) return LDA_ERR_WORKSPACE;
  return LDA_OK;
}

unsigned fill_grid(int64_t n) {
  const int64_t b = (n + 255) / 256;
  return (unsigned)(b < 4096 ? (b > 0 ? b : 1) : 4096);
}

}  // namespace
}  // namespace lda

extern "C" size_t lda_word_index_bytes(int64_t N, int32_t V) {
  if (N < 0 || V <= 0 || N > LDA_COUNT_MAX_N || V > LDA_WORD_INDEX_MAX_V) return 0;
  return word_index_layout(N, V).bytes;
}

extern "C" int lda_word_index_build(const int32_t *word_id, int64_t N, int32_t V, void *index,
                                    size_t index_bytes, void *stream) {
  const int st = check_word_index(N, V, index, index_bytes);
  if (st != LDA_OK) return st;
  if (N > 0 && !word_id) return LDA_ERR_NULL;
  if (reinterpret_cast<uintptr_t>(word_id) & 3u) return LDA_ERR_ALIGN;
  const WordIndexLayout L = word_index_layout(N, V);
  char *b = static_cast<char *>(index);
  int32_t *off = reinterpret_cast<int32_t *>(b + L.off);
  int32_t *cursor = reinterpret_cast<int32_t *>(b + L.cursor);
  int32_t *sums = reinterpret_cast<int32_t *>(b + L.sums);
  int32_t *perm = reinterpret_cast<int32_t *>(b + L.perm);
  int32_t *wsorted = reinterpret_cast<int32_t *>(b + L.wsorted);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int run = index_run(N);
  const int64_t per = (int64_t)run * kCountChunk;
  const unsigned runs = (unsigned)((N + per - 1) / per);
  // histogram of the words into cursor, then its exclusive scan into off
  const int64_t counters = (int64_t)V * kCounterStride;
  index_fill<<<fill_grid(counters), 256, 0, s>>>(cursor, counters, 0);
  if (N > 0) index_hist<<<runs, kCountThreads, 0, s>>>(word_id, N, V, run, cursor);
  const int64_t items = (int64_t)V + 1;
  const unsigned nb = (unsigned)((items + kScanItems - 1) / kScanItems);
  index_scan_local<<<nb, kScanThreads, 0, s>>>(cursor, V, kCounterStride, items, off, sums);
  index_scan_sums<<<1, kScanThreads, 0, s>>>(sums, (int32_t)nb);
  index_scan_add<<<nb, kScanThreads, 0, s>>>(off, items, sums);
  // the tokens placed word by word
  index_fill<<<fill_grid(counters), 256, 0, s>>>(cursor, counters, 0);
  if (N > 0)
    index_scatter<<<runs, kCountThreads, 0, s>>>(word_id, N, V, run, off, cursor, perm, wsorted,
                                                 N);
  return finish_launch();
}

extern "C" int lda_count_topics_indexed(const int64_t *doc_offsets, const int32_t *word_id,
                                        const int32_t *z, int64_t N, int32_t M, int32_t V,
                                        int32_t K, const void *index, size_t index_bytes,
                                        int32_t *ndk, int32_t *nwk, void *stream) {
  if (N < 0 || M <= 0 || V <= 0 || K <= 0) return LDA_ERR_SHAPE;
  if (K > LDA_MAX_K) return LDA_ERR_UNSUPPORTED;
  // (as lda_count_topics_docs: only nwk is limited)
  if ((int64_t)V * K * 4 > LDA_MAX_COUNT_TABLE_BYTES) return LDA_ERR_UNSUPPORTED;
  const int st = check_word_index(N, V, index, index_bytes);
  if (st != LDA_OK) return st;
  if (!ndk || !nwk || !doc_offsets) return LDA_ERR_NULL;
  if (N > 0 && (!word_id || !z)) return LDA_ERR_NULL;
  const void *ptrs[] = {ndk, nwk, word_id, z};
  for (const void *p : ptrs)
    if (reinterpret_cast<uintptr_t>(p) & 3u) return LDA_ERR_ALIGN;
  if (reinterpret_cast<uintptr_t>(doc_offsets) & 7u) return LDA_ERR_ALIGN;
  const WordIndexLayout L = word_index_layout(N, V);
  const char *b = static_cast<const char *>(index);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t cells = (int64_t)V * K;
  const int64_t blocks = (cells / 4 + 255) / 256;
  count_clear<<<(unsigned)(blocks < 4096 ? (blocks > 0 ? blocks : 1) : 4096), 256, 0, s>>>(
      nwk, cells);
  const size_t lds = (size_t)kDocWaves * (size_t)K * sizeof(uint32_t);
  count_docs_kernel<<<doc_grid(M), kDocWaves * 64, lds, s>>>(doc_offsets, word_id, z, N, M, V,
                                                              K, ndk);
  if (N > 0) {
    const int run = index_run(N);
    const int64_t per = (int64_t)run * kCountChunk;
    count_words_indexed<<<(unsigned)((N + per - 1) / per), kCountThreads, 0, s>>>(
        reinterpret_cast<const int32_t *>(b + L.perm), reinterpret_cast<const int32_t *>(b + L.wsorted),
        reinterpret_cast<const int32_t *>(b + L.off), z, N, V, K, run, nwk);
  }
  return finish_launch();
}

extern "C" int lda_butterfly_width(int32_t K) {
  if (K <= 0) return LDA_ERR_SHAPE;
  if (K > LDA_MAX_K) return LDA_ERR_UNSUPPORTED;
  return width_for(K);
}

extern "C" const char *lda_status_string(int status) {
  switch (status) {
    case LDA_OK: return "ok";
    case LDA_ERR_NULL: return "a required pointer is NULL";
    case LDA_ERR_SHAPE: return "invalid shape (N < 0, M <= 0, V <= 0 or K <= 0)";
    case LDA_ERR_UNSUPPORTED:
      return "unsupported size (K > LDA_MAX_K, N > LDA_MAX_N, a table larger than the entry "
             "point takes, or a K or N the entry point does not take)";
    case LDA_ERR_HIP: return "HIP runtime error";
    case LDA_ERR_ALIGN: return "a pointer is not aligned (4 bytes; 8 for offsets and workspaces)";
    case LDA_ERR_WORKSPACE:
      return "routing workspace too small, or the route does not belong to these tokens";
    default: return "unknown status";
  }
}

extern "C" const char *lda_last_hip_error(void) {
  return hipGetErrorString(g_last_hip);
}

extern "C" int lda_version(void) { return 300; }
