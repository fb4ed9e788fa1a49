// HIP kernels and C ABI of the per-token LDA topic draw (gfx950).
//
// lda_draw_naive      Algorithm 1 + Algorithm 3, one lane per token.
// lda_draw_butterfly  Algorithm 7 (+ 5, 8, 9, 10) for 64-lane wavefronts.
// lda_butterfly_table the butterfly-patterned tables (Fig. 1, right).
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "butterfly.hpp"
#include "lda_draw.h"

namespace lda {
namespace {

constexpr int kWavesPerBlock = 4;
constexpr int kBlockThreads = kWavesPerBlock * kWave;

// ---------------------------------------------------------------------------
// Naive kernel (Algorithm 1 with Algorithm 3).  Lane n walks the K topics of
// its own token, keeps the full prefix table p[K] in its private segment and
// binary-searches it for the first entry above stop = S * u.
template <int KMAX>
__global__ __launch_bounds__(256) void naive_kernel(
    const float *__restrict__ theta, const float *__restrict__ phi,
    const int32_t *__restrict__ doc_id, const int32_t *__restrict__ word_id,
    const float *__restrict__ u, int32_t *__restrict__ z, int64_t N, int K) {
  const int64_t n = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (n >= N) return;
  const float *th = theta + (int64_t)doc_id[n] * K;
  const float *ph = phi + (int64_t)word_id[n] * K;
  float p[KMAX];
  float sum = 0.0f;
  for (int k = 0; k < K; ++k) {
    sum = prefix_step(sum, th[k], ph[k]);
    p[k] = sum;
  }
  const float stop = sum * u[n];
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

// LDS floats per wavefront of the butterfly kernel: the block-end prefixes
// (NB rows of 64 lanes) during the sweep, then the rebuilt table of one block
// (W - 1 rows of 64 lanes) during the search.
__host__ __device__ constexpr int region_rows(int NB, int W) {
  return NB > W - 1 ? NB : W - 1;
}

// ---------------------------------------------------------------------------
// Butterfly kernel.  Wavefront g takes tokens [64 g, 64 g + 64); lanes past N
// repeat token N - 1 so that every lane takes part in every exchange (the
// paper's "staying awake" rule) and skip the store.
//
// Sweep (Algorithm 8 without the table): per block, the transposed tile,
// the butterfly, and the running prefix at the block's end, kept in LDS.
// Search (Algorithm 9): binary search over the block ends for stop = S * u.
// Rebuild: one tile in which every token contributes its own chosen block;
// the butterfly's rows go to LDS.  In-block search (Algorithm 10): at level b
// lane r reads row (r & mask) | (bit - 1) of column r xor flip directly from
// LDS, which is the entry the search-assist loop of the paper delivers with
// shuffles.  Remnant: Algorithm 9's linear fallback.
template <int W>
__global__ __launch_bounds__(kBlockThreads) void butterfly_kernel(
    const float *__restrict__ theta, const float *__restrict__ phi,
    const int32_t *__restrict__ doc_id, const int32_t *__restrict__ word_id,
    const float *__restrict__ u, int32_t *__restrict__ z, int64_t N, int K) {
  extern __shared__ float lds[];
  constexpr int LOG2W = (W == 64) ? 6 : 5;
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  const int64_t first = ((int64_t)blockIdx.x * kWavesPerBlock + wave) * kWave;
  if (first >= N) return;  // whole wavefront past the end
  const int64_t n = first + lane < N ? first + lane : N - 1;
  const bool valid = first + lane < N;
  const int r = lane & (W - 1);

  const int doc = doc_id[n];
  const int word = word_id[n];
  const float un = u[n];
  const int R = K % W;
  const int NB = K / W;
  float *region = lds + wave * region_rows(NB, W) * kWave;
  const int doc0 = __builtin_amdgcn_readfirstlane(doc);
  const bool one_doc = __builtin_amdgcn_ballot_w64(doc == doc0) == ~0ull;

  // Remnant: untransposed running sum of the first R topics.
  const float *th_row = theta + (int64_t)doc * K;
  const float *ph_row = phi + (int64_t)word * K;
  float sum = 0.0f;
  for (int j = 0; j < R; ++j) sum = prefix_step(sum, th_row[j], ph_row[j]);
  const float p_rem = sum;

  // Sweep over the blocks.
  for (int b = 0; b < NB; ++b) {
    float a[W];
    load_tile<W>(a, theta, phi, K, R, doc, word, b, r, one_doc, true);
    butterfly_block<W>(a, r, NoStore{});
    sum += a[W - 1];
    region[b * kWave + lane] = sum;
  }

  const float stop = sum * un;
  int j;
  if (NB == 0) {
    j = remnant_search(th_row, ph_row, R, stop, K - 1);
  } else {
    // Algorithm 9: binary search over the last row of each block.
    int lo = 0, hi = NB - 1;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (stop < region[mid * kWave + lane])
        hi = mid;
      else
        lo = mid + 1;
    }
    float low = lo > 0 ? region[(lo - 1) * kWave + lane] : p_rem;
    float high = region[lo * kWave + lane];
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    // Rebuild the chosen block of every token and keep its table in LDS.
    {
      float a[W];
      const int blk0 = __builtin_amdgcn_readfirstlane(lo);
      const bool one_blk = __builtin_amdgcn_ballot_w64(lo == blk0) == ~0ull;
      load_tile<W>(a, theta, phi, K, R, doc, word, lo, r, one_doc, one_blk);
      butterfly_block<W>(a, r, RowStore{region + lane, kWave, true});
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    // Algorithm 10: butterfly search within the block.
    const int gbase = lane & ~(W - 1);
    int flip = 0;
#pragma unroll
    for (int lvl = 0; lvl < LOG2W; ++lvl) {
      const int bit = (W / 2) >> lvl;
      const int mask = ((W - 1) * (2 * bit)) & (W - 1);
      const int d = (r & mask) | (bit - 1);
      const float y = region[d * kWave + gbase + (r ^ flip)];
      const float cmp = (r & bit) ? high - y : low + y;
      if (stop < cmp) {
        high = cmp;
        flip ^= bit & r;
      } else {
        low = cmp;
        flip ^= bit & ~r;
      }
    }
    j = R + lo * W + (flip ^ r);
    if (lo == 0 && R > 0 && stop < p_rem)
      j = remnant_search(th_row, ph_row, R, stop, K - 1);
  }
  if (valid) z[n] = j;
}

// ---------------------------------------------------------------------------
// Table dump: the per-lane table p[K] of Algorithm 7 for every token.
template <int W>
__global__ __launch_bounds__(kBlockThreads) void table_kernel(
    const float *__restrict__ theta, const float *__restrict__ phi,
    const int32_t *__restrict__ doc_id, const int32_t *__restrict__ word_id,
    float *__restrict__ table, int64_t N, int K) {
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  const int64_t first = ((int64_t)blockIdx.x * kWavesPerBlock + wave) * kWave;
  if (first >= N) return;
  const int64_t n = first + lane < N ? first + lane : N - 1;
  const bool valid = first + lane < N;
  const int r = lane & (W - 1);
  const int doc = doc_id[n];
  const int word = word_id[n];
  const int R = K % W;
  const int NB = K / W;
  const int doc0 = __builtin_amdgcn_readfirstlane(doc);
  const bool one_doc = __builtin_amdgcn_ballot_w64(doc == doc0) == ~0ull;
  float *out = table + n * (int64_t)K;

  const float *th_row = theta + (int64_t)doc * K;
  const float *ph_row = phi + (int64_t)word * K;
  float sum = 0.0f;
  for (int j = 0; j < R; ++j) {
    sum = prefix_step(sum, th_row[j], ph_row[j]);
    if (valid) out[j] = sum;
  }
  for (int b = 0; b < NB; ++b) {
    float a[W];
    load_tile<W>(a, theta, phi, K, R, doc, word, b, r, one_doc, true);
    butterfly_block<W>(a, r, RowStore{out + R + b * W, 1, valid});
    sum += a[W - 1];
    if (valid) out[R + b * W + W - 1] = sum;
  }
}

// ---------------------------------------------------------------------------
thread_local hipError_t g_last_hip = hipSuccess;

int check_args(const void *theta, const void *phi, const void *doc_id,
               const void *word_id, const void *u, const void *z, int64_t N,
               int32_t M, int32_t V, int32_t K) {
  if (N < 0 || M <= 0 || V <= 0 || K <= 0) return LDA_ERR_SHAPE;
  if (K > LDA_MAX_K) return LDA_ERR_UNSUPPORTED;
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

int width_for(int32_t K) { return K >= 64 ? 64 : 32; }

dim3 wave_grid(int64_t N) {
  const int64_t waves = (N + kWave - 1) / kWave;
  return dim3((unsigned)((waves + kWavesPerBlock - 1) / kWavesPerBlock));
}

template <int KMAX>
void launch_naive(const float *theta, const float *phi, const int32_t *d,
                  const int32_t *w, const float *u, int32_t *z, int64_t N,
                  int32_t K, hipStream_t s) {
  const dim3 grid((unsigned)((N + 255) / 256));
  naive_kernel<KMAX><<<grid, 256, 0, s>>>(theta, phi, d, w, u, z, N, K);
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
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (K <= 64)
    launch_naive<64>(theta, phi, doc_id, word_id, u, z, N, K, s);
  else if (K <= 256)
    launch_naive<256>(theta, phi, doc_id, word_id, u, z, N, K, s);
  else if (K <= 1024)
    launch_naive<1024>(theta, phi, doc_id, word_id, u, z, N, K, s);
  else
    launch_naive<LDA_MAX_K>(theta, phi, doc_id, word_id, u, z, N, K, s);
  return finish_launch();
}

extern "C" int lda_draw_butterfly(const float *theta, const float *phi,
                                  const int32_t *doc_id, const int32_t *word_id,
                                  const float *u, int32_t *z, int64_t N,
                                  int32_t M, int32_t V, int32_t K,
                                  void *stream) {
  const int st = check_args(theta, phi, doc_id, word_id, u, z, N, M, V, K);
  if (st != LDA_OK || N == 0) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int W = width_for(K);
  const size_t lds = (size_t)kWavesPerBlock * region_rows(K / W, W) * kWave *
                     sizeof(float);
  if (W == 64)
    butterfly_kernel<64><<<wave_grid(N), kBlockThreads, lds, s>>>(
        theta, phi, doc_id, word_id, u, z, N, K);
  else
    butterfly_kernel<32><<<wave_grid(N), kBlockThreads, lds, s>>>(
        theta, phi, doc_id, word_id, u, z, N, K);
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
  if (width_for(K) == 64)
    table_kernel<64><<<wave_grid(N), kBlockThreads, 0, s>>>(
        theta, phi, doc_id, word_id, table, N, K);
  else
    table_kernel<32><<<wave_grid(N), kBlockThreads, 0, s>>>(
        theta, phi, doc_id, word_id, table, N, K);
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
    case LDA_ERR_UNSUPPORTED: return "K exceeds LDA_MAX_K";
    case LDA_ERR_HIP: return "HIP runtime error";
    case LDA_ERR_ALIGN: return "a pointer is not 4-byte aligned";
    default: return "unknown status";
  }
}

extern "C" const char *lda_last_hip_error(void) {
  return hipGetErrorString(g_last_hip);
}

extern "C" int lda_version(void) { return 100; }
