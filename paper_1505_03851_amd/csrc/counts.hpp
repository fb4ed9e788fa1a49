// Topic counts of a set of draws (gfx950): the statistics the update of theta
// and phi consumes once every z has been drawn (Section 1: draw a topic for
// every word, then update theta and phi; Section 2: the uncollapsed sampler).
//
//   ndk[d][k] = tokens of document d drawn to topic k     int32 [M][K]
//   nwk[w][k] = tokens of word w drawn to topic k         int32 [V][K]
//
// (nwk word-major, the layout of phi).  A token whose document, word or topic
// is out of range is not counted.
//
// Two kernels on the caller's stream: count_clear zeroes both tables (a
// kernel, not a memset, so that the call can be captured into a graph), then
// count_kernel adds the tokens.  Device-wide atomics on each token's cells
// would serialise on the frequent words' cells (a Zipf vocabulary puts a
// tenth of all tokens on one word, most of them on a few of its topics), so
// each workgroup first aggregates a chunk of tokens in an LDS hash table keyed
// by the flat cell index, then adds each distinct cell's count with one
// device-wide atomic: a cell receives at most one atomic per chunk.  The
// document table is aggregated first, then the word table, in the same LDS.
// With documents given as offsets (contiguous), each document's row is
// counted by one wavefront in LDS and written whole instead (count_docs_kernel):
// no clearing and no atomics for that table.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "config.hpp"

namespace LDA_NS {
namespace {

constexpr int kCountThreads = 256;                     // threads per workgroup
constexpr int kCountPer = 8;                           // tokens per thread and chunk
constexpr int kCountChunk = kCountThreads * kCountPer;  // tokens per workgroup
constexpr int kCountSlots = 2 * kCountChunk;           // hash slots (load <= 1/2)
constexpr uint32_t kCountEmpty = 0xffffffffu;          // an unused slot's key

// Zero n ints with 16-byte stores (the body) and 4-byte stores (the ends).
__global__ __launch_bounds__(256) void count_clear(int32_t *p, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  // ints before the first 16-byte boundary
  const int64_t head = (int64_t)((16u - (reinterpret_cast<uintptr_t>(p) & 15u)) & 15u) / 4;
  const int64_t h = head < n ? head : n;
  if (t < h) p[t] = 0;
  int4 *body = reinterpret_cast<int4 *>(p + h);
  const int64_t quads = (n - h) / 4;
  for (int64_t i = t; i < quads; i += stride) body[i] = int4{0, 0, 0, 0};
  const int64_t tail0 = h + 4 * quads;
  if (t < n - tail0) p[tail0 + t] = 0;
}

// Slot of `key` in the table (linear probing from a multiplicative hash);
// adds one to its count.
__device__ __forceinline__ void count_insert(uint32_t *keys, uint32_t *cnt, uint32_t key) {
  uint32_t s = (key * 2654435761u) >> (32 - __builtin_ctz(kCountSlots));
  while (true) {
    const uint32_t prev = atomicCAS(&keys[s], kCountEmpty, key);
    if (prev == kCountEmpty || prev == key) {
      atomicAdd(&cnt[s], 1u);
      return;
    }
    s = (s + 1) & (kCountSlots - 1);
  }
}

// The same, returning whether the insert took a free slot (a key new to the
// table).
__device__ __forceinline__ bool count_insert_new(uint32_t *keys, uint32_t *cnt, uint32_t key) {
  uint32_t s = (key * 2654435761u) >> (32 - __builtin_ctz(kCountSlots));
  while (true) {
    const uint32_t prev = atomicCAS(&keys[s], kCountEmpty, key);
    if (prev == kCountEmpty || prev == key) {
      atomicAdd(&cnt[s], 1u);
      return prev == kCountEmpty;
    }
    s = (s + 1) & (kCountSlots - 1);
  }
}

// The same, returning the slot and, in `rank`, the key's count before this
// insert (the insert's rank among the chunk's inserts of the key).
__device__ __forceinline__ uint32_t count_insert_ranked(uint32_t *keys, uint32_t *cnt,
                                                        uint32_t key, uint32_t &rank) {
  uint32_t s = (key * 2654435761u) >> (32 - __builtin_ctz(kCountSlots));
  while (true) {
    const uint32_t prev = atomicCAS(&keys[s], kCountEmpty, key);
    if (prev == kCountEmpty || prev == key) {
      rank = atomicAdd(&cnt[s], 1u);
      return s;
    }
    s = (s + 1) & (kCountSlots - 1);
  }
}

// Add every occupied slot's count to its cell of `out` and empty the table.
__device__ __forceinline__ void count_flush(uint32_t *keys, uint32_t *cnt, int32_t *out) {
  for (int s = threadIdx.x; s < kCountSlots; s += kCountThreads) {
    const uint32_t key = keys[s];
    if (key != kCountEmpty) {
      atomicAdd(&out[key], (int32_t)cnt[s]);
      keys[s] = kCountEmpty;
      cnt[s] = 0;
    }
  }
}

// One workgroup per chunk of kCountChunk consecutive tokens.  Cells are
// addressed by d K + k and w K + k, below 2^32 - 1 (each table holds at most
// 2^32 - 1 cells), so never equal to kCountEmpty.
__global__ __launch_bounds__(kCountThreads) void count_kernel(
    const int32_t *__restrict__ doc_id, const int32_t *__restrict__ word_id,
    const int32_t *__restrict__ z, int64_t N, int32_t M, int32_t V, int32_t K,
    int32_t *__restrict__ ndk, int32_t *__restrict__ nwk) {
  __shared__ uint32_t keys[kCountSlots];
  __shared__ uint32_t cnt[kCountSlots];
  for (int s = threadIdx.x; s < kCountSlots; s += kCountThreads) {
    keys[s] = kCountEmpty;
    cnt[s] = 0;
  }
  // this thread's tokens (consecutive threads, consecutive tokens), loaded
  // before any is used; kCountEmpty marks a token not counted
  const int64_t c0 = (int64_t)blockIdx.x * kCountChunk + threadIdx.x;
  uint32_t dk[kCountPer], wk[kCountPer];
#pragma unroll
  for (int i = 0; i < kCountPer; ++i) {
    const int64_t n = c0 + (int64_t)i * kCountThreads;
    int32_t d = -1, w = -1, k = -1;
    if (n < N) {
      d = doc_id[n];
      w = word_id[n];
      k = z[n];
    }
    const bool ok = (uint32_t)d < (uint32_t)M && (uint32_t)w < (uint32_t)V &&
                    (uint32_t)k < (uint32_t)K;
    dk[i] = ok ? (uint32_t)d * (uint32_t)K + (uint32_t)k : kCountEmpty;
    wk[i] = ok ? (uint32_t)w * (uint32_t)K + (uint32_t)k : kCountEmpty;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kCountPer; ++i)
    if (dk[i] != kCountEmpty) count_insert(keys, cnt, dk[i]);
  __syncthreads();
  count_flush(keys, cnt, ndk);
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kCountPer; ++i)
    if (wk[i] != kCountEmpty) count_insert(keys, cnt, wk[i]);
  __syncthreads();
  count_flush(keys, cnt, nwk);
}

// The word table alone (count_kernel's second half), for the offsets form.
__global__ __launch_bounds__(kCountThreads) void count_words_kernel(
    const int32_t *__restrict__ word_id, const int32_t *__restrict__ z, int64_t N, int32_t V,
    int32_t K, int32_t *__restrict__ nwk) {
  __shared__ uint32_t keys[kCountSlots];
  __shared__ uint32_t cnt[kCountSlots];
  for (int s = threadIdx.x; s < kCountSlots; s += kCountThreads) {
    keys[s] = kCountEmpty;
    cnt[s] = 0;
  }
  const int64_t c0 = (int64_t)blockIdx.x * kCountChunk + threadIdx.x;
  uint32_t wk[kCountPer];
#pragma unroll
  for (int i = 0; i < kCountPer; ++i) {
    const int64_t n = c0 + (int64_t)i * kCountThreads;
    int32_t w = -1, k = -1;
    if (n < N) {
      w = word_id[n];
      k = z[n];
    }
    const bool ok = (uint32_t)w < (uint32_t)V && (uint32_t)k < (uint32_t)K;
    wk[i] = ok ? (uint32_t)w * (uint32_t)K + (uint32_t)k : kCountEmpty;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kCountPer; ++i)
    if (wk[i] != kCountEmpty) count_insert(keys, cnt, wk[i]);
  __syncthreads();
  count_flush(keys, cnt, nwk);
}

// The document table from documents given as offsets (document m = tokens
// doc_offsets[m] .. doc_offsets[m+1] - 1, contiguous): one wavefront per
// document counts its tokens' topics in an LDS row of K bins and writes the
// whole row, at a 64-bit address (ndk may hold any number of cells), so that
// the table needs neither clearing nor atomics in memory.  A token is counted
// when its word and topic are in range (as in count_kernel).  Offsets outside
// [0, N] are clamped, never dereferenced.  Workgroup b takes documents
// b kDocWaves .. b kDocWaves + kDocWaves - 1, then the same again every
// gridDim.x kDocWaves documents: the grid is capped at kDocGridMax
// workgroups, since one dispatch holds fewer than 2^32 work-items.
constexpr int kDocWaves = 4;             // documents (wavefronts) per workgroup
constexpr int64_t kDocGridMax = 1 << 20;  // workgroups per launch (2^28 work-items)
__global__ __launch_bounds__(kDocWaves * 64) void count_docs_kernel(
    const int64_t *__restrict__ doc_offsets, const int32_t *__restrict__ word_id,
    const int32_t *__restrict__ z, int64_t N, int32_t M, int32_t V, int32_t K,
    int32_t *__restrict__ ndk) {
  extern __shared__ __align__(16) uint32_t rows[];  // kDocWaves rows of K bins
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  uint32_t *bins = rows + (size_t)wave * (size_t)K;
  // (K divisible by 4: the row's bins are 16-byte aligned in LDS)
  const bool quads = (K & 3) == 0;
  // (m0 is the same for the whole workgroup: every barrier is reached by all)
  for (int64_t m0 = (int64_t)blockIdx.x * kDocWaves; m0 < M;
       m0 += (int64_t)gridDim.x * kDocWaves) {
    const int64_t m = m0 + wave;
    if (quads)
      for (int k = 4 * lane; k < K; k += 4 * 64)
        *reinterpret_cast<uint4 *>(bins + k) = uint4{0u, 0u, 0u, 0u};
    else
      for (int k = lane; k < K; k += 64) bins[k] = 0;
    __syncthreads();
    if (m < M) {
      int64_t lo = doc_offsets[m], hi = doc_offsets[m + 1];
      lo = lo < 0 ? 0 : (lo > N ? N : lo);
      hi = hi < lo ? lo : (hi > N ? N : hi);
      for (int64_t n = lo + lane; n < hi; n += 64) {
        const int32_t w = word_id[n], k = z[n];
        if ((uint32_t)w < (uint32_t)V && (uint32_t)k < (uint32_t)K) atomicAdd(&bins[k], 1u);
      }
    }
    __syncthreads();
    if (m < M) {
      int32_t *row = ndk + m * (int64_t)K;
      if (quads && (reinterpret_cast<uintptr_t>(row) & 15u) == 0) {
        for (int k = 4 * lane; k < K; k += 4 * 64) {
          const uint4 v = *reinterpret_cast<const uint4 *>(bins + k);
          *reinterpret_cast<int4 *>(row + k) =
              int4{(int32_t)v.x, (int32_t)v.y, (int32_t)v.z, (int32_t)v.w};
        }
      } else {
        for (int k = lane; k < K; k += 64) row[k] = (int32_t)bins[k];
      }
    }
    __syncthreads();  // (the row is read out before the next documents clear it)
  }
}

}  // namespace
}  // namespace LDA_NS
