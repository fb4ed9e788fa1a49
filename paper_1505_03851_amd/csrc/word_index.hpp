// The tokens grouped by word (gfx950), and the word-topic counts taken in
// that order.
//
// The word table nwk of the topic counts (counts.hpp) is scattered over V K
// cells; counted in token order, each chunk of tokens touches cells all over
// it, and every distinct cell costs one device-wide atomic, executed on the
// memory side.  A word index, built once per corpus (the word ids do not
// change from sweep to sweep), lists the tokens word by word:
//
//   off[w] .. off[w+1] - 1   the positions of word w's tokens   int32 [V + 1]
//   perm[p]                  the token at position p              int32 [N]
//   wsorted[p]               its word                             int32 [N]
//
// (a counting sort: a histogram of the words, an exclusive scan, then the
// tokens summed in a workgroup's LDS table reserve a run of positions per
// distinct word with one atomic and are placed there; the order of a word's
// tokens is not fixed).
// Tokens whose word id lies outside [0, V) are left out.  The counts then
// take the positions in runs of chunks: a cell's tokens are aggregated in LDS
// as in count_kernel, and at each flush of the table a cell of a word whose
// tokens all lie in the positions taken since the last flush is written with
// a plain store (no other workgroup touches it); only words that straddle
// flushes (the frequent ones, and at most two per flush at its ends) add
// with atomics.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "config.hpp"
#include "counts.hpp"

namespace LDA_NS {
namespace {

constexpr int kScanThreads = 256;
constexpr int kScanPer = 16;                             // items per thread
constexpr int kScanItems = kScanThreads * kScanPer;      // items per workgroup
constexpr int kScanMaxBlocks = kScanItems;               // one workgroup scans the sums

// Fill n ints with v (a kernel, so that the build can be captured).
__global__ __launch_bounds__(256) void index_fill(int32_t *p, int64_t n, int32_t v) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = v;
}

// Each workgroup of the build and of the indexed counts takes a run of
// `run` chunks (index_run: up to kIndexRun, while the grid keeps
// kIndexGroups workgroups) and keeps one LDS table across them, flushing it
// (to memory, with one atomic or store per distinct key) only when it holds
// more than kFlushAt keys (so that after the next chunk it is at most 3/4
// full) and at the end of the run: a frequent word's counter or cell then
// takes one atomic per flush rather than per chunk, and atomics on one
// address are executed one after another on the memory side.
constexpr int kIndexRun = 8;
constexpr int64_t kIndexGroups = 2048;
constexpr uint32_t kFlushAt = kCountSlots / 2 - kCountChunk / 2;

// The build's per-word counters (the histogram, then the cursors of the
// scatter) lie kCounterStride ints apart, one to a 64-byte line: atomics on
// one line are executed one after another on the memory side, and the
// frequent words' counters, adjacent when the vocabulary is sorted by
// frequency, would otherwise share lines (measured on MI355X: the build of
// the 16.8M-token corpus takes 0.88 ms with them apart, 3.15 ms packed).
#ifndef LDA_COUNTER_STRIDE
#define LDA_COUNTER_STRIDE 16
#endif
constexpr int kCounterStride = LDA_COUNTER_STRIDE;

// Chunks per workgroup for N tokens.
__host__ __device__ inline int index_run(int64_t N) {
  const int64_t chunks = (N + kCountChunk - 1) / kCountChunk;
  const int64_t r = chunks / kIndexGroups;
  return r < 1 ? 1 : (r > kIndexRun ? kIndexRun : (int)r);
}

// Tokens per word (word ids in [0, V)), aggregated per run in LDS, added to
// counts[w kCounterStride] (zero beforehand) with one atomic per distinct
// word and flush.
__global__ __launch_bounds__(kCountThreads) void index_hist(const int32_t *__restrict__ word_id,
                                                             int64_t N, int32_t V, int run,
                                                             int32_t *__restrict__ counts) {
  __shared__ uint32_t keys[kCountSlots];
  __shared__ uint32_t cnt[kCountSlots];
  __shared__ uint32_t used;  // keys in the table
  for (int s = threadIdx.x; s < kCountSlots; s += kCountThreads) {
    keys[s] = kCountEmpty;
    cnt[s] = 0;
  }
  if (threadIdx.x == 0) used = 0;
  const int64_t run0 = (int64_t)blockIdx.x * run * kCountChunk;
  for (int c = 0; c < run; ++c) {
    const int64_t c0 = run0 + (int64_t)c * kCountChunk;
    if (c0 >= N) break;
    int32_t w[kCountPer];
#pragma unroll
    for (int i = 0; i < kCountPer; ++i) {
      const int64_t n = c0 + threadIdx.x + (int64_t)i * kCountThreads;
      w[i] = n < N ? word_id[n] : -1;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kCountPer; ++i)
      if ((uint32_t)w[i] < (uint32_t)V && count_insert_new(keys, cnt, (uint32_t)w[i]))
        atomicAdd(&used, 1u);
    __syncthreads();
    if (used > kFlushAt || c == run - 1 || c0 + kCountChunk >= N) {
      for (int s = threadIdx.x; s < kCountSlots; s += kCountThreads) {
        const uint32_t key = keys[s];
        if (key != kCountEmpty) {
          atomicAdd(&counts[(size_t)key * kCounterStride], (int32_t)cnt[s]);
          keys[s] = kCountEmpty;
          cnt[s] = 0;
        }
      }
      __syncthreads();
      if (threadIdx.x == 0) used = 0;
    }
  }
}

// Exclusive scan of the kScanThreads values v of a workgroup (one per
// thread); returns this thread's prefix and leaves the total in `total`.
__device__ __forceinline__ int32_t block_exclusive_scan(int32_t v, int32_t &total) {
  __shared__ int32_t part[kScanThreads];
  const int t = threadIdx.x;
  part[t] = v;
  __syncthreads();
  for (int d = 1; d < kScanThreads; d <<= 1) {
    const int32_t add = t >= d ? part[t - d] : 0;
    __syncthreads();
    part[t] += add;
    __syncthreads();
  }
  total = part[kScanThreads - 1];
  const int32_t incl = part[t];
  __syncthreads();
  return incl - v;
}

// Exclusive scan of in[0], in[stride], ... (n_in items) into out[0 .. n),
// per workgroup of kScanItems items (each thread kScanPer consecutive ones);
// the workgroup's total goes to sums[blockIdx.x].  Items at or past n_in
// count as 0 (so that scanning n = V + 1 items of V counts leaves the grand
// total in out[V]).
__global__ __launch_bounds__(kScanThreads) void index_scan_local(const int32_t *__restrict__ in,
                                                                  int64_t n_in, int stride,
                                                                  int64_t n,
                                                                  int32_t *__restrict__ out,
                                                                  int32_t *__restrict__ sums) {
  const int64_t i0 = ((int64_t)blockIdx.x * kScanThreads + threadIdx.x) * kScanPer;
  int32_t v[kScanPer];
  int32_t run = 0;
#pragma unroll
  for (int j = 0; j < kScanPer; ++j) {
    v[j] = i0 + j < n_in ? in[(i0 + j) * stride] : 0;
    run += v[j];
  }
  int32_t total;
  int32_t pre = block_exclusive_scan(run, total);
#pragma unroll
  for (int j = 0; j < kScanPer; ++j) {
    if (i0 + j < n) out[i0 + j] = pre;
    pre += v[j];
  }
  if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

// Exclusive scan, in place, of the nb <= kScanMaxBlocks workgroup sums (one
// workgroup).
__global__ __launch_bounds__(kScanThreads) void index_scan_sums(int32_t *sums, int32_t nb) {
  const int i0 = threadIdx.x * kScanPer;
  int32_t v[kScanPer];
  int32_t run = 0;
#pragma unroll
  for (int j = 0; j < kScanPer; ++j) {
    v[j] = i0 + j < nb ? sums[i0 + j] : 0;
    run += v[j];
  }
  int32_t total;
  int32_t pre = block_exclusive_scan(run, total);
#pragma unroll
  for (int j = 0; j < kScanPer; ++j) {
    if (i0 + j < nb) sums[i0 + j] = pre;
    pre += v[j];
  }
}

// Add each workgroup's scanned sum to its items.
__global__ __launch_bounds__(kScanThreads) void index_scan_add(int32_t *__restrict__ out,
                                                                int64_t n,
                                                                const int32_t *__restrict__ sums) {
  const int64_t i0 = ((int64_t)blockIdx.x * kScanThreads + threadIdx.x) * kScanPer;
  const int32_t add = sums[blockIdx.x];
#pragma unroll
  for (int j = 0; j < kScanPer; ++j)
    if (i0 + j < n) out[i0 + j] += add;
}

// Place the tokens, run by run: the tokens since the last flush are counted
// per word in LDS; at a flush each distinct word reserves a run of positions
// with one atomic on cursor[w kCounterStride] (zero beforehand), then those
// tokens are read
// again and each writes perm and wsorted at off[w] + run start + its rank
// among the word's tokens there.  The token set is index_hist's (n < N, word
// id in [0, V)), so every word's positions end at off[w + 1]; a position past
// `limit` (offsets that do not belong to these tokens) is not written.
__global__ __launch_bounds__(kCountThreads) void index_scatter(
    const int32_t *__restrict__ word_id, int64_t N, int32_t V, int run,
    const int32_t *__restrict__ off, int32_t *__restrict__ cursor, int32_t *__restrict__ perm,
    int32_t *__restrict__ wsorted, int64_t limit) {
  __shared__ uint32_t keys[kCountSlots];
  __shared__ uint32_t cnt[kCountSlots];
  __shared__ int32_t start[kCountSlots];
  __shared__ uint32_t used;
  for (int s = threadIdx.x; s < kCountSlots; s += kCountThreads) {
    keys[s] = kCountEmpty;
    cnt[s] = 0;
  }
  if (threadIdx.x == 0) used = 0;
  const int64_t run0 = (int64_t)blockIdx.x * run * kCountChunk;
  int64_t from = run0;  // first token since the last flush
  for (int c = 0; c < run; ++c) {
    const int64_t c0 = run0 + (int64_t)c * kCountChunk;
    if (c0 >= N) break;
    int32_t w[kCountPer];
#pragma unroll
    for (int i = 0; i < kCountPer; ++i) {
      const int64_t n = c0 + threadIdx.x + (int64_t)i * kCountThreads;
      w[i] = n < N ? word_id[n] : -1;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kCountPer; ++i)
      if ((uint32_t)w[i] < (uint32_t)V && count_insert_new(keys, cnt, (uint32_t)w[i]))
        atomicAdd(&used, 1u);
    __syncthreads();
    const int64_t to = c0 + kCountChunk < N ? c0 + kCountChunk : N;
    if (used > kFlushAt || c == run - 1 || to >= N) {
      for (int s = threadIdx.x; s < kCountSlots; s += kCountThreads) {
        if (keys[s] != kCountEmpty)
          start[s] = atomicAdd(&cursor[(size_t)keys[s] * kCounterStride], (int32_t)cnt[s]);
        cnt[s] = 0;
      }
      __syncthreads();
      for (int64_t p0 = from; p0 < to; p0 += kCountChunk) {
#pragma unroll
        for (int i = 0; i < kCountPer; ++i) {
          const int64_t n = p0 + threadIdx.x + (int64_t)i * kCountThreads;
          const int32_t wn = n < to ? word_id[n] : -1;
          if ((uint32_t)wn < (uint32_t)V) {
            uint32_t rank;
            const uint32_t slot = count_insert_ranked(keys, cnt, (uint32_t)wn, rank);
            const int64_t p = (int64_t)off[wn] + start[slot] + rank;
            if (p >= 0 && p < limit) {
              perm[p] = (int32_t)n;
              wsorted[p] = wn;
            }
          }
        }
      }
      __syncthreads();
      for (int s = threadIdx.x; s < kCountSlots; s += kCountThreads) {
        keys[s] = kCountEmpty;
        cnt[s] = 0;
      }
      if (threadIdx.x == 0) used = 0;
      from = to;
    }
  }
}

// The word table from the index: one workgroup per run of `run` chunks of
// kCountChunk positions (positions past off[V] hold no token).
// A token counts when its topic is in [0, K); its cell w K + k.  At a flush,
// a cell of a word whose positions all lie in the positions since the last
// flush is stored, the others added atomically, into nwk (zero beforehand).
// Positions past N, perm entries outside [0, N) and words outside [0, V) (an
// index that does not belong to these tokens) are skipped.
__global__ __launch_bounds__(kCountThreads) void count_words_indexed(
    const int32_t *__restrict__ perm, const int32_t *__restrict__ wsorted,
    const int32_t *__restrict__ off, const int32_t *__restrict__ z, int64_t N, int32_t V,
    int32_t K, int run, int32_t *__restrict__ nwk) {
  __shared__ uint32_t keys[kCountSlots];
  __shared__ uint32_t cnt[kCountSlots];
  __shared__ uint32_t used;
  const int64_t run0 = (int64_t)blockIdx.x * run * kCountChunk;
  // (at most N positions, whatever an index of other tokens says)
  const int64_t total = off[V] < N ? off[V] : N;
  if (run0 >= total) return;  // (uniform: the whole workgroup leaves)
  for (int s = threadIdx.x; s < kCountSlots; s += kCountThreads) {
    keys[s] = kCountEmpty;
    cnt[s] = 0;
  }
  if (threadIdx.x == 0) used = 0;
  int64_t from = run0;  // first position since the last flush
  for (int c = 0; c < run; ++c) {
    const int64_t lo = run0 + (int64_t)c * kCountChunk;
    if (lo >= total) break;
    const int64_t hi = lo + kCountChunk < total ? lo + kCountChunk : total;
    uint32_t key[kCountPer];
#pragma unroll
    for (int i = 0; i < kCountPer; ++i) {
      const int64_t p = lo + threadIdx.x + (int64_t)i * kCountThreads;
      int32_t n = -1, w = -1, k = -1;
      if (p < hi) {
        n = perm[p];
        w = wsorted[p];
      }
      if ((uint64_t)(int64_t)n < (uint64_t)N) k = z[n];
      const bool ok = (uint32_t)w < (uint32_t)V && (uint32_t)k < (uint32_t)K;
      key[i] = ok ? (uint32_t)w * (uint32_t)K + (uint32_t)k : kCountEmpty;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kCountPer; ++i)
      if (key[i] != kCountEmpty && count_insert_new(keys, cnt, key[i])) atomicAdd(&used, 1u);
    __syncthreads();
    if (used > kFlushAt || c == run - 1 || hi >= total) {
      for (int s = threadIdx.x; s < kCountSlots; s += kCountThreads) {
        const uint32_t kk = keys[s];
        if (kk != kCountEmpty) {
          const uint32_t w = kk / (uint32_t)K;
          const bool whole = off[w] >= from && off[w + 1] <= hi;
          if (whole)
            nwk[kk] = (int32_t)cnt[s];
          else
            atomicAdd(&nwk[kk], (int32_t)cnt[s]);
          keys[s] = kCountEmpty;
          cnt[s] = 0;
        }
      }
      __syncthreads();
      if (threadIdx.x == 0) used = 0;
      from = hi;
    }
  }
}

}  // namespace
}  // namespace LDA_NS
