// Routing of tokens to the XCDs of the GPU by word (gfx950).
//
// The GPU dispatches workgroups to its eight XCDs round robin (workgroup b on
// XCD b mod 8), and each XCD has its own L2.  In token order every XCD reads
// rows of phi from the whole vocabulary.  Routing splits the words into 256
// classes by a hash, assigns the classes to the XCDs so that every XCD gets
// about the same number of tokens, and lays the tokens out as eight lists,
// list x holding (in their original order) the tokens whose word class went to
// XCD x.  A draw whose workgroup b takes its tokens from list b mod 8 then
// keeps one eighth of the vocabulary in each L2.
//
// The routing depends on the word and document ids only, so a sampler builds
// it once and reuses it for every sweep over the corpus.
//
// Routed position i holds token perm[i] (-1: padding) with word rword[i] and
// document rdoc[i].  List x starts at start[x] and is padded to a multiple
// of 64 positions (a padding position repeats the list's last token and is
// drawn but not stored).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "config.hpp"

#include <algorithm>

namespace LDA_NS {

constexpr int kRouteXcds = 8;           // lists (XCDs of the MI355X)
constexpr int kRouteClasses = 256;      // word classes
constexpr int kRouteThreads = 256;      // threads of the builder's workgroups
constexpr int kRouteChunk = 4096;       // tokens per chunk of the count/scatter
constexpr int kRoutePer = kRouteChunk / kRouteThreads;  // tokens per thread and chunk
constexpr int kRoutePad = 64;           // lists are padded to whole wavefronts

// Word class: bits 16..23 of the word id times 2654435761 (Knuth's
// multiplicative hash), modulo 2^32.
__host__ __device__ __forceinline__ int route_class(int32_t word) {
  return (int)(((uint32_t)word * 2654435761u) >> 16) & (kRouteClasses - 1);
}

// Device part of the routing plan, inside the caller's workspace.
struct RoutePlan {
  int32_t *perm, *rword, *rdoc;  // [Np] each
  int32_t *chunk_off;            // [nchunks][8] exclusive offsets in each list
  int32_t *counts;               // [256] tokens per word class
  int32_t *map;                  // [256] XCD of each word class
  int64_t *lists;                // tokens[8], start[8], length[8]
  int32_t *chunk_hist;           // [nchunks][256] tokens per word class in each chunk
};

// Fill n ints with v (used instead of a memset so the builder can be captured).
__global__ void route_fill(int32_t *p, int64_t n, int32_t v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

// Tokens per word class, in each chunk of kRouteChunk tokens and in all:
// each workgroup takes every gridDim.x-th chunk (each thread's loads of a
// chunk issued before any is used) into an LDS histogram, writes it out as
// the chunk's and adds it to its own totals, which it then adds to the counts
// with one atomic per class.  A token counts when its index is below N,
// whatever its word id, exactly as route_scatter places it: the two passes
// must agree on the token set, or a list would receive more tokens than
// its counted length.
__global__ __launch_bounds__(kRouteThreads) void route_hist(const int32_t *__restrict__ word,
                                                            int64_t N, int64_t nchunks,
                                                            int32_t *chunk_hist, int32_t *counts) {
  __shared__ int32_t h[kRouteClasses];
  const int t = threadIdx.x;
  h[t] = 0;
  int32_t total = 0;
  __syncthreads();
  for (int64_t ch = blockIdx.x; ch < nchunks; ch += gridDim.x) {
    const int64_t c0 = ch * kRouteChunk + t;
    int32_t w[kRoutePer];
#pragma unroll
    for (int k = 0; k < kRoutePer; ++k) {
      const int64_t i = c0 + (int64_t)k * kRouteThreads;
      w[k] = i < N ? word[i] : 0;
    }
#pragma unroll
    for (int k = 0; k < kRoutePer; ++k)
      if (c0 + (int64_t)k * kRouteThreads < N) atomicAdd(&h[route_class(w[k])], 1);
    __syncthreads();
    const int32_t v = h[t];
    chunk_hist[ch * kRouteClasses + t] = v;
    total += v;
    h[t] = 0;
    __syncthreads();
  }
  if (total) atomicAdd(&counts[t], total);
}

// The class map and the list layout, computed on the host from the class
// counts (route_assign) and handed to the device as kernel arguments.
struct RouteAssignment {
  int32_t map[kRouteClasses];    // XCD of each word class
  int64_t lists[3 * kRouteXcds];  // tokens[8], start[8], padded length[8]
};

// Rank the classes by token count (largest first, ties by class), then assign
// them in that order, each to the list with the fewest tokens so far (ties:
// the lowest list), and lay the lists out one after another, each padded to
// a multiple of 64 positions.  (A serial pass of 256 steps: a few
// microseconds on the host, where one GPU thread took tens.)
inline RouteAssignment route_assign(const int32_t (&counts)[kRouteClasses]) {
  // one 64-bit key per class, (2^31 - 1 - count, class): ascending keys give
  // the ranking (counts lie in [0, 2^31))
  uint64_t key[kRouteClasses];
  for (int c = 0; c < kRouteClasses; ++c)
    key[c] = ((uint64_t)(uint32_t)(0x7fffffff - counts[c]) << 32) | (uint32_t)c;
  std::sort(key, key + kRouteClasses);
  RouteAssignment a;
  int64_t load[kRouteXcds] = {};
  for (int r = 0; r < kRouteClasses; ++r) {
    const int c = (int)(key[r] & 0xffffffffu);
    int best = 0;
    for (int x = 1; x < kRouteXcds; ++x)
      if (load[x] < load[best]) best = x;
    a.map[c] = best;
    load[best] += counts[c];
  }
  int64_t start = 0;
  for (int x = 0; x < kRouteXcds; ++x) {
    const int64_t len = (load[x] + kRoutePad - 1) / kRoutePad * kRoutePad;
    a.lists[x] = load[x];
    a.lists[kRouteXcds + x] = start;
    a.lists[2 * kRouteXcds + x] = len;
    start += len;
  }
  return a;
}

// The assignment into the workspace (one workgroup of 256 threads).
__global__ __launch_bounds__(kRouteThreads) void route_set(const RouteAssignment a, int32_t *map,
                                                           int64_t *lists) {
  map[threadIdx.x] = a.map[threadIdx.x];
  if (threadIdx.x < 3 * kRouteXcds) lists[threadIdx.x] = a.lists[threadIdx.x];
}

// Tokens of each list in each chunk, from the chunk's class histogram (one
// workgroup per chunk).
__global__ __launch_bounds__(kRouteThreads) void route_count(const int32_t *__restrict__ chunk_hist,
                                                             const int32_t *__restrict__ map,
                                                             int32_t *chunk_count) {
  __shared__ int32_t c[kRouteXcds];
  const int t = threadIdx.x;
  if (t < kRouteXcds) c[t] = 0;
  __syncthreads();
  const int32_t v = chunk_hist[(int64_t)blockIdx.x * kRouteClasses + t];
  if (v) atomicAdd(&c[map[t]], v);
  __syncthreads();
  if (t < kRouteXcds) chunk_count[(int64_t)blockIdx.x * kRouteXcds + t] = c[t];
}

// Exclusive prefix over the chunks, in place: workgroup x scans list x.  Each
// pass loads 256 x kScanPer chunk counts (all loads issued first), then scans
// them: per thread sequentially, across the workgroup through LDS.
constexpr int kScanPer = 16;
__global__ __launch_bounds__(kRouteThreads) void route_scan(int32_t *chunk_off, int64_t nchunks) {
  __shared__ int32_t part[kRouteThreads];
  const int x = blockIdx.x, t = threadIdx.x;
  int64_t carry = 0;
  for (int64_t b = 0; b < nchunks; b += (int64_t)kRouteThreads * kScanPer) {
    int32_t v[kScanPer];
    const int64_t k0 = b + (int64_t)t * kScanPer;  // this thread's kScanPer chunks
#pragma unroll
    for (int j = 0; j < kScanPer; ++j)
      v[j] = k0 + j < nchunks ? chunk_off[(k0 + j) * kRouteXcds + x] : 0;
    int32_t sum = 0;
#pragma unroll
    for (int j = 0; j < kScanPer; ++j) sum += v[j];
    part[t] = sum;
    __syncthreads();
    // inclusive scan of the 256 thread sums (Hillis-Steele in LDS)
    for (int d = 1; d < kRouteThreads; d <<= 1) {
      const int32_t o = t >= d ? part[t - d] : 0;
      __syncthreads();
      part[t] += o;
      __syncthreads();
    }
    int64_t run = carry + part[t] - sum;
#pragma unroll
    for (int j = 0; j < kScanPer; ++j) {
      if (k0 + j < nchunks) chunk_off[(k0 + j) * kRouteXcds + x] = (int32_t)run;
      run += v[j];
    }
    carry += part[kRouteThreads - 1];
    __syncthreads();
  }
}

// Stable scatter: per chunk, tokens are taken in order, 256 at a time; a
// token's position in its list is the list's start, plus the tokens of the
// list in earlier chunks, earlier rounds of this chunk, earlier wavefronts of
// this round and earlier lanes of its wavefront.
__global__ __launch_bounds__(kRouteThreads) void route_scatter(
    const int32_t *__restrict__ word, const int32_t *__restrict__ doc, int64_t N,
    const int32_t *__restrict__ map, const int32_t *__restrict__ chunk_off,
    const int64_t *__restrict__ lists, int32_t *perm, int32_t *rword, int32_t *rdoc) {
  constexpr int kWaves = kRouteThreads / 64;
  __shared__ int32_t wave_count[kWaves][kRouteXcds];
  __shared__ int64_t next[kRouteXcds];
  __shared__ int32_t m[kRouteClasses];
  const int lane = threadIdx.x & 63, wave = threadIdx.x / 64;
  const int64_t c0 = (int64_t)blockIdx.x * kRouteChunk;
  m[threadIdx.x] = map[threadIdx.x];
  if (threadIdx.x < kRouteXcds)
    next[threadIdx.x] = lists[kRouteXcds + threadIdx.x] +
                        chunk_off[(int64_t)blockIdx.x * kRouteXcds + threadIdx.x];
  // this thread's tokens of every round, loaded before any is used
  int32_t ws[kRoutePer], ds[kRoutePer];
#pragma unroll
  for (int k = 0; k < kRoutePer; ++k) {
    const int64_t i = c0 + (int64_t)k * kRouteThreads + threadIdx.x;
    ws[k] = i < N ? word[i] : 0;
    ds[k] = i < N ? doc[i] : 0;
  }
  __syncthreads();
  const uint64_t below = (1ull << lane) - 1ull;
#pragma unroll
  for (int r = 0; r < kRoutePer; ++r) {
    const int64_t i = c0 + (int64_t)r * kRouteThreads + threadIdx.x;
    const bool valid = i < N;
    const int32_t w = ws[r];
    const int x = valid ? m[route_class(w)] : -1;
    int rank = 0;
    for (int y = 0; y < kRouteXcds; ++y) {
      const uint64_t mask = __ballot(x == y);
      if (x == y) rank = __popcll(mask & below);
      if (lane == 0) wave_count[wave][y] = __popcll(mask);
    }
    __syncthreads();
    if (valid) {
      int64_t pos = next[x] + rank;
      for (int v = 0; v < wave; ++v) pos += wave_count[v][x];
      perm[pos] = (int32_t)i;
      rword[pos] = w;
      rdoc[pos] = ds[r];
    }
    __syncthreads();
    if (threadIdx.x < kRouteXcds)
      for (int v = 0; v < kWaves; ++v) next[threadIdx.x] += wave_count[v][threadIdx.x];
    __syncthreads();
  }
}

// Padding positions of every list: no token (-1), the word and document of
// the list's last token.
__global__ void route_pad(const int64_t *__restrict__ lists, int32_t *perm, int32_t *rword,
                          int32_t *rdoc) {
  const int x = blockIdx.x;
  const int64_t tokens = lists[x], start = lists[kRouteXcds + x],
                len = lists[2 * kRouteXcds + x];
  if (tokens == 0) return;  // an empty list has no positions
  const int64_t last = start + tokens - 1;
  for (int64_t p = start + tokens + threadIdx.x; p < start + len; p += blockDim.x) {
    perm[p] = -1;
    rword[p] = rword[last];
    rdoc[p] = rdoc[last];
  }
}

}  // namespace LDA_NS
