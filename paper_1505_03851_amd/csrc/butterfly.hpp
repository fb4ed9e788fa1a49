// Device building blocks of the butterfly draw for gfx950 (wave64).
//
// Notation follows Sections 3 and 4 of the paper: W lanes form a group, lane r
// of the group owns one token, topics are split into a leading remnant of
// K mod W topics and K / W blocks of W topics.  In a block, register a[k] of
// lane r holds the product of token k of the group at topic (block base + r):
// the transposed tile that cooperative, coalesced loads produce.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lda {

constexpr int kWave = 64;

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

// Value of `x` held by lane (lane xor BIT), BIT a power of two below 64.
// xor 1 and 2 are DPP quad permutations, xor 4..16 ds_swizzle in bit-mask
// mode (within 32 lanes), xor 32 a ds_bpermute.
template <int BIT>
__device__ __forceinline__ float xor_lane(float x) {
  static_assert(BIT > 0 && BIT < kWave && (BIT & (BIT - 1)) == 0, "bad BIT");
  int v = __builtin_bit_cast(int, x);
  if constexpr (BIT == 1) {
    v = __builtin_amdgcn_mov_dpp(v, 0xB1, 0xF, 0xF, false);  // [1,0,3,2]
  } else if constexpr (BIT == 2) {
    v = __builtin_amdgcn_mov_dpp(v, 0x4E, 0xF, 0xF, false);  // [2,3,0,1]
  } else if constexpr (BIT <= 16) {
    v = __builtin_amdgcn_ds_swizzle(v, 0x1F | (BIT << 10));
  } else {
    v = __builtin_amdgcn_ds_bpermute((lane_id() ^ BIT) << 2, v);
  }
  return __builtin_bit_cast(float, v);
}

// Store policies for the table rows a stage finishes.
struct NoStore {
  __device__ __forceinline__ void operator()(int, float) const {}
};

// Row d of the block goes to base[d * stride] (LDS or global).
struct RowStore {
  float *base;
  int stride;
  bool enabled;
  __device__ __forceinline__ void operator()(int d, float v) const {
    if (enabled) base[d * stride] = v;
  }
};

// One set of replacements (Section 4): rows d and d + BIT, d = 2*BIT*i + BIT-1,
// lanes r and r xor BIT.  [a b; c d] -> [a d; a+b c+d]: the lane with BIT set
// keeps its row-(d+BIT) value in row d, and row d + BIT receives the sum of
// the kept value and the value the partner lane sends.
template <int W, int BIT, class Store>
__device__ __forceinline__ void butterfly_stages(float (&a)[W], int r,
                                                 const Store &store) {
  if constexpr (BIT < W) {
    const bool hi = (r & BIT) != 0;
#pragma unroll
    for (int i = 0; i < W / (2 * BIT); ++i) {
      const int d = 2 * BIT * i + (BIT - 1);
      const float send = hi ? a[d] : a[d + BIT];
      const float recv = xor_lane<BIT>(send);
      const float keep = hi ? a[d + BIT] : a[d];
      a[d] = keep;
      a[d + BIT] = keep + recv;
      store(d, keep);
    }
    butterfly_stages<W, BIT * 2, Store>(a, r, store);
  }
}

// Algorithm 8's butterfly for one block: afterwards a[0..W-2] hold lane r's
// column of the butterfly-patterned block (row d in a[d]) and a[W-1] holds
// the sum of lane r's own token over the block.
template <int W, class Store>
__device__ __forceinline__ void butterfly_block(float (&a)[W], int r,
                                                const Store &store) {
  butterfly_stages<W, 1, Store>(a, r, store);
}

// Value of `v` in lane (group base + k): uniform across the wave when W = 64.
template <int W>
__device__ __forceinline__ int group_value(int v, int k) {
  if constexpr (W == kWave) {
    return __builtin_amdgcn_readlane(v, k);
  } else {
    static_assert(W == 32, "W is 32 or 64");
    const int lo = __builtin_amdgcn_readlane(v, k);
    const int hi = __builtin_amdgcn_readlane(v, 32 + k);
    return lane_id() < 32 ? lo : hi;
  }
}

// Transposed tile of one block per token (Algorithm 8's product loop, with
// Algorithm 5's transposed theta access): a[k] = theta[doc_k][c_k] *
// phi[word_k][c_k] with c_k = R + blk_k * W + r, where doc_k, word_k, blk_k
// are the document, word and block of token k of the group.  Each k is one
// coalesced load of W consecutive floats per group.  With `one_doc` (every
// token of the wave in document doc0) and `one_blk` (every token on the same
// block) theta is one load per lane instead of W.
template <int W>
__device__ __forceinline__ void load_tile(float (&a)[W],
                                          const float *__restrict__ theta,
                                          const float *__restrict__ phi, int K,
                                          int R, int doc, int word, int blk,
                                          int r, bool one_doc, bool one_blk) {
  if (one_doc && one_blk) {
    const int doc0 = __builtin_amdgcn_readfirstlane(doc);
    const int blk0 = __builtin_amdgcn_readfirstlane(blk);
    const int col = R + blk0 * W + r;
    const float th = theta[(int64_t)doc0 * K + col];
#pragma unroll
    for (int k = 0; k < W; ++k) {
      const int wk = group_value<W>(word, k);
      a[k] = th * phi[(int64_t)wk * K + col];
    }
  } else {
#pragma unroll
    for (int k = 0; k < W; ++k) {
      const int wk = group_value<W>(word, k);
      const int dk = group_value<W>(doc, k);
      const int col = R + group_value<W>(blk, k) * W + r;
      a[k] = theta[(int64_t)dk * K + col] * phi[(int64_t)wk * K + col];
    }
  }
}

// One step of the untransposed running sum of the remnant (and of the naive
// kernel): sum + theta * phi.  Written once so that every recomputation of a
// remnant prefix rounds identically.
__device__ __forceinline__ float prefix_step(float sum, float th, float ph) {
  return __builtin_fmaf(th, ph, sum);
}

// Linear search of the remnant (Algorithm 9's fallback, Algorithm 2's loop):
// recompute the prefix of topics 0..R-1 and return the first j with
// stop < prefix_j, or `none` if there is no such j.
__device__ __forceinline__ int remnant_search(const float *__restrict__ th_row,
                                              const float *__restrict__ ph_row,
                                              int R, float stop, int none) {
  float s = 0.0f;
  for (int j = 0; j < R; ++j) {
    s = prefix_step(s, th_row[j], ph_row[j]);
    if (stop < s) return j;
  }
  return none;
}

}  // namespace lda
