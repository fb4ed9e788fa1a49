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

#include "config.hpp"

namespace LDA_NS {

constexpr int kWave = 64;

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

__device__ __forceinline__ int as_int(float x) { return __builtin_bit_cast(int, x); }
__device__ __forceinline__ float as_float(int x) { return __builtin_bit_cast(float, x); }

// ---------------------------------------------------------------------------
// Cross-lane primitives.

// Value of `x` held by lane (lane xor BIT), BIT a power of two below 64:
// the paper's shuffleXor with a constant mask.  xor 1 and 2 are DPP quad
// permutations, xor 4..16 ds_swizzle in bit-mask mode (within 32 lanes),
// xor 32 a ds_bpermute.
template <int BIT>
__device__ __forceinline__ float xor_lane(float x) {
  static_assert(BIT > 0 && BIT < kWave && (BIT & (BIT - 1)) == 0, "bad BIT");
  int v = as_int(x);
  if constexpr (BIT == 1) {
    v = __builtin_amdgcn_mov_dpp(v, 0xB1, 0xF, 0xF, false);  // [1,0,3,2]
  } else if constexpr (BIT == 2) {
    v = __builtin_amdgcn_mov_dpp(v, 0x4E, 0xF, 0xF, false);  // [2,3,0,1]
  } else if constexpr (BIT <= 16) {
    v = __builtin_amdgcn_ds_swizzle(v, 0x1F | (BIT << 10));
  } else {
    v = __builtin_amdgcn_ds_bpermute((lane_id() ^ BIT) << 2, v);
  }
  return as_float(v);
}

// The paper's shuffleXor with a per-lane mask: value of `x` in lane
// (lane xor m), m < 64.
__device__ __forceinline__ float xor_lane_var(float x, int m) {
  return as_float(__builtin_amdgcn_ds_bpermute((lane_id() ^ m) << 2, as_int(x)));
}

// Half exchange between lanes l and l xor BIT of two registers x, y: lanes
// with BIT clear keep x and receive the partner's x in y; lanes with BIT set
// keep y and receive the partner's y in x.  Afterwards x + y is, in every
// lane, the pair sum of one token (the lane's "kept" register).
//   BIT 32, 16: one v_permlane32_swap / v_permlane16_swap (gfx950);
//   BIT 8, 4:   two DPP row shifts whose bank masks pick the receiving lanes.
template <int BIT>
__device__ __forceinline__ void half_swap(float &x, float &y) {
  if constexpr (BIT == 32) {
    auto s = __builtin_amdgcn_permlane32_swap(as_int(x), as_int(y), false, false);
    x = as_float(s[0]);
    y = as_float(s[1]);
  } else if constexpr (BIT == 16) {
    auto s = __builtin_amdgcn_permlane16_swap(as_int(x), as_int(y), false, false);
    x = as_float(s[0]);
    y = as_float(s[1]);
  } else {
    static_assert(BIT == 8 || BIT == 4, "half_swap: BIT in {4, 8, 16, 32}");
    // row_shr:BIT (lane i reads i - BIT) into the lanes with BIT set,
    // row_shl:BIT (lane i reads i + BIT) into the lanes with BIT clear.
    constexpr int hi_banks = BIT == 8 ? 0xC : 0xA;
    constexpr int lo_banks = BIT == 8 ? 0x3 : 0x5;
    const int xi = as_int(x), yi = as_int(y);
    const int xn = __builtin_amdgcn_update_dpp(xi, yi, 0x110 + BIT, 0xF, hi_banks, false);
    const int yn = __builtin_amdgcn_update_dpp(yi, xi, 0x100 + BIT, 0xF, lo_banks, false);
    x = as_float(xn);
    y = as_float(yn);
  }
}

// Pair sum for BIT 1, 2 (within a DPP bank): lanes with BIT clear return
// x + partner's x, lanes with BIT set return y + partner's y.
template <int BIT>
__device__ __forceinline__ float pair_sum(float x, float y) {
  const bool hi = (lane_id() & BIT) != 0;
  const float send = hi ? x : y;
  const float keep = hi ? y : x;
  return keep + xor_lane<BIT>(send);
}

// ---------------------------------------------------------------------------
// Block totals for the sweep: a reduce-scatter of the W x W tile.  Stage BIT
// pairs registers k and k + BIT (k < BIT) across lanes l and l xor L, L the
// stage's lane bit; after the stages for BIT = W/2 .. 1 lane l holds the sum
// of its own token over the block's W topics in a[0].  The tile registers are
// consumed from the top, so the caller can refill a[BIT..2*BIT-1] as soon as
// stage BIT has finished.
//
// Lane bits: with HALF = false, L = BIT (lane bits W/2 .. 1).  With HALF
// (W = 64), L = 16, 8, 4, 2, 1 and then 32: the lanes first sum over aligned
// groups of topics inside each half of the block, so that just before the last
// stage every lane holds its token's sum over each half.  Register k then
// holds token reg_token(k), the register index with its bits moved to the
// matching lane bits.
template <int W, int BIT, bool HALF>
__host__ __device__ constexpr int stage_lane_bit() {
  return HALF ? (BIT == 1 ? W / 2 : BIT / 2) : BIT;
}

template <int W, bool HALF>
__host__ __device__ constexpr int reg_token(int k) {
  return HALF ? ((k >> 1) | ((k & 1) ? W / 2 : 0)) : k;
}

template <int W, int BIT, bool HALF = false>
__device__ __forceinline__ void reduce_stage(float (&a)[W]) {
  constexpr int L = stage_lane_bit<W, BIT, HALF>();
  if constexpr (L >= 4) {
#pragma unroll
    for (int k = BIT - 1; k >= 0; --k) {
      half_swap<L>(a[k], a[k + BIT]);
      a[k] = a[k] + a[k + BIT];
    }
  } else {
#pragma unroll
    for (int k = 0; k < BIT; ++k) a[k] = pair_sum<L>(a[k], a[k + BIT]);
  }
}

// The last stage of the HALF order (lane bit W/2), which also returns the
// lane's token sum over the lower half of the block: after the exchange a[0]
// holds the lower half's sum and a[1] the upper half's, in every lane.
template <int W>
__device__ __forceinline__ float reduce_last_half(float (&a)[W]) {
  half_swap<W / 2>(a[0], a[1]);
  const float lower = a[0];
  a[0] = a[0] + a[1];
  return lower;
}

// ---------------------------------------------------------------------------
// Algorithm 8's butterfly for one block (the paper's replacement rule, with
// stages in the paper's order bit = 1, 2, ..., W/2).  Set for BIT: rows d and
// d + BIT, d = 2*BIT*i + BIT - 1, lanes r and r xor BIT; [a b; c d] becomes
// [a d; a+b c+d]: the lane with BIT set keeps its row-(d+BIT) value in row d,
// and row d + BIT receives the kept value plus what the partner sends.
// Afterwards a[0..W-2] hold lane r's column of the butterfly-patterned block
// (row d in a[d]) and a[W-1] holds the sum of lane r's own token.
//
// ALT applies the other rule the paper mentions, [a b; c d] -> [a c; a+b c+d]:
// the lane with BIT set takes its partner's row-(d+BIT) value into row d, one
// more select after the exchange.  Its row d (s trailing ones) then holds, in
// column r, the sum of token (d & ~(2^(s+1)-1)) + (r & (2^(s+1)-1)) over the
// left half of the aligned 2^(s+1) topics that contain topic r.
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

template <int W, int BIT, bool ALT, class Store>
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
      const float row_d = ALT ? (hi ? recv : a[d]) : keep;
      a[d] = row_d;
      a[d + BIT] = keep + recv;
      store(d, row_d);
    }
    butterfly_stages<W, BIT * 2, ALT, Store>(a, r, store);
  }
}

template <int W, bool ALT = false, class Store>
__device__ __forceinline__ void butterfly_block(float (&a)[W], int r,
                                                const Store &store) {
  butterfly_stages<W, 1, ALT, Store>(a, r, store);
}

// ---------------------------------------------------------------------------
// Memory access through buffer resources: a per-wave base and size in SGPRs,
// a per-lane byte offset (VGPR) and a per-token byte offset (SGPR).
using rsrc_t = __amdgpu_buffer_rsrc_t;

__device__ __forceinline__ rsrc_t make_rsrc(const void *base, uint32_t bytes) {
  // dword3: 32-bit raw data (same value the CDNA3/CDNA4 libraries use)
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, bytes,
                                           0x00020000);
}

// (the builtin returns the 32 loaded bits as an unsigned integer)
__device__ __forceinline__ float load_f32(rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0));
}

// Four consecutive floats per lane (one 16-byte buffer load): a leaf of
// kLeaf topics.
using f4 = float __attribute__((ext_vector_type(4)));
using f2 = float __attribute__((ext_vector_type(2)));
constexpr int kLeaf = 4;

__device__ __forceinline__ f4 load_f32x4(rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_bit_cast(f4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}

// ---------------------------------------------------------------------------
// A table (theta [M][K] or phi [V][K]) as the draw kernels address it: a
// 32-bit row handle (`row(id)`) plus a lane offset in bytes (the topics
// within the row).  The kernels only pass handles on (also across lanes).
//  * LDA_WIDE_TABLES 0, tables below 4 GiB: a buffer resource over the table;
//    the handle is the row's byte offset, and the resource's range check
//    returns 0 for a read past the table, so an id out of range reads zeros
//    and cannot fault.
//  * LDA_WIDE_TABLES 1, any size (fewer than 2^31 rows): the table's base
//    pointer; the handle is the row index, and each load forms the 64-bit
//    address base + row K + the lane offset.  row() clamps the id to the
//    table's last row, so that here too every read stays inside the table.
// `extent` is the table's size in the handles' unit (bytes, or rows).
// ld / ld4 take a handle that is uniform across the wavefront (a scalar
// operand), ldv / ld4v one that differs between lanes.
__host__ __device__ constexpr uint32_t table_extent(int64_t rows, int32_t K) {
  return LDA_WIDE_TABLES ? (uint32_t)rows : (uint32_t)(rows * (int64_t)K * 4);
}

#if LDA_WIDE_TABLES
// 16-byte loads at 4-byte alignment (a table's base need only be 4-byte aligned)
using f4u = float __attribute__((ext_vector_type(4), aligned(4)));

struct Table {
  const float *base;
  uint32_t step;   // floats per row (K)
  uint32_t last;   // the last row
  __device__ __forceinline__ uint32_t row(uint32_t id) const { return id < last ? id : last; }
  __device__ __forceinline__ const char *at(uint32_t voff, uint32_t row) const {
    return reinterpret_cast<const char *>(base + (uint64_t)row * step) + voff;
  }
  __device__ __forceinline__ float ld(uint32_t voff, uint32_t row) const {
    return *reinterpret_cast<const float *>(at(voff, row));
  }
  __device__ __forceinline__ float ldv(uint32_t voff, uint32_t row) const { return ld(voff, row); }
  __device__ __forceinline__ f4 ld4(uint32_t voff, uint32_t row) const {
    return *reinterpret_cast<const f4u *>(at(voff, row));
  }
  __device__ __forceinline__ f4 ld4v(uint32_t voff, uint32_t row) const { return ld4(voff, row); }
};

__device__ __forceinline__ Table make_table(const float *base, uint32_t extent, int K) {
  return Table{base, (uint32_t)K, extent - 1u};
}
#else
struct Table {
  rsrc_t rs;
  uint32_t step;   // bytes per row (4 K)
  __device__ __forceinline__ uint32_t row(uint32_t id) const { return id * step; }
  __device__ __forceinline__ float ld(uint32_t voff, uint32_t row) const {
    return load_f32(rs, voff, row);
  }
  __device__ __forceinline__ float ldv(uint32_t voff, uint32_t row) const {
    return load_f32(rs, voff + row, 0);
  }
  __device__ __forceinline__ f4 ld4(uint32_t voff, uint32_t row) const {
    return load_f32x4(rs, voff, row);
  }
  __device__ __forceinline__ f4 ld4v(uint32_t voff, uint32_t row) const {
    return load_f32x4(rs, voff + row, 0);
  }
};

__device__ __forceinline__ Table make_table(const float *base, uint32_t extent, int K) {
  return Table{make_rsrc(base, extent), (uint32_t)K * 4u};
}
#endif

// Sum of the four theta-phi products of a leaf of four topics, in topic order
// (the products of topics 1..3 are fused multiply-adds onto the running sum).
__device__ __forceinline__ float dot4(f4 t, f4 x) {
  return __builtin_fmaf(t.w, x.w, __builtin_fmaf(t.z, x.z, __builtin_fmaf(t.y, x.y, t.x * x.x)));
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

// How a wavefront's tokens map to documents, for the theta factor of the
// tile: one document (one theta value per lane per block), two documents in
// two contiguous runs (two values and a per-token choice), any mix (one
// theta load per token), or (leaf kernel on routed tokens) a few runs of
// documents whose theta leaves are staged in LDS once per block.
enum ThetaMode : int { kOneDoc = 0, kTwoDocs = 1, kAnyDocs = 2, kFewDocs = 3 };

// One step of an untransposed running sum (the naive kernel, the remnant of
// the table dump): sum + theta * phi.
__device__ __forceinline__ float prefix_step(float sum, float th, float ph) {
  return __builtin_fmaf(th, ph, sum);
}


}  // namespace LDA_NS
