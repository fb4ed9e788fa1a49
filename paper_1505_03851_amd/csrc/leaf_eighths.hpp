// Leaf kernel with 32-topic prefix rows (gfx950).
#pragma once

#include "tile.hpp"

namespace LDA_NS {
namespace {

// Leaf kernel with 32-topic prefix rows (K divisible by 4, from
// LDA_EIGHTHS_MIN_K topics to LDA_EIGHTHS_MAX_BLOCKS 256-topic blocks,
// N >= 64; when K is not a multiple of 256 the first block begins with
// 256 - K mod 256 empty topics, as the remnant block of butterfly_kernel).
//
// The sweep reads every token's phi row with 16-byte loads: lane l takes the
// leaf of topics [4l, 4l + 4) of each 256-topic block, so one load
// instruction brings one token's 256 topics, and the lane sums its leaf's
// four products (dot4).  The 64 leaf sums of a token are then combined across
// lanes as single products are in butterfly_kernel, but the reduce-scatter
// first sums over lane bits 2, 1, 0 (the eight lanes of a 32-topic "eighth"
// of the block) and then only exchanges over lane bits 3, 4, 5, so that every
// lane ends with its own token's eight eighth sums rather than their total.
// The running prefixes at the 8 NB eighth ends go to LDS; Algorithm 9's
// search runs over them, and the chosen 32-topic chunk is rebuilt with
// Algorithm 8's butterfly and searched with Algorithm 10, by the W = 32
// machinery of the half-block tail (two tokens per load instruction).  Against
// the one-topic sweep this reads the same bytes with four times fewer load
// instructions (a 64-lane dword load costs the memory pipeline about as many
// cycles as a 16-byte one), and the rebuild reads 128 B of phi per token
// (its theta from LDS where one document's row was staged during the sweep).
//
// Register slot s of the sweep holds token eighth_slot_token(s): with the
// stage order above, lane l ends with slot (l5 l4 l3 l0 l1 l2) (bits listed
// from bit 0 up), so slots are loaded with the inverse permutation and lane l
// finishes with token l.  Afterwards eighth q of the lane's token is in
// register bitrev3(q).
constexpr int kBlock4 = kWave * kLeaf;  // topics per block

__host__ __device__ constexpr int eighth_slot_token(int s) {
  return ((s >> 3) & 1) | (((s >> 4) & 1) << 1) | (((s >> 5) & 1) << 2) |
         (((s >> 2) & 1) << 3) | (((s >> 1) & 1) << 4) | ((s & 1) << 5);
}
__host__ __device__ constexpr int bitrev3(int q) { return ((q & 1) << 2) | (q & 2) | ((q >> 2) & 1); }

// Slots of a sweep block are taken in pair order 0, 32, 1, 33, ...: as soon
// as slots s and s + 32 have their leaf sums, the first reduce-scatter stage
// combines them, so only 32 partial sums stay live.
__device__ __host__ constexpr int pair_token(int i) { return (i >> 1) + ((i & 1) << 5); }

// Sums registers k and k + BIT (k < BIT) across lanes l and l xor L: lanes
// with L clear keep token k's sum, lanes with L set token k + BIT's.
template <int L, int BIT, int N>
__device__ __forceinline__ void pair_stage(float (&a)[N]) {
#pragma unroll
  for (int k = 0; k < BIT; ++k) {
    if constexpr (L >= 4) {
      half_swap<L>(a[k], a[k + BIT]);
      a[k] = a[k] + a[k + BIT];
    } else {
      a[k] = pair_sum<L>(a[k], a[k + BIT]);
    }
  }
}

// First topic of this lane's leaf in block `blk` (negative in the front
// padding of block 0 when K is not a multiple of 256), and the byte offset its
// loads use (padding leaves read topics 0..3; their products are replaced by
// zero where they are used).
__device__ __forceinline__ int leaf_topic(int c0, int blk, int r) {
  return c0 + blk * kBlock4 + kLeaf * r;
}
__device__ __forceinline__ uint32_t leaf_bytes(int c0, int blk, int r) {
  const int t = leaf_topic(c0, blk, r);
  return (uint32_t)(t > 0 ? t : 0) * 4u;
}

// Theta leaf of block `blk` at row offset `row`; zero for a padding leaf.
template <bool PAD>
__device__ __forceinline__ f4 theta_leaf(const Table &tt, int c0, int blk, int r, uint32_t row) {
  const f4 t = tt.ld4(leaf_bytes(c0, blk, r), row);
  if constexpr (PAD) {
    const f4 zero = {0.0f, 0.0f, 0.0f, 0.0f};
    return leaf_topic(c0, blk, r) >= 0 ? t : zero;
  }
  return t;
}

// Theta leaves of a wavefront whose tokens form D <= kFewMax runs of documents
// (kFewDocs): per block, each run's leaf at this lane's topics is loaded once
// and staged in LDS, leaf `lane` of run d and block b at lds[d rstride +
// b bstride + lane]; each token then reads its run's leaf from LDS instead of
// from memory.  With rstride = 64 and bstride = 0 every block's leaves replace
// the last ones; with rstride = 64 NB and bstride = 64 the runs' whole rows
// stay, for the rebuild.
constexpr int kFewMax = 4;
struct FewDocs {
  f4 *lds;                 // this wavefront's staged leaves (one-document
                           // sweeps that stage the theta row: that row)
  int D;                   // runs of documents in the wavefront, uniform
  uint32_t row[kFewMax];   // their theta row offsets, uniform
  int slot;                // this lane's run
  int rstride, bstride;    // staging layout, uniform (in leaves)
};

// Loads of block `blk`'s leaves of the wavefront's runs (to be staged later).
template <bool PAD>
__device__ __forceinline__ void few_load(const FewDocs &fd, const Table &tt, int c0, int blk, int r,
                                         f4 (&st)[kFewMax]) {
#pragma unroll
  for (int d = 0; d < kFewMax; ++d)
    if (d < fd.D) st[d] = theta_leaf<PAD>(tt, c0, blk, r, fd.row[d]);
}

// Stage the loaded leaves in LDS.  The wavefront's earlier LDS reads are
// issued before these writes and LDS executes one wavefront's operations in
// order, so the writes may replace leaves the wavefront has read already.
__device__ __forceinline__ void few_stage(const FewDocs &fd, const f4 (&st)[kFewMax], int lane,
                                          int blk) {
#pragma unroll
  for (int d = 0; d < kFewMax; ++d)
    if (d < fd.D) fd.lds[d * fd.rstride + blk * fd.bstride + lane] = st[d];
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// The staged leaf of token t's run in block blk.
__device__ __forceinline__ f4 few_leaf(const FewDocs &fd, int t, int lane, int blk) {
  return fd.lds[__builtin_amdgcn_readlane(fd.slot, t) * fd.rstride + blk * fd.bstride + lane];
}

// Sweep step for one 256-topic block: win[] holds (or awaits) the phi leaves
// of the first C slots in pair order, twin[] their theta leaves (any
// documents; with a few documents, those of the first CT slots, read from
// LDS), th[] the theta leaves of the first / last document.  With PREFETCH
// the windows and thn[] are refilled with block `next` as the block drains.
// rows[q * 64] receives the running prefix at the end of eighth q; returns the
// prefix at the block's end.  c0 is the first topic of block 0 (PAD: K is not
// a multiple of 256 and block 0 begins with 256 - K mod 256 empty topics).
// With TS (one document) the block's theta leaves also go to LDS, leaf l at
// fd.lds[blk * 64 + l]: the whole row, in topic order from c0, for the rebuild.
template <int MODE, bool PREFETCH, int C, int CT, bool PAD, bool TS = false>
__device__ __forceinline__ float sweep8_block(const Wave<kWave, false> &w, const FewDocs &fd,
                                              f4 (&win)[C], f4 (&twin)[CT], f4 (&th)[2],
                                              f4 (&thn)[2], int c0, int blk, int next,
                                              float *rows, float prefix) {
  static_assert(kWave % C == 0, "the window size must divide 64");
  const uint32_t vcur = leaf_bytes(c0, blk, w.r);
  const uint32_t vnext = leaf_bytes(c0, next, w.r);
  // any documents: theta comes per token, so padding leaves are zeroed per product
  const bool real = !PAD || leaf_topic(c0, blk, w.r) >= 0;
  const int kb = MODE == kTwoDocs ? launder_int(w.kb) : kWave;
  const int lane = lane_id();
  // kFewDocs: the next block's run leaves, loaded now and staged in LDS once
  // this block's last reads of the staged leaves have been issued (CT slots
  // before the block's end)
  f4 st[kFewMax];
  if constexpr (MODE == kFewDocs && PREFETCH) few_load<PAD>(fd, w.th, c0, next, w.r, st);
  if constexpr (TS && MODE == kOneDoc) fd.lds[blk * kWave + lane] = th[0];
  float s[kWave / 2];
  float lo = 0.0f;
#pragma unroll
  for (int i = 0; i < kWave; ++i) {
    const int slot = pair_token(i);
    const int t = eighth_slot_token(slot);
    f4 tv;
    if constexpr (MODE == kAnyDocs)
      tv = twin[i % C];
    else if constexpr (MODE == kFewDocs)
      tv = twin[i % CT];
    else if constexpr (MODE == kTwoDocs)
      tv = t < kb ? th[0] : th[1];
    else
      tv = th[0];
    float v = dot4(tv, win[i % C]);
    if constexpr (PAD && MODE == kAnyDocs) v = real ? v : 0.0f;
    if (i & 1) {
      float hi = v;
      half_swap<4>(lo, hi);
      s[slot - 32] = lo + hi;
    } else {
      lo = v;
    }
    const bool refill = i + C < kWave;
    if (refill || PREFETCH) {
      const int tn = eighth_slot_token(pair_token(refill ? i + C : i + C - kWave));
      const uint32_t voff = refill ? vcur : vnext;
      if (!refill && (MODE == kOneDoc || MODE == kTwoDocs) && i + C == kWave) {
        thn[0] = theta_leaf<PAD>(w.th, c0, next, w.r, w.th_off0);
        if constexpr (MODE == kTwoDocs) thn[1] = theta_leaf<PAD>(w.th, c0, next, w.r, w.th_off1);
      }
      win[i % C] = w.ph.ld4(voff, __builtin_amdgcn_readlane(w.ph_lane, tn));
      if constexpr (MODE == kAnyDocs)
        twin[i % C] = w.th.ld4(voff, __builtin_amdgcn_readlane(w.th_lane, tn));
    }
    if constexpr (MODE == kFewDocs) {
      const bool trefill = i + CT < kWave;
      if (trefill || PREFETCH) {
        if (!trefill && i + CT == kWave) few_stage(fd, st, lane, next);
        const int tt = eighth_slot_token(pair_token(trefill ? i + CT : i + CT - kWave));
        twin[i % CT] = few_leaf(fd, tt, lane, trefill ? blk : next);
      }
    }
    // keep the window rolling: no load is hoisted past this point (hoisting
    // them all would need 4 registers per token of the block)
    __builtin_amdgcn_sched_barrier(0);
  }
  pair_stage<2, 16>(s);
  pair_stage<1, 8>(s);
#pragma unroll
  for (int j = 0; j < 4; ++j) half_swap<8>(s[j], s[j + 4]);
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    half_swap<16>(s[j], s[j + 2]);
    half_swap<16>(s[j + 4], s[j + 6]);
  }
#pragma unroll
  for (int j = 0; j < 8; j += 2) half_swap<32>(s[j], s[j + 1]);
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    prefix += s[bitrev3(q)];
    rows[q * kWave] = prefix;
  }
  if constexpr (PREFETCH && (MODE == kOneDoc || MODE == kTwoDocs)) {
    th[0] = thn[0];
    if constexpr (MODE == kTwoDocs) th[1] = thn[1];
  }
  return prefix;
}

// The whole sweep over NB blocks; rows[r * 64] receives the prefix at the end
// of eighth r.  Returns the token's total.
// A sweep8 hook that does nothing.
struct NoHook {
  __device__ __forceinline__ void operator()() const {}
};

template <int MODE, int C, bool PAD, int CF = C, class Hook = NoHook, bool TS = false>
__device__ __forceinline__ float sweep8(const Wave<kWave, false> &w, const FewDocs &fd, int NB,
                                        int c0, float *rows, Hook hook = Hook{}) {
  static_assert(CF <= C && kWave % CF == 0, "the theta window divides 64 and is at most C");
  constexpr int CT = MODE == kAnyDocs ? C : (MODE == kFewDocs ? CF : 1);
  f4 win[C], twin[CT], th[2], thn[2];
  const uint32_t v0 = leaf_bytes(c0, 0, w.r);
  if constexpr (MODE == kOneDoc || MODE == kTwoDocs) {
    th[0] = theta_leaf<PAD>(w.th, c0, 0, w.r, w.th_off0);
    th[1] = MODE == kTwoDocs ? theta_leaf<PAD>(w.th, c0, 0, w.r, w.th_off1) : th[0];
  }
  if constexpr (MODE == kFewDocs) {
    f4 st[kFewMax];
    few_load<PAD>(fd, w.th, c0, 0, w.r, st);
    few_stage(fd, st, lane_id(), 0);
  }
#pragma unroll
  for (int i = 0; i < C; ++i) {
    const int t = eighth_slot_token(pair_token(i));
    win[i] = w.ph.ld4(v0, __builtin_amdgcn_readlane(w.ph_lane, t));
    if constexpr (MODE == kAnyDocs)
      twin[i] = w.th.ld4(v0, __builtin_amdgcn_readlane(w.th_lane, t));
    if constexpr (MODE == kFewDocs)
      if (i < CT) twin[i % CT] = few_leaf(fd, t, lane_id(), 0);
  }
  // hook() runs once, after the first block's step (loads it issues are in
  // flight during the other blocks)
  float prefix = 0.0f;
  for (int b = 0; b < NB - 1; ++b) {
    prefix = sweep8_block<MODE, true, C, CT, PAD, TS>(w, fd, win, twin, th, thn, c0, b, b + 1,
                                                      rows + 8 * b * kWave, prefix);
    if (b == 0) hook();
  }
  prefix = sweep8_block<MODE, false, C, CT, PAD, TS>(w, fd, win, twin, th, thn, c0, NB - 1, 0,
                                                     rows + 8 * (NB - 1) * kWave, prefix);
  if (NB == 1) hook();
  return prefix;
}

// The rebuild's tile of a one-document wavefront whose theta row is staged in
// LDS (trow: the row's floats from topic c0, zero in the padding): as
// load_tile_blocks for W = 32, with theta read from LDS.
template <bool PADDED>
__device__ __forceinline__ void load_chunk_staged(const Wave<kWave / 2, false> &w,
                                                  float (&a)[kWave / 2], int blk, int first,
                                                  const float *trow) {
#pragma unroll
  for (int k = 0; k < kWave / 2; ++k) {
    const int bk = group_value<kWave / 2>(blk, k);
    const int i = bk * (kWave / 2) + w.r;  // topic first + i
    const int t = first + i;
    const uint32_t voff = (uint32_t)(PADDED && t < 0 ? 0 : t) * 4u;
    const uint32_t poff = (uint32_t)group_value<kWave / 2>((int)w.ph_lane, k);
    a[k] = trow[i] * load_row<kWave / 2>(w.ph, voff, poff);
  }
}

// LDS floats per wavefront: the 8 NB prefix rows, and with TS the theta row.
__host__ __device__ constexpr int eighths_lds_floats(int NB, bool TS) {
  return 8 * NB * kWave + (TS ? NB * kBlock4 : 0);
}

// TS: one-document wavefronts stage their theta row in LDS during the sweep
// and the rebuild reads theta from there.
template <int C, int WPB, int WPEU, bool PAD, bool TS>
__global__ __launch_bounds__(WPB * kWave) __attribute__((amdgpu_waves_per_eu(WPEU)))
void leaf_eighths_kernel(const float *__restrict__ theta, const float *__restrict__ phi,
                         DocSource docs, const int32_t *__restrict__ word_id,
                         UniformSource u, int32_t *__restrict__ z, int64_t N, int K,
                         uint32_t theta_extent, uint32_t phi_extent) {
  extern __shared__ float lds[];
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int64_t first = ((int64_t)blockIdx.x * WPB + wave) * kWave;
  if (first >= N) return;  // whole wavefront past the end
  // Window of 64 tokens as in butterfly_kernel (N >= 64 here).
  const int64_t t0 = first + kWave <= N ? first : N - kWave;
  const int64_t n = t0 + lane;
  const bool store = n >= first;

  const int doc = docs.wave_doc(n, t0, t0 + kWave - 1);
  const int word = word_id[n];
  const float un = u(n);
  // 256-topic blocks; with PAD block 0 starts at topic c0 < 0 (a remnant of
  // K mod 256 topics behind 256 - K mod 256 empty ones, as in butterfly_kernel)
  const int NB = (K + kBlock4 - 1) / kBlock4;
  const int c0 = K - NB * kBlock4;
  Wave<kWave, false> w;
  init_wave<kWave, false>(w, theta, phi, theta_extent, phi_extent, word_id, t0, kWave - 1, K,
                          lane, doc, word);
  float *region = lds + wave * eighths_lds_floats(NB, TS);
  FewDocs stage{};
  if constexpr (TS) stage.lds = reinterpret_cast<f4 *>(region + 8 * NB * kWave);
  const FewDocs none{};
  float sum;
  if (w.mode == kOneDoc)
    sum = sweep8<kOneDoc, C, PAD, C, NoHook, TS>(w, stage, NB, c0, region + lane);
  else if (w.mode == kTwoDocs)
    sum = sweep8<kTwoDocs, C, PAD>(w, none, NB, c0, region + lane);
  else
    sum = sweep8<kAnyDocs, (C > 2 ? C / 2 : C), PAD>(w, none, NB, c0, region + lane);
  const float stop = sum * un;
  // Algorithm 9 over the ends of the 8 NB eighths.
  int lo = 0, hi = 8 * NB - 1;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (stop < region[mid * kWave + lane])
      hi = mid;
    else
      lo = mid + 1;
  }
  const int chunk = lo;
  float low = lo > 0 ? region[(lo - 1) * kWave + lane] : 0.0f;
  float high = region[lo * kWave + lane];
  // Rebuild every token's chosen 32-topic chunk (W = 32 groups) and search it
  // with Algorithm 10.  Empty topics have the prefix 0 <= stop, but the
  // search's rebuilt prefixes (high - y) may round to a tiny nonzero value
  // there, so a stop of 0 (u = 0) or of a few ulps of S can end the search
  // among them: the draw is then topic 0 (inside the rounding band).  With
  // S = 0 every comparison fails and the result is K - 1.
  const Wave<kWave / 2, false> wh = half_wave(w, lane);
  float h[kWave / 2];
  if (TS && w.mode == kOneDoc) {
    lds_order();
    load_chunk_staged<PAD>(wh, h, chunk, c0, reinterpret_cast<const float *>(stage.lds));
  } else {
    load_tile_blocks<kWave / 2, false, PAD>(wh, h, chunk, c0);
  }
  butterfly_block<kWave / 2>(h, wh.r, NoStore{});
  const int j = c0 + chunk * (kWave / 2) +
                inblock_search<kWave / 2, false>(h, nullptr, wh.r, wh.gbase, stop, low, high);
  if (store) z[n] = j < 0 ? 0 : j;
}

}  // namespace
}  // namespace LDA_NS
