// Leaf kernel on tokens routed to the XCDs (gfx950).
#pragma once

#include "leaf_eighths.hpp"
#include "route.hpp"

namespace LDA_NS {
namespace {

// The leaf kernel on routed tokens.  Workgroups are dispatched to the GPU's
// eight XCDs round robin (workgroup b on XCD b mod 8), and each XCD has its
// own L2.  Routing gives list x of the tokens -- those whose word falls in the
// word classes assigned to XCD x -- to the workgroups b with b mod 8 = x, so
// that each L2 caches the phi rows of one eighth of the vocabulary.  Routed
// position i holds token perm[i] (-1: padding, drawn but not stored) with
// word rword[i] and document rdoc[i]; list x is [lists[x], lists[x] +
// lists[8 + x]), a multiple of 64 long, in the original token order, so that
// the documents of a wavefront form a few runs (kFewDocs).
constexpr int kXcds = kRouteXcds;

struct RoutedTokens {
  const int32_t *perm, *rword, *rdoc;
  int64_t base[kXcds], len[kXcds];  // list starts and lengths
};

// Up to kRowsMaxBlocks 256-topic blocks, a wavefront whose tokens form at
// most kRowsMax runs of documents keeps the runs' whole theta rows in LDS
// (staged leaf by leaf during the sweep), and the rebuild reads its theta
// values there rather than from memory.
constexpr int kRowsMax = 3;
constexpr int kRowsMaxBlocks = 4;

// LDS floats per wavefront of the routed kernel: the prefix rows, then the
// staged theta leaves of up to kFewMax runs, or the kRowsMax runs' rows.
__host__ __device__ constexpr int routed_lds_floats(int NB) {
  const int leaves = kFewMax * kWave * 4;
  const int rows = NB <= kRowsMaxBlocks ? kRowsMax * NB * kBlock4 : 0;
  return 8 * NB * kWave + (rows > leaves ? rows : leaves);
}

// The rebuild's tile (load_tile_blocks for W = 32) with theta read from the
// runs' rows staged in LDS: token k's topic first + i of run s_k at
// trow[s_k * row + i] (zero in the padding).
template <bool PADDED>
__device__ __forceinline__ void load_chunk_rows(const Wave<kWave / 2, false> &w,
                                                float (&a)[kWave / 2], int blk, int first,
                                                const float *trow, int slot, int row) {
#pragma unroll
  for (int k = 0; k < kWave / 2; ++k) {
    const int bk = group_value<kWave / 2>(blk, k);
    const int sk = group_value<kWave / 2>(slot, k);
    const int i = bk * (kWave / 2) + w.r;  // topic first + i
    const int t = first + i;
    const uint32_t voff = (uint32_t)(PADDED && t < 0 ? 0 : t) * 4u;
    const uint32_t poff = (uint32_t)group_value<kWave / 2>((int)w.ph_lane, k);
    a[k] = trow[sk * row + i] * load_row<kWave / 2>(w.ph, voff, poff);
  }
}

// One wavefront of the leaf kernel over 64 listed tokens: lane `lane` draws
// token n (document doc, word word) and stores z[n] if `store`.  The tokens
// need not be consecutive; their documents usually form a few runs
// (kFewDocs).  region: the wavefront's routed_lds_floats(NB) floats of LDS.
template <int C, bool PAD>
__device__ __forceinline__ void draw_listed(const float *__restrict__ theta,
                                            const float *__restrict__ phi, uint32_t theta_extent,
                                            uint32_t phi_extent, int K, const int32_t *wp,
                                            int64_t first, int lane, float *region, int64_t n,
                                            bool store, int doc, int word, const UniformSource &u,
                                            int32_t *__restrict__ z) {
  const int NB = (K + kBlock4 - 1) / kBlock4;
  const int c0 = K - NB * kBlock4;
  FewDocs fd;
  fd.lds = reinterpret_cast<f4 *>(region + 8 * NB * kWave);
  Wave<kWave, false> w;
  init_wave<kWave, false>(w, theta, phi, theta_extent, phi_extent, wp, first, kWave - 1, K, lane,
                          doc, word);
  // runs of documents among the wavefront's tokens
  const int prev = __builtin_amdgcn_ds_bpermute(((lane + kWave - 1) & (kWave - 1)) << 2, doc);
  const uint64_t starts = __builtin_amdgcn_ballot_w64(lane == 0 || doc != prev);
  fd.D = __builtin_amdgcn_readfirstlane(__builtin_popcountll(starts));
  fd.slot = __builtin_popcountll(starts & ((2ull << lane) - 1ull)) - 1;
  const bool rows = NB <= kRowsMaxBlocks && fd.D <= kRowsMax;
  fd.rstride = rows ? NB * kWave : kWave;
  fd.bstride = rows ? kWave : 0;
  uint64_t m = starts;
#pragma unroll
  for (int d = 0; d < kFewMax; ++d) {
    fd.row[d] = 0;
    if (m) {
      const int ln = __builtin_ctzll(m);
      m &= m - 1;
      fd.row[d] = w.th.row((uint32_t)__builtin_amdgcn_readlane(doc, ln));
    }
  }
  // The uniform's load depends on the token index's; issued before the
  // sweep it would hold up every in-order wait for the sweep's loads, so
  // it is issued after the first block's step.
  float un = 0.0f;
  const auto load_u = [&]() { un = u(n); };
  region += lane;
  float sum;
  if (fd.D == 1 && rows)
    sum = sweep8<kOneDoc, C, PAD, C, decltype(load_u), true>(w, fd, NB, c0, region, load_u);
  else if (fd.D == 1)
    sum = sweep8<kOneDoc, C, PAD>(w, fd, NB, c0, region, load_u);
  else if (fd.D <= kFewMax)
    sum = sweep8<kFewDocs, LDA_ROUTED_FEW_WINDOW, PAD, LDA_ROUTED_FEW_THETA>(w, fd, NB, c0,
                                                                           region, load_u);
  else
    sum = sweep8<kAnyDocs, (C > 2 ? C / 2 : C), PAD>(w, fd, NB, c0, region, load_u);
  const float stop = sum * un;
  // Algorithm 9 over the ends of the 8 NB eighths.
  int lo = 0, hi = 8 * NB - 1;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (stop < region[mid * kWave])
      hi = mid;
    else
      lo = mid + 1;
  }
  const int chunk = lo;
  float low = lo > 0 ? region[(lo - 1) * kWave] : 0.0f;
  float high = region[lo * kWave];
  // Rebuild and Algorithm 10 on the chosen 32-topic chunk, as in
  // leaf_eighths_kernel.
  const Wave<kWave / 2, false> wh = half_wave(w, lane);
  float h[kWave / 2];
  if (rows) {
    lds_order();
    load_chunk_rows<PAD>(wh, h, chunk, c0, reinterpret_cast<const float *>(fd.lds), fd.slot,
                         NB * kBlock4);
  } else {
    load_tile_blocks<kWave / 2, false, PAD>(wh, h, chunk, c0);
  }
  butterfly_block<kWave / 2>(h, wh.r, NoStore{});
  const int j = c0 + chunk * (kWave / 2) +
                inblock_search<kWave / 2, false>(h, nullptr, wh.r, wh.gbase, stop, low, high);
  // (a search ending among the empty topics: topic 0, as in leaf_eighths_kernel)
  if (store) z[n] = j < 0 ? 0 : j;
}

template <int C, int WPB, int WPEU, bool PAD>
__global__ __launch_bounds__(WPB * kWave) __attribute__((amdgpu_waves_per_eu(WPEU)))
void routed_eighths_kernel(const float *__restrict__ theta, const float *__restrict__ phi,
                           RoutedTokens rt, UniformSource u, int32_t *__restrict__ z, int K,
                           uint32_t theta_extent, uint32_t phi_extent) {
  extern __shared__ float lds[];
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int x = blockIdx.x % kXcds;
  const int64_t base = rt.base[x];
  const int64_t len = rt.len[x];
  const int NB = (K + kBlock4 - 1) / kBlock4;
  // One tile of WPB wavefronts of its list per workgroup (the grid holds as
  // many tiles per list as the longest list needs).
  const int64_t first = ((int64_t)(blockIdx.x / kXcds) * WPB + wave) * kWave;
  if (first >= len) return;
  const int64_t i = base + first + lane;
  const int n = rt.perm[i];
  draw_listed<C, PAD>(theta, phi, theta_extent, phi_extent, K, rt.rword + base, first, lane,
                      lds + wave * routed_lds_floats(NB), n >= 0 ? n : 0, n >= 0, rt.rdoc[i],
                      rt.rword[i], u, z);
}

}  // namespace
}  // namespace LDA_NS
