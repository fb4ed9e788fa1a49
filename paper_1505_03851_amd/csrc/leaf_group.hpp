// Leaf-group kernel for K up to 256, and with 8-topic leaves up to 508
// (gfx950).
#pragma once

#include "tile.hpp"

namespace LDA_NS {
namespace {

// Leaf groups for K up to 256 (K divisible by 4, at most 4 G topics for a
// group size G of 8, 16, 32 or 64 lanes; N >= 64), and with leaves of 4 H
// topics (H quads) up to 4 H G; below, H = 1.  Sections 3 and 4 with a
// 4-topic leaf in the place of a topic: a wavefront holds 64 / G groups of G
// tokens, lane r of a group owns token r of the group and, in the tile, leaf
// r (topics c0 + 4r .. c0 + 4r + 3, c0 = K - 4G <= 0: the first 4G - K
// topics are empty) of every token of its group.  Load k brings leaf r of
// token k of every group into lane r of that group, so each load instruction
// reads the whole rows (16 G bytes) of 64 / G tokens.  Register a[k] is the
// leaf sum (dot4) of token k; Algorithm 8's butterfly over the G leaves
// leaves the table and the lane's own token's total; Algorithm 10 finds the
// leaf whose prefix range holds u * S, and the leaf's four products,
// reloaded for the lane's own token, give the topic by a scan from the
// prefix before the leaf. The theta leaf comes once per lane when each
// group's tokens share one document (GROUP_DOCS), else with every phi leaf.
// How the theta leaves of a group's tokens are found: every group's tokens in
// one document (one leaf per lane, loaded once), in at most kMaxGroupRuns<G>
// runs of documents (each run's leaf loaded once per lane; token k takes the
// leaf of its run: for groups of 64 lanes, up to 4 runs, from LDS where the
// leaves are staged, read a few tokens ahead; below, up to 2 runs, by a
// select in registers), or any mix (a leaf per token, loaded with its phi
// leaf).  In the first two cases every run's leaves are also staged in LDS,
// and the final reload takes its theta leaf from there (one LDS read in the
// place of a gather from memory).
enum GroupTheta : int { kGroupOne = 0, kGroupRuns = 1, kGroupAny = 2 };
template <int G>
constexpr int kMaxGroupRuns = G == kWave ? 4 : 2;
constexpr int kRunAhead = 4;  // tokens whose staged theta leaves are read ahead
// Runs read from LDS in the tile (measured: 5-15% faster for 64-lane groups
// than four selects per token; for 32-lane groups, up to 12% slower than one
// select)
template <int G>
constexpr bool kStageRuns = G == kWave;
// Groups of at most LDA_GROUP_KEEP_MAX_G lanes with 4-topic leaves keep, in
// LDS, each leaf's running sums after its first three topics for every token
// of the group (the dot4's intermediate values), so that the final scan
// reads them there instead of reloading the chosen leaf from memory:
// 12 (G + 1) bytes per token (rows padded by one leaf against LDS bank
// conflicts).
template <int G, int H>
constexpr bool kKeepLeaves = H == 1 && G <= LDA_GROUP_KEEP_MAX_G;

// LDS bytes per wavefront of the leaf-group kernel: the staged theta leaves
// of up to kMaxGroupRuns<G> runs, or the kept leaf sums.
template <int G, int H>
constexpr int group_lds_bytes() {
  if constexpr (kKeepLeaves<G, H>) return kWave * (G + 1) * 3 * (int)sizeof(float);
  return kMaxGroupRuns<G> * H * kWave * (int)sizeof(f4);
}

// A leaf of L = 4 H consecutive topics: H 16-byte quads.
template <int H>
struct Leaf {
  f4 q[H];
};

// Sum of the leaf's L theta-phi products, in topic order (the first a
// product, the others fused multiply-adds onto the running sum).
template <int H>
__device__ __forceinline__ float leaf_dot(const Leaf<H> &t, const Leaf<H> &p) {
  float s = dot4(t.q[0], p.q[0]);
#pragma unroll
  for (int h = 1; h < H; ++h) {
    s = __builtin_fmaf(t.q[h].x, p.q[h].x, s);
    s = __builtin_fmaf(t.q[h].y, p.q[h].y, s);
    s = __builtin_fmaf(t.q[h].z, p.q[h].z, s);
    s = __builtin_fmaf(t.q[h].w, p.q[h].w, s);
  }
  return s;
}

// The tile of a group: a[k] = this lane's leaf sum of token k of its group.
// voff[h]: byte offset of quad h of this lane's leaf in a row; real[h]: the
// quad holds topics (false: front padding, its theta is zero).  With
// kKeepLeaves, the running sums after the leaf's first one, two and three
// topics go to keep2[t (G + 1) + r] (the first two) and keep1[t (G + 1) + r]
// for the wavefront's token t = gbase + k and this lane's leaf r.
template <int G, int H, int C, int MODE>
__device__ __forceinline__ void group_tile(float (&a)[G], const Table &th_t, const Table &ph_t,
                                           const uint32_t (&voff)[H], const bool (&real)[H],
                                           uint32_t ph_lane, uint32_t th_lane, int gbase,
                                           uint64_t gstarts, f4 *stage, f2 *keep2,
                                           float *keep1) {
  constexpr bool KEEP = kKeepLeaves<G, H>;
  static_assert(G % C == 0, "the window size must divide G");
  constexpr int R = MODE == kGroupRuns ? kMaxGroupRuns<G> : 1;
  const f4 zero = {0.0f, 0.0f, 0.0f, 0.0f};
  // leaf of token k of the group at row offset `row` of that token (held by
  // the lane that owns the token): with G = 64 the row is uniform and goes in
  // the scalar offset, else it is fetched per lane
  const auto leaf_of = [&](const Table &t, uint32_t row, int k) {
    Leaf<H> l;
    if constexpr (G == kWave) {
      const uint32_t srow = (uint32_t)__builtin_amdgcn_readlane((int)row, k);
#pragma unroll
      for (int h = 0; h < H; ++h) l.q[h] = t.ld4(voff[h], srow);
    } else {
      const uint32_t vrow = (uint32_t)__builtin_amdgcn_ds_bpermute((gbase + k) << 2, (int)row);
#pragma unroll
      for (int h = 0; h < H; ++h) l.q[h] = t.ld4v(voff[h], vrow);
    }
    return l;
  };
  const auto mask = [&](Leaf<H> l) {
#pragma unroll
    for (int h = 0; h < H; ++h) l.q[h] = real[h] ? l.q[h] : zero;
    return l;
  };
  // kGroupRuns: gstarts bit p (0 < p < G) marks the group's token p as the
  // first of a run; run j's leaf is that of the token opening it
  Leaf<H> th[R];
  if constexpr (MODE == kGroupOne) {
    Leaf<H> l;
#pragma unroll
    for (int h = 0; h < H; ++h) l.q[h] = th_t.ld4v(voff[h], th_lane);
    th[0] = mask(l);
  } else if constexpr (MODE == kGroupRuns) {
    uint64_t m = gstarts;
    th[0] = mask(leaf_of(th_t, th_lane, 0));
#pragma unroll
    for (int j = 1; j < R; ++j) {
      const int p = m ? (int)__builtin_ctzll(m) : 0;
      m &= m - 1;
      th[j] = mask(leaf_of(th_t, th_lane, p));
    }
  }
  if constexpr (MODE != kGroupAny && !KEEP) {
    // stage the runs' leaves: quad h of run j at stage[(j H + h) 64 + lane]
    const int lane = lane_id();
#pragma unroll
    for (int j = 0; j < R; ++j)
#pragma unroll
      for (int h = 0; h < H; ++h) stage[(j * H + h) * kWave + lane] = th[j].q[h];
    lds_order();
  }
  const auto run_of = [&](int k) {
    // runs opened at the group's tokens 1 .. k
    const uint64_t upto = k == 63 ? ~0ull : ((2ull << k) - 1ull);
    return __builtin_popcountll(gstarts & upto);
  };
  const auto staged = [&](int k) {
    Leaf<H> l;
    const int base = run_of(k) * H * kWave + lane_id();
#pragma unroll
    for (int h = 0; h < H; ++h) l.q[h] = stage[base + h * kWave];
    return l;
  };
  constexpr bool STAGED = MODE == kGroupRuns && kStageRuns<G>;
  constexpr int CT = MODE == kGroupAny ? C : (STAGED ? kRunAhead : 1);
  Leaf<H> win[C], twin[CT];
#pragma unroll
  for (int k = 0; k < C; ++k) {
    win[k] = leaf_of(ph_t, ph_lane, k);
    if constexpr (MODE == kGroupAny) twin[k] = leaf_of(th_t, th_lane, k);
  }
  if constexpr (STAGED) {
#pragma unroll
    for (int k = 0; k < CT; ++k) twin[k] = staged(k);
  }
#pragma unroll
  for (int k = 0; k < G; ++k) {
    Leaf<H> tv;
    if constexpr (MODE == kGroupAny) {
      tv = mask(twin[k % C]);
    } else if constexpr (STAGED) {
      tv = twin[k % CT];
    } else if constexpr (MODE == kGroupRuns) {
      const int j = run_of(k);
      tv = th[0];
#pragma unroll
      for (int i = 1; i < R; ++i)
#pragma unroll
        for (int h = 0; h < H; ++h) tv.q[h] = j == i ? th[i].q[h] : tv.q[h];
    } else {
      tv = th[0];
    }
    if constexpr (KEEP) {
      // dot4's steps, the first three sums kept
      const f4 t = tv.q[0], p = win[k % C].q[0];
      const float s0 = t.x * p.x;
      const float s1 = __builtin_fmaf(t.y, p.y, s0);
      const float s2 = __builtin_fmaf(t.z, p.z, s1);
      a[k] = __builtin_fmaf(t.w, p.w, s2);
      const int at = (gbase + k) * (G + 1) + (lane_id() & (G - 1));
      keep2[at] = f2{s0, s1};
      keep1[at] = s2;
    } else {
      a[k] = leaf_dot(tv, win[k % C]);
    }
    if (k + C < G) {
      win[k % C] = leaf_of(ph_t, ph_lane, k + C);
      if constexpr (MODE == kGroupAny) twin[k % C] = leaf_of(th_t, th_lane, k + C);
    }
    if constexpr (STAGED)
      if (k + CT < G) twin[k % CT] = staged(k + CT);
    __builtin_amdgcn_sched_barrier(0);
  }
  if constexpr (KEEP) lds_order();
}

// L = 4 H topics per lane: groups of G lanes cover 4 H G topics.
template <int G, int H, int C, int WPEU, bool PAD>
__global__ __launch_bounds__(kBlockThreads) __attribute__((amdgpu_waves_per_eu(WPEU)))
void leaf_group_kernel(const float *__restrict__ theta, const float *__restrict__ phi,
                       DocSource docs, const int32_t *__restrict__ word_id,
                       UniformSource u, int32_t *__restrict__ z, int64_t N, int K,
                       uint32_t theta_extent, uint32_t phi_extent) {
  constexpr int L = kLeaf * H;
  constexpr bool KEEP = kKeepLeaves<G, H>;
  extern __shared__ float lds[];
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  float *region = lds + wave * (group_lds_bytes<G, H>() / (int)sizeof(float));
  f4 *stage = reinterpret_cast<f4 *>(region);
  f2 *keep2 = reinterpret_cast<f2 *>(region);
  float *keep1 = region + 2 * kWave * (G + 1);
  const int64_t first = ((int64_t)blockIdx.x * kWavesPerBlock + wave) * kWave;
  if (first >= N) return;  // whole wavefront past the end
  // Window of 64 tokens as in butterfly_kernel (N >= 64 here).
  const int64_t t0 = first + kWave <= N ? first : N - kWave;
  const int64_t n = t0 + lane;
  const bool store = n >= first;
  const int doc = docs.wave_doc(n, t0, t0 + kWave - 1);
  const int word = word_id[n];
  const float un = u(n);

  const Table th_t = make_table(theta, theta_extent, K);
  const Table ph_t = make_table(phi, phi_extent, K);
  const uint32_t ph_lane = ph_t.row((uint32_t)word);
  const uint32_t th_lane = th_t.row((uint32_t)doc);
  const int r = lane & (G - 1), gbase = lane & ~(G - 1);
  const int c0 = K - L * G;  // first topic of leaf 0 (< 0: front padding)
  uint32_t voff[H];
  bool real[H];
#pragma unroll
  for (int h = 0; h < H; ++h) {
    const int topic = c0 + L * r + kLeaf * h;
    real[h] = !PAD || topic >= 0;
    voff[h] = (uint32_t)(real[h] ? topic : 0) * 4u;
  }
  // runs of documents inside each group: bit l of `starts` marks lane l's
  // token as the first of a run (not counting the group's first token)
  // (lane l's previous document by a DPP wavefront shift right by one lane:
  // no LDS round trip before the first loads; lane 0 keeps its own)
  const int prev = __builtin_amdgcn_update_dpp(doc, doc, 0x138, 0xF, 0xF, false);
  const uint64_t starts = __builtin_amdgcn_ballot_w64(r != 0 && doc != prev);
  const uint64_t gmask = G == kWave ? ~0ull : ((1ull << G) - 1ull);
  const uint64_t gstarts = (starts >> gbase) & gmask;  // this lane's group, bit p = token p
  // the most runs in any group (groups of G lanes: at most 64 / G of them)
  int most = 0;
#pragma unroll
  for (int g = 0; g < kWave / G; ++g)
    most = max(most, __builtin_popcountll((starts >> (g * G)) & gmask));

  float a[G];
  if (most == 0)
    group_tile<G, H, C, kGroupOne>(a, th_t, ph_t, voff, real, ph_lane, th_lane, gbase, 0,
                                   stage, keep2, keep1);
  else if (most < kMaxGroupRuns<G>)
    group_tile<G, H, C, kGroupRuns>(a, th_t, ph_t, voff, real, ph_lane, th_lane, gbase,
                                    gstarts, stage, keep2, keep1);
  else
    group_tile<G, H, C, kGroupAny>(a, th_t, ph_t, voff, real, ph_lane, th_lane, gbase, 0,
                                   stage, keep2, keep1);
  butterfly_block<G>(a, r, NoStore{});
  const float total = a[G - 1];
  const float stop = total * un;
  float low = 0.0f, high = total;
  int q = inblock_search<G, false>(a, nullptr, r, gbase, stop, low, high);
  // The search rebuilds prefixes as low + y or high - y.  Where the true
  // prefix is 0 (up to the first real topic) high - y may round to a tiny
  // nonzero value, and a stop of 0 (u = 0) or of a few ulps of S may then
  // end the search in a padding leaf.  The true prefix before the leaf
  // holding topic 0 is exactly 0, so the search never ends before that leaf,
  // and from there it scans from exactly 0.
  if constexpr (PAD) {
    const int qmin = (-c0) / L;  // leaf holding topic 0
    if (q <= qmin) {
      q = qmin;
      low = 0.0f;
    }
  }
  // Leaf q of the lane's own token, scanned from the prefix before it: the
  // first of its L topics whose running sum exceeds stop, else the last.
  // Padding topics (front of leaf qmin when L does not divide K) have zero
  // weight and a running sum of exactly 0 <= stop, so they are never chosen;
  // with S = 0 every comparison fails and the result is K - 1.
  // The theta leaf: staged in LDS by lane gbase + q for the run of the
  // lane's own token (padding quads already zero there), unless the group's
  // documents were too many runs.
  const int tq = c0 + L * q;
  if constexpr (KEEP) {
    // the kept sums of leaf q of this lane's token (nondecreasing: the
    // products are not negative), added to the prefix before the leaf
    const int at = lane * (G + 1) + q;
    const f2 s01 = keep2[at];
    const float s2 = keep1[at];
    const int i = stop < low + s01.x ? 0 : stop < low + s01.y ? 1 : stop < low + s2 ? 2 : 3;
    if (store) z[n] = tq + i;
    return;
  }
  const bool staged = most < kMaxGroupRuns<G>;
  const int run = __builtin_popcountll(gstarts & ((2ull << r) - 1ull));
  float sum = low;
  int i = L - 1;
#pragma unroll
  for (int h = 0; h < H; ++h) {
    const int topic = tq + kLeaf * h;
    const uint32_t qoff = (uint32_t)(topic > 0 ? topic : 0) * 4u;
    f4 tl;
    if (staged) {
      tl = stage[(run * H + h) * kWave + gbase + q];
    } else {
      tl = th_t.ld4v(qoff, th_lane);
      if (PAD && topic < 0) tl = f4{0.0f, 0.0f, 0.0f, 0.0f};
    }
    const f4 pl = ph_t.ld4v(qoff, ph_lane);
#pragma unroll
    for (int e = 0; e < kLeaf; ++e) {
      const int idx = kLeaf * h + e;
      if (idx == L - 1) break;  // the leaf's last topic needs no comparison
      sum = __builtin_fmaf(tl[e], pl[e], sum);
      if (i == L - 1 && stop < sum) i = idx;
    }
  }
  if (store) z[n] = tq + i;
}

}  // namespace
}  // namespace LDA_NS
