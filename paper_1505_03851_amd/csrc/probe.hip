// Measurement probes (gfx950): a memory-only copy of the draw's access
// pattern, and a streaming read.  They draw nothing; they exist to measure
// the floor the memory system sets for the draw and the rates at which HBM
// and the MALL serve reads (include/lda_probe.h).
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "lda_draw.h"
#include "lda_probe.h"
#include "butterfly.hpp"

namespace lda {
namespace {

constexpr int kLdsPerCu = 160 * 1024;  // LDS of one CU (bytes)

__device__ __forceinline__ float sum4(f4 v) { return (v.x + v.y) + (v.z + v.w); }

// Memory-only floor of the draw for rows read by groups of G lanes (G < 64:
// one load reads the rows, K <= 4 G topics, of 64 / G tokens) or, with G =
// 64, in blocks of 256 topics, one token per load.  Per wavefront of 64
// consecutive tokens (the last wavefront takes the final 64 tokens, as the
// draw does): the phi leaves of every token, the theta leaves of a token whose
// document differs from the previous token's, u; z written where the draw
// stores.  C loads are issued before their values are summed.
template <int G, int C>
__global__ __launch_bounds__(4 * kWave) void floor_kernel(
    const float *__restrict__ theta, const float *__restrict__ phi,
    const int32_t *__restrict__ doc_id, const int32_t *__restrict__ word_id,
    const float *__restrict__ u, int32_t *__restrict__ z, int64_t N, int K, int wpb,
    uint32_t theta_bytes, uint32_t phi_bytes) {
  extern __shared__ float occupancy_pad[];  // never touched: caps workgroups per CU
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int64_t first = ((int64_t)blockIdx.x * wpb + wave) * kWave;
  if (first >= N) return;
  const int64_t t0 = first + kWave <= N ? first : N - kWave;
  const int64_t n = t0 + lane;
  const bool store = n >= first;
  const int doc = doc_id[n];
  const int word = word_id[n];
  float acc = u[n];
  const rsrc_t th_rs = make_rsrc(theta, theta_bytes);
  const rsrc_t ph_rs = make_rsrc(phi, phi_bytes);
  const uint32_t row_bytes = (uint32_t)K * 4u;
  const uint32_t ph_lane = (uint32_t)word * row_bytes;
  const uint32_t th_lane = (uint32_t)doc * row_bytes;
  if constexpr (G == kWave) {
    const int nb = (K + 4 * kWave - 1) / (4 * kWave);
    const int c0 = K - 4 * kWave * nb;  // first topic of block 0 (<= 0)
    for (int b = 0; b < nb; ++b) {
      const int topic = c0 + 4 * kWave * b + 4 * lane;
      const uint32_t voff = (uint32_t)(topic > 0 ? topic : 0) * 4u;
      for (int k0 = 0; k0 < kWave; k0 += C) {
        f4 v[C];
#pragma unroll
        for (int j = 0; j < C; ++j) {
          const uint32_t srow = (uint32_t)__builtin_amdgcn_readlane((int)ph_lane, k0 + j);
          v[j] = load_f32x4(ph_rs, voff, srow);
        }
#pragma unroll
        for (int j = 0; j < C; ++j) {
          const int k = k0 + j;
          const int dk = __builtin_amdgcn_readlane(doc, k);
          const int dp = __builtin_amdgcn_readlane(doc, k > 0 ? k - 1 : 0);
          if (k == 0 || dk != dp)
            acc += sum4(load_f32x4(th_rs, voff, (uint32_t)__builtin_amdgcn_readlane((int)th_lane, k)));
          acc += sum4(v[j]);
        }
      }
    }
  } else {
    const int r = lane & (G - 1), gbase = lane & ~(G - 1);
    const int topic = K - 4 * G + 4 * r;
    const uint32_t voff = (uint32_t)(topic > 0 ? topic : 0) * 4u;
    for (int k0 = 0; k0 < G; k0 += C) {
      f4 v[C];
#pragma unroll
      for (int j = 0; j < C; ++j) {
        const uint32_t vrow =
            (uint32_t)__builtin_amdgcn_ds_bpermute((gbase + k0 + j) << 2, (int)ph_lane);
        v[j] = load_f32x4(ph_rs, voff + vrow, 0);
      }
#pragma unroll
      for (int j = 0; j < C; ++j) {
        const int k = k0 + j;
        const int dk = __builtin_amdgcn_ds_bpermute((gbase + k) << 2, doc);
        const int dp = __builtin_amdgcn_ds_bpermute((gbase + (k > 0 ? k - 1 : 0)) << 2, doc);
        if (k == 0 || dk != dp)
          acc += sum4(load_f32x4(th_rs, voff + (uint32_t)dk * row_bytes, 0));
        acc += sum4(v[j]);
      }
    }
  }
  if (store) z[n] = __builtin_bit_cast(int32_t, acc);
}

// Streaming read: every 16 bytes of buf, `passes` times.  Workgroup b reads
// its own contiguous span of the buffer (the last span takes the remainder),
// 16 loads of 16 bytes in flight per lane; all LDA_PROBE_READ_GROUPS
// workgroups are resident at once (8 per CU), so between two passes over a
// span every XCD streams its whole share of the buffer.
constexpr int kReadInFlight = 16;
__global__ __launch_bounds__(256) void read_kernel(const f4 *__restrict__ buf, int64_t n4,
                                                   int passes, float *__restrict__ out) {
  const int64_t per = n4 / gridDim.x;
  const int64_t lo = (int64_t)blockIdx.x * per;
  const int64_t hi = blockIdx.x + 1 == gridDim.x ? n4 : lo + per;
  constexpr int64_t step = (int64_t)kReadInFlight * 256;
  float acc = 0.0f;
  for (int p = 0; p < passes; ++p) {
    int64_t i = lo + threadIdx.x;
    for (; i + (kReadInFlight - 1) * 256 < hi; i += step) {
      f4 v[kReadInFlight];
#pragma unroll
      for (int j = 0; j < kReadInFlight; ++j) v[j] = buf[i + j * 256];
#pragma unroll
      for (int j = 0; j < kReadInFlight; ++j) acc += sum4(v[j]);
    }
    for (; i < hi; i += 256) acc += sum4(buf[i]);
  }
  out[(int64_t)blockIdx.x * blockDim.x + threadIdx.x] = acc;
}

template <int G, int C>
int launch_floor(const float *theta, const float *phi, const int32_t *doc_id,
                 const int32_t *word_id, const float *u, int32_t *z, int64_t N, int32_t M,
                 int32_t V, int32_t K, int wpb, int waves_per_cu, hipStream_t s) {
  size_t pad = 0;
  if (waves_per_cu > 0) {
    const int groups = waves_per_cu / wpb > 0 ? waves_per_cu / wpb : 1;
    pad = (size_t)(kLdsPerCu / groups) & ~(size_t)255;
    if (pad > 65536 &&
        hipFuncSetAttribute(reinterpret_cast<const void *>(&floor_kernel<G, C>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)pad) != hipSuccess)
      return LDA_ERR_HIP;
  }
  const int64_t waves = (N + kWave - 1) / kWave;
  const dim3 grid((unsigned)((waves + wpb - 1) / wpb));
  floor_kernel<G, C><<<grid, wpb * kWave, pad, s>>>(
      theta, phi, doc_id, word_id, u, z, N, K, wpb, (uint32_t)((int64_t)M * K * 4),
      (uint32_t)((int64_t)V * K * 4));
  return LDA_OK;
}

template <int C>
int dispatch_floor(const float *theta, const float *phi, const int32_t *doc_id,
                   const int32_t *word_id, const float *u, int32_t *z, int64_t N, int32_t M,
                   int32_t V, int32_t K, int wpb, int waves_per_cu, hipStream_t s) {
  if (K <= 32)
    return launch_floor<8, 8>(theta, phi, doc_id, word_id, u, z, N, M, V, K, wpb, waves_per_cu, s);
  if (K <= 64)
    return launch_floor<16, C < 16 ? C : 16>(theta, phi, doc_id, word_id, u, z, N, M, V, K, wpb,
                                             waves_per_cu, s);
  if (K <= 128)
    return launch_floor<32, C>(theta, phi, doc_id, word_id, u, z, N, M, V, K, wpb, waves_per_cu, s);
  return launch_floor<kWave, C>(theta, phi, doc_id, word_id, u, z, N, M, V, K, wpb, waves_per_cu,
                                s);
}

thread_local hipError_t g_probe_hip = hipSuccess;

int finish(int st) {
  if (st != LDA_OK) return st;
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    g_probe_hip = e;
    return LDA_ERR_HIP;
  }
  return LDA_OK;
}

}  // namespace
}  // namespace lda

using namespace lda;

extern "C" int lda_probe_draw_floor(const float *theta, const float *phi, const int32_t *doc_id,
                                    const int32_t *word_id, const float *u, int32_t *z,
                                    int64_t N, int32_t M, int32_t V, int32_t K, int32_t window,
                                    int32_t waves_per_group, int32_t waves_per_cu,
                                    void *stream) {
  if (N < 0 || M <= 0 || V <= 0 || K <= 0) return LDA_ERR_SHAPE;
  if (K % 4 || K > 2048 || N < kWave || N > LDA_MAX_N) return LDA_ERR_UNSUPPORTED;
  if ((window != 8 && window != 16) || (waves_per_group != 2 && waves_per_group != 4) ||
      waves_per_cu < 0 || waves_per_cu > 32)
    return LDA_ERR_UNSUPPORTED;
  if ((int64_t)M * K * 4 > LDA_MAX_TABLE_BYTES || (int64_t)V * K * 4 > LDA_MAX_TABLE_BYTES)
    return LDA_ERR_UNSUPPORTED;
  const void *ptrs[] = {theta, phi, doc_id, word_id, u, z};
  for (const void *p : ptrs) {
    if (!p) return LDA_ERR_NULL;
    if (reinterpret_cast<uintptr_t>(p) & 3u) return LDA_ERR_ALIGN;
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int st = window == 8 ? dispatch_floor<8>(theta, phi, doc_id, word_id, u, z, N, M, V, K,
                                                 waves_per_group, waves_per_cu, s)
                             : dispatch_floor<16>(theta, phi, doc_id, word_id, u, z, N, M, V, K,
                                                  waves_per_group, waves_per_cu, s);
  return finish(st);
}

extern "C" int lda_probe_read(const void *buf, int64_t bytes, int32_t passes, float *out,
                              void *stream) {
  if (bytes < 0 || passes < 1) return LDA_ERR_SHAPE;
  if (bytes == 0) return LDA_OK;
  if (!buf || !out) return LDA_ERR_NULL;
  if ((reinterpret_cast<uintptr_t>(buf) & 15u) || (bytes & 15) ||
      (reinterpret_cast<uintptr_t>(out) & 3u))
    return LDA_ERR_ALIGN;
  read_kernel<<<LDA_PROBE_READ_GROUPS, 256, 0, static_cast<hipStream_t>(stream)>>>(
      static_cast<const f4 *>(buf), bytes / 16, passes, out);
  return finish(LDA_OK);
}
