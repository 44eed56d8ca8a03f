// Block-level statistics of one row slice: max, lowest-index argmax and the exp2 sum of a
// temperature softmax. Shared by the evaluation kernel and hs_softmax_stats.
#pragma once

#include <climits>

#include "hs_internal.h"

namespace hs {

template <bool NEED_SUM, bool NEED_ARG>
__device__ inline SliceStat block_reduce_stat(float m, int idx, float o, float s) {
  __shared__ SliceStat sh[kWaves];
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    float m2 = __shfl_xor(m, off, 64);
    if (NEED_ARG) {
      int i2 = __shfl_xor(idx, off, 64);
      argmax_combine(m, idx, m2, i2);
    } else {
      m = fmaxf(m, m2);
    }
    if (NEED_SUM) {
      float o2 = __shfl_xor(o, off, 64);
      float s2 = __shfl_xor(s, off, 64);
      lse2_combine(o, s, o2, s2);
    }
  }
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  if (lane == 0) sh[wv] = SliceStat{m, idx, o, s};
  __syncthreads();
  SliceStat r = sh[0];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) {
    SliceStat x = sh[w];
    if (NEED_ARG) argmax_combine(r.m, r.idx, x.m, x.idx);
    else r.m = fmaxf(r.m, x.m);
    if (NEED_SUM) lse2_combine(r.o, r.s, x.o, x.s);
  }
  __syncthreads();
  return r;
}

// Statistics of vectors [v0, v1) of a row whose first logit is at rowp (V logits in the row).
// The exp2 sum is taken against the thread's own offset fl(m_t * c) and combined exactly
// across threads, so the slice result is sum_v exp2(z_v c - fl(m c)) for the slice max m.
template <int DT, bool NEED_SUM, bool NEED_ARG>
__device__ inline SliceStat row_slice_stats(const char* rowp, int64_t v0, int64_t v1, int64_t V,
                                            float c) {
  using Vt = Vec<DT>;
  constexpr int E = Vt::kElems, U = Vt::kU;
  const int t = threadIdx.x;
  float z[U][E];
#pragma unroll
  for (int j = 0; j < U; ++j) {
    int64_t vi = v0 + (int64_t)j * kThreads + t;
    if (vi < v1) {
      Vt::load(rowp, vi, V, z[j]);
    } else {
#pragma unroll
      for (int e = 0; e < E; ++e) z[j][e] = -INFINITY;
    }
  }
  float m = -INFINITY;
  int idx = INT_MAX;
#pragma unroll
  for (int j = 0; j < U; ++j) {
#pragma unroll
    for (int e = 0; e < E; ++e) {
      float x = z[j][e];
      if (NEED_ARG) {
        if (x > m) {
          m = x;
          idx = (int)((v0 + (int64_t)j * kThreads + t) * E + e);
        }
      } else {
        m = fmaxf(m, x);
      }
    }
  }
  // a thread whose logits are all -inf still owns its lowest valid index
  if (NEED_ARG && idx == INT_MAX && v0 + t < v1) idx = (int)((v0 + t) * E);
  float o = -INFINITY, s = 0.0f;
  if (NEED_SUM && m != -INFINITY) {
    o = m * c;  // rounded product; consumers recompute exactly this value (no contraction)
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < U; ++j)
#pragma unroll
      for (int e = 0; e < E; ++e) acc[e & 3] += __builtin_amdgcn_exp2f(fmaf(z[j][e], c, -o));
    s = (acc[0] + acc[1]) + (acc[2] + acc[3]);
  }
  return block_reduce_stat<NEED_SUM, NEED_ARG>(m, idx, o, s);
}

}  // namespace hs
