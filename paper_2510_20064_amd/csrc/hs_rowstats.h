// Block-level reduction of per-thread row statistics: max, lowest-index argmax and exp2 sums
// taken against per-thread offsets, combined onto the largest offset (hs_softmax_stats).
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

}  // namespace hs
