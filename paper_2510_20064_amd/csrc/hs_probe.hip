// Streaming-read probe: reads every 16-byte vector of a buffer once and writes one word per
// wave (the XOR of the words it read, so that no load can be dropped). It does none of the
// method's arithmetic; it gives the rate at which this device streams a resident buffer, the
// ceiling that the evaluation kernels' achieved bandwidth is compared with.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "hs_internal.h"

namespace hs {
namespace {

constexpr int kProbeThreads = 256;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <int U, bool NT>
__global__ __launch_bounds__(kProbeThreads) void stream_read_kernel(const u32x4* __restrict__ x,
                                                                    uint64_t n, uint32_t* out) {
  const uint64_t stride = (uint64_t)gridDim.x * kProbeThreads;
  uint64_t i = (uint64_t)blockIdx.x * kProbeThreads + threadIdx.x;
  uint32_t acc = 0;
  // U loads in flight per thread, each wave's load one contiguous KiB
  for (; i + (U - 1) * stride < n; i += U * stride) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = NT ? __builtin_nontemporal_load(x + i + u * stride) : x[i + u * stride];
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; i < n; i += stride) {
    const u32x4 v = x[i];
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) acc ^= __shfl_xor(acc, o);
  if ((threadIdx.x & 63) == 0) out[blockIdx.x * (kProbeThreads / 64) + (threadIdx.x >> 6)] = acc;
}

template <int U, bool NT>
int launch_one(const void* x, uint64_t n, int grid, uint32_t* out, hipStream_t s) {
  stream_read_kernel<U, NT><<<grid, kProbeThreads, 0, s>>>(static_cast<const u32x4*>(x), n, out);
  return hipGetLastError() == hipSuccess ? HS_OK : HS_ERR_HIP;
}

}  // namespace

int launch_stream_read(const void* x, uint64_t vectors, int grid, int unroll, bool nontemporal,
                       uint32_t* out, hipStream_t s) {
  switch (unroll * 2 + (nontemporal ? 1 : 0)) {
    case 2: return launch_one<1, false>(x, vectors, grid, out, s);
    case 3: return launch_one<1, true>(x, vectors, grid, out, s);
    case 4: return launch_one<2, false>(x, vectors, grid, out, s);
    case 5: return launch_one<2, true>(x, vectors, grid, out, s);
    case 8: return launch_one<4, false>(x, vectors, grid, out, s);
    case 9: return launch_one<4, true>(x, vectors, grid, out, s);
    case 16: return launch_one<8, false>(x, vectors, grid, out, s);
    case 17: return launch_one<8, true>(x, vectors, grid, out, s);
    default: return HS_ERR_ARG;
  }
}

}  // namespace hs
