// Standalone learner kernel (hs_accept_len, hs_hedge_update, hs_normalhedge_update):
// one wave64 per query, running the learner step of hs_learner.h.
#include "hs_learner.h"

namespace hs {

__global__ __launch_bounds__(64) void hs_tail_kernel(TailArgs a) {
  extern __shared__ double lds[];
  tail_query(a, blockIdx.x, lds);
}

int launch_tail(const TailArgs& a, hipStream_t stream) {
  const size_t lds = sizeof(double) * (size_t)tail_lds_doubles(a);
  hs_tail_kernel<<<a.B, 64, lds, stream>>>(a);
  return hipGetLastError() == hipSuccess ? HS_OK : HS_ERR_HIP;
}

}  // namespace hs
