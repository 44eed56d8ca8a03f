// Standalone learner kernel (hs_accept_len, hs_hedge_update, hs_normalhedge_update):
// one wave64 per query, running the learner step of hs_learner.h.
#include "hs_learner.h"

namespace hs {

__global__ __launch_bounds__(64) void hs_tail_kernel(TailArgs a) {
  extern __shared__ double lds[];
  if (a.round_fail) {
    // the evaluation launch before this one advanced the epoch once, at its end; its fail
    // word carries that call's tag when one of its waits gave up: then its alpha and
    // agreement are marked invalid, and the learner state must stay as it is
    const uint32_t tag = tag_of_epoch(*a.round_epoch - 1u);
    const uint64_t fw = *a.round_fail;
    if ((uint32_t)fw == tag && (fw >> 32) != 0) {
      mark_query_failed(a, blockIdx.x);
      return;
    }
  }
  tail_query(a, blockIdx.x, lds);
}

int launch_tail(const TailArgs& a, hipStream_t stream) {
  const size_t lds = sizeof(double) * (size_t)tail_lds_doubles(a);
  hs_tail_kernel<<<a.B, 64, lds, stream>>>(a);
  return hipGetLastError() == hipSuccess ? HS_OK : HS_ERR_HIP;
}

}  // namespace hs
