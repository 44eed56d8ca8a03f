// hs_candidate_mass: Theorem 2 with EAGLE-2's dynamic pruning. When the draft tree is
// pruned, the acceptance probability at a node is the target's mass on the node's kept
// children rather than on Top_L(q); the caller, which grew and pruned the tree, passes the
// kept children. One wave per output (query, drafter, position): lane j gathers the target
// logit of candidate j (and j + 64, ...), p_v = 2^(z_v c - lse log2 e) with c = log2(e) / T
// and the row's natural-log normaliser lse, and the wave sums them in a fixed order.
// Latency-bound: a few loads per output, against the row statistics the caller already has.
#include "hs_internal.h"
#include "hs_wave.h"

namespace hs {

namespace {

struct CmArgs {
  const char* tptr;    // target logits, row (b, k) at tptr + (b sb + k sk) element_size
  int64_t sb, sk;      // strides in elements
  const float* lse;    // [B][K] natural-log normalisers of the target rows at T
  const int32_t* cand; // [B][N][K][C] token indices; negative = empty slot
  float* gamma;        // [B][N][K]
  int N, K, C;
  int64_t V, rows;     // rows = B N K outputs
  float c;             // log2(e) / T
  FastDiv divK, divN;
};

template <int DT>
__device__ inline float logit_at(const char* row, int64_t v) {
  if constexpr (DT == HS_F32) return reinterpret_cast<const float*>(row)[v];
  else return Vec<DT>::lo(reinterpret_cast<const uint16_t*>(row)[v]);
}

template <int DT>
__global__ __launch_bounds__(kThreads) void hs_cmass_kernel(CmArgs A) {
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t r = (int64_t)blockIdx.x * kWaves + wv;
  if (r >= A.rows) return;  // wave-uniform; no barrier below
  const uint32_t r32 = (uint32_t)r;  // rows < 2^31
  const uint32_t bn = fdiv(r32, A.divK);
  const int k = (int)(r32 - bn * (uint32_t)A.K);
  const int b = (int)fdiv(bn, A.divN);
  const char* row =
      A.tptr + ((int64_t)b * A.sb + (int64_t)k * A.sk) * (int64_t)Vec<DT>::kBytes;
  const float nl = -A.lse[(int64_t)b * A.K + k] * 1.44269504088896340736f;
  const int32_t* cr = A.cand + r * A.C;
  float e = 0.0f;
  bool bad = false;
  for (int j = lane; j < A.C; j += 64) {
    const int32_t v = cr[j];
    if (v >= 0) {
      if (v >= A.V) bad = true;
      else e += __builtin_amdgcn_exp2f(fmaf(logit_at<DT>(row, v), A.c, nl));
    }
  }
  const float tot = wave_sum_f(e);
  const bool any_bad = __ballot(bad) != 0;
  if (lane == 0) A.gamma[r] = any_bad ? NAN : tot;
}

}  // namespace

int launch_candidate_mass(const void* tptr, int64_t sb, int64_t sk, int dtype, int B, int N,
                          int K, int64_t V, int C, float c, const float* lse,
                          const int32_t* cand, float* gamma, hipStream_t stream) {
  CmArgs A;
  A.tptr = reinterpret_cast<const char*>(tptr);
  A.sb = sb;
  A.sk = sk;
  A.lse = lse;
  A.cand = cand;
  A.gamma = gamma;
  A.N = N;
  A.K = K;
  A.C = C;
  A.V = V;
  A.rows = (int64_t)B * N * K;
  A.c = c;
  A.divK = make_fastdiv((uint32_t)K);
  A.divN = make_fastdiv((uint32_t)N);
  const unsigned grid = (unsigned)((A.rows + kWaves - 1) / kWaves);
  if (dtype == HS_F32) hs_cmass_kernel<HS_F32><<<grid, kThreads, 0, stream>>>(A);
  else if (dtype == HS_F16) hs_cmass_kernel<HS_F16><<<grid, kThreads, 0, stream>>>(A);
  else hs_cmass_kernel<HS_BF16><<<grid, kThreads, 0, stream>>>(A);
  return hipGetLastError() == hipSuccess ? HS_OK : HS_ERR_HIP;
}

}  // namespace hs
