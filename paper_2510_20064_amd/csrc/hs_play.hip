// Drafter play and regret bookkeeping, one wave64 per query.
//   hs_play_kernel   : the action of QFI-D's round (Appendix, algorithm "Queued Full-Information
//                      with Delays": play a_t according to p, by its argmax or a sample).
//   hs_regret_kernel : Regret_T = sum_t f_t[i_t] - min_i sum_t f_t[i] (Section 3.1), and the
//                      played drafter's expected accepted length summed over rounds.
// Every sum whose value decides an integer or is compared with a reference runs left to right
// in fp64 (the total and prefix sums of the play over the drafters, the cumulative losses per
// drafter in loss order), so it is reproducible bit for bit.
#include "hs_internal.h"

namespace hs {

namespace {

__device__ inline double lane_d(double x, int l) {
  const uint64_t u = __double_as_longlong(x);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), l);
  return __longlong_as_double(((long long)hi << 32) | lo);
}

// One coalesced load of the query's weights (lane i: drafter i), then every lane walks them
// left to right from broadcasts, so each lane forms the same fp64 sums in the order the
// definition gives.
__global__ __launch_bounds__(64) void hs_play_kernel(const double* w, int B, int N, int how,
                                                     const double* u, int32_t* choice) {
  const int b = blockIdx.x, i = threadIdx.x;
  const double wi = i < N ? w[(int64_t)b * N + i] : 0.0;
  const double ub = how == HS_PLAY_SAMPLE ? u[b] : 0.0;
  double tot = 0.0;
  for (int j = 0; j < N; ++j) tot += lane_d(wi, j);
  int c = -1;
  if (tot > 0.0 && isfinite(tot)) {
    if (how == HS_PLAY_ARGMAX) {
      c = 0;
      double best = lane_d(wi, 0);
      for (int j = 1; j < N; ++j) {
        const double x = lane_d(wi, j);
        if (x > best) {  // strict: the lowest index of the largest weight
          best = x;
          c = j;
        }
      }
    } else {
      // inverse CDF: the smallest i whose prefix sum exceeds u * total
      const double thr = ub * tot;
      double acc = 0.0;
      c = N - 1;  // rounding can leave the last prefix at or below thr
      for (int j = 0; j < N; ++j) {
        acc += lane_d(wi, j);
        if (acc > thr) {
          c = j;
          break;
        }
      }
    }
  }
  if (i == 0) choice[b] = c;
}

__global__ __launch_bounds__(64) void hs_regret_kernel(const double* loss, int L, int B, int N,
                                                       const int32_t* played, double* cum,
                                                       double* played_sum, double* regret,
                                                       const double* eal, double* eal_sum) {
  const int b = blockIdx.x, i = threadIdx.x;
  const bool act = i < N;
  double ci = act ? cum[(int64_t)b * N + i] : 0.0;
  double ps = played_sum[b];
  for (int l = 0; l < L; ++l) {
    const double* f = loss + ((int64_t)l * B + b) * N;
    if (act) ci += f[i];
    const int it = played[(int64_t)l * B + b];
    ps += (it >= 0 && it < N) ? f[it] : NAN;  // every lane the same value, in loss order
  }
  // min over drafters (exact; a NaN counts as +inf, as a failed comparison does)
  double v = act && !isnan(ci) ? ci : INFINITY;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmin(v, __shfl_xor(v, o, 64));
  if (act) cum[(int64_t)b * N + i] = ci;
  if (i == 0) {
    played_sum[b] = ps;
    regret[b] = ps - v;
    if (eal && eal_sum && L > 0) {
      const int it = played[(int64_t)(L - 1) * B + b];
      eal_sum[b] += (it >= 0 && it < N) ? eal[(int64_t)b * N + it] : NAN;
    }
  }
}

}  // namespace

int launch_play(const double* w, int B, int N, int how, const double* u, int32_t* choice,
                hipStream_t stream) {
  hs_play_kernel<<<B, 64, 0, stream>>>(w, B, N, how, u, choice);
  return hipGetLastError() == hipSuccess ? HS_OK : HS_ERR_HIP;
}

int launch_regret(const double* loss, int L, int B, int N, const int32_t* played, double* cum,
                  double* played_sum, double* regret, const double* eal, double* eal_sum,
                  hipStream_t stream) {
  hs_regret_kernel<<<B, 64, 0, stream>>>(loss, L, B, N, played, cum, played_sum, regret, eal,
                                         eal_sum);
  return hipGetLastError() == hipSuccess ? HS_OK : HS_ERR_HIP;
}

}  // namespace hs
