// Delayed feedback (Section 3.3, "HedgeSpec: Loss functions and Delayed Feedback"; Appendix,
// algorithm "Queued Full-Information with Delays"): the token-level length loss
//   f_s[i] = 1 - EAL(gamma_s .. gamma_{s+K-1})[i] / (K + 1)
// (Theorem 3's estimator on the window of K tokens that starts at token s) becomes known only
// once the feedback of all K tokens of its window has arrived. With hybrid losses (Appendix,
// "Practical heuristics") a query's first H tokens take the acceptance loss 1 - gamma_s
// instead, known at once. Each call appends the feedback
// of a query's newest tokens to its history ring and feeds every window that is now complete,
// in token order, to Hedge and NormalHedge before anything else happens: the base learners
// see a delay-free loss stream in their own clock, and a call that completes no window leaves
// them untouched. One wave64 per query, lane i = drafter i, fp64.
#include "hs_learner.h"

namespace hs {

__global__ __launch_bounds__(64) void hs_delayed_kernel(DelayArgs a) {
  // LDS: the window losses [K][N] doubles, the learners' scratch, then the feedback of tokens
  // t_used .. t_new - 1 (at most 2K - 1 of them) as [2K][N] floats
  extern __shared__ double lossv[];
  const int b = blockIdx.x, i = threadIdx.x;
  const int N = a.N, K = a.K, W = 2 * K;
  const bool act = i < N;
  double* scratch = lossv + K * N;
  float* gw = reinterpret_cast<float*>(scratch + kLearnScratch);
  TailArgs st{};  // only the learner-state fields, for load_learner_in
  st.N = N;
  st.M = K;
  st.logw = a.logw;
  st.R = a.R;
  st.p = a.p;
  st.c = a.c;
  const LearnerIn in = load_learner_in(st, b);
  // (a clock that is not a valid state, e.g. never zero-filled, is clamped into range: wrong
  // numbers, but every ring and LDS index stays in bounds)
  const int64_t t_next = max(a.clock[2 * b], (int64_t)0);
  const int64_t t_used = min(t_next, max(a.clock[2 * b + 1], t_next - K));
  const int m = min(max(a.count[b], 0), K);  // counts outside [0, K] are clamped
  float* hb = a.hist + (int64_t)b * W * N;
  const int64_t t_new = t_next + m;
  // the ring holds tokens t_used .. t_next - 1 (at most K of them), the call brings
  // t_next .. t_new - 1 (at most K): at most 2K tokens in all, so no two share a ring slot
  const int nold = (int)(t_next - t_used);
  if (act) {
    for (int j = 0; j < nold; ++j) gw[j * N + i] = hb[(int)((t_used + j) % W) * N + i];
    for (int j = 0; j < m; ++j) {
      const int64_t o = ((int64_t)b * N + i) * K + j;
      const float g = a.gamma_src == 1 ? a.alpha[o] : (float)a.agree[o];
      gw[(nold + j) * N + i] = g;
      hb[(int)((t_next + j) % W) * N + i] = g;
    }
  }
  // the tokens whose loss is known form a prefix of the stream: those before H (acceptance
  // loss) as soon as they arrive, a later token s once its window s .. s+K-1 is in. The new
  // ones are t_used .. ready - 1, at most m of them.
  // (With the same H on every call at most m tokens become ready. If a caller raises H
  // mid-stream more may; taking at most K per call keeps the unused tokens at most K, so the
  // ring of 2K and the LDS buffers always hold them, and the rest follow in later calls.)
  const int64_t H = a.hybrid;
  const int64_t ready = t_new <= H ? t_new : H + max((int64_t)0, t_new - K + 1 - H);
  const int L = (int)min((int64_t)K, max((int64_t)0, ready - t_used));
  for (int l = 0; l < L; ++l) {
    double f;
    if (t_used + l < H) {
      f = 1.0 - (act ? (double)gw[l * N + i] : 0.0);
    } else {
      double pp = 1.0, sp = 0.0;
      for (int j = 0; j < K; ++j) {
        pp *= act ? (double)gw[(l + j) * N + i] : 0.0;
        sp += pp;
      }
      f = 1.0 - (1.0 + sp) / (double)(K + 1);
    }
    if (act) {
      lossv[l * N + i] = f;
      if (a.loss) a.loss[((int64_t)l * a.B + b) * N + i] = f;
    }
  }
  if (L > 0)
    learner_update(a.logw, a.w, a.eta, a.R, a.p, a.c, b, N, L, in, scratch,
                   [&](int l) -> double { return act ? lossv[l * N + i] : 0.0; });
  if (i == 0) {
    a.clock[2 * b] = t_new;
    a.clock[2 * b + 1] = t_used + L;
    if (a.nloss) a.nloss[b] = L;
  }
}

int launch_delayed(const DelayArgs& a, hipStream_t stream) {
  const size_t lds = sizeof(double) * ((size_t)a.K * a.N + kLearnScratch) +
                     sizeof(float) * 2 * (size_t)a.K * a.N;
  hs_delayed_kernel<<<a.B, 64, lds, stream>>>(a);
  return hipGetLastError() == hipSuccess ? HS_OK : HS_ERR_HIP;
}

}  // namespace hs
