// Learner kernel: acceptance length, loss, Hedge and NormalHedge for one query per wave64.
//
// Lane i owns drafter i (N <= 64). Everything is fp64; the per-query state
// (log-weights, regrets, NormalHedge distribution) stays in device memory between rounds.
//   gamma        : alpha (speculative sampling, Theorem 1) or argmax agreement (greedy)
//   prefix[n]    : gamma[n] * prefix[parent[n]]   (chain: parent[n] = n - 1)
//   EAL          : 1 + sum of prefix over the path root -> path_end, which equals Theorem 3's
//                  sum_{k=1}^{K+1} k (1 - gamma_k) prod_{j<k} gamma_j with gamma_{K+1} = 0
//   loss         : length, token-level acceptance, or chunk acceptance (HS_LOSS_*)
//   Hedge        : logw -= eta * loss per vector, w = softmax(logw)
//   NormalHedge  : regret update R_i += l_A - l_i, scale c from (1/N) sum exp(r^2 / 2c) = e,
//                  p ~ (r/c) exp(r^2/2c)
#include <math.h>

#include "hs_internal.h"

namespace hs {

__device__ inline double wsum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ inline double wmax(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o, 64));
  return v;
}

// NormalHedge's scale. With a_i = r_i^2 / 2 and s = 1/c, phi(s) = log((1/N) sum exp(a_i s)) - 1
// is convex and increasing; its root s* lies in [2/M, 2(1 + ln N)/M], M = max r_i^2 (at the
// upper end every exponent is <= 1 + ln N). Newton's method started at the upper end moves
// monotonically down to s* (the tangent of a convex function lies below it), converging
// quadratically. Returns s*.
__device__ inline double normalhedge_inv_scale(double a, bool act, int N, double M) {
  double s = 2.0 * (1.0 + log((double)N)) / M;
  for (int it = 0; it < 100; ++it) {
    double ex = act ? exp(a * s) : 0.0;
    double E = wsum(ex);
    double F = wsum(act ? a * ex : 0.0);
    double phi = log(E / (double)N) - 1.0;
    if (!(phi > 0.0) || !(F > 0.0)) break;
    double ds = phi * E / F;
    double sn = s - ds;
    if (!(sn < s) || !(sn > 0.0)) break;
    s = sn;
    if (ds <= 1e-16 * s) break;
  }
  return s;
}

__global__ __launch_bounds__(64) void hs_tail_kernel(TailArgs a) {
  const int b = blockIdx.x;
  const int i = threadIdx.x;
  const bool act = i < a.N;
  const int M = a.M;
  __shared__ double gam[HS_MAX_POSITIONS][64];   // gamma, then prefix products, [node][lane]
  __shared__ double lossv[HS_MAX_POSITIONS][64]; // loss vectors [l][lane]
  int L = a.L;

  if (a.gamma_src != 0) {
    // gamma of this lane's drafter at every node
    for (int n = 0; n < M; ++n) {
      double g = 0.0;
      if (act) {
        const int64_t o = ((int64_t)b * a.N + i) * M + n;
        g = (a.gamma_src == 1) ? (double)a.alpha[o] : (double)a.agree[o];
      }
      gam[n][i] = g;
    }
    const int end = a.path_end ? a.path_end[b] : M - 1;
    const bool ok = end >= 0 && end < M;
    // loss terms that need the raw gamma along the path
    double sum1mg = 0.0;
    int len = 0;
    if (ok) {
      for (int n = end; n >= 0; n = a.tree ? a.parent[n] : n - 1) {
        sum1mg += 1.0 - gam[n][i];
        ++len;
      }
    }
    if (a.loss_kind == HS_LOSS_ACCEPT_TOKEN) {
      for (int n = 0; n < M; ++n) lossv[n][i] = 1.0 - gam[n][i];
    }
    // prefix products in node order (parents precede children)
    for (int n = 0; n < M; ++n) {
      const int pn = a.tree ? a.parent[n] : n - 1;
      const double pp = pn >= 0 ? gam[pn][i] : 1.0;
      gam[n][i] = gam[n][i] * pp;
    }
    double eal = NAN;
    if (ok) {
      double sp = 0.0;
      for (int n = end; n >= 0; n = a.tree ? a.parent[n] : n - 1) sp += gam[n][i];
      eal = 1.0 + sp;
    }
    if (act) {
      a.eal[(int64_t)b * a.N + i] = eal;
      if (a.prefix)
        for (int n = 0; n < M; ++n) a.prefix[((int64_t)b * a.N + i) * M + n] = gam[n][i];
    }
    if (a.loss_kind == HS_LOSS_LENGTH) {
      lossv[0][i] = ok ? 1.0 - eal / (double)(len + 1) : NAN;
      L = 1;
    } else if (a.loss_kind == HS_LOSS_ACCEPT_CHUNK) {
      lossv[0][i] = ok ? sum1mg / (double)len : NAN;
      L = 1;
    } else {
      L = M;
    }
    if (!act)
      for (int l = 0; l < L; ++l) lossv[l][i] = 0.0;
    if (a.loss_out && act)
      for (int l = 0; l < L; ++l) a.loss_out[((int64_t)l * a.B + b) * a.N + i] = lossv[l][i];
  }

  auto loss_at = [&](int l) -> double {
    if (a.gamma_src != 0) return lossv[l][i];
    return act ? a.loss_in[((int64_t)l * a.B + b) * a.N + i] : 0.0;
  };

  // ---- Hedge ----
  if (a.logw) {
    double lw = act ? a.logw[(int64_t)b * a.N + i] : -INFINITY;
    for (int l = 0; l < L; ++l) lw -= a.eta * loss_at(l);
    const double mx = wmax(act ? lw : -INFINITY);
    const double e = act ? exp(lw - mx) : 0.0;
    const double se = wsum(e);
    if (act) {
      a.logw[(int64_t)b * a.N + i] = lw - mx;
      a.w[(int64_t)b * a.N + i] = e / se;
    }
  }

  // ---- NormalHedge ----
  if (a.R) {
    double Rv = act ? a.R[(int64_t)b * a.N + i] : 0.0;
    double pv = act ? a.p[(int64_t)b * a.N + i] : 0.0;
    double cc = 0.0;
    for (int l = 0; l < L; ++l) {
      const double li = loss_at(l);
      // l_A - l_i as sum_j p_j (l_j - l_i): equal to it because sum_j p_j = 1, and exactly
      // zero when every drafter that carries weight has this drafter's loss
      double dR = 0.0;
      for (int j = 0; j < a.N; ++j) dR += __shfl(pv, j, 64) * (__shfl(li, j, 64) - li);
      if (act) Rv += dR;
      const double r = (act && Rv > 0.0) ? Rv : 0.0;
      const double M2 = wmax(r * r);
      if (!(M2 > 0.0)) {
        pv = act ? 1.0 / (double)a.N : 0.0;
        cc = 0.0;
        continue;
      }
      const double ai = 0.5 * r * r;
      const double s = normalhedge_inv_scale(ai, act, a.N, M2);
      const double u = act ? r * exp(ai * s) : 0.0;
      const double su = wsum(u);
      pv = u / su;
      cc = 1.0 / s;
    }
    if (act) {
      a.R[(int64_t)b * a.N + i] = Rv;
      a.p[(int64_t)b * a.N + i] = pv;
    }
    if (i == 0) a.c[b] = cc;
  }
}

int launch_tail(const TailArgs& a, hipStream_t stream) {
  hs_tail_kernel<<<a.B, 64, 0, stream>>>(a);
  return hipGetLastError() == hipSuccess ? HS_OK : HS_ERR_HIP;
}

}  // namespace hs
