// Per-query learner step, run by one wave64 (lane i = drafter i, N <= 64), all in fp64:
//   gamma       : alpha (speculative sampling, Theorem 1) or argmax agreement (greedy)
//   prefix[n]   : gamma[n] * prefix[parent[n]]   (chain: parent[n] = n - 1)
//   EAL         : 1 + sum of prefix over the path root -> path_end. Summing Theorem 3's
//                 k (1 - gamma_k) prod_{j<k} gamma_j by parts (gamma_{K+1} = 0) gives this form.
//   loss        : HS_LOSS_LENGTH 1 - EAL/(K_path + 1); HS_LOSS_ACCEPT_CHUNK mean of
//                 (1 - gamma) over the path; HS_LOSS_ACCEPT_TOKEN the K vectors 1 - gamma_k
//                 (zero vectors past a chain's k_h = end + 1 verified tokens)
//   Hedge       : logw -= eta * loss for each vector in order; w = softmax(logw)
//   NormalHedge : per vector, R_i += l_A - l_i; c solves (1/N) sum exp([R]_+^2 / 2c) = e;
//                 p_i ~ ([R_i]_+ / c) exp([R_i]_+^2 / 2c)
// The wave is the only user of the query's state (logw, w, R, p, c) within a launch.
#pragma once

#include <math.h>

#include "hs_internal.h"

namespace hs {


// Wave64 reductions of doubles on the DPP network (no LDS crossbar round trip): pairs and
// quads by quad_perm, 8- and 16-lane groups by the half-row and row mirrors, then the four
// row results are read into scalars. Every lane gets the same value; all 64 lanes must be active.
template <int CTRL>
__device__ inline double dpp_d(double x) {
  const long long b = __double_as_longlong(x);
  const int lo = __builtin_amdgcn_mov_dpp((int)b, CTRL, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_mov_dpp((int)(b >> 32), CTRL, 0xF, 0xF, false);
  return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}
__device__ inline double lane_d(double x, int lane) {
  const long long b = __double_as_longlong(x);
  const int lo = __builtin_amdgcn_readlane((int)b, lane);
  const int hi = __builtin_amdgcn_readlane((int)(b >> 32), lane);
  return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}
__device__ inline double wsum(double v) {
  v += dpp_d<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp_d<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp_d<0x141>(v);  // row_half_mirror
  v += dpp_d<0x140>(v);  // row_mirror
  return (lane_d(v, 0) + lane_d(v, 16)) + (lane_d(v, 32) + lane_d(v, 48));
}
__device__ inline double wmax(double v) {
  v = fmax(v, dpp_d<0xB1>(v));
  v = fmax(v, dpp_d<0x4E>(v));
  v = fmax(v, dpp_d<0x141>(v));
  v = fmax(v, dpp_d<0x140>(v));
  return fmax(fmax(lane_d(v, 0), lane_d(v, 16)), fmax(lane_d(v, 32), lane_d(v, 48)));
}

// NormalHedge's scale. With a_i = r_i^2 / 2 and s = 1/c, phi(s) = log((1/N) sum exp(a_i s)) - 1
// is convex and increasing; its root s* lies in [2/M, 2(1+ln N)/M], M = max r_i^2 (at the
// upper end every exponent is <= 1 + ln N, so nothing overflows, and phi >= 0 there). Newton's
// method decreases monotonically to s* from any point right of it (the tangent of a convex
// function lies below it). From a point left of s* the step overshoots to the right; an
// overshoot past the bracket restarts from the bracket's right end instead, so every later
// iterate lies right of s* (bisection would land left again and again: up to 55 iterations
// instead of 6 on random loss streams of 64 drafters). The start is the previous round's scale
// when it lies in the bracket (regrets move little per round), else the right end. Returns s*.
__device__ inline double normalhedge_inv_scale(double a, bool act, int N, double M, double s0) {
  double lo = 2.0 / M;
  const double hi = 2.0 * (1.0 + log((double)N)) / M;
  double s = (s0 > lo && s0 < hi) ? s0 : hi;
  for (int it = 0; it < 100; ++it) {
    const double ex = act ? exp(a * s) : 0.0;
    const double E = wsum(ex);
    const double F = wsum(act ? a * ex : 0.0);
    // near the root (mean exp within 1e-4 of e) Newton's step on psi(s) = E / N - e instead:
    // also convex and increasing, with the same root and sign, and no log to evaluate
    const double Ne = (double)N * 2.718281828459045;
    const double d = E - Ne;
    const bool near = fabs(d) < 1e-4 * Ne;
    const double phi = near ? d : log(E / (double)N) - 1.0;
    if (phi == 0.0 || !(F > 0.0)) break;
    double sn = s - (near ? d / F : phi * E / F);
    if (phi < 0.0) {
      lo = s;
      if (!(sn < hi)) sn = hi;
    } else if (!(sn > lo)) {  // rounding only: a right-side step stays right of s* > lo
      sn = 0.5 * (lo + s);
    }
    const double ds = fabs(sn - s);
    s = sn;
    if (ds <= 4e-16 * s) break;
  }
  return s;
}

// LDS doubles learner_update uses as scratch: p and the loss vector of every drafter.
constexpr int kLearnScratch = 2 * 64;

// LDS doubles tail_query needs: gamma / prefix products [M][N], losses [L][N], then the
// learner's scratch.
__host__ __device__ inline int tail_lds_doubles(const TailArgs& a) {
  if (a.gamma_src == 0) return kLearnScratch;
  const int L = a.loss_kind == HS_LOSS_ACCEPT_TOKEN ? a.M : 1;
  return a.M * a.N + L * a.N + kLearnScratch;
}

// The state the learner step of query b reads (lane i: drafter i), loaded before the step
// so that the loads can fly while gamma is gathered.
struct LearnerIn {
  double lw0, R0, p0, c_prev;
  int end;
};
__device__ __forceinline__ LearnerIn load_learner_in(const TailArgs& a, int b) {
  const int i = threadIdx.x & 63;
  const bool act = i < a.N;
  const int64_t si = (int64_t)b * a.N + i;
  LearnerIn s;
  s.lw0 = (a.logw && act) ? a.logw[si] : 0.0;
  s.R0 = (a.R && act) ? a.R[si] : 0.0;
  s.p0 = (a.R && act) ? a.p[si] : 0.0;
  s.c_prev = a.R ? a.c[b] : 0.0;  // warm start of the scale search
  s.end = (a.gamma_src != 0 && a.path_end) ? a.path_end[b] : a.M - 1;
  return s;
}

// The base learners of query b take the L loss vectors loss_at(0 .. L-1) in order (lane i:
// drafter i, all 64 lanes of the wave; `in` holds the state as loaded by load_learner_in;
// scratch: kLearnScratch doubles of LDS used by this wave only):
//   Hedge       : logw -= eta * loss for each vector; w = softmax(logw) (logw and w may be NULL)
//   NormalHedge : per vector, R_i += l_A - l_i, c solves the scale equation, p from R and c
//                 (R, p and c may be NULL)
template <typename LossAt>
__device__ __forceinline__ void learner_update(double* logw, double* w, double eta, double* R,
                                               double* p, double* c, int b, int N, int L,
                                               const LearnerIn& in, double* scratch,
                                               LossAt loss_at) {
  const int i = threadIdx.x & 63;
  const bool act = i < N;
  // ---- Hedge ----
  if (logw) {
    double lw = act ? in.lw0 : -INFINITY;
    for (int l = 0; l < L; ++l) lw -= eta * loss_at(l);
    const double mx = wmax(act ? lw : -INFINITY);
    const double e = act ? exp(lw - mx) : 0.0;
    const double se = wsum(e);
    if (act) {
      logw[(int64_t)b * N + i] = lw - mx;
      w[(int64_t)b * N + i] = e / se;
    }
  }

  // ---- NormalHedge ----
  if (R) {
    double Rv = in.R0;
    double pv = in.p0;
    double cc = 0.0;
    for (int l = 0; l < L; ++l) {
      const double li = loss_at(l);
      // l_A - l_i as sum_j p_j (l_j - l_i): equal to it because sum_j p_j = 1, and exactly
      // zero when every drafter that carries weight has this drafter's loss. Every lane reads
      // all (p_j, l_j) from LDS (the wave's own writes: LDS operations of a wave execute in
      // order), in four interleaved partial sums combined in a fixed order.
      scratch[i] = pv;
      scratch[64 + i] = li;
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      double d0 = 0.0, d1 = 0.0, d2 = 0.0, d3 = 0.0;
      int j = 0;
      for (; j + 4 <= N; j += 4) {
        d0 += scratch[j] * (scratch[64 + j] - li);
        d1 += scratch[j + 1] * (scratch[64 + j + 1] - li);
        d2 += scratch[j + 2] * (scratch[64 + j + 2] - li);
        d3 += scratch[j + 3] * (scratch[64 + j + 3] - li);
      }
      for (; j < N; ++j) d0 += scratch[j] * (scratch[64 + j] - li);
      const double dR = (d0 + d1) + (d2 + d3);
      __builtin_amdgcn_wave_barrier();  // every lane has read before the next vector's writes
      if (act) Rv += dR;
      const double r = (act && Rv > 0.0) ? Rv : 0.0;
      const double M2 = wmax(r * r);
      if (!(M2 > 0.0)) {
        pv = act ? 1.0 / (double)N : 0.0;
        cc = 0.0;
        continue;
      }
      const double ai = 0.5 * r * r;
      const double s = normalhedge_inv_scale(
          ai, act, N, M2, cc > 0.0 ? 1.0 / cc : (in.c_prev > 0.0 ? 1.0 / in.c_prev : 0.0));
      const double u = act ? r * exp(ai * s) : 0.0;
      const double su = wsum(u);
      pv = u / su;
      cc = 1.0 / s;
    }
    if (act) {
      R[(int64_t)b * N + i] = Rv;
      p[(int64_t)b * N + i] = pv;
    }
    if (i == 0) c[b] = cc;
  }
}

// Outputs of query b when its step is skipped because its gamma depends on a word the
// evaluation lost: EAL, prefix products and losses NaN; the learner state is not touched.
// Run by all 64 lanes of one wave.
__device__ inline void mark_query_failed(const TailArgs& a, int b) {
  const int i = threadIdx.x & 63;
  if (i >= a.N || a.gamma_src == 0) return;
  const int64_t qi = (int64_t)b * a.N + i;
  a.eal[qi] = NAN;
  if (a.prefix)
    for (int n = 0; n < a.M; ++n) a.prefix[qi * a.M + n] = NAN;
  if (a.loss_out) {
    const int L = a.loss_kind == HS_LOSS_ACCEPT_TOKEN ? a.M : 1;
    for (int l = 0; l < L; ++l) a.loss_out[((int64_t)l * a.B + b) * a.N + i] = NAN;
  }
}

// Learner step for query b, executed by all 64 lanes of one wave (uniform control flow).
// gamma_lds (optional): the query's gamma as [N][M] floats in LDS, instead of a.alpha / a.agree.
// pre (optional): the state, already loaded by load_learner_in.
// Every input is loaded before anything is stored, so the loads are in flight together.
__device__ __forceinline__ void tail_query(const TailArgs& a, int b, double* lds,
                                           const float* gamma_lds = nullptr,
                                           const LearnerIn* pre = nullptr) {
  const int i = threadIdx.x & 63;
  const int N = a.N, M = a.M;
  const bool act = i < N;
  double* gam = lds;            // [M][N]: gamma, then prefix products
  double* lossv = lds + M * N;  // [L][N]
  int L = a.L;

  const LearnerIn in = pre ? *pre : load_learner_in(a, b);
  const int end = in.end;

  if (a.gamma_src != 0) {
    const bool ok = end >= 0 && end < M;
    double sum1mg = 0.0, eal = NAN;
    int len = 0;
    auto gamma_at = [&](int n) -> double {
      const int64_t o = ((int64_t)b * N + i) * M + n;
      return gamma_lds ? (double)gamma_lds[i * M + n]
                       : (a.gamma_src == 1) ? (double)a.alpha[o] : (double)a.agree[o];
    };
    if (act && !a.tree) {
      // chain: one pass in position order, the prefix product carried in a register
      double pp = 1.0, sp = 0.0;
      for (int n = 0; n < M; ++n) {
        const double g = gamma_at(n);
        // one token loss per verified token of the chunk (k_h = end + 1 of them), zero
        // vectors (no change to either learner) after them
        if (a.loss_kind == HS_LOSS_ACCEPT_TOKEN) lossv[n * N + i] = !ok ? NAN : n <= end ? 1.0 - g : 0.0;
        pp *= g;
        if (a.prefix) a.prefix[((int64_t)b * N + i) * M + n] = pp;
        if (n <= end) {
          sp += pp;
          sum1mg += 1.0 - g;
        }
      }
      len = ok ? end + 1 : 0;
      if (ok) eal = 1.0 + sp;
      a.eal[(int64_t)b * N + i] = eal;
      if (a.loss_kind == HS_LOSS_LENGTH)
        lossv[i] = ok ? 1.0 - eal / (double)(len + 1) : NAN;
      else if (a.loss_kind == HS_LOSS_ACCEPT_CHUNK)
        lossv[i] = ok ? sum1mg / (double)len : NAN;
    } else if (act) {
      for (int n = 0; n < M; ++n) gam[n * N + i] = gamma_at(n);
      if (ok)
        for (int n = end; n >= 0; n = a.tree ? a.parent[n] : n - 1) {
          sum1mg += 1.0 - gam[n * N + i];
          ++len;
        }
      if (a.loss_kind == HS_LOSS_ACCEPT_TOKEN)
        for (int n = 0; n < M; ++n) lossv[n * N + i] = 1.0 - gam[n * N + i];
      // prefix products in node order (a parent precedes its children)
      for (int n = 0; n < M; ++n) {
        const int pn = a.tree ? a.parent[n] : n - 1;
        const double pp = pn >= 0 ? gam[pn * N + i] : 1.0;
        gam[n * N + i] = gam[n * N + i] * pp;
      }
      if (ok) {
        double sp = 0.0;
        for (int n = end; n >= 0; n = a.tree ? a.parent[n] : n - 1) sp += gam[n * N + i];
        eal = 1.0 + sp;
      }
      a.eal[(int64_t)b * N + i] = eal;
      if (a.prefix)
        for (int n = 0; n < M; ++n) a.prefix[((int64_t)b * N + i) * M + n] = gam[n * N + i];
      if (a.loss_kind == HS_LOSS_LENGTH)
        lossv[i] = ok ? 1.0 - eal / (double)(len + 1) : NAN;
      else if (a.loss_kind == HS_LOSS_ACCEPT_CHUNK)
        lossv[i] = ok ? sum1mg / (double)len : NAN;
    }
    L = (a.loss_kind == HS_LOSS_ACCEPT_TOKEN) ? M : 1;
    if (a.loss_out && act)
      for (int l = 0; l < L; ++l) a.loss_out[((int64_t)l * a.B + b) * N + i] = lossv[l * N + i];
  }

  auto loss_at = [&](int l) -> double {
    if (!act) return 0.0;
    if (a.gamma_src != 0) return lossv[l * N + i];
    return a.loss_in[((int64_t)l * a.B + b) * N + i];
  };
  learner_update(a.logw, a.w, a.eta, a.R, a.p, a.c, b, N, L, in,
                 lds + tail_lds_doubles(a) - kLearnScratch, loss_at);
}

}  // namespace hs
