/*
 * Float64 CPU oracle for the HedgeSpec drafter-evaluation path.
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product path may link, load or call
 * this file; only the tests, the smoke check and the bench's CPU-baseline leg do.
 * It shares no code, header or constant with the GPU library: the only thing
 * both sides share is the input bytes written by the seeded generator.
 *
 * Every routine is the plain definition from the paper (arXiv 2510.20064),
 * evaluated in fp64 with straightforward loops, no blocking and no reordering
 * beyond what the definition states. Each routine names the passage it follows.
 * Built with -O2 -fno-fast-math -ffp-contract=off.
 *
 * Parity status of each routine (pins live in the CPU test suite):
 *   or_decode               : pinned (every fp16 bit pattern against numpy's binary16 type;
 *                             fp16 inputs give exactly the fp32 results for the same values).
 *   or_row_stats, or_alpha  : pinned (identities of Theorem 1, closed form for a
 *                             boosted token, brute-force enumeration of the
 *                             speculative-decoding box, disjoint supports).
 *   or_eal_path, or_accept_len : pinned (Theorem 3 against brute force,
 *                             worked example of the censoring appendix, constant-gamma
 *                             closed form, range [1, K+1]).
 *   or_topl                 : pinned (closed-form top-L masses of a target built from a
 *                             known distribution, full vocabulary gives 1, brute-force
 *                             enumeration of the dominating L-subset, ties and signed
 *                             zeros by index, invariance under exact rescaling of the
 *                             drafter, L = 1 greedy hit equals argmax agreement).
 *   or_candidate_mass       : pinned (the kept children equal to Top_L reproduce or_topl's
 *                             mass, every token gives 1, no token 0, a target built from a
 *                             known distribution gives that distribution's mass).
 *   or_hybrid_losses        : pinned (H = 0 is the window loss, H >= T the acceptance loss,
 *                             the appendix's K = 8 example with a first chunk of 4 tokens).
 *   or_play                 : pinned (point masses, empirical frequencies on a uniform grid
 *                             of draws, argmax ties by index, zero rows).
 *   or_regret_update        : pinned (hand-computed stream, always playing one drafter,
 *                             chunked updates equal one update, the played EAL sum).
 *   or_window_losses        : pinned (all-accept and all-reject windows, K = 1, constant
 *                             gamma geometric sum, the censoring appendix's worked example).
 *   or_hedge                : pinned (closed form w ~ exp(-eta * cumulative loss),
 *                             Hedge's expected-regret bound ln N / eta + eta T / 8).
 *   or_normalhedge          : pinned (closed-form c for one or m equal positive
 *                             regrets, scale covariance, sum_i p_i dR_i = 0, and
 *                             the weights equal the normalised gradient in R of the
 *                             scale equation's left side at the solved c, taken by
 *                             finite differences, with several distinct regrets).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_F32 0
#define OR_BF16 1
#define OR_F16 2

#define OR_LOSS_LENGTH 0
#define OR_LOSS_ACCEPT_TOKEN 1
#define OR_LOSS_ACCEPT_CHUNK 2

/*
 * Exact decode of one stored logit to fp64: bf16 is the top half of an fp32; fp16 (the
 * precision the paper's models were served in, Section "Experiment setup and baselines") is
 * IEEE 754 binary16: 1 sign bit, 5 exponent bits with bias 15, 10 fraction bits; exponent
 * field 0 holds zero and the subnormals f 2^-24, field 31 infinity (f = 0) and NaN.
 */
static double or_decode(const void* base, int dtype, int64_t idx) {
  if (dtype == OR_F32) return (double)((const float*)base)[idx];
  if (dtype == OR_F16) {
    const uint16_t h = ((const uint16_t*)base)[idx];
    const int ex = (h >> 10) & 0x1F, fr = h & 0x3FF;
    const double sg = (h & 0x8000) ? -1.0 : 1.0;
    if (ex == 0x1F) return fr ? NAN : sg * INFINITY;
    if (ex == 0) return sg * ldexp((double)fr, -24);
    return sg * ldexp(1024.0 + fr, ex - 25);
  }
  uint32_t u = (uint32_t)((const uint16_t*)base)[idx] << 16;
  float f;
  memcpy(&f, &u, 4);
  return (double)f;
}

/*
 * Row statistics of a temperature softmax p = softmax(z / T).
 *   max    : max_v z_v
 *   argmax : the lowest v with z_v = max (left-to-right scan, strict >)
 *   lse    : log sum_v exp(z_v / T) = max/T + log sum_v exp((z_v - max)/T)
 * Greedy decoding picks the argmax of the raw logits, so the argmax does not
 * depend on T. A row whose entries are all -inf has no distribution (lse = NaN).
 */
void or_row_stats(const void* row, int dtype, int64_t V, double T, double* max_out,
                  int64_t* argmax_out, double* lse_out) {
  double m = -INFINITY;
  int64_t am = 0;
  for (int64_t v = 0; v < V; ++v) {
    double z = or_decode(row, dtype, v);
    if (z > m) {
      m = z;
      am = v;
    }
  }
  double s = 0.0;
  for (int64_t v = 0; v < V; ++v) s += exp((or_decode(row, dtype, v) - m) / T);
  if (max_out) *max_out = m;
  if (argmax_out) *argmax_out = am;
  if (lse_out) *lse_out = (m == -INFINITY) ? NAN : m / T + log(s);
}

/*
 * Acceptance probability of speculative sampling (Theorem 1, Leviathan et al.
 * Thm 3.5, restated in Section 2.2): alpha = sum_v min(p(v), q(v)) = 1 - TV(p, q),
 * with p = softmax(z_t / T) and q = softmax(z_i / T). Clamped to [0, 1].
 * lse_t / lse_i are the row log-normalisers from or_row_stats. Theorem 1 takes two
 * distributions: a row with no finite logit has none (lse = NaN), and alpha is NaN.
 */
double or_alpha(const void* zt, const void* zi, int dtype, int64_t V, double T, double lse_t,
                double lse_i) {
  if (isnan(lse_t) || isnan(lse_i)) return NAN;
  double a = 0.0;
  for (int64_t v = 0; v < V; ++v) {
    double p = exp(or_decode(zt, dtype, v) / T - lse_t);
    double q = exp(or_decode(zi, dtype, v) / T - lse_i);
    a += (p < q) ? p : q;
  }
  if (a < 0.0) a = 0.0;
  if (a > 1.0) a = 1.0;
  return a;
}

/*
 * Evaluation of all drafters on G (query, position) groups.
 * logits : [R][G][ld] stored logits, R = N + 1, row 0 = target, row 1 + i = drafter i.
 * Outputs (any may be NULL):
 *   alpha  [G][N]  : or_alpha of (target, drafter i)            (Theorem 1)
 *   agree  [G][N]  : 1 if argmax target == argmax drafter i       (greedy form of Theorem 1)
 *   argmax [G][R]  : argmax of every row
 *   rmax, rlse [G][R] : row max and log-normaliser
 * want_alpha = 0 skips the softmax work (greedy indicators only).
 */
int or_eval(const void* logits, int dtype, int64_t ld, int R, int64_t G, int64_t V, double T,
            int want_alpha, double* alpha, uint8_t* agree, int64_t* argmax, double* rmax,
            double* rlse) {
  if (R < 2 || G < 1 || V < 1 || ld < V) return -1;
  if (want_alpha && !(T > 0.0)) return -2;
  int N = R - 1;
  double* lse = (double*)malloc(sizeof(double) * (size_t)(R * G));
  double* mx = (double*)malloc(sizeof(double) * (size_t)(R * G));
  int64_t* am = (int64_t*)malloc(sizeof(int64_t) * (size_t)(R * G));
  double Ts = want_alpha ? T : 1.0;
  size_t es = (dtype == OR_F32) ? 4 : 2;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t x = 0; x < (int64_t)R * G; ++x) {
    int64_t r = x / G, g = x % G;
    const char* row = (const char*)logits + (size_t)((r * G + g) * ld) * es;
    or_row_stats(row, dtype, V, Ts, &mx[g * R + r], &am[g * R + r], &lse[g * R + r]);
  }
  if (want_alpha && alpha) {
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t x = 0; x < (int64_t)N * G; ++x) {
      int64_t g = x / N;
      int i = (int)(x % N);
      const char* zt = (const char*)logits + (size_t)((0 * G + g) * ld) * es;
      const char* zi = (const char*)logits + (size_t)(((1 + i) * G + g) * ld) * es;
      alpha[g * N + i] = or_alpha(zt, zi, dtype, V, T, lse[g * R + 0], lse[g * R + 1 + i]);
    }
  }
  for (int64_t g = 0; g < G; ++g) {
    for (int r = 0; r < R; ++r) {
      if (argmax) argmax[g * R + r] = am[g * R + r];
      if (rmax) rmax[g * R + r] = mx[g * R + r];
      if (rlse) rlse[g * R + r] = want_alpha ? lse[g * R + r] : NAN;
    }
    if (agree)
      for (int i = 0; i < N; ++i) agree[g * N + i] = (uint8_t)(am[g * R + 0] == am[g * R + 1 + i]);
  }
  free(lse);
  free(mx);
  free(am);
  return 0;
}

/*
 * EAGLE acceptance probability (Theorem 2, proof in the appendix "Theorem 2 proof"):
 * the greedy draft tree gives the node reached after the verified prefix the L children
 * Top_L(q), the L tokens that the drafter ranks highest, and the next token is accepted
 * when the target's sample is one of them:
 *   gamma = sum_{v in Top_L(q)} p(v),   p = softmax(z_t / T).
 * The drafter's ranking is that of its raw logits (a softmax at any temperature keeps it).
 * Equal logits rank by lower token index first, as for the greedy argmax; -0 equals +0.
 * Top_L is taken by L passes over the row, each picking the best unpicked token.
 * Greedy decoding (one-hot p at the target's argmax): hit = 1 if that argmax is in Top_L.
 *   logits     : [R][G][ld] as in or_eval (row 0 target, row 1 + i drafter i).
 *   gamma      : [G][N] (when want_mass; needs T > 0), hit: [G][N], idx: [G][N][L] (Top_L in
 *                rank order). Any output may be NULL.
 */
int or_topl(const void* logits, int dtype, int64_t ld, int R, int64_t G, int64_t V, int L,
            double T, int want_mass, double* gamma, uint8_t* hit, int32_t* idx) {
  if (R < 2 || G < 1 || V < 1 || ld < V || L < 1 || L > V) return -1;
  if (want_mass && !(T > 0.0)) return -2;
  int N = R - 1;
  size_t es = (dtype == OR_F32) ? 4 : 2;
  int rc = 0;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t x = 0; x < (int64_t)N * G; ++x) {
    int64_t g = x / N;
    int i = (int)(x % N);
    const char* zt = (const char*)logits + (size_t)((0 * G + g) * ld) * es;
    const char* zq = (const char*)logits + (size_t)(((1 + i) * G + g) * ld) * es;
    uint8_t* picked = (uint8_t*)calloc((size_t)V, 1);
    int64_t* top = (int64_t*)malloc(sizeof(int64_t) * (size_t)L);
    if (!picked || !top) {
      rc = -3;
    } else {
      for (int r = 0; r < L; ++r) {
        int64_t best = -1;
        double qb = 0.0;
        for (int64_t v = 0; v < V; ++v) {
          if (picked[v]) continue;
          double q = or_decode(zq, dtype, v);
          if (best < 0 || q > qb) {
            best = v;
            qb = q;
          }
        }
        picked[best] = 1;
        top[r] = best;
      }
      double m, lse;
      int64_t am;
      or_row_stats(zt, dtype, V, want_mass ? T : 1.0, &m, &am, &lse);
      if (want_mass && gamma) {
        double s = 0.0, in = 0.0;
        for (int64_t v = 0; v < V; ++v) s += exp((or_decode(zt, dtype, v) - m) / T);
        for (int r = 0; r < L; ++r) in += exp((or_decode(zt, dtype, top[r]) - m) / T);
        gamma[g * N + i] = in / s;
      }
      if (hit) hit[g * N + i] = picked[am];
      if (idx)
        for (int r = 0; r < L; ++r) idx[(g * N + i) * L + r] = (int32_t)top[r];
    }
    free(picked);
    free(top);
  }
  return rc;
}

/*
 * Theorem 2 with EAGLE-2's dynamic pruning: when the draft tree is pruned, the acceptance
 * probability at a node is the target's mass on the node's kept children instead of on
 * Top_L(q). Here the kept children are given: for group g (a query and position) and drafter
 * i, cand[(g * N + i) * C + j], j < C, lists token indices; a negative entry is an empty slot,
 * and each listed index counts once per listing. gamma[g * N + i] = sum over the listed v of
 * softmax(z_t / T)_v, with z_t the target row of group g; an index >= V makes it NaN.
 *   target : [G][ld] stored logits, one target row per group.
 */
int or_candidate_mass(const void* target, int dtype, int64_t ld, int64_t G, int64_t V, int N,
                      int C, const int32_t* cand, double T, double* gamma) {
  if (G < 1 || V < 1 || ld < V || N < 1 || C < 1 || !(T > 0.0)) return -1;
  size_t es = (dtype == OR_F32) ? 4 : 2;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t g = 0; g < G; ++g) {
    const char* zt = (const char*)target + (size_t)(g * ld) * es;
    double m, lse;
    int64_t am;
    or_row_stats(zt, dtype, V, T, &m, &am, &lse);
    for (int i = 0; i < N; ++i) {
      double s = 0.0;
      for (int j = 0; j < C; ++j) {
        int32_t v = cand[(g * N + i) * C + j];
        if (v < 0) continue;
        if (v >= V) {
          s = NAN;
          break;
        }
        s += exp(or_decode(zt, dtype, v) / T - lse);
      }
      gamma[g * N + i] = s;
    }
  }
  return 0;
}

/* Row statistics of `rows` rows of a [rows][ld] tensor (one temperature softmax each). */
int or_softmax_stats(const void* x, int dtype, int64_t rows, int64_t V, int64_t ld, double T,
                     double* rmax, int64_t* rargmax, double* rlse) {
  if (rows < 1 || V < 1 || ld < V || !(T > 0.0)) return -1;
  size_t es = (dtype == OR_F32) ? 4 : 2;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t r = 0; r < rows; ++r)
    or_row_stats((const char*)x + (size_t)(r * ld) * es, dtype, V, T, &rmax[r], &rargmax[r],
                 &rlse[r]);
  return 0;
}

/*
 * The node path root -> end of a draft tree given by parent pointers
 * (parent[0] = -1, parent[n] < n). Node n carries the feedback gamma of the
 * token that follows the prefix ending at n (Section 3.2: gamma_{j,i} for the
 * j-th verified position). Writes the path root first; returns its length.
 */
int or_path(const int32_t* parent, int M, int end, int32_t* path) {
  int len = 0;
  int32_t tmp[4096];
  for (int n = end; n >= 0; n = parent[n]) {
    if (len >= 4096 || n >= M) return -1;
    tmp[len++] = n;
  }
  for (int j = 0; j < len; ++j) path[j] = tmp[len - 1 - j];
  return len;
}

/*
 * Theorem 3 (one-step counterfactual AcceptLength estimator), taken literally:
 *   EAL = sum_{k=1}^{K+1} k (1 - gamma_k) prod_{j=1}^{k-1} gamma_j,  gamma_{K+1} = 0.
 * gamma[0..K-1] holds gamma_1..gamma_K. The value lies in [1, K+1] (Section 3.2).
 */
double or_eal_path(const double* gamma, int K) {
  double eal = 0.0;
  for (int k = 1; k <= K + 1; ++k) {
    double gk = (k <= K) ? gamma[k - 1] : 0.0;
    double prod = 1.0;
    for (int j = 1; j <= k - 1; ++j) prod *= gamma[j - 1];
    eal += (double)k * (1.0 - gk) * prod;
  }
  return eal;
}

/*
 * Token-level length loss (Section 3.3, "HedgeSpec: Loss functions and Delayed Feedback"):
 * for token s and drafter i, f_s[i] = 1 - EAL(gamma_s .. gamma_{s+K-1})[i] / (K + 1), i.e.
 * Theorem 3's estimator on the window of K tokens that starts at s (the window's (K+1)-th
 * term takes gamma := 0, as in the chunk definition above).
 * gamma: [T][N] token stream; loss: [T - K + 1][N], one vector per complete window in token
 * order. Returns the number of windows (0 when T < K).
 */
int or_window_losses(const double* gamma, int T, int N, int K, double* loss) {
  int nw = T - K + 1;
  if (nw < 0) nw = 0;
  double g[4096];
  for (int s = 0; s < nw; ++s)
    for (int i = 0; i < N; ++i) {
      for (int j = 0; j < K; ++j) g[j] = gamma[(size_t)(s + j) * N + i];
      loss[(size_t)s * N + i] = 1.0 - or_eal_path(g, K) / (double)(K + 1);
    }
  return nw;
}

/*
 * Hybrid losses (Appendix "Practical heuristics: hybrid losses, skipping update"): the first H
 * tokens of a stream take the acceptance-probability loss 1 - gamma_s, known as soon as token
 * s's feedback is in; later tokens take the token-level length loss of or_window_losses, known
 * once the K tokens of their window are in. gamma: [T][N]; loss: [T][N]. Writes, in token
 * order, the losses of every token whose loss is known after T tokens and returns their number
 * (they form a prefix of the stream: min(T, H) + max(0, T - K + 1 - H) when T > H).
 */
int or_hybrid_losses(const double* gamma, int T, int N, int K, int64_t H, double* loss) {
  int n = 0;
  for (int s = 0; s < T; ++s) {
    if (s < H) {
      for (int i = 0; i < N; ++i) loss[(size_t)n * N + i] = 1.0 - gamma[(size_t)s * N + i];
    } else {
      if (s + K > T) break;
      double g[4096];
      for (int i = 0; i < N; ++i) {
        for (int j = 0; j < K; ++j) g[j] = gamma[(size_t)(s + j) * N + i];
        loss[(size_t)n * N + i] = 1.0 - or_eal_path(g, K) / (double)(K + 1);
      }
    }
    ++n;
  }
  return n;
}

/*
 * Drafter play (Appendix, algorithm QFI-D: play action a_t according to p, by sampling from p
 * or by taking its argmax). weights: [B][N], non-negative, not necessarily normalised.
 *   how = 0: choice = the lowest index of the largest weight;
 *   how = 1: choice = the smallest i with w_0 + ... + w_i > u[b] (w_0 + ... + w_{N-1}), the
 *            prefix sums taken left to right; u[b] in [0, 1) is the query's uniform draw.
 * A row whose weights sum to 0 (or are not finite) gives -1.
 */
void or_play(const double* weights, int B, int N, int how, const double* u, int32_t* choice) {
  for (int b = 0; b < B; ++b) {
    const double* w = weights + (size_t)b * N;
    double tot = 0.0;
    for (int i = 0; i < N; ++i) tot += w[i];
    int c = -1;
    if (tot > 0.0 && isfinite(tot)) {
      if (how == 0) {
        c = 0;
        for (int i = 1; i < N; ++i)
          if (w[i] > w[c]) c = i;
      } else {
        const double thr = u[b] * tot;
        double acc = 0.0;
        c = N - 1;  /* rounding can leave the last prefix at or below thr */
        for (int i = 0; i < N; ++i) {
          acc += w[i];
          if (acc > thr) {
            c = i;
            break;
          }
        }
      }
    }
    choice[b] = c;
  }
}

/*
 * Regret bookkeeping (Section 3.1): Regret_T = sum_t f_t[i_t] - min_i sum_t f_t[i], with the
 * drafter i_t that was played when loss vector f_t applied. For each of the L vectors in order:
 * cum[b][i] += f[b][i]; played_sum[b] += f[b][i_t]. Then regret[b] = played_sum[b] -
 * min_i cum[b][i]. A played index outside [0, N) makes that query's sums NaN. With eal [B][N]
 * given, eal_sum[b] += eal[b][i] for the drafter i played with the last vector (the round's
 * expected accepted length, whose mean over rounds is the mean accepted length).
 */
void or_regret_update(const double* loss, int L, int B, int N, const int32_t* played,
                      double* cum, double* played_sum, double* regret, const double* eal,
                      double* eal_sum) {
  for (int b = 0; b < B; ++b) {
    for (int l = 0; l < L; ++l) {
      const double* f = loss + ((size_t)l * B + b) * N;
      const int it = played[(size_t)l * B + b];
      for (int i = 0; i < N; ++i) cum[(size_t)b * N + i] += f[i];
      played_sum[b] += (it >= 0 && it < N) ? f[it] : NAN;
    }
    double mn = INFINITY;
    for (int i = 0; i < N; ++i)
      if (cum[(size_t)b * N + i] < mn) mn = cum[(size_t)b * N + i];
    regret[b] = played_sum[b] - mn;
    if (eal && eal_sum && L > 0) {
      const int it = played[(size_t)(L - 1) * B + b];
      eal_sum[b] += (it >= 0 && it < N) ? eal[(size_t)b * N + it] : NAN;
    }
  }
}

/*
 * Expected acceptance length and losses for B queries and N drafters.
 * gamma   : [B][N][M] feedback per node (chain: M = K positions).
 * parent  : [M] or NULL for a chain (parent[k] = k - 1).
 * path_end: [B] or NULL (node M - 1). For a chain this is the chunk's verified length:
 *           k_h = path_end[b] + 1 (Appendix "Chunk-Level vs Token-Level", chunks of length k_h).
 * eal     : [B][N] Theorem 3 along the path root -> path_end[b].
 * prefix  : [B][N][M] or NULL: product of gamma over the path root -> n, for every node n.
 * loss    : [L][B][N] or NULL, by loss_kind:
 *   LENGTH        : 1 - EAL / (K_path + 1)                      (chunk length loss, Appendix "Chunk-Level Games")
 *   ACCEPT_TOKEN  : L = M vectors, l_k = 1 - gamma_k for the k_h tokens of the chunk and zero
 *                   vectors after them (chain only) (acceptance-probability loss, Section 3.3)
 *   ACCEPT_CHUNK  : (1/K_path) sum_k (1 - gamma_k)               (chunk acceptance loss, Appendix "Chunk-Level Games")
 * Returns 0, or -1 on an invalid path.
 */
int or_accept_len(const double* gamma, int B, int N, int M, const int32_t* parent,
                  const int32_t* path_end, double* eal, double* prefix, int loss_kind,
                  double* loss) {
  int32_t* chainpar = NULL;
  if (!parent) {
    chainpar = (int32_t*)malloc(sizeof(int32_t) * (size_t)M);
    for (int k = 0; k < M; ++k) chainpar[k] = k - 1;
    parent = chainpar;
  }
  int bad = 0;
  for (int b = 0; b < B; ++b) {
    int end = path_end ? path_end[b] : M - 1;
    int32_t path[4096];
    int len = (end >= 0 && end < M) ? or_path(parent, M, end, path) : -1;
    for (int i = 0; i < N; ++i) {
      const double* g = gamma + ((size_t)b * N + i) * M;
      if (len < 1) {
        bad = 1;
        eal[b * N + i] = NAN;
        if (loss) {
          if (loss_kind == OR_LOSS_ACCEPT_TOKEN)
            for (int k = 0; k < M; ++k) loss[((size_t)k * B + b) * N + i] = NAN;
          else
            loss[b * N + i] = NAN;
        }
        continue;
      }
      double gp[4096];
      for (int j = 0; j < len; ++j) gp[j] = g[path[j]];
      double e = or_eal_path(gp, len);
      eal[b * N + i] = e;
      if (prefix) {
        for (int n = 0; n < M; ++n) {
          int32_t pn[4096];
          int ln = or_path(parent, M, n, pn);
          double pr = 1.0;
          for (int j = 0; j < ln; ++j) pr *= g[pn[j]];
          prefix[((size_t)b * N + i) * M + n] = pr;
        }
      }
      if (loss) {
        if (loss_kind == OR_LOSS_LENGTH) {
          loss[b * N + i] = 1.0 - e / (double)(len + 1);
        } else if (loss_kind == OR_LOSS_ACCEPT_CHUNK) {
          double s = 0.0;
          for (int j = 0; j < len; ++j) s += 1.0 - gp[j];
          loss[b * N + i] = s / (double)len;
        } else {
          /* chains only: one vector per verified token of the chunk (k_h = end + 1 of them);
             the rows past the chunk are zero vectors, which leave both learners unchanged */
          for (int k = 0; k < M; ++k) loss[((size_t)k * B + b) * N + i] = k <= end ? 1.0 - g[k] : 0.0;
        }
      }
    }
  }
  free(chainpar);
  return bad ? -1 : 0;
}

/*
 * Hedge (Appendix "Online Learning with Delayed Feedback", remark on Hedge):
 * Update applies w_i <- w_i exp(-eta l_i) for each of the L loss vectors in
 * FIFO order; Predict returns the normalised weights. w is [B][N], one learner
 * per query, and holds normalised weights on entry and exit.
 */
void or_hedge(double* w, const double* loss, int L, int B, int N, double eta) {
  for (int b = 0; b < B; ++b) {
    double* wb = w + (size_t)b * N;
    for (int l = 0; l < L; ++l) {
      const double* lb = loss + ((size_t)l * B + b) * N;
      double s = 0.0;
      for (int i = 0; i < N; ++i) {
        wb[i] = wb[i] * exp(-eta * lb[i]);
        s += wb[i];
      }
      for (int i = 0; i < N; ++i) wb[i] /= s;
    }
  }
}

/* (1/N) sum_i exp(r_i^2 / (2c)), the left side of NormalHedge's scale equation. */
static double nh_g(const double* r, int N, double c) {
  double s = 0.0;
  for (int i = 0; i < N; ++i) s += exp(r[i] * r[i] / (2.0 * c));
  return s / (double)N;
}

/*
 * NormalHedge (Appendix "Variants of Hedging Algorithmic choice", figure
 * "The workflow of NormalHedge"), one learner per query, for each of the L loss
 * vectors in order:
 *   l_A = sum_i p_i l_i
 *   R_i <- R_i + (l_A - l_i)      (evaluated as sum_j p_j (l_j - l_i), see below)
 *   find c > 0 with (1/N) sum_i exp([R_i]_+^2 / (2c)) = e
 *   p_i <- ([R_i]_+ / c) exp([R_i]_+^2 / (2c)), normalised.
 * The left side decreases strictly in c; with M = max_i [R_i]_+^2 it is <= e at
 * c = M/2 and >= e at c = M/(2(1 + ln N)), so the root is found by bisection on
 * that bracket, run until the bracket's relative width is below 1e-15.
 * When every [R_i]_+ is 0 the equation has no root; p is then uniform and c = 0.
 * R, p: [B][N] in/out; c: [B] out (value of the last update).
 */
void or_normalhedge(double* R, double* p, double* c, const double* loss, int L, int B, int N) {
  const double E = exp(1.0);
  double* r = (double*)malloc(sizeof(double) * (size_t)N);
  double* dR = (double*)malloc(sizeof(double) * (size_t)N);
  for (int b = 0; b < B; ++b) {
    double* Rb = R + (size_t)b * N;
    double* pb = p + (size_t)b * N;
    double cb = 0.0;
    for (int l = 0; l < L; ++l) {
      const double* lb = loss + ((size_t)l * B + b) * N;
      /* l_A - l_i evaluated as sum_j p_j (l_j - l_i): the same quantity because the p_j sum
         to 1, and exactly 0 whenever every drafter in the support of p has drafter i's loss,
         so ties cannot create spurious regrets out of rounding. */
      double M = 0.0;
      for (int i = 0; i < N; ++i) dR[i] = 0.0;
      for (int i = 0; i < N; ++i)
        for (int j = 0; j < N; ++j) dR[i] += pb[j] * (lb[j] - lb[i]);
      for (int i = 0; i < N; ++i) {
        Rb[i] = Rb[i] + dR[i];
        r[i] = Rb[i] > 0.0 ? Rb[i] : 0.0;
        if (r[i] * r[i] > M) M = r[i] * r[i];
      }
      if (M == 0.0) {
        for (int i = 0; i < N; ++i) pb[i] = 1.0 / (double)N;
        cb = 0.0;
        continue;
      }
      double lo = M / (2.0 * (1.0 + log((double)N))), hi = M / 2.0;
      for (int it = 0; it < 4000 && hi - lo > 1e-15 * hi; ++it) {
        double mid = 0.5 * (lo + hi);
        if (mid <= lo || mid >= hi) break;
        if (nh_g(r, N, mid) > E)
          lo = mid;
        else
          hi = mid;
      }
      cb = 0.5 * (lo + hi);
      double s = 0.0;
      for (int i = 0; i < N; ++i) {
        pb[i] = (r[i] / cb) * exp(r[i] * r[i] / (2.0 * cb));
        s += pb[i];
      }
      for (int i = 0; i < N; ++i) pb[i] /= s;
    }
    c[b] = cb;
  }
  free(r);
  free(dR);
}

/* Residual (1/N) sum exp(r^2/2c) - e for a given regret row; exposed for the pins. */
double or_normalhedge_residual(const double* R, int N, double c) {
  double* r = (double*)malloc(sizeof(double) * (size_t)N);
  for (int i = 0; i < N; ++i) r[i] = R[i] > 0.0 ? R[i] : 0.0;
  double g = nh_g(r, N, c) - exp(1.0);
  free(r);
  return g;
}
