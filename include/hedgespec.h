/*
 * hedgespec.h - C ABI of libhedgespec.so, the MI355X (gfx950) drafter-evaluation
 * hot path of HedgeSpec (arXiv 2510.20064, "Not-a-Bandit: Provably No-Regret
 * Drafter Selection in Speculative Decoding for LLMs").
 *
 * One verification round of the full-information evaluation phase (Section 3.2):
 * for B queries, K verified positions (or M draft-tree nodes) and N drafters, the
 * target's and every drafter's logits become temperature softmaxes; every
 * (query, drafter, position) gets its acceptance probability and greedy
 * agreement; every (query, drafter) gets Theorem 3's expected acceptance length
 * and a loss; per-query Hedge and NormalHedge learners are updated.
 *
 * Conventions shared by every entry point
 *   - Pointers are DEVICE pointers unless the name ends in _host.
 *   - Every call is asynchronous: it validates its arguments on the host, then
 *     enqueues its kernels on `stream` (a hipStream_t; NULL = the null stream)
 *     and returns without synchronising.
 *   - The caller owns every buffer and keeps it alive until the stream work has
 *     completed. The library keeps no pointer after a call returns and
 *     allocates no memory; scratch space is a caller-provided workspace.
 *   - Validation is complete and happens before anything is enqueued: on an
 *     error code nothing has been enqueued and no output has been touched. (The
 *     one check that asks the device, how many evaluation workgroups it holds at
 *     once, comes last.)
 *   - Device-side faults surface at the caller's next synchronisation.
 *   - Calls that share a workspace must not overlap in time (same stream, or
 *     ordered by events).
 */
#ifndef HEDGESPEC_H
#define HEDGESPEC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes (every entry point returns one) ---------------------------------------- */
#define HS_OK 0
#define HS_ERR_NULL 1        /* a required pointer is NULL                                   */
#define HS_ERR_SHAPE 2       /* B, N, K, V, L or a stride out of range                       */
#define HS_ERR_DTYPE 3       /* unknown storage type                                         */
#define HS_ERR_ALIGN 4       /* a logits row is not 16-byte aligned                          */
#define HS_ERR_TEMPERATURE 5 /* temperature not finite and > 0 where a softmax is needed     */
#define HS_ERR_TREE 6        /* invalid parent array, or a loss kind a tree does not support */
#define HS_ERR_WORKSPACE 7   /* workspace NULL or smaller than the queried size              */
#define HS_ERR_LIMIT 8       /* a size above the library's limits (see below)                */
#define HS_ERR_HIP 9         /* the HIP runtime refused a launch                             */
#define HS_ERR_ARG 10        /* unknown mode or loss kind                                    */

/* ---- limits ------------------------------------------------------------------------------- */
#define HS_MAX_DRAFTERS 64 /* N: one wave64 lane per drafter in the learner kernel  */
#define HS_MAX_POSITIONS 64 /* K (chain positions) or M (tree nodes)                */
#define HS_MAX_QUERIES 65535
#define HS_MAX_TOPL 32      /* L: children per draft-tree node in hs_eval_topl           */
#define HS_MAX_CANDIDATES 1024 /* C: candidate slots per node in hs_candidate_mass       */
/* V: at most 512 * 256 16-byte vectors per row (1048576 bf16 or fp16, or 524288 fp32
   logits), and the device must hold ceil(V / 2048) (bf16, fp16) or ceil(V / 1024) (fp32)
   evaluation workgroups at once: hs_eval_alpha returns HS_ERR_LIMIT otherwise. */

/* ---- enumerations ------------------------------------------------------------------------- */
#define HS_F32 0  /* fp32 logits                            */
#define HS_BF16 1 /* bf16 logits (upper half of an fp32)    */
#define HS_F16 2  /* fp16 logits (IEEE 754 binary16), the precision the paper's models were
                     served in (Section "Experiment setup and baselines") */

#define HS_SAMPLE 0 /* gamma = alpha, speculative sampling at temperature T (Theorem 1)        */
#define HS_GREEDY 1 /* gamma = argmax agreement, Theorem 1 with one-hot p and q (greedy)       */

#define HS_PLAY_ARGMAX 0 /* play the drafter of largest weight (lowest index on ties)   */
#define HS_PLAY_SAMPLE 1 /* sample the drafter from the weights with a given draw        */

#define HS_LOSS_LENGTH 0       /* 1 - EAL/(K_path + 1): chunk length loss (Appendix "Chunk-Level Games") */
#define HS_LOSS_ACCEPT_TOKEN 1 /* K vectors 1 - gamma_k, in order (Section 3.3, acceptance loss)         */
#define HS_LOSS_ACCEPT_CHUNK 2 /* (1/K_path) sum_k (1 - gamma_k) (Appendix "Chunk-Level Games")           */

/*
 * A [B][K][V] logits tensor: element (b, k, v) is at
 * ptr + (b * stride_b + k * stride_k + v) * element_size. V is contiguous.
 * Strides are in elements. ptr and every row start must be 16-byte aligned
 * (strides multiples of 4 for fp32 and of 8 for bf16 and fp16).
 */
typedef struct hs_view {
  const void* ptr;
  int64_t stride_b;
  int64_t stride_k;
} hs_view;

/*
 * hs_softmax_stats - statistics of `rows` temperature softmaxes p = softmax(z/T).
 * The softmax of the target and of every drafter is the first step of Theorem 1
 * (Section 2.2); the temperature form follows the non-greedy experiments (T = 0.5,
 * Appendix "Non-greedy results").
 *   logits     : [rows][ld] of `dtype`, V <= ld, row starts 16-byte aligned.
 *   row_max    : [rows] max_v z_v (raw logits), or NULL.
 *   row_lse    : [rows] natural-log normaliser log sum_v exp(z_v / T), or NULL.
 *   row_argmax : [rows] lowest v with z_v = max (raw logits, so independent of T), or NULL.
 * Needs T finite and > 0. A row whose entries are all -inf yields lse = NaN.
 */
int hs_softmax_stats(const void* logits, int dtype, int64_t rows, int64_t V, int64_t ld,
                     float temperature, float* row_max, float* row_lse, int32_t* row_argmax,
                     void* stream);

/* Bytes of device workspace hs_eval_alpha needs for this shape (0 on invalid shapes). */
size_t hs_eval_alpha_workspace_size(int B, int N, int K, int64_t V, int dtype);

/*
 * hs_eval_alpha - full-information evaluation of N drafters (Section 3.2).
 * For every query b, position k and drafter i:
 *   alpha[b][i][k] = sum_v min(p(v), q_i(v)) = 1 - TV(p, q_i)      (Theorem 1)
 *     with p = softmax(target[b][k] / T), q_i = softmax(drafter_i[b][k] / T),
 *     accumulated in fp32 and clamped to [0, 1]; NaN when either row has no finite
 *     logit or holds a NaN logit (it defines no distribution);
 *   agree[b][i][k]  = 1 if argmax target[b][k] == argmax drafter_i[b][k] else 0;
 *   argmax_t[b][k], argmax_d[b][i][k] = lowest index of the row maximum (raw logits).
 * target       : host pointer to one view; drafters_host: host array of N views.
 * alpha        : [B][N][K] fp32 or NULL. Needs T finite and > 0 when non-NULL.
 * agree        : [B][N][K] uint8 or NULL.
 * argmax_t     : [B][K] int32 or NULL; argmax_d: [B][N][K] int32 or NULL.
 * mode         : HS_SAMPLE or HS_GREEDY. Only selects which outputs are required:
 *                HS_SAMPLE requires alpha, HS_GREEDY requires agree; any other
 *                non-NULL output is filled as well.
 * K            : positions per query (chain) or tree nodes M; 1 <= K <= 64.
 * workspace    : at least hs_eval_alpha_workspace_size() bytes of device memory,
 *                256-byte aligned, ZERO-FILLED before its first use (e.g. hipMemset),
 *                and afterwards written only by these calls. The library keeps a call
 *                counter in it (the epoch, uint32 at byte 0) and tags every word it
 *                exchanges between workgroups with a 31-bit tag derived from it, so the
 *                workspace is reused for any shape without clearing; its counters (bytes
 *                16 and 24) carry the tag too, so a stale count of an earlier call is
 *                never taken for the current one. Memory that other code wrote may hold
 *                words that look current: such a workspace gives undefined results (but
 *                never a hang). After a device fault or an HS_ERR_HIP return, zero it again.
 * Waits      : every wait of one workgroup for another's words is bounded (about 0.5 s,
 *                see hs_set_wait_limit). A wait that gives up (a device too busy with
 *                other work to hold a whole team of workgroups at once) makes the call
 *                mark every output invalid: alpha NaN, agree 0, argmax -2.
 * Logit range  : fp32 accuracy for finite logits z with |z| log2(e) / T <= 2^28 (for
 *                example |z| <= 1.8e8 at T = 1). A logit far below its row's maximum
 *                contributes its exact probability, which underflows to 0, however large
 *                its magnitude: masks such as -1e9 or the storage type's most negative
 *                finite value are fine next to ordinary logits. A row whose largest
 *                logit is outside the range is treated as having no distribution (NaN).
 * Each logit is read from HBM once per call, in one launch. Results are
 * deterministic (fixed reduction order) for a given shape.
 */
int hs_eval_alpha(const hs_view* target, const hs_view* drafters_host, int N, int B, int K,
                  int64_t V, int dtype, float temperature, int mode, float* alpha, uint8_t* agree,
                  int32_t* argmax_t, int32_t* argmax_d, void* workspace, size_t workspace_bytes,
                  void* stream);

/*
 * hs_eval_alpha_noalloc - hs_eval_alpha for callers that cannot allocate device memory or
 * pass a workspace: code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc. Arguments, outputs, results and errors are those of hs_eval_alpha (same kernels)
 * without the workspace: the exchange words live in a fixed array of
 * hs_eval_alpha_noalloc_max_workspace() bytes (64 MiB) that the library's code object holds
 * on every device it runs on until the process ends (zero when loaded, and never in need of
 * clearing: its words are tagged per call). A shape whose workspace
 * (hs_eval_alpha_workspace_size) is larger gets HS_ERR_WORKSPACE before anything is enqueued.
 * The first call on a device looks up that device's copy (hipGetSymbolAddress); no call
 * allocates. Calls on one device share the array: calls that overlap in time on one device
 * (different streams, or threads without ordering) race and give undefined results; calls
 * ordered on one stream are safe.
 */
int hs_eval_alpha_noalloc(const hs_view* target, const hs_view* drafters_host, int N, int B,
                          int K, int64_t V, int dtype, float temperature, int mode, float* alpha,
                          uint8_t* agree, int32_t* argmax_t, int32_t* argmax_d, void* stream);
size_t hs_eval_alpha_noalloc_max_workspace(void);

/* Bytes of device workspace hs_eval_topl needs for this shape (0 on invalid shapes). */
size_t hs_eval_topl_workspace_size(int B, int N, int K, int64_t V, int L, int dtype);

/*
 * hs_eval_topl - EAGLE acceptance probabilities of N drafters (Theorem 2; Section 2.3 and
 * Section 3.2's gamma for EAGLE's greedy draft tree). The tree gives the node after a
 * verified prefix the drafter's L highest-ranked tokens as children, Top_L(q_i), and the
 * target accepts one of them with probability
 *   gamma[b][i][k] = sum_{v in Top_L(drafter_i[b][k])} p(v),  p = softmax(target[b][k] / T),
 * accumulated in fp32 and clamped to [0, 1]. The ranking is that of the raw drafter logits
 * (a softmax at any temperature keeps it); equal logits rank lower token index first, and
 * -0 ranks as +0.
 *   hit[b][i][k]      = 1 if the target's argmax (lowest index of its row maximum) is in
 *                       Top_L, else 0: gamma of greedy decoding (one-hot p).
 *   children[b][i][k] = Top_L in rank order, L int32 token indices.
 * A drafter row holding a NaN logit has no ranking: its children, hit and gamma are
 * unspecified. A target row holding one gives gamma = NaN.
 * target, drafters_host, N, B, K, V, dtype: as in hs_eval_alpha (K positions or tree nodes).
 * L            : children per node, 1 <= L <= min(V, HS_MAX_TOPL) (EAGLE's default is 10).
 * gamma        : [B][N][K] fp32 or NULL. Needs T finite and > 0 when non-NULL.
 * hit          : [B][N][K] uint8 or NULL.
 * children     : [B][N][K][L] int32 or NULL.
 * mode         : HS_SAMPLE requires gamma, HS_GREEDY requires hit; any other non-NULL
 *                output is filled as well.
 * workspace    : at least hs_eval_topl_workspace_size() bytes of device memory, 256-byte
 *                aligned; scratch only (no initialisation needed, contents undefined after).
 * Two launches: each logit is read from HBM once, by the first (per 2048-logit slice of each
 * row: the target's softmax statistics, or a drafter's L best keys, 8 L bytes); the second
 * merges each drafter row's candidates and reads the target logits of its L winners.
 * Deterministic for a given shape.
 * EAGLE-2's dynamic pruning, whose candidate set is the pruned subtree: hs_candidate_mass.
 */
int hs_eval_topl(const hs_view* target, const hs_view* drafters_host, int N, int B, int K,
                 int64_t V, int dtype, int L, float temperature, int mode, float* gamma,
                 uint8_t* hit, int32_t* children, void* workspace, size_t workspace_bytes,
                 void* stream);

/*
 * hs_candidate_mass - Theorem 2 with EAGLE-2's dynamic pruning: when the draft tree is pruned,
 * the candidate set at a node is the node's kept children (the pruned set of descendants)
 * instead of Top_L(q), and the target accepts one of them with probability
 *   gamma[b][i][k] = sum_{j < C, cand[b][i][k][j] >= 0} p(cand[b][i][k][j]),
 *   p = softmax(target[b][k] / T),
 * accumulated in fp32 in a fixed order, not clamped (a listed index counts once per listing).
 * target, B, K, V, dtype: as in hs_eval_alpha.
 * target_lse   : [B][K] fp32 device, log sum_v exp(target[b][k][v] / T) (natural log), e.g.
 *                hs_softmax_stats' row_lse over the target rows at the same T.
 * cand         : [B][N][K][C] int32 device, the kept children (hs_eval_topl's `children`
 *                after pruning); a negative entry is an empty slot. An index >= V makes that
 *                gamma NaN.
 * C            : slots per node, 1 <= C <= HS_MAX_CANDIDATES.
 * gamma        : [B][N][K] fp32 device.
 * One launch, one wave per output; it reads the C indices and the target logits they name.
 */
int hs_candidate_mass(const hs_view* target, int N, int B, int K, int64_t V, int dtype,
                      float temperature, const float* target_lse, const int32_t* cand, int C,
                      float* gamma, void* stream);

/*
 * hs_accept_len - Theorem 3's one-step counterfactual acceptance-length
 * estimator for every (query, drafter), and the learner's loss.
 * gamma is alpha (HS_SAMPLE; `alpha` [B][N][K] fp32) or the agreement
 * indicator (HS_GREEDY; `agree` [B][N][K] uint8).
 * Chains (parent_host = NULL): EAL = sum_{k=1}^{K+1} k (1-gamma_k) prod_{j<k} gamma_j
 *   = 1 + sum_{k=1}^{K} prod_{j<=k} gamma_j, with gamma_{K+1} = 0.
 * Trees (parent_host = host int32[K], parent[0] = -1, 0 <= parent[n] < n):
 *   node n carries the feedback of the token after its prefix (Section 3.2);
 *   prefix[n] = gamma[n] * prefix[parent[n]] (root: gamma[0]); the path is
 *   root -> path_end[b]; EAL = 1 + sum of prefix over the path's K_path nodes.
 * path_end     : [B] int32 device array or NULL (node K-1). An index outside
 *                [0, K) gives NaN for that query's EAL and loss. For a chain it is the
 *                chunk's verified length k_h - 1 (Appendix "Chunk-Level vs Token-Level":
 *                chunks of ragged length k_h use Theorem 3 with K = k_h).
 * eal          : [B][N] fp64 (required).
 * prefix       : [B][N][K] fp64 or NULL.
 * loss         : [L][B][N] fp64 or NULL; L = K for HS_LOSS_ACCEPT_TOKEN (chains
 *                only: rows past a query's k_h verified tokens are zero vectors, which
 *                leave Hedge and NormalHedge unchanged), else L = 1. See HS_LOSS_* for the
 *                definitions.
 */
int hs_accept_len(const float* alpha, const uint8_t* agree, int mode, int B, int N, int K,
                  const int32_t* parent_host, const int32_t* path_end, double* eal,
                  double* prefix, int loss_kind, double* loss, void* stream);

/*
 * hs_hedge_update - Hedge, one learner per query (Appendix "Online Learning with
 * Delayed Feedback", Hedge remark): for each of the L loss vectors in order,
 * w_i <- w_i exp(-eta loss_i); Predict returns the normalised weights.
 * Kept in the log domain: logw_i -= eta * loss_i, re-centred so max_i logw_i = 0,
 * then w = softmax(logw).
 * logw : [B][N] fp64 in/out (initialise to 0); w: [B][N] fp64 out.
 * loss : [L][B][N] fp64, expected in [0, 1] (not checked: device data). L >= 1.
 */
int hs_hedge_update(double* logw, double* w, const double* loss, int L, int B, int N, double eta,
                    void* stream);

/*
 * hs_normalhedge_update - NormalHedge, one learner per query (Appendix "Variants
 * of Hedging Algorithmic choice", figure "The workflow of NormalHedge"). For each
 * of the L loss vectors in order:
 *   l_A = sum_i p_i l_i;  R_i += l_A - l_i;  r_i = max(R_i, 0);
 *   c solves (1/N) sum_i exp(r_i^2 / (2c)) = e;
 *   p_i = (r_i / c) exp(r_i^2 / (2c)) / normaliser.
 * If every r_i is 0 the equation has no root: p = 1/N and c = 0.
 * R : [B][N] fp64 in/out (initialise to 0); p: [B][N] fp64 in/out (initialise to 1/N);
 * c : [B] fp64 in/out: on entry only a starting point for the search of c (any value
 *     works; the previous call's output makes it fastest), on exit the value of the
 *     last update; loss: [L][B][N] fp64.
 */
int hs_normalhedge_update(double* R, double* p, double* c, const double* loss, int L, int B,
                          int N, void* stream);

/*
 * hs_delayed_update - the token-level game with delayed feedback (Section 3.3,
 * "HedgeSpec: Loss functions and Delayed Feedback"; Appendix, algorithm QFI-D,
 * "Queued Full-Information with Delays", with Hedge and NormalHedge as base learners).
 * The token-level length loss of token s for drafter i,
 *   f_s[i] = 1 - EAL(gamma_s .. gamma_{s+K-1})[i] / (K + 1),
 * is Theorem 3's estimator on the window of K tokens that starts at s (the window's
 * (K+1)-th term takes gamma = 0, as in hs_accept_len). It is known only once the
 * feedback of all K tokens of its window has arrived. Per query b, this call appends
 * the feedback of the query's next count[b] tokens to the history ring, then feeds
 * every window that is now complete and not yet used to the base learners, in token
 * order, before returning: the learners see a delay-free loss stream in their own
 * clock. A query whose call completes no window keeps its learner state unchanged.
 * alpha / agree : [B][N][K] gamma of this round (HS_SAMPLE: alpha fp32; HS_GREEDY:
 *                 agree uint8); token j of the call is position j, j < count[b].
 * count         : [B] int32 device; values outside [0, K] are clamped to it.
 * hybrid_tokens : H >= 0. Hybrid losses (Appendix "Practical heuristics: hybrid losses"): the
 *                 first H tokens of every query's stream take the acceptance-probability loss
 *                 1 - gamma_s instead, known as soon as the token's feedback arrives (against
 *                 the cold start); 0 = the length loss throughout. The tokens whose loss is
 *                 known always form a prefix of the stream, so the FIFO order is unchanged.
 *                 Use the same H for every call of a stream (a change shifts the switch; a
 *                 call then uses at most K of the losses that became known, the rest later).
 * hist          : [B][2K][N] fp32 device, the history ring (caller-owned, zero-filled
 *                 before the first call of a stream, not read by the caller).
 * clock         : [B][2] int64 device, zero-filled before the first call: tokens
 *                 received and windows used so far, per query.
 * logw, w, eta  : Hedge state (both or neither); R, p, c: NormalHedge state (all or
 *                 none), as in hs_hedge_update / hs_normalhedge_update.
 * loss          : [K][B][N] fp64 or NULL: the window losses used by this call, in
 *                 order (rows past nloss[b] are not written).
 * nloss         : [B] int32 or NULL: how many loss vectors each query used (at most count[b]).
 * One launch, one wave per query. Errors: HS_ERR_SHAPE / HS_ERR_LIMIT on B, N, K;
 * HS_ERR_ARG on mode or a non-finite eta; HS_ERR_NULL on missing inputs or unpaired
 * learner state. Nothing is enqueued on error.
 */
int hs_delayed_update(const float* alpha, const uint8_t* agree, int mode, int B, int N, int K,
                      const int32_t* count, int64_t hybrid_tokens, float* hist, int64_t* clock,
                      double* logw, double* w, double eta, double* R, double* p, double* c,
                      double* loss, int32_t* nloss, void* stream);

/*
 * hs_play - the drafter each query plays next (Appendix, algorithm QFI-D, "Queued
 * Full-Information with Delays": after the queued losses are in, play a_t according to p, by
 * sampling from p or by its argmax).
 * weights : [B][N] fp64 device, non-negative (Hedge's w or NormalHedge's p; need not sum to 1).
 * how     : HS_PLAY_ARGMAX, or HS_PLAY_SAMPLE: the smallest i with w_0 + ... + w_i >
 *           u[b] * (w_0 + ... + w_{N-1}), prefix sums taken left to right in fp64.
 * u       : [B] fp64 device uniform draws in [0, 1) (required for HS_PLAY_SAMPLE; the caller
 *           owns the random stream).
 * choice  : [B] int32 device out; -1 for a row whose weights do not sum to a positive finite
 *           number. One launch, one wave per query.
 */
int hs_play(const double* weights, int B, int N, int how, const double* u, int32_t* choice,
            void* stream);

/*
 * hs_regret_update - regret bookkeeping (Section 3.1): Regret_T = sum_t f_t[i_t] -
 * min_i sum_t f_t[i], with i_t the drafter played when loss vector f_t applied. For each of
 * the L loss vectors in order: cum_loss[b][i] += f[b][i] and played_loss[b] += f[b][i_t]; then
 * regret[b] = played_loss[b] - min_i cum_loss[b][i] (the sums run in loss order, in fp64).
 * loss        : [L][B][N] fp64 device (as hs_accept_len writes it), L >= 1.
 * played      : [L][B] int32 device: the drafter played for each vector. An index outside
 *               [0, N) makes that query's played_loss and regret NaN from then on.
 * cum_loss    : [B][N] fp64 in/out, played_loss: [B] fp64 in/out (zero-fill to start);
 *               regret: [B] fp64 out.
 * eal, eal_sum: both or neither. eal [B][N] (this round's expected accepted lengths);
 *               eal_sum[b] += eal[b][i] for the drafter played with the last vector, so that
 *               eal_sum / rounds is the played drafters' mean accepted length.
 */
int hs_regret_update(const double* loss, int L, int B, int N, const int32_t* played,
                     double* cum_loss, double* played_loss, double* regret, const double* eal,
                     double* eal_sum, void* stream);

/*
 * hs_round - one verification round of the whole path: the work of hs_eval_alpha,
 * then per query hs_accept_len's work, the loss, and the Hedge and NormalHedge
 * updates with that loss (same workspace contract as hs_eval_alpha). In sample mode
 * the learner step runs inside the evaluation launch when its LDS (gamma, losses and
 * scratch of one query) fits in the evaluation kernel's: one launch. Otherwise, and
 * in greedy mode, it is a second launch, one wave per query. Arguments mean what they
 * mean in the calls above. Learner state pointers may be NULL to skip that learner (logw
 * and w together; R, p and c together). eal is required; alpha/agree as hs_eval_alpha
 * requires them for `mode`.
 * A round whose evaluation lost a word (a wait gave up, see hs_eval_alpha) never feeds it
 * to a learner: each query whose gamma depends on a lost word (with the second launch:
 * every query) keeps its learner state unchanged and gets NaN eal, prefix and loss; the
 * call still returns HS_OK (the failure happens on the device, after the call returned).
 */
typedef struct hs_round_args {
  hs_view target;
  const hs_view* drafters_host; /* host array of N views */
  int N, B, K;
  int64_t V;
  int dtype;
  float temperature;
  int mode;
  float* alpha;
  uint8_t* agree;
  int32_t* argmax_t;
  int32_t* argmax_d;
  const int32_t* parent_host;
  const int32_t* path_end;
  double* eal;
  double* prefix;
  int loss_kind;
  double* loss;
  double* logw;
  double* w;
  double eta;
  double* R;
  double* p;
  double* c;
  void* workspace;
  size_t workspace_bytes;
} hs_round_args;

int hs_round(const hs_round_args* args, void* stream);

/* Name of a status code; the thread's last error message; library version (major*10000+minor*100+patch). */
const char* hs_status_string(int status);
const char* hs_last_error(void);
int hs_version(void);

/*
 * hs_set_wait_limit - polls (about 2 us apart) before a wait of one evaluation workgroup
 * for another's words gives up, for every hs_eval_alpha / hs_round launched after this call
 * in the process. Negative restores the default (2^18, about 0.5 s). 0 makes every such wait
 * give up at once, whatever the words hold: every call then takes its failure path (outputs
 * marked invalid, learner state unchanged) while every kernel still ends normally, which is
 * how that path is tested. Not synchronised with calls in flight on other threads.
 */
void hs_set_wait_limit(int polls);

/*
 * hs_stream_read - measurement aid, not a step of the method: reads every 16-byte vector of a
 * device buffer once and writes, for each wave, the XOR of the 32-bit words it read. Timed
 * over a buffer far larger than the 256 MB Infinity Cache, it gives the rate at which this
 * device streams resident data from HBM: the practical ceiling the evaluation kernels'
 * achieved bandwidth is compared with (they, too, read every logit once).
 *   x:      device pointer, 16-byte aligned; bytes: its size, a positive multiple of 16.
 *   grid:   workgroups of 256 threads (1..65536); they stride over the buffer together.
 *   unroll: 1, 2, 4 or 8 loads of 16 bytes in flight per thread.
 *   nontemporal: nonzero for loads that tell the caches not to keep the data.
 *   out:    device pointer to grid * 4 uint32 words (written; the caller owns it).
 *   stream: hipStream_t or NULL. Asynchronous; errors: HS_ERR_NULL, HS_ERR_ALIGN,
 *           HS_ERR_SHAPE, HS_ERR_ARG, HS_ERR_HIP.
 */
int hs_stream_read(const void* x, size_t bytes, int grid, int unroll, int nontemporal,
                   uint32_t* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* HEDGESPEC_H */
