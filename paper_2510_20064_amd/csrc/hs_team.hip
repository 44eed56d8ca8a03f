// Drafter evaluation with one read of every logit, in one launch: softmax statistics,
// alpha = sum_v min(p, q_i) for every drafter (Theorem 1), greedy argmax and agreement, and
// for hs_round the learner step.
//
// min(p_v, q_v) needs both rows' normalisers, which depend on the whole row, so the
// slices of a row have to meet before any min can be taken. Here they meet on chip: a
// work item is (row set, slice) = the target slice and the slices of up to D drafters of
// one (query, position) group, 256 16-byte vectors each, held in the registers of one
// 256-thread workgroup (thread t owns vector t of every row). The S items of a row set form
// a team that is resident at the same time:
//   1. every item reduces its rows (max, lowest argmax, exp2 sum against the slice offset
//      o, an integer-valued float at or above m c, c = log2(e) / T) and publishes them as
//      tagged words;
//   2. item s folds the S slice statistics of row s (rows s, s + S, ... when S is smaller
//      than the row count) into the row's log2 normaliser L = hi + lo and publishes it;
//   3. every item reads the normalisers and forms its slice's part of sum_v min(p_v, q_v)
//      for each drafter: from the e_v kept in registers when the workgroup holds one item
//      (one multiply, one min and one add per drafter logit), else from the logits again
//      (one fma, one min, one exp2 and one add); the partials are published;
//   4. slot d mod S sums drafter d's S slice partials in slice order into alpha.
// Within a workgroup every reduction over the slice goes through LDS: each thread stores its
// per-row value, then one 16-lane group per row reduces the row's 256 values and the result
// is known to the whole group, so no wave reduces all rows on its own.
// A workgroup with several items overlaps them: while item j's normalisers are exchanged it
// runs the statistics of item j + 1, and the loads of item j + 2 go out as soon as item j's
// min-sums have freed its registers.
//
// The grid holds as many teams as the device keeps resident at once, so all members of a
// team run together and waiting on one cannot deadlock. Words crossing workgroups carry the
// call's tag; the last team to finish advances the epoch the tag derives from. Every wait is
// bounded: a word that never arrives yields NaN (argmax -2), no hang, and everything computed
// from it carries a taint mark, so the learner step of such a round leaves the learner state
// unchanged.
#include <algorithm>
#include <atomic>
#include <cstdio>

#include "hs_learner.h"
#include "hs_wave.h"

namespace hs {

constexpr int kPollSleep = 2;  // s_sleep units (64 clocks) between polls
constexpr int kCritPrio = 2;   // wave priority of the exchange-critical stages (s_setprio)
constexpr int kFoldPrio = 3;   // and of the pipelined kernel's row folds, which gate the team
// The wave that holds no row of the group reductions (16-lane group r reduces row r, so the at
// most kMaxSetDrafters + 1 rows sit in the other waves) takes a member's first fold duty and
// the normaliser wait: their load round trips then overlap the other waves' group reductions
// instead of following them, and wave 0 keeps thread 0's claims and counts.
constexpr int kDutyWave = kWaves - 1;
static_assert(kMaxSetDrafters + 1 <= 4 * kDutyWave, "the duty wave must hold no reduction row");

struct TeamArgs {
  // What every workgroup reads before its first loads comes first: the first 128 bytes of the
  // kernel arguments, two scalar-cache lines, requested together at entry. The row table
  // follows at the end.
  int B, N, K, nsub, S, items;
  int teams;         // workgroups of the launch / S
  // drafter rows at one constant distance (uni != 0): row bases from these scalars instead of
  // the row table, so the kernel does not wait for the table at its start
  int uni;
  FastDiv divS, divK;  // by S and K
  int64_t V;
  int64_t dd;          // bytes from drafter i's row (b, k) to drafter i + 1's
  const void* base0;   // the target's rows (rows.ptr[0] and its strides)
  const void* base1;   // drafter 0's rows (rows.ptr[1] and its strides)
  int64_t sb0, sk0, sb1, sk1;
  uint32_t* epoch;     // advanced by the last workgroup to finish
  // ---- 128 bytes ----
  int64_t nvec;
  float c;
  FastDiv divNsub;     // by nsub
  uint64_t* fail;      // set, with the call's tag, by the first wait that gives up
  uint32_t polls;      // polls before a wait gives up (0: every wait gives up at once)
  uint32_t* next_set;  // row sets claimed beyond each team's fixed ones
  uint64_t* finished;  // teams of this launch that have finished (a tagged count)
  uint64_t* mbox;      // [teams][4]: the row set of each team's coming items
  uint64_t* stat;  // [sets][D + 1][S][3]
  uint64_t* norm;  // [sets][D + 1][3] (the single-item kernel's other copies: norm_copy)
  uint64_t* part;  // [G][N][S]
  float* alpha;
  int32_t* argmax_t;
  int32_t* argmax_d;
  uint8_t* agree;
  // learner step in the same launch (learn != 0; alpha kernels only): gamma words gw [B][N][K]
  // are written by the folders (gamma = alpha when learn == 1, agreement when learn == 2), and
  // workgroup b (mod the grid) runs query b's step once it has finished its own items
  int learn;
  uint64_t* gw;
  TailArgs tail;
  RowTable rows;
};


// (a vector load: a scalar one would hold up the kernel-argument loads waited on with it)
__device__ inline uint32_t call_tag(const uint32_t* epoch) {
  const uint32_t e =
      __hip_atomic_load(const_cast<uint32_t*>(epoch), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return (uint32_t)__builtin_amdgcn_readfirstlane((int)tag_of_epoch(e));
}

// Adds 1 to the count that the word w keeps for the call with this tag and returns the
// count before (0 for the first add of a call): the word holds (count << 32) | tag, and a
// word with another tag, from an earlier call or never written, counts as 0. So nothing has
// to be reset between calls, and whatever a word held before cannot skew this call's count.
// The call that completes a count leaves the word at (0 << 32) | the next call's tag
// (count_team), so each add of the next call is a single fetch-and-add, which leaves the tag
// half alone and costs every adder one round trip however many add at once. An add that
// finds another tag (the first call on a zeroed workspace) goes on by compare-and-swap: the
// first exchange replaces the whole word, so its earlier fetch-and-adds on the stale word do
// not count, and every adder is counted once, by its fetch-and-add or by its exchange.
__device__ inline uint32_t tagged_add(uint64_t* w, uint32_t tag) {
  const uint64_t old =
      __hip_atomic_fetch_add(w, 1ull << 32, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if ((uint32_t)old == tag) return (uint32_t)(old >> 32);
  uint64_t cur = get_word(w);
  for (;;) {  // each failed exchange means another add succeeded: this ends
    const uint32_t n = (uint32_t)cur == tag ? (uint32_t)(cur >> 32) : 0u;
    uint64_t expect = cur;
    if (__hip_atomic_compare_exchange_strong(w, &expect, ((uint64_t)(n + 1u) << 32) | tag,
                                             __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT))
      return n;
    cur = expect;
  }
}

// The word at w once it carries tag (its taint mark, if any, kept). Bounded: after `polls`
// polls, or as soon as another wait of this call has given up, the value is 0xFFFFFFFE (a NaN
// as float, -2 as int), tainted; the first wait to give up raises the call's fail flag, so one
// lost word costs one time-out, not one per wait. polls = 0 (set from the host, to test the
// failure path) makes every wait give up at once.
__device__ inline uint64_t await_word(const uint64_t* w, uint32_t tag, const TeamArgs& A) {
  constexpr uint64_t kLost = (0xFFFFFFFEull << 32) | kTaint;
  if (A.polls == 0) {
    put_word(A.fail, word_of(1, tag));
    return kLost | tag;
  }
  uint64_t v = get_word(w);
  for (uint32_t n = 1; tag_of(v) != tag; ++n) {
    if (n >= A.polls) {
      put_word(A.fail, word_of(1, tag));
      return kLost | tag;
    }
    if ((n & 255) == 0 && (uint32_t)get_word(A.fail) == tag) return kLost | tag;
    __builtin_amdgcn_s_sleep(kPollSleep);
    v = get_word(w);
  }
  return v;
}

// Mailbox word of a team's item j: the row set in bits 38..63, j mod 64 in bits 32..37, the
// call's tag below, so neither an earlier item's word in the same ring slot nor an earlier
// call's word is taken for it.
__device__ inline uint64_t mbox_word(uint32_t set, int j, uint32_t tag) {
  return ((uint64_t)((set << 6) | ((uint32_t)j & 63u)) << 32) | tag;
}
// The row set posted for item j (bounded as await_word: `none` after a time-out, raising the
// fail flag).
__device__ inline uint32_t await_mbox(const uint64_t* w, int j, uint32_t tag, const TeamArgs& A,
                                      uint32_t none) {
  auto ok = [&](uint64_t v) {
    return (uint32_t)v == tag && ((uint32_t)(v >> 32) & 63u) == ((uint32_t)j & 63u);
  };
  if (A.polls == 0) {
    put_word(A.fail, word_of(1, tag));
    return none;
  }
  uint64_t v = get_word(w);
  for (uint32_t n = 1; !ok(v); ++n) {
    if (n >= A.polls || ((n & 255) == 0 && (uint32_t)get_word(A.fail) == tag)) {
      put_word(A.fail, word_of(1, tag));
      return none;
    }
    __builtin_amdgcn_s_sleep(kPollSleep);
    v = get_word(w);
  }
  return (uint32_t)(v >> 38);
}

// Copy c of the normaliser words: the first at A.norm, the others after the gamma words (the
// single-item kernel only, whose row sets are its teams).
__device__ inline uint64_t* norm_copy(const TeamArgs& A, int c, int rows) {
  if (c == 0) return A.norm;
  const uintptr_t end = reinterpret_cast<uintptr_t>(A.gw + (int64_t)A.B * A.N * A.K);
  return reinterpret_cast<uint64_t*>((end + 255) & ~(uintptr_t)255) +
         (c - 1) * norm_copy_words(A.teams, rows);
}

// Fold of row rr of row set `set`: the S slice statistics, two slices per lane per pass
// (lane j takes slices j, j + 64, ... in order), then the wave. Publishes the row's log2
// normaliser as hi + lo (in NC copies) and its argmax; writes the argmax and agreement
// outputs. The published words are tainted when any slice word was lost.
template <int D, bool NEED_SUM, bool NEED_ARG, int NC = 1>
__device__ __forceinline__ void fold_row(const TeamArgs& A, int set, int rr, int b, int k, int sub,
                                uint32_t tag, int lane) {
  constexpr int RM = D + 1;
  const int S = A.S;
  const uint64_t* base = A.stat + ((int64_t)set * RM + rr) * S * 3;
  float m = -INFINITY, o = -INFINITY, sum = 0.0f;
  int idx = INT_MAX;
  bool lost = false;
  for (int j0 = 0; j0 < S; j0 += 128) {
    uint64_t w[2][3];
#pragma unroll
    for (int h = 0; h < 2; ++h) {  // issue every load of the pass before waiting on any
      const int j = j0 + lane + 64 * h;
      if (j < S) {
        w[h][0] = get_word(base + 3 * j);
        if (NEED_SUM) w[h][1] = get_word(base + 3 * j + 1);
        if (NEED_ARG) w[h][2] = get_word(base + 3 * j + 2);
      }
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int j = j0 + lane + 64 * h;
      if (j < S) {
        if (tag_of(w[h][0]) != tag) w[h][0] = await_word(base + 3 * j, tag, A);
        lost |= tainted(w[h][0]);
        const float ms = word_f(w[h][0]);
        if (NEED_ARG) {
          if (tag_of(w[h][2]) != tag) w[h][2] = await_word(base + 3 * j + 2, tag, A);
          lost |= tainted(w[h][2]);
          argmax_combine(m, idx, ms, word_i(w[h][2]));
        } else {
          m = fmaxf(m, ms);
        }
        if (NEED_SUM) {
          if (tag_of(w[h][1]) != tag) w[h][1] = await_word(base + 3 * j + 1, tag, A);
          lost |= tainted(w[h][1]);
          lse2_combine(o, sum, exp_offset_of(ms, A.c), word_f(w[h][1]));
        }
      }
    }
  }
  wave_max<NEED_ARG>(m, idx);
  if (NEED_SUM) wave_lse(o, sum);
  const uint32_t tt = tag | taint_bits(__ballot(lost) != 0);
  uint64_t* nw = A.norm + ((int64_t)set * RM + rr) * 3;
  if (NEED_SUM) {
    // log2 normaliser o + log2(sum) as an unevaluated sum hi + lo (TwoSum); lane c writes
    // copy c
    const float l2 = log2f(sum);
    const float hi = o + l2;
    const float bb = hi - o;
    const float lo = (o - (hi - bb)) + (l2 - bb);
    if (lane < NC) {
      uint64_t* cw = norm_copy(A, lane, RM) + ((int64_t)set * RM + rr) * 3;
      put_word(cw, word_of(hi, tt));
      put_word(cw + 1, word_of(lo, tt));
    }
  }
  if (lane != 0) return;
  if (NEED_ARG) {
    put_word(nw + 2, word_of(idx, tt));
    if (rr == 0) {
      if (sub == 0 && A.argmax_t) A.argmax_t[(int64_t)b * A.K + k] = idx;
    } else {
      const int64_t oi = ((int64_t)b * A.N + sub * D + rr - 1) * A.K + k;
      if (A.argmax_d) A.argmax_d[oi] = idx;
      if (A.agree) {
        const uint64_t tw = await_word(A.norm + (int64_t)set * RM * 3 + 2, tag, A);
        const int it = word_i(tw);
        const bool ag = idx == it && it >= 0;
        A.agree[oi] = (uint8_t)ag;
        if (A.learn == 2) put_word(A.gw + oi, word_of(ag ? 1.0f : 0.0f, tt | ((uint32_t)tw & kTaint)));
      }
    }
  }
}

// Position of work item (set, slot): row set, slice, group (b, k), drafters n in the set, and
// the calling thread's vector index within the row.
struct ItemPos {
  int set, s, g, sub, b, k, n;
  int vi;  // a row holds fewer than 2^31 logits
};
__device__ inline ItemPos item_pos(const TeamArgs& A, uint32_t set, int slot, int D) {
  ItemPos q;
  q.set = (int)set;
  q.s = slot;
  if (A.nsub == 1) {
    q.g = q.set;
    q.sub = 0;
  } else {
    q.g = (int)fdiv(set, A.divNsub);
    q.sub = q.set - q.g * A.nsub;
  }
  q.b = (int)fdiv((uint32_t)q.g, A.divK);
  q.k = q.g - q.b * A.K;
  q.n = min(D, A.N - q.sub * D);
  q.vi = q.s * kThreads + (int)threadIdx.x;
  return q;
}

// LDS of a team workgroup. Per-thread values of every row are stored transposed, [row][thread],
// so that one 16-lane group reduces one row (group_read) instead of every wave reducing every
// row on its own. Slice offsets are double-buffered by item parity: an item's min-sum runs
// after the statistics of its successor.
template <int D, bool NEED_ARG, bool PT = false>
struct TeamLds {
  float xt[D + 1][kThreads];                  // per-thread max keys / maxima, then exp2 sums
  int xi[NEED_ARG ? D + 1 : 1][kThreads];     // per-thread argmax
  float xs[PT ? D + 1 : 1][kThreads];         // per-thread exp2 sums against the thread's offset
  int xo[PT ? D + 1 : 1][kThreads];           // that offset (saturated to int32)
  float xp[D][kThreads];                      // per-thread min-sums of each drafter
  float o[2][D + 1];                          // slice offsets exp_offset_of(m, c)
  float no[2][D + 1];                         // -exp_offset(o): the addend of the exponents
  float nw[D];     // from the logits: -exp_offset(o_d) - (a_t - a_d), a_x = (o_x - hi_x) - lo_x
  float dl[D];     // from the logits: a_t - a_d
  uint32_t wide;   // from the logits: some drafter's |offset| is too large for nw to be exact
  float G[D];      // kept e_v: 2^(a_t - a_d)
  float F[D];      // factor of drafter d's group sum: 2^(a_d) (kept e_v), else 2^(a_t)
  uint32_t next;  // a row set of the team's coming items, posted by thread 0
  uint32_t taint;  // the item's normalisers include a lost word: its partials are tainted
  // the row table, copied from the kernel arguments once (lane-parallel loads instead of a
  // chain of dependent scalar loads per item)
  const char* ptr[kMaxRows];
  int64_t sb[kMaxRows];
  int64_t sk[kMaxRows];
};

// Issue the loads of item q into dst: exactly D + 1 unconditional 16-byte loads, so that the
// number of loads in flight is the same on every path and a later wait for an older item's
// registers can leave these outstanding. Each comes from an address clamped into the row's
// complete vectors (lanes past the row end are masked to -inf before use, mask_tail); rows
// past the set's last drafter, and every row when !valid, read 16 bytes of the workspace's
// control block instead (a cache-resident dummy, never used). The one partial vector at the
// end of a row (V not a multiple of the vector width) is then re-read element by element, in
// a branch taken only by the slice that holds it.
template <int DT, int D, bool UNI = false, typename L>
__device__ __forceinline__ void fetch_item(const TeamArgs& A, const ItemPos& q, bool valid,
                                           const L& sh, typename Vec<DT>::Raw (&dst)[D + 1]) {
  using Vt = Vec<DT>;
  constexpr int E = Vt::kElems;
  const int64_t vfull = A.V / E;  // complete 16-byte vectors per row
  const uint64_t dummy = reinterpret_cast<uint64_t>(A.epoch);
  uint64_t rb[D + 1];
  if (UNI && A.uni) {
    // drafters at a constant distance: uniform scalar arithmetic
    rb[0] = valid ? reinterpret_cast<uint64_t>(A.base0) +
                        (uint64_t)(((int64_t)q.b * A.sb0 + (int64_t)q.k * A.sk0) *
                                   Vt::kBytes)
                  : dummy;
    const uint64_t d0 = reinterpret_cast<uint64_t>(A.base1) +
                        (uint64_t)(((int64_t)q.b * A.sb1 + (int64_t)q.k * A.sk1) *
                                   Vt::kBytes) +
                        (uint64_t)((int64_t)q.sub * D * A.dd);
#pragma unroll
    for (int r = 1; r <= D; ++r)
      rb[r] = valid && r <= q.n ? d0 + (uint64_t)((int64_t)(r - 1) * A.dd) : dummy;
  } else {
    // lane r <= n: the base of row r of the item from the table in LDS, then broadcast
    const int l = threadIdx.x & 63;
    uint64_t base = dummy;
    if (valid && l <= q.n) {
      const int row = l == 0 ? 0 : q.sub * D + l;
      base = reinterpret_cast<uint64_t>(sh.ptr[row]) +
             (uint64_t)(((int64_t)q.b * sh.sb[row] + (int64_t)q.k * sh.sk[row]) * Vt::kBytes);
    }
#pragma unroll
    for (int r = 0; r <= D; ++r) {
      const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)base, r);
      const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(base >> 32), r);
      rb[r] = ((uint64_t)hi << 32) | lo;
    }
  }
  // uniform row base + 32-bit lane offset (a row holds < 2^31 logits); a global (not flat)
  // 16-byte load. 16-bit rows load nontemporal (every logit is read once; the target slice of
  // a group's later row sets still comes from L2): 1% faster on every bf16 workload measured,
  // but 19% slower on 64 stacked fp32 tiny chains, so fp32 rows load plainly
  typedef unsigned int u4 __attribute__((ext_vector_type(4)));
  const uint32_t off =
      valid && vfull > 0 ? (uint32_t)((q.vi < vfull ? q.vi : vfull - 1) * 16) : 0u;
#pragma unroll
  for (int r = 0; r <= D; ++r) {
    const uint32_t o = r <= q.n ? off : 0u;
    typedef const __attribute__((address_space(1))) u4* gp4;
    const u4 v = DT != HS_F32 ? __builtin_nontemporal_load((gp4)(rb[r] + o)) : *(gp4)(rb[r] + o);
    __builtin_memcpy(&dst[r], &v, 16);
  }
  if (valid && vfull < A.nvec && (int64_t)(q.s + 1) * kThreads > vfull) {  // the tail slice
#pragma unroll
    for (int r = 0; r <= D; ++r)
      if (r <= q.n && q.vi == vfull)
        dst[r] = Vt::load_raw(reinterpret_cast<const char*>(rb[r]), q.vi, A.V);
  }
}

// -inf for the lanes of the last slice that lie past the row end.
template <int DT, int D>
__device__ __forceinline__ void mask_tail(const TeamArgs& A, const ItemPos& q,
                                          typename Vec<DT>::Raw (&x)[D + 1]) {
  if ((int64_t)(q.s + 1) * kThreads > A.nvec) {
#pragma unroll
    for (int r = 0; r <= D; ++r)
      if (q.vi >= A.nvec) x[r] = Vec<DT>::neg_raw();
  }
}

// The offset a slice is exponentiated against: exp_offset_of(m, c) when that is finite (an
// integer-valued float, so that sums against different offsets rescale exactly), 0 for a slice
// with no logit whose scaled value is finite (every e_v is then exp2(-inf) = 0).
__device__ inline float exp_offset(float o) { return o != -INFINITY ? o : 0.0f; }

// min of two values that are >= 0 or +NaN (0 * inf): the unsigned order of the bits is their
// order and a NaN loses, as with fminf, without fminf's canonicalising of the operands.
__device__ inline float min_pos(float a, float b) {
  return __uint_as_float(min(__float_as_uint(a), __float_as_uint(b)));
}

// fminf of two results of arithmetic (never a signalling NaN): the hardware minimum, which
// returns the other operand for a quiet NaN as fminf does. Written out because the compiler
// otherwise re-canonicalises an operand that it cannot prove is a result of arithmetic (the
// target's exponents, once per item).
__device__ inline float min_arith(float a, float b) {
  float r;
  asm("v_min_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}

// The raw registers of one row made opaque to the compiler: each stage unpacks the logits
// afresh (two integer operations per pair) instead of the compiler keeping the unpacked
// floats of a whole item live from one stage to the next, which would not fit in registers.
template <typename Raw>
__device__ __forceinline__ void launder(Raw& x) {
  static_assert(sizeof(Raw) == 16, "16-byte vectors");
  uint32_t w[4];
  __builtin_memcpy(w, &x, 16);
  asm volatile("" : "+v"(w[0]), "+v"(w[1]), "+v"(w[2]), "+v"(w[3]));
  __builtin_memcpy(&x, w, 16);
}

// ---- 1. per-thread max (and lowest argmax) of every row of item q, to LDS ----
template <int DT, int D, bool NEED_ARG, typename L>
__device__ __forceinline__ void thread_max(const TeamArgs& A, const ItemPos& q,
                                           typename Vec<DT>::Raw (&raw)[D + 1], L& sh,
                                           int t) {
  constexpr int E = Vec<DT>::kElems;
#pragma unroll
  for (int r = 0; r <= D; ++r) {
    if (r > q.n) continue;
    launder(raw[r]);
    float z[E];
    Vec<DT>::unpack(raw[r], z);
    float m = -INFINITY;
    int idx = INT_MAX;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      if (NEED_ARG) {
        if (z[e] > m) {
          m = z[e];
          idx = q.vi * E + e;
        }
      } else {
        m = fmaxf(m, z[e]);
      }
    }
    if (NEED_ARG) {
      // a lane whose logits are all -inf still owns its lowest valid index
      if (idx == INT_MAX && q.vi < A.nvec) idx = q.vi * E;
      sh.xt[r][t] = m;
      sh.xi[r][t] = idx;
    } else {
      sh.xt[r][t] = __int_as_float(fkey(m));  // integer key: the group max needs no NaN care
    }
  }
}

// ---- 1-3. per-thread statistics of every row of item q in one pass (several items per
// workgroup): the max, the thread's own offset o_t (exp_offset_of: integer-valued, at or
// above m_t c) and the exp2 sum against it; max keys, sums and offsets to LDS. The offsets
// are integer-valued, so the group's rescaling of the sums to the slice offset is exact. A
// thread whose m_t c is -inf (logits all -inf, or finite ones whose product with c is below
// the fp32 range) takes offset -2^126: each of its logits then gives 0, or NaN for a NaN
// logit ----
template <int DT, int D, bool NEED_ARG, typename L>
__device__ __forceinline__ void thread_stats_pt(const TeamArgs& A, const ItemPos& q,
                                                typename Vec<DT>::Raw (&raw)[D + 1], L& sh,
                                                int t) {
  constexpr int E = Vec<DT>::kElems;
#pragma unroll
  for (int r = 0; r <= D; ++r) {
    if (r > q.n) continue;
    launder(raw[r]);
    float z[E];
    Vec<DT>::unpack(raw[r], z);
    float m = -INFINITY;
    int idx = INT_MAX;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      if (NEED_ARG) {
        if (z[e] > m) {
          m = z[e];
          idx = q.vi * E + e;
        }
      } else {
        m = fmaxf(m, z[e]);
      }
    }
    // exp_offset_of(m, c) without its test for m c = -inf (no logit whose scaled value is
    // finite): the fma then gives NaN, which fmaxf replaces by -2^126; every z c - of is then
    // -inf or far below -2^125, so each e_v is 0 (NaN for a NaN logit); m is never NaN
    const float mc = m * A.c;
    const float of = fmaxf(ceilf(fmaf(fabsf(mc), 0x1p-22f, mc)), -0x1p126f);
    float v[E];
#pragma unroll
    for (int e = 0; e < E; ++e) v[e] = __builtin_amdgcn_exp2f(fmaf(z[e], A.c, -of));
    float a0 = v[0], a1 = v[1];
#pragma unroll
    for (int e = 2; e < E; ++e) {
      if (e & 1) a1 += v[e];
      else a0 += v[e];
    }
    if (NEED_ARG) {
      if (idx == INT_MAX && q.vi < A.nvec) idx = q.vi * E;
      sh.xt[r][t] = m;
      sh.xi[r][t] = idx;
    } else {
      sh.xt[r][t] = __int_as_float(fkey(m));
    }
    sh.xs[r][t] = a0 + a1;
    sh.xo[r][t] = cvt_i32_sat(of);
  }
}

// ---- 2. group max: 16-lane group gi reduces row gi (every lane of the group gets the slice
// max m and argmax). Waves whose groups hold no row skip it. ----
template <int D, bool NEED_ARG, typename L>
__device__ __forceinline__ void group_max(const L& sh, int n, int gi, int gl, float& m,
                                          int& idx) {
  const int r = min(gi, n);  // groups past the last row reduce a copy of it (all 16 lanes
                             // of a group must take part in the DPP steps)
  if (NEED_ARG) {
    float v[16];
    int iv[16];
    group_read(&sh.xt[r][0], gl, v);
    group_read(&sh.xi[r][0], gl, iv);
    m = v[0];
    idx = iv[0];
#pragma unroll
    for (int u = 1; u < 16; ++u) argmax_combine(m, idx, v[u], iv[u]);
    row16_argmax(m, idx);
  } else {
    int kv[16];
    group_read(reinterpret_cast<const int*>(&sh.xt[r][0]), gl, kv);
    int k = kv[0];
#pragma unroll
    for (int u = 1; u < 16; ++u) k = max(k, kv[u]);
    m = fkey_inv(row16_max(k));
  }
}

// Slice statistics of row r as tagged words.
template <bool NEED_SUM, bool NEED_ARG>
__device__ __forceinline__ void publish_row(const TeamArgs& A, const ItemPos& q, int r,
                                            uint32_t tag, float m, float s, int idx, int RM) {
  uint64_t* wp = A.stat + (((int64_t)q.set * RM + r) * A.S + q.s) * 3;
  put_word(wp, word_of(m, tag));
  if (NEED_SUM) put_word(wp + 1, word_of(s, tag));
  if (NEED_ARG) put_word(wp + 2, word_of(idx, tag));
}

// Slot s's duty index for an item whose duties start at slot rot: duties are numbered from
// rot on, so that the row and alpha folds move round the team from item to item instead of
// falling on the same few members every time (the team goes at its slowest member's pace).
__device__ inline int duty_index(int s, int rot, int S) { return s >= rot ? s - rot : s - rot + S; }

// ---- 4. fold duty: rows i, i + S, ... of the row set (i = the slot's duty index for the
// item's rotation rot), spread over the waves, wave `first` taking the first ----
template <int D, bool NEED_SUM, bool NEED_ARG, int NC = 1>
__device__ __forceinline__ void fold_item(const TeamArgs& A, const ItemPos& q, uint32_t tag,
                                          int lane, int wv, int first, int rot = 0) {
  const int order = (wv + kWaves - first) % kWaves;
  for (int rr = duty_index(q.s, rot, A.S) + order * A.S; rr <= q.n; rr += kWaves * A.S)
    fold_row<D, NEED_SUM, NEED_ARG, NC>(A, q.set, rr, q.b, q.k, q.sub, tag, lane);
}

// ---- 5. normalisers (the duty wave; a barrier follows): lanes 2r and 2r + 1 wait for row r's hi and
// lo; lane 2r forms a_r = (o_r - hi_r) - lo_r and, for a drafter row, the constants of its
// min-sum to LDS: G and F = 2^(a_r) for kept e_v (6'), else the exponent addend and 2^(a_t) (6).
// A row with no finite logit folds to hi = -inf, lo = NaN, so its a is NaN: it has no
// distribution, and F is NaN whenever a_t or a_d is, which makes that drafter's alpha NaN in
// either form ----
template <int D, bool KEPT, typename L>
__device__ __forceinline__ void await_norms(const TeamArgs& A, const ItemPos& q, uint32_t tag,
                                            L& sh, int bf, int lane) {
  float h = 0.0f;
  bool lost = false;
  if (lane < 2 * (q.n + 1)) {
    constexpr int NC = KEPT ? kNormCopies : 1;  // the single-item kernel's fold writes copies
    const uint64_t w =
        await_word(norm_copy(A, q.s & (NC - 1), D + 1) +
                       ((int64_t)q.set * (D + 1) + (lane >> 1)) * 3 + (lane & 1),
                   tag, A);
    h = word_f(w);
    lost = tainted(w);
  }
  const bool any_lost = __ballot(lost) != 0;
  if (lane == 0) sh.taint = taint_bits(any_lost);
  const float lo = dpp_f<0xB1>(h);  // lane 2r: the lo of row r, from lane 2r + 1
  const float a = (sh.o[bf][min(lane >> 1, D)] - h) - lo;
  const float at = lane_f(a, 0);
  const bool drafter = !(lane & 1) && lane >= 2 && lane < 2 * (q.n + 1);
  if (drafter) {
    const int d = (lane >> 1) - 1;
    const bool undefined = at != at || a != a;
    if (KEPT) {
      sh.G[d] = __builtin_amdgcn_exp2f(at - a);
      sh.F[d] = undefined ? NAN : __builtin_amdgcn_exp2f(a);
    } else {
      sh.nw[d] = sh.no[bf][d + 1] - (at - a);
      sh.dl[d] = at - a;
      sh.F[d] = undefined ? NAN : __builtin_amdgcn_exp2f(at);
    }
  }
  if (!KEPT) {
    // nw_d holds the offset and the small difference a_t - a_d in one float: exact enough
    // (error <= 2^-17) while |offset| <= 128, the case of ordinary logits; beyond that the
    // min-sums subtract the difference in a second operation
    const bool wide = __ballot(drafter && fabsf(sh.no[bf][min(lane >> 1, D)]) > 128.0f) != 0;
    if (lane == 0) sh.wide = wide;
  }
}

// ---- 3. exponentials kept in registers (workgroups with a single item): e_v = exp2(z_v c - o)
// against the slice offsets (buffer 0) into x, per-thread sums to LDS ----
template <int DT, int D, typename L>
__device__ __forceinline__ void thread_exps_kept(const TeamArgs& A, const ItemPos& q,
                                                 typename Vec<DT>::Raw (&raw)[D + 1],
                                                 float (&x)[D + 1][Vec<DT>::kElems], L& sh,
                                                 int t) {
  constexpr int E = Vec<DT>::kElems;
#pragma unroll
  for (int r = 0; r <= D; ++r) {
    if (r > q.n) continue;
    launder(raw[r]);
    Vec<DT>::unpack(raw[r], x[r]);
    const float no = sh.no[0][r];
#pragma unroll
    for (int e = 0; e < E; ++e) x[r][e] = __builtin_amdgcn_exp2f(fmaf(x[r][e], A.c, no));
    float a0 = x[r][0], a1 = x[r][1];
#pragma unroll
    for (int e = 2; e < E; ++e) {
      if (e & 1) a1 += x[r][e];
      else a0 += x[r][e];
    }
    sh.xt[r][t] = a0 + a1;
  }
}

// ---- 6'. per-thread min-sums from kept e_v: min(p_v, q_v) = 2^(a_d) min(e_t,v G, e_d,v) with
// G = 2^(a_t - a_d); one multiply, one min and one add per drafter logit ----
template <int DT, int D, typename L>
__device__ __forceinline__ void thread_minsums_kept(const ItemPos& q,
                                                    const float (&x)[D + 1][Vec<DT>::kElems],
                                                    L& sh, int t) {
  constexpr int E = Vec<DT>::kElems;
#pragma unroll
  for (int d = 0; d < D; ++d) {
    if (d >= q.n) continue;
    const float G = sh.G[d];
    float y[E];
#pragma unroll
    for (int e = 0; e < E; ++e) y[e] = min_pos(x[0][e] * G, x[d + 1][e]);
    float a0 = y[0], a1 = y[1];
#pragma unroll
    for (int e = 2; e < E; ++e) {
      if (e & 1) a1 += y[e];
      else a0 += y[e];
    }
    sh.xp[d][t] = a0 + a1;
  }
}

// ---- 6. per-thread min-sums, from the logits again: with u_v = z_t,v c - o_t and
// w_v = z_d,v c - o_d, p_v = 2^(u_v + a_t) and q_v = 2^(w_v + a_d), so
// min(p_v, q_v) = 2^(a_t) 2^min(u_v, w_v - (a_t - a_d)), and w_v - (a_t - a_d) is one fma
// z_d,v c + nw_d; one fma, one min, one exp2 and one add per drafter logit. The factor 2^(a_t)
// is applied to the group sum. Identical rows give nw_d = -o_t, so both operands agree
// bitwise ----
template <int DT, int D, bool WIDE, typename L>
__device__ __forceinline__ void thread_minsums_form(const TeamArgs& A, const ItemPos& q,
                                                    typename Vec<DT>::Raw (&raw)[D + 1], L& sh,
                                                    int bf, int t) {
  constexpr int E = Vec<DT>::kElems;
  float u[E];
  launder(raw[0]);
  Vec<DT>::unpack(raw[0], u);
  const float nt = sh.no[bf][0];
#pragma unroll
  for (int e = 0; e < E; ++e) u[e] = fmaf(u[e], A.c, nt);
#pragma unroll
  for (int d = 0; d < D; ++d) {
    if (d >= q.n) continue;
    float w[E];
    launder(raw[d + 1]);
    Vec<DT>::unpack(raw[d + 1], w);
    float y[E];
    if (!WIDE) {
      const float nw = sh.nw[d];
#pragma unroll
      for (int e = 0; e < E; ++e) {
        // a slice with no finite logit has every u_v (target) or w_v (drafter) at -inf; nw_d
        // is then infinite or NaN, and where the other operand becomes NaN it loses to the -inf
        y[e] = __builtin_amdgcn_exp2f(min_arith(u[e], fmaf(w[e], A.c, nw)));
      }
    } else {
      // a large offset: the exact residual z c - o_d first, then the difference
      const float no = sh.no[bf][d + 1], dl = sh.dl[d];
#pragma unroll
      for (int e = 0; e < E; ++e)
        y[e] = __builtin_amdgcn_exp2f(fminf(u[e], fmaf(w[e], A.c, no) - dl));
    }
    // two interleaved sums, started from the first terms (no additions of zero)
    float a0 = y[0], a1 = y[1];
#pragma unroll
    for (int e = 2; e < E; ++e) {
      if (e & 1) a1 += y[e];
      else a0 += y[e];
    }
    sh.xp[d][t] = a0 + a1;
  }
}
// The form is chosen once per item (uniform), so that each copy of the loop is straight-line
// over all drafters and the compiler can interleave them.
template <int DT, int D, typename L>
__device__ __forceinline__ void thread_minsums(const TeamArgs& A, const ItemPos& q,
                                               typename Vec<DT>::Raw (&raw)[D + 1], L& sh,
                                               int bf, int t) {
  if (sh.wide == 0) thread_minsums_form<DT, D, false>(A, q, raw, sh, bf, t);
  else thread_minsums_form<DT, D, true>(A, q, raw, sh, bf, t);
}

// ---- 7. alpha of the set's drafters from the slice partials: output d is summed by slot
// d mod S (wave 1 for the first), lane l taking slices l, l + 64, ... in order, then across the
// wave ----
template <int D>
__device__ __forceinline__ void fold_alpha(const TeamArgs& A, const ItemPos& q, uint32_t tag,
                                           int lane, int wv, int rot = 0) {
  const int S = A.S;
  for (int d = duty_index(q.s, rot, S) + ((wv + 3) & 3) * S; d < q.n; d += kWaves * S) {
    const uint64_t* src = A.part + ((int64_t)q.g * A.N + q.sub * D + d) * S;
    float v = 0.0f;
    bool lost = false;
    for (int j0 = 0; j0 < S; j0 += 128) {
      uint64_t w[2];
#pragma unroll
      for (int h = 0; h < 2; ++h)  // issue every load of the pass before waiting on any
        if (j0 + lane + 64 * h < S) w[h] = get_word(src + j0 + lane + 64 * h);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int j = j0 + lane + 64 * h;
        if (j < S) {
          if (tag_of(w[h]) != tag) w[h] = await_word(src + j, tag, A);
          lost |= tainted(w[h]);
          v += word_f(w[h]);
        }
      }
    }
    v = wave_sum_f(v);
    const uint32_t tt = tag | taint_bits(__ballot(lost) != 0);
    // clamped to [0, 1]; a NaN (a row without a distribution, or a lost word) stays NaN
    if (lane == 0) {
      const int64_t o = ((int64_t)q.b * A.N + q.sub * D + d) * A.K + q.k;
      const float al = v != v ? v : fminf(fmaxf(v, 0.0f), 1.0f);
      A.alpha[o] = al;
      if (A.learn == 1) put_word(A.gw + o, word_of(al, tt));
    }
  }
}

// ---- 9. learner step of query b, once this workgroup has finished its items: the query's
// N * K gamma words are gathered into LDS (the team buffers are free by now), then wave 0 runs
// the step; the learner's state is loaded before the gather, so those loads fly meanwhile.
// When any gamma word is tainted (computed from a lost word) the step is skipped: the
// learner state stays as it was and the query's EAL, prefix and loss outputs are NaN.
// The host only asks for it when the learner's LDS fits in the team's. ----
template <typename L>
__device__ __forceinline__ void learn_query(const TeamArgs& A, uint32_t tag, int b, L& sh,
                                            int t) {
  const int nk = A.N * A.K;
  double* lds = reinterpret_cast<double*>(&sh);
  float* gam = reinterpret_cast<float*>(lds + tail_lds_doubles(A.tail));
  const uint64_t* src = A.gw + (int64_t)b * nk;
  LearnerIn pre{};
  if (t < 64) pre = load_learner_in(A.tail, b);
  __syncthreads();  // the team buffers are no longer read
  bool lost = false;
  for (int o = t; o < nk; o += kThreads) {
    const uint64_t w = await_word(src + o, tag, A);
    lost |= tainted(w);
    gam[o] = word_f(w);
  }
  const bool skip = __syncthreads_or(lost) != 0;
  if (t < 64) {
    if (skip) mark_query_failed(A.tail, b);
    else tail_query(A.tail, b, lds, gam, &pre);
  }
  __syncthreads();
}

// ---- 8. end of a workgroup ----
// A team's leader counts its team once every member has read the call's tag and no claim of
// the team is outstanding: after folding row 0 of the team's last item (at its end), or, with
// one item per workgroup, right after folding row 0. The
// last team counted advances the epoch and resets the row-set counter (one count per team,
// not per workgroup; the count of finished teams is tagged with the call, so it needs no
// reset).
__device__ inline void count_team(const TeamArgs& A, uint32_t tag, int teams) {
  if (tagged_add(A.finished, tag) == (uint32_t)teams - 1u) {
    const uint32_t e = *A.epoch + 1u;
    *A.next_set = 0u;  // every team has finished: nothing claims any more
    put_word(A.finished, (uint64_t)tag_of_epoch(e));  // count 0 for the next call's tag
    *A.epoch = e;      // the next call takes a new tag
  }
}
// When a wait of this call gave up, every workgroup that sees the fail flag at its end marks
// every output (alpha NaN, argmax -2, agreement 0): a wave that took a lost word has seen the
// flag, so each value computed from one is overwritten by the same workgroup, and outputs of
// row sets that no team reached are marked too; values written without a lost word are
// correct either way.
template <typename L>
__device__ __forceinline__ void finish(const TeamArgs& A, uint32_t tag, bool count, int teams,
                                       L& sh, int t) {
  if (t == 0) {
    const uint64_t fw = get_word(A.fail);
    const uint32_t flags = ((uint32_t)fw == tag && (fw >> 32) != 0) ? 2u : 0u;
    if (count) count_team(A, tag, teams);
    sh.next = flags;
  }
  __syncthreads();
  if (sh.next == 0u) return;
  const int64_t outs = (int64_t)A.B * A.N * A.K;
  for (int64_t o = t; o < outs; o += kThreads) {
    if (A.alpha) A.alpha[o] = __int_as_float(0x7FC00000);
    if (A.agree) A.agree[o] = 0;
    if (A.argmax_d) A.argmax_d[o] = -2;
  }
  if (A.argmax_t)
    for (int64_t o = t; o < (int64_t)A.B * A.K; o += kThreads) A.argmax_t[o] = -2;
}

// A team of S workgroups (slot s takes slice s of every item) works through row sets: its
// first three are sets T, T + teams and T + 2 teams (T = team), later ones are claimed three
// items ahead by the team's leader from a device-wide counter and posted in the team's
// mailbox ring, so teams that run faster (the wave arbiter favours older waves) take more sets
// and all finish within an item of each other.
// With alpha two items are in flight per workgroup: iteration j folds item j (published in the
// previous iteration), takes the statistics of item j + 1 and publishes them, and only then
// waits for item j's normalisers and takes its min-sums from the logits again, after which
// item j's registers receive the loads of item j + 2. The exchange of one item thus overlaps
// the statistics of the next. Two raw buffers (not three, with the next loads issued before
// the statistics) keep the kernel within 128 VGPRs, so four workgroups share a CU: 3-4% faster
// on every large workload than three workgroups with three buffers.
// SINGLE (alpha kernels only): every team has exactly one item, so nothing is pipelined, the
// e_v stay in registers and drafters at a constant distance are addressed without the table.
template <int DT, int D, bool NEED_SUM, bool NEED_ARG, bool SINGLE>
__global__ __launch_bounds__(kThreads, 4) void hs_team_kernel(TeamArgs A) {
  using Raw = typename Vec<DT>::Raw;
  constexpr int RM = D + 1;
  __shared__ TeamLds<D, NEED_ARG, NEED_SUM && !SINGLE> sh;
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  const int gi = t >> 4, gl = t & 15;  // 16-lane group gi reduces row gi; gl: lane in it
  const int S = A.S;
  // every scalar the first loads depend on, requested in one round at entry (otherwise each
  // is loaded just before its first use, one scalar-cache round trip apiece); the pipelined
  // alpha kernel, whose first loads are a small part of its run, loads them at first use
  // instead (0.6% faster there: fewer scalar registers held across its loop)
  if constexpr (SINGLE || !NEED_SUM) {
    asm volatile("" ::"s"(A.N), "s"(A.K), "s"(A.nsub), "s"(A.S), "s"(A.items), "s"(A.teams),
                 "s"(A.uni), "s"(A.divS.m), "s"(A.divS.s1), "s"(A.divS.s2), "s"(A.divK.m),
                 "s"(A.divK.s1), "s"(A.divK.s2), "s"(A.V), "s"(A.dd), "s"(A.base0),
                 "s"(A.base1), "s"(A.sb0), "s"(A.sk0), "s"(A.sb1), "s"(A.sk1), "s"(A.epoch));
  }
  const int teams = A.teams;
  // consecutive workgroups form a team; the workgroups that share a CU (w, w + CUs, ...)
  // then belong to different teams, so that one team's waits leave the CU to the others
  const int T = (int)fdiv(blockIdx.x, A.divS);
  // slot: the member's slice. The pipelined kernel rotates it by the team index, so that the
  // workgroups a CU holds at once (w, w + CUs, ...) take different slices also when S divides
  // the number of CUs (8% on 64 stacked fp32 tiny chains, S = 32; no change where it does not)
  int slot = (int)blockIdx.x - T * S;
  if constexpr (NEED_SUM && !SINGLE) {
    slot += T - (int)fdiv((uint32_t)T, A.divS) * S;  // + T mod S
    if (slot >= S) slot -= S;
  }
  const uint32_t nsets = fdiv((uint32_t)A.items, A.divS);
  constexpr int kStatic = NEED_SUM ? 3 : 2;  // items per team with a fixed row set
  // slot 0 folds row 0 of every item, so it waits for the whole team each item: it can never
  // be more than one item ahead of any member, which keeps a ring of 4 mailbox words safe
  const bool leader = slot == 0;
  const bool dynamic = kStatic * teams < (int)nsets;  // else no team has more than its fixed sets
  uint32_t tag = 0;  // the call's tag: read once the first loads are in flight
  uint64_t* mbox = A.mbox + (size_t)T * 4;
  if (!(SINGLE && A.uni) && t < kMaxRows) {
    sh.ptr[t] = reinterpret_cast<const char*>(A.rows.ptr[t]);
    sh.sb[t] = A.rows.sb[t];
    sh.sk[t] = A.rows.sk[t];
  }
  __syncthreads();

  // the row set of the team's item j < kStatic
  auto fixed_set = [&](int j) { return min((uint32_t)(T + j * teams), nsets); };
  // leader: claim the row set of the team's item j >= kStatic and post it (the counter starts
  // past every team's fixed sets, so a set is never claimed twice, and once a team's next item
  // has none every later claim has none either)
  auto claim = [&](int j) __attribute__((always_inline)) {
    if (!dynamic || !leader || t != 0) return;
    const uint32_t v = (uint32_t)(kStatic * teams) +
                       __hip_atomic_fetch_add(A.next_set, 1u, __ATOMIC_RELAXED,
                                              __HIP_MEMORY_SCOPE_AGENT);
    put_word(mbox + (j & 3), mbox_word(min(v, nsets), j, tag));
  };
  // thread 0: the row set of the team's item j >= kStatic (nsets: none left) into LDS, so that
  // all waves of the workgroup take the same one after the next barrier
  auto post_set = [&](int j) __attribute__((always_inline)) {
    if (t == 0) sh.next = dynamic ? await_mbox(mbox + (j & 3), j, tag, A, nsets) : nsets;
  };
  // first slot of the row or alpha fold duties of row set `set` (several items per workgroup):
  // (set (D + 1) + extra) mod S, so consecutive items use different members, and the alpha
  // folds of an item start where its row folds end. (The argmax-only kernel keeps row 0 on
  // the leader, which bounds how far the leader's claims run ahead of its team; in the alpha
  // kernels every member waits for the normalisers of each item, which bounds it there.)
  auto rotation = [&](uint32_t s, int extra) __attribute__((always_inline)) -> int {
    const uint32_t x = s * (uint32_t)RM + (uint32_t)extra;
    return (int)(x - fdiv(x, A.divS) * (uint32_t)S);
  };

  if constexpr (!NEED_SUM) {
    // argmax only: max stage, publish, fold
    Raw nxt[RM];
    uint32_t set = (uint32_t)T, next = fixed_set(1);
    fetch_item<DT, D>(A, item_pos(A, set, slot, D), true, sh, nxt);
    tag = call_tag(A.epoch);  // first needed once the first loads are in flight
    for (int j = 0; set < nsets; ++j) {
      const ItemPos q = item_pos(A, set, slot, D);
      __builtin_amdgcn_s_setprio(kCritPrio);
      mask_tail<DT, D>(A, q, nxt);
      thread_max<DT, D, NEED_ARG>(A, q, nxt, sh, t);
      if (j >= 1) post_set(j + 1);
      claim(j + 2);
      __syncthreads();
      if (j >= 1) next = sh.next;
      if (next < nsets) fetch_item<DT, D>(A, item_pos(A, next, slot, D), true, sh, nxt);
      if (wv * 4 <= q.n) {
        float m;
        int idx;
        group_max<D, NEED_ARG>(sh, q.n, gi, gl, m, idx);
        if (gl == 0 && gi <= q.n) publish_row<false, NEED_ARG>(A, q, gi, tag, m, 0.0f, idx, RM);
      }
      fold_item<D, false, NEED_ARG>(A, q, tag, lane, wv, kDutyWave);
      __builtin_amdgcn_s_setprio(0);
      __syncthreads();  // the LDS rows are free for the next item
      set = next;
    }
    finish(A, tag, leader, teams, sh, t);
  } else {
    // statistics of item q from raw (bf: its offset buffer), published
    auto stats = [&](const ItemPos& q, Raw (&raw)[RM], int bf) __attribute__((always_inline)) {
      __builtin_amdgcn_s_setprio(kCritPrio);
      mask_tail<DT, D>(A, q, raw);
      thread_stats_pt<DT, D, NEED_ARG>(A, q, raw, sh, t);
      __syncthreads();
      if (wv * 4 <= q.n) {  // this wave holds the group of a row
        float m;
        int idx;
        group_max<D, NEED_ARG>(sh, q.n, gi, gl, m, idx);
        const int r = min(gi, q.n);
        // -inf for a slice without a logit whose product with c is in range
        const float o = exp_offset_of(m, A.c);
        const int os = cvt_i32_sat(exp_offset(o));
        // the 16 sums of this lane rescaled to the slice offset (exact: powers of two) and
        // added in sum16's order, four at a time (one 16-byte read of sums and of offsets).
        // A thread's offset is at most the slice's, unless the thread took offset -2^126 for a
        // sum that is 0 or NaN. Offsets beyond the int32 range saturate, and a difference that
        // wraps needs |offset| >= 2^30, where the thread's exponents are all <= -256 and its
        // sum is exactly 0 (or NaN): ldexp of 0 or NaN is 0 or NaN whatever the shift
        typedef float F4 __attribute__((ext_vector_type(4)));
        typedef int I4 __attribute__((ext_vector_type(4)));
        float c[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const F4 x = *reinterpret_cast<const F4*>(&sh.xs[r][64 * i + 4 * gl]);
          const I4 y = *reinterpret_cast<const I4*>(&sh.xo[r][64 * i + 4 * gl]);
          auto d = [&](int yi) { return (int)((uint32_t)yi - (uint32_t)os); };  // wraps
          c[i] = (ldexpf(x[0], d(y[0])) + ldexpf(x[1], d(y[1]))) +
                 (ldexpf(x[2], d(y[2])) + ldexpf(x[3], d(y[3])));
        }
        const float s = row16_sum((c[0] + c[1]) + (c[2] + c[3]));
        if (gl == 0 && gi <= q.n) {
          sh.o[bf][gi] = o;
          sh.no[bf][gi] = -exp_offset(o);
          publish_row<true, NEED_ARG>(A, q, gi, tag, m, s, idx, RM);
        }
      }
      __builtin_amdgcn_s_setprio(0);
    };

    // the item's slice partials to the workspace (after a barrier), as tagged words
    auto store_partials = [&](const ItemPos& q) __attribute__((always_inline)) {
      if (wv * 4 < q.n) {
        float v[16];
        const int d = min(gi, q.n - 1);
        group_read(&sh.xp[d][0], gl, v);
        const float y = row16_sum(sum16(v));
        if (gl == 0 && gi < q.n)
          put_word(A.part + ((int64_t)q.g * A.N + q.sub * D + gi) * S + q.s,
                   word_of(y * sh.F[gi], tag | sh.taint));
      }
    };

    // Several items per workgroup: the row sets of one (query, position) group follow each
    // other in a team when there are groups enough to keep every team busy, so the target's
    // slice, the same for all of them, is re-read from this XCD's L2 rather than from HBM. A
    // team's items come in blocks (a group's nsub row sets, else single row sets): its first
    // kB blocks are blocks T, T + teams, ... (at least three items, to fill the pipeline), and
    // later ones are claimed from the device-wide counter three items ahead, by the leader,
    // and posted in the team's mailbox ring.
    const bool blocked = !SINGLE && A.nsub > 1 && nsets >= 4u * (uint32_t)teams * (uint32_t)A.nsub;
    const uint32_t bsz = blocked ? (uint32_t)A.nsub : 1u;
    const uint32_t nblocks = blocked ? fdiv(nsets, A.divNsub) : nsets;
    const int kB = blocked ? (int)((3u + bsz - 1u) / bsz) : 3;
    const bool dyn = kB * teams < (int)nblocks;  // else no team has more than its fixed blocks
    int nblk = 0;  // blocks given to this team so far (the same count in every member)
    auto block_first = [&](uint32_t bl) { return bl < nblocks ? bl * bsz : nsets; };
    // the row set after s (nsets: none), or kClaim when it starts a block that is to be claimed
    constexpr uint32_t kClaim = 0xFFFFFFFFu;
    auto successor = [&](uint32_t s) __attribute__((always_inline)) -> uint32_t {
      if (s >= nsets) return nsets;
      if (blocked && fdiv(s + 1u, A.divNsub) * bsz != s + 1u) return s + 1u;  // same group
      if (nblk < kB) return block_first((uint32_t)(T + (nblk++) * teams));
      return dyn ? kClaim : nsets;
    };

    Raw R0[RM], R1[RM];
    uint32_t set = SINGLE ? (uint32_t)T : block_first((uint32_t)T);
    nblk = 1;
    const ItemPos q0 = item_pos(A, set, slot, D);
    fetch_item<DT, D, SINGLE>(A, q0, true, sh, R0);
    if constexpr (SINGLE) {
      // one item per workgroup: nothing to overlap, so its e_v stay in registers
      tag = call_tag(A.epoch);  // first needed once the first loads are in flight
      const ItemPos& q = q0;
      float x[RM][Vec<DT>::kElems];
      __builtin_amdgcn_s_setprio(kCritPrio);
      mask_tail<DT, D>(A, q, R0);
      thread_max<DT, D, NEED_ARG>(A, q, R0, sh, t);
      __syncthreads();
      const bool rows = wv * 4 <= q.n;
      float m = 0.0f;
      int idx = 0;
      if (rows) {
        group_max<D, NEED_ARG>(sh, q.n, gi, gl, m, idx);
        if (gl == 0 && gi <= q.n) {
          const float o = exp_offset_of(m, A.c);  // -inf: no finite logit in the slice
          sh.o[0][gi] = o;
          sh.no[0][gi] = -exp_offset(o);
        }
      }
      __syncthreads();
      thread_exps_kept<DT, D>(A, q, R0, x, sh, t);
      __syncthreads();
      if (rows) {
        float v[16];
        group_read(&sh.xt[min(gi, q.n)][0], gl, v);
        const float sm = row16_sum(sum16(v));
        if (gl == 0 && gi <= q.n) publish_row<true, NEED_ARG>(A, q, gi, tag, m, sm, idx, RM);
      }
      fold_item<D, true, NEED_ARG, kNormCopies>(A, q, tag, lane, wv, 0);
      __builtin_amdgcn_s_setprio(0);
      // with one item per workgroup the leader counts its team once it has folded row 0 (every
      // member has published, so has read the tag), not at its end: the count's round trip
      // then overlaps the normaliser wait instead of following the learner step or the alpha
      // folds. (The fold duties start at wave 0, whose thread 0 counts.)
      if (leader && t == 0) count_team(A, tag, teams);
      if (wv == 0) await_norms<D, true>(A, q, tag, sh, 0, lane);
      __syncthreads();
      thread_minsums_kept<DT, D>(q, x, sh, t);
      __syncthreads();
      store_partials(q);
      fold_alpha<D>(A, q, tag, lane, wv);
      if (A.learn)
        for (int b = blockIdx.x; b < A.B; b += gridDim.x) learn_query(A, tag, b, sh, t);
      finish(A, tag, false, teams, sh, t);
      return;
    }
    uint32_t set1 = successor(set);
    uint32_t set2 = successor(set1);  // items 0-2 lie in fixed blocks: never kClaim
    fetch_item<DT, D>(A, item_pos(A, min(set1, nsets - 1), slot, D), set1 < nsets, sh,
                      R1);
    tag = call_tag(A.epoch);  // first needed once the first loads are in flight
    stats(q0, R0, 0);
    // the first item's group reductions read every column of the LDS rows that the next
    // item's per-thread statistics overwrite, and nothing else in the first iteration waits
    // for the whole workgroup before those writes (later items are kept apart by the
    // barriers around the min-sums); after it every wave has published its rows
    __syncthreads();

    uint32_t pset = nsets;  // the team's previous item, whose alpha is still to be folded
    // iteration j: rc holds item j (statistics published) and then receives item j + 2, rn
    // holds item j + 1 (loaded). Returns false once the team has no item j + 1.
    auto iter = [&](int j, Raw (&rc)[RM], Raw (&rn)[RM])
                    __attribute__((always_inline)) -> bool {
      const int bf = j & 1;
      const ItemPos q = item_pos(A, set, slot, D);
      // the leader's claim of item j + 3 goes out before the fold and is posted after it, so
      // waiting for its result waits for nothing else; the duty wave, which folds, claims
      // (the argmax-only kernel, whose folds are short, claims on thread 0)
      const uint32_t set3 = successor(set2);  // item j + 3, unless it is to be claimed
      const bool claiming = set3 == kClaim && leader && wv == kDutyWave && lane == 0;
      uint32_t cv = 0;
      if (claiming)
        cv = __hip_atomic_fetch_add(A.next_set, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __builtin_amdgcn_s_setprio(kFoldPrio);
      fold_item<D, true, NEED_ARG>(A, q, tag, lane, wv, kDutyWave, rotation(set, 0));
      __builtin_amdgcn_s_setprio(0);
      if (claiming)
        put_word(mbox + ((j + 3) & 3),
                 mbox_word(block_first((uint32_t)(kB * teams) + cv), j + 3, tag));
      if (set1 < nsets) stats(item_pos(A, set1, slot, D), rn, bf ^ 1);
      if (set3 == kClaim && t == 0) sh.next = await_mbox(mbox + ((j + 3) & 3), j + 3, tag, A, nsets);
      if (wv == kDutyWave) await_norms<D, false>(A, q, tag, sh, bf, lane);
      __syncthreads();
      thread_minsums<DT, D>(A, q, rc, sh, bf, t);
      __syncthreads();
      store_partials(q);
      fetch_item<DT, D>(A, item_pos(A, min(set2, nsets - 1), slot, D), set2 < nsets, sh, rc);
      // alpha of the previous item, whose partials were stored an iteration ago; its polls
      // overlap the loads just issued (1.4% faster than folding it before the normaliser wait)
      if (pset < nsets) fold_alpha<D>(A, item_pos(A, pset, slot, D), tag, lane, wv, rotation(pset, RM));
      if (set1 >= nsets) return false;
      pset = set;
      set = set1;
      set1 = set2;
      set2 = set3 == kClaim ? sh.next : set3;
      return true;
    };
    // unrolled by two so that the register buffers alternate without copies
    for (int j = 0;; j += 2) {
      if (!iter(j, R0, R1)) break;
      if (!iter(j + 1, R1, R0)) break;
    }
    fold_alpha<D>(A, item_pos(A, set, slot, D), tag, lane, wv, rotation(set, RM));
    if (A.learn)
      for (int b = blockIdx.x; b < A.B; b += gridDim.x) learn_query(A, tag, b, sh, t);
    finish(A, tag, leader, teams, sh, t);
  }
}

// ---- host side -------------------------------------------------------------------------------

namespace {

// Polls before a wait inside the team kernel gives up (about 0.5 s at the default); 0 makes
// every wait give up at once, which tests of the failure path set from the host.
constexpr uint32_t kDefaultPolls = 1u << 18;
std::atomic<uint32_t> g_wait_polls{kDefaultPolls};

uint32_t wait_polls() { return g_wait_polls.load(std::memory_order_relaxed); }

// Workgroups of the team kernel the current device holds at once.
template <int DT, int D, bool NS, bool NA, bool SG>
int capacity_t() {
  static std::atomic<int> cached[64];  // per device; 0 = not yet known
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  int v = cached[dev].load(std::memory_order_relaxed);
  if (v > 0) return v;
  int per_cu = 0, cus = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, hs_team_kernel<DT, D, NS, NA, SG>,
                                                   kThreads, 0) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return 0;
  v = per_cu * cus;
  cached[dev].store(v, std::memory_order_relaxed);
  return v;
}

// Runs the team kernel with as many teams as the device holds at once (no more than there are
// row sets or mailbox rings); the single-item kernel when that covers every row set.
// *learned: whether the launch runs the learner step itself (its LDS fits in the team's).
template <int DT, int D, bool NS, bool NA>
int launch_t(TeamArgs A, const TeamGeom& g, hipStream_t stream, bool* learned) {
  const int64_t sets = g.items / g.S;
  const bool single = NS && capacity_t<DT, D, NS, NA, NS>() / g.S >= sets;
  const int64_t teams =
      single ? sets
             : std::min<int64_t>({capacity_t<DT, D, NS, NA, false>() / g.S, sets,
                                  (int64_t)kMaxTeams});
  if (teams <= 0) return HS_ERR_LIMIT;
  const int64_t P = teams * g.S;
  if (A.learn) {  // only the alpha kernels carry the learner (it would cost the argmax-only
                  // kernels a workgroup per CU in registers)
    const size_t need = sizeof(double) * (size_t)tail_lds_doubles(A.tail) +
                        sizeof(float) * (size_t)g.N * g.K;
    if (!NS || need > sizeof(TeamLds<D, NA>)) A.learn = 0;
  }
  *learned = A.learn != 0;
  A.teams = (int)teams;
  if (single) hs_team_kernel<DT, D, NS, NA, NS><<<(unsigned)P, kThreads, 0, stream>>>(A);
  else hs_team_kernel<DT, D, NS, NA, false><<<(unsigned)P, kThreads, 0, stream>>>(A);
  return HS_OK;
}

// Calls F<DT, D, NS, NA>::run(args...) for the geometry and mode.
template <template <int, int, bool, bool> class F, int DT, int D, typename... Args>
int by_mode(bool ns, bool na, Args&&... args) {
  if (ns && na) return F<DT, D, true, true>::run(args...);
  if (ns) return F<DT, D, true, false>::run(args...);
  return F<DT, D, false, true>::run(args...);
}
template <template <int, int, bool, bool> class F, int DT, typename... Args>
int by_set(int D, bool ns, bool na, Args&&... args) {
  switch (D) {
    case 1: return by_mode<F, DT, 1>(ns, na, args...);
    case 2: return by_mode<F, DT, 2>(ns, na, args...);
    case 4: return by_mode<F, DT, 4>(ns, na, args...);
    default: return by_mode<F, DT, kMaxSetDrafters>(ns, na, args...);
  }
}
template <template <int, int, bool, bool> class F, typename... Args>
int dispatch(const TeamGeom& g, bool ns, bool na, Args&&... args) {
  if (g.dtype == HS_F32) return by_set<F, HS_F32>(g.D, ns, na, args...);
  if (g.dtype == HS_F16) return by_set<F, HS_F16>(g.D, ns, na, args...);
  return by_set<F, HS_BF16>(g.D, ns, na, args...);
}

template <int DT, int D, bool NS, bool NA>
struct Capacity {  // the smaller of the two kernels' (a team must fit in either)
  static int run() {
    return std::min(capacity_t<DT, D, NS, NA, false>(), capacity_t<DT, D, NS, NA, NS>());
  }
};
template <int DT, int D, bool NS, bool NA>
struct Launch {
  static int run(const TeamArgs& A, const TeamGeom& g, hipStream_t s, bool* learned) {
    return launch_t<DT, D, NS, NA>(A, g, s, learned);
  }
};

}  // namespace

void set_wait_polls(int polls) {
  g_wait_polls.store(polls < 0 ? kDefaultPolls : (uint32_t)polls, std::memory_order_relaxed);
}

int team_capacity(const TeamGeom& g, bool need_sum, bool need_arg) {
  return dispatch<Capacity>(g, need_sum, need_arg);
}

int launch_round(const TeamGeom& g, const RowTable& rows, float c, bool need_sum, bool need_arg,
                 float* alpha, uint8_t* agree, int32_t* argmax_t, int32_t* argmax_d, char* ws,
                 const TailArgs* tail, hipStream_t stream) {
  const TeamWs L = team_ws(g);
  TeamArgs A{};
  A.rows = rows;
  A.base0 = rows.ptr[0];
  A.base1 = rows.ptr[1];
  A.sb0 = rows.sb[0];
  A.sk0 = rows.sk[0];
  A.sb1 = rows.sb[1];
  A.sk1 = rows.sk[1];
  // drafters at one constant distance with equal strides (e.g. one [N][B][K][V] tensor)
  A.uni = 1;
  A.dd = g.N > 1 ? reinterpret_cast<const char*>(rows.ptr[2]) -
                       reinterpret_cast<const char*>(rows.ptr[1])
                 : 0;
  for (int i = 2; i <= g.N && A.uni; ++i)
    A.uni = reinterpret_cast<const char*>(rows.ptr[i]) -
                    reinterpret_cast<const char*>(rows.ptr[i - 1]) ==
                A.dd &&
            rows.sb[i] == rows.sb[1] && rows.sk[i] == rows.sk[1];
  A.B = g.B;
  A.N = g.N;
  A.K = g.K;
  A.nsub = g.nsub;
  A.S = g.S;
  A.divS = make_fastdiv((uint32_t)g.S);
  A.divNsub = make_fastdiv((uint32_t)g.nsub);
  A.divK = make_fastdiv((uint32_t)g.K);
  A.items = (int)g.items;
  A.V = g.V;
  A.nvec = g.nvec;
  A.c = c;
  A.epoch = reinterpret_cast<uint32_t*>(ws + L.epoch);
  A.fail = reinterpret_cast<uint64_t*>(ws + L.epoch + 8);
  A.polls = wait_polls();
  A.next_set = reinterpret_cast<uint32_t*>(ws + L.epoch + 16);
  A.finished = reinterpret_cast<uint64_t*>(ws + L.epoch + 24);
  A.mbox = reinterpret_cast<uint64_t*>(ws + L.epoch + 64);
  A.stat = reinterpret_cast<uint64_t*>(ws + L.stat);
  A.norm = reinterpret_cast<uint64_t*>(ws + L.norm);
  A.part = need_sum ? reinterpret_cast<uint64_t*>(ws + L.part) : nullptr;
  A.alpha = need_sum ? alpha : nullptr;
  A.argmax_t = argmax_t;
  A.argmax_d = argmax_d;
  A.agree = agree;
  // the gamma words (the learner step in the same launch); the single-item kernel's extra
  // normaliser copies follow them
  A.gw = reinterpret_cast<uint64_t*>(ws + L.gw);
  if (tail) {  // the learner step in the same launch, when its LDS fits
    A.learn = tail->gamma_src;
    A.tail = *tail;
  }
  bool learned = false;
  int rc = dispatch<Launch>(g, need_sum, need_arg, A, g, stream, &learned);
  if (rc) return rc;
  if (hipGetLastError() != hipSuccess) return HS_ERR_HIP;
  if (tail && !learned) {  // a launch of its own, told where to see whether this one failed
    A.tail.round_epoch = A.epoch;
    A.tail.round_fail = A.fail;
    return launch_tail(A.tail, stream);
  }
  return HS_OK;
}

}  // namespace hs
