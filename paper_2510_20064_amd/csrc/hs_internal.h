// Internal declarations of libhedgespec: kernel geometry, workspace layout and
// device helpers shared by the evaluation, statistics and learner kernels.
// gfx950 (CDNA4): wave64, 256-thread workgroups, 16-byte global loads.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "hedgespec.h"

namespace hs {

constexpr int kThreads = 256;          // workgroup size of the streaming kernels (4 waves)
constexpr int kWaves = kThreads / 64;
constexpr int kSliceElems = 4096;      // logits per workgroup pass in hs_softmax_stats
constexpr int kMaxRows = HS_MAX_DRAFTERS + 1;
constexpr int kMaxSetDrafters = 8;     // drafters held on chip with the target by one workgroup
constexpr int kMaxTeamSlices = 512;    // slices per row (one workgroup each) in one team
constexpr int kMaxTeams = 4096;        // teams resident at once (one mailbox ring each)
// copies of each row's published normaliser (a power of two): with one item per workgroup
// every member of a team polls its row set's normaliser words at once, so each copy is read
// by a quarter of them
constexpr int kNormCopies = 4;

// Per-storage-type 16-byte vector: 4 fp32 or 8 bf16 or fp16 logits.
template <int DT>
struct Vec;
template <>
struct Vec<HS_F32> {
  static constexpr int kElems = 4;
  static constexpr int kBytes = 4;
  static constexpr int kU = kSliceElems / (kThreads * kElems);  // vectors per thread per slice
  using Raw = float4;
  // raw 16-byte vector vi of a row (logits at or beyond V read as -inf)
  __device__ static inline Raw load_raw(const char* rowp, int64_t vi, int64_t V) {
    if ((vi + 1) * kElems <= V) return *reinterpret_cast<const float4*>(rowp + vi * 16);
    const float* p = reinterpret_cast<const float*>(rowp);
    float z[kElems];
#pragma unroll
    for (int e = 0; e < kElems; ++e) z[e] = vi * kElems + e < V ? p[vi * kElems + e] : -INFINITY;
    return make_float4(z[0], z[1], z[2], z[3]);
  }
  __device__ static inline Raw zero_raw() { return make_float4(0.f, 0.f, 0.f, 0.f); }
  __device__ static inline Raw neg_raw() {
    return make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
  }
  __device__ static inline void unpack(const Raw& x, float* z) {
    z[0] = x.x; z[1] = x.y; z[2] = x.z; z[3] = x.w;
  }
  __device__ static inline void load(const char* rowp, int64_t vi, int64_t V, float* z) {
    if ((vi + 1) * kElems <= V) {
      float4 x = *reinterpret_cast<const float4*>(rowp + vi * 16);
      z[0] = x.x; z[1] = x.y; z[2] = x.z; z[3] = x.w;
    } else {
      const float* p = reinterpret_cast<const float*>(rowp);
#pragma unroll
      for (int e = 0; e < kElems; ++e) {
        int64_t idx = vi * kElems + e;
        z[e] = idx < V ? p[idx] : -INFINITY;
      }
    }
  }
};
// 8 16-bit logits per vector: bf16 (the upper half of an fp32) or fp16 (IEEE 754 binary16,
// converted exactly by the hardware's half-to-float conversion).
template <bool F16>
struct Vec16 {
  static constexpr int kElems = 8;
  static constexpr int kBytes = 2;
  static constexpr int kU = kSliceElems / (kThreads * kElems);
  static constexpr uint32_t kNegInf = F16 ? 0xFC00u : 0xFF80u;  // -inf
  // the value of the low (lo) or high (hi) half of a 32-bit word
  __device__ static inline float lo(uint32_t w) {
    if constexpr (F16) return (float)__builtin_bit_cast(_Float16, (uint16_t)w);
    else return __uint_as_float(w << 16);
  }
  __device__ static inline float hi(uint32_t w) {
    if constexpr (F16) return (float)__builtin_bit_cast(_Float16, (uint16_t)(w >> 16));
    else return __uint_as_float(w & 0xFFFF0000u);
  }
  using Raw = uint4;
  // raw 16-byte vector vi of a row (logits beyond V read as -inf)
  __device__ static inline Raw load_raw(const char* rowp, int64_t vi, int64_t V) {
    if ((vi + 1) * kElems <= V) return *reinterpret_cast<const uint4*>(rowp + vi * 16);
    const uint16_t* p = reinterpret_cast<const uint16_t*>(rowp);
    uint32_t h[kElems];
#pragma unroll
    for (int e = 0; e < kElems; ++e) h[e] = vi * kElems + e < V ? p[vi * kElems + e] : kNegInf;
    return make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16),
                      h[6] | (h[7] << 16));
  }
  __device__ static inline Raw zero_raw() { return make_uint4(0u, 0u, 0u, 0u); }
  __device__ static inline Raw neg_raw() {  // four pairs of -inf
    constexpr uint32_t w = kNegInf | (kNegInf << 16);
    return make_uint4(w, w, w, w);
  }
  __device__ static inline void unpack(const Raw& x, float* z) {
    z[0] = lo(x.x); z[1] = hi(x.x); z[2] = lo(x.y); z[3] = hi(x.y);
    z[4] = lo(x.z); z[5] = hi(x.z); z[6] = lo(x.w); z[7] = hi(x.w);
  }
  __device__ static inline void load(const char* rowp, int64_t vi, int64_t V, float* z) {
    if ((vi + 1) * kElems <= V) {
      uint4 x = *reinterpret_cast<const uint4*>(rowp + vi * 16);
      unpack(x, z);
    } else {
      const uint16_t* p = reinterpret_cast<const uint16_t*>(rowp);
#pragma unroll
      for (int e = 0; e < kElems; ++e) {
        int64_t idx = vi * kElems + e;
        z[e] = idx < V ? lo(p[idx]) : -INFINITY;
      }
    }
  }
};
template <>
struct Vec<HS_BF16> : Vec16<false> {};
template <>
struct Vec<HS_F16> : Vec16<true> {};

// Division of a 32-bit value by a divisor fixed for the launch, by a multiply-high and two
// shifts (Granlund and Montgomery, "Division by invariant integers using multiplication",
// 1994): with l = ceil(log2 d) and m = floor(2^32 (2^l - d) / d) + 1,
// q = (t + ((n - t) >> 1)) >> (l - 1), t = mulhi(m, n); d = 1 uses shifts 0 and 0.
struct FastDiv {
  uint32_t m, s1, s2;
};
inline FastDiv make_fastdiv(uint32_t d) {
  uint32_t l = 0;
  while (l < 32 && ((uint64_t)1 << l) < d) ++l;
  FastDiv f;
  f.m = (uint32_t)((((uint64_t)1 << 32) * (((uint64_t)1 << l) - d)) / d + 1);
  f.s1 = l > 0 ? 1 : 0;
  f.s2 = l > 0 ? l - 1 : 0;
  return f;
}
__device__ inline uint32_t fdiv(uint32_t n, const FastDiv& f) {
  const uint32_t t = __umulhi(f.m, n);
  return (t + ((n - t) >> f.s1)) >> f.s2;
}

// The R = N + 1 logits rows of a (query, position) group: row 0 target, row 1 + i drafter i.
struct RowTable {
  const void* ptr[kMaxRows];
  int64_t sb[kMaxRows];
  int64_t sk[kMaxRows];
};

// Geometry of the evaluation. A group is one (query, position): the target row and the N
// drafter rows. Its drafters are split into row sets of up to D (1, 2, 4 or 8), and each row
// is cut into S slices of kThreads 16-byte vectors. One work item = (row set, slice): the
// target slice and its row set's drafter slices, held by one workgroup.
struct TeamGeom {
  int B, N, K, G;     // G = B * K groups
  int D, nsub;        // drafters per row set, row sets per group
  int S;              // slices per row
  int64_t V, nvec;    // logits and 16-byte vectors per row
  int dtype;
  int64_t items;      // G * nsub * S
};

inline int team_set_size(int N) { return N <= 1 ? 1 : N <= 2 ? 2 : N <= 4 ? 4 : kMaxSetDrafters; }

// false if the shape is outside the limits of the evaluation kernel
inline bool team_geom(int B, int N, int K, int64_t V, int dtype, TeamGeom* g) {
  if (B < 1 || N < 1 || K < 1 || V < 1) return false;
  if (B > HS_MAX_QUERIES || N > HS_MAX_DRAFTERS || K > HS_MAX_POSITIONS || V > INT32_MAX)
    return false;
  if (dtype != HS_F32 && dtype != HS_BF16 && dtype != HS_F16) return false;
  const int E = dtype == HS_F32 ? 4 : 8;
  g->B = B;
  g->N = N;
  g->K = K;
  g->G = B * K;
  g->D = team_set_size(N);
  g->nsub = (N + g->D - 1) / g->D;
  g->V = V;
  g->nvec = (V + E - 1) / E;
  g->dtype = dtype;
  const int64_t S = (g->nvec + kThreads - 1) / kThreads;
  if (S > kMaxTeamSlices) return false;
  g->S = (int)S;
  g->items = (int64_t)g->G * g->nsub * g->S;
  // items index with int; row sets fit the 26 bits a mailbox word gives them
  return g->items < ((int64_t)1 << 31) && (int64_t)g->G * g->nsub < ((int64_t)1 << 26);
}

// Statistics of one row slice, in log2 units: offset o = fl(m * c) with c = log2(e)/T and
// s = sum_v exp2(z_v * c - o); every exponent is formed by one fused multiply-add against the
// same offset, so slices and threads combine exactly whatever the rounding of o.
struct SliceStat {
  float m;   // max of the raw logits
  int idx;   // lowest index attaining m
  float o;   // offset
  float s;   // sum of exp2(z c - o)
};

// Workspace of the evaluation (byte offsets, 256-aligned). Words exchanged between
// workgroups are 64-bit (value, tag) pairs; the tag is the call's epoch, kept in the
// workspace and advanced once per call, so words of earlier calls are never mistaken for
// current ones and nothing has to be cleared.
struct TeamWs {
  size_t epoch;  // control block: uint32 call counter at +0, the call's fail flag (word) at
                 // +8, the row-set count (tagged word) at +16, the count of teams that have
                 // finished (tagged word) at +24, then a ring of 4 mailbox words per team at +64
  size_t stat;   // [G * nsub][D + 1][S][3] words: slice max, exp2 sum, argmax
  size_t norm;   // [G * nsub][D + 1][3] words: log2 normaliser hi, lo, argmax
  size_t norm_copy;  // bytes of one copy of them (kNormCopies - 1 more follow the gamma words)
  size_t part;   // [G][N][S] words: per-slice sums of min(p, q_i)
  size_t gw;     // [B][N][K] words: gamma (alpha or agreement) for a learner in the same launch
  size_t total;
};

__host__ __device__ inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Tag of the evaluation call with epoch e: 31 bits (bit 31 of a word's tag half is its taint
// mark), never 0, the content of a zero-filled workspace.
__host__ __device__ inline uint32_t tag_of_epoch(uint32_t e) { return (e % 0x7FFFFFFFu) + 1u; }

// Words from one copy of the normaliser words to the next, for `sets` row sets of `rows` rows
// (the single-item kernel has one row set per team, so it passes its team count).
__host__ __device__ inline int64_t norm_copy_words(int64_t sets, int rows) {
  return (int64_t)align256((size_t)(24 * sets * rows)) / 8;
}

inline TeamWs team_ws(const TeamGeom& g) {
  TeamWs L;
  const size_t sets = (size_t)g.G * g.nsub, rows = (size_t)g.D + 1;
  size_t off = 0;
  L.epoch = off;
  off = align256(off + 64 + 32 * (size_t)kMaxTeams);
  L.stat = off;
  off = align256(off + 24 * sets * rows * g.S);
  L.norm = off;
  L.norm_copy = 8 * (size_t)norm_copy_words((int64_t)sets, (int)rows);
  off += L.norm_copy;
  L.part = off;
  off = align256(off + 8 * (size_t)g.G * g.N * g.S);
  L.gw = off;
  off = align256(off + 8 * (size_t)g.B * g.N * g.K);
  off += (kNormCopies - 1) * L.norm_copy;  // the normaliser words' other copies
  L.total = off;
  return L;
}

// ---- device reductions -------------------------------------------------------------------

__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Lexicographic (value descending, index ascending) argmax combine.
__device__ inline void argmax_combine(float& m, int& idx, float m2, int idx2) {
  if (m2 > m || (m2 == m && idx2 < idx)) {
    m = m2;
    idx = idx2;
  }
}

// The offset that the exp2 sums of a part of a row are taken against, m the part's largest
// logit: an integer-valued float at or above the exact product m c. fl(m c) can lie below it
// by half an ulp, which for |m c| >= 2^31 would put the largest exponent z c - offset (one
// fma, exactly rounded) above 128; the nudge by a factor 1 +- 2^-22 (at least 1.5 ulp)
// keeps every exponent <= 0, so no exp2 and no sum of them overflows, whatever the logits.
// The largest exponent is then >= -(1 + |m c| 2^-22): exact to fp32 accuracy while
// |m c| <= 2^28; beyond that a part's sum underflows towards 0 (such a part contributes
// as a masked one). -inf when m c is -inf: the part has no logit whose scaled value is finite.
__device__ inline float exp_offset_of(float m, float c) {
  const float mc = m * c;
  return mc > -INFINITY ? ceilf(fmaf(fabsf(mc), 0x1p-22f, mc)) : -INFINITY;
}

// fp32 -> int32 with the hardware's saturation (out-of-range values clamp to INT_MIN or
// INT_MAX, NaN gives 0), which the C++ conversion does not promise.
__device__ inline int cvt_i32_sat(float x) {
  int r;
  asm("v_cvt_i32_f32 %0, %1" : "=v"(r) : "v"(x));
  return r;
}

// Combine two (offset, sum) pairs of exp2 sums: sum_a 2^(o_a - o) + sum_b 2^(o_b - o).
// A pair whose offset is -inf has no finite logit: its sum is 0, or NaN when it saw a NaN
// logit, and it is carried as s * 0 so that the NaN survives.
__device__ inline void lse2_combine(float& o, float& s, float o2, float s2) {
  float on = fmaxf(o, o2);
  float a = (o == -INFINITY) ? s * 0.0f : s * __builtin_amdgcn_exp2f(o - on);
  float b = (o2 == -INFINITY) ? s2 * 0.0f : s2 * __builtin_amdgcn_exp2f(o2 - on);
  o = on;
  s = a + b;
}

}  // namespace hs

// Launchers (host side), defined next to their kernels.
namespace hs {
int launch_softmax_stats(const void* x, int dtype, int64_t rows, int64_t V, int64_t ld, float c,
                         float* row_max, float* row_lse, int32_t* row_argmax, hipStream_t stream);

struct TailArgs {
  const float* alpha;
  const uint8_t* agree;
  int gamma_src;  // 0: losses come from loss_in; 1: gamma = alpha; 2: gamma = agree
  int B, N, M;
  int tree;
  int32_t parent[HS_MAX_POSITIONS];
  const int32_t* path_end;
  double* eal;
  double* prefix;
  int loss_kind;
  double* loss_out;
  const double* loss_in;
  int L;
  double* logw;
  double* w;
  double eta;
  double* R;
  double* p;
  double* c;
  // set when this step follows an evaluation launch of its own: that launch's workspace
  // epoch (advanced once by it) and fail word; a failed evaluation skips the step
  const uint32_t* round_epoch;
  const uint64_t* round_fail;
};
int launch_tail(const TailArgs& a, hipStream_t stream);

// Delayed feedback: the token-level length loss over a sliding window of K tokens, fed to the
// base learners as each window completes (hs_delayed.hip).
struct DelayArgs {
  const float* alpha;    // [B][N][K] (gamma_src 1)
  const uint8_t* agree;  // [B][N][K] (gamma_src 2)
  int gamma_src;
  int B, N, K;
  const int32_t* count;  // [B]: tokens whose feedback arrives now (positions 0 .. count - 1)
  int64_t hybrid;        // tokens 0 .. hybrid - 1 of each stream take the acceptance loss
  float* hist;           // [B][2K][N]: feedback of the last 2K tokens, by token index mod 2K
  int64_t* clock;        // [B][2]: tokens received, windows used
  double* logw;
  double* w;
  double eta;
  double* R;
  double* p;
  double* c;
  double* loss;    // [K][B][N] or NULL: the window losses used, in order
  int32_t* nloss;  // [B] or NULL: how many
};
int launch_delayed(const DelayArgs& a, hipStream_t stream);
// EAGLE acceptance mass (hs_topl.hip): per-slice candidates, then the merge. Workspace bytes
// for a shape, and the two launches.
size_t topl_ws_bytes(const TeamGeom& g, int L);
bool topl_fits(const TeamGeom& g);  // work units and rows index with 31 bits
int launch_topl(const TeamGeom& g, const RowTable& rows, int L, float c, bool want_sum,
                float* gamma, uint8_t* hit, int32_t* idx, char* ws, hipStream_t stream);
// Drafter play and regret bookkeeping (hs_play.hip).
int launch_play(const double* w, int B, int N, int how, const double* u, int32_t* choice,
                hipStream_t stream);
int launch_regret(const double* loss, int L, int B, int N, const int32_t* played, double* cum,
                  double* played_sum, double* regret, const double* eal, double* eal_sum,
                  hipStream_t stream);
// Evaluation of one round: the team kernel (which also advances the workspace epoch) and, when
// tail != nullptr, the learner step on its alpha or agreement.
int launch_round(const TeamGeom& g, const RowTable& rows, float c, bool need_sum, bool need_arg,
                 float* alpha, uint8_t* agree, int32_t* argmax_t, int32_t* argmax_d, char* ws,
                 const TailArgs* tail, hipStream_t stream);
// Workgroups of the team kernel that one device holds at once for this shape and mode (0 if
// unknown); the launch needs at least S of them.
int team_capacity(const TeamGeom& g, bool need_sum, bool need_arg);
// Polls before a wait inside the team kernel gives up, for launches after this call (negative:
// the default; 0: every wait gives up at once).
void set_wait_polls(int polls);
}  // namespace hs
