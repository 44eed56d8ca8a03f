// hs_eval_topl: EAGLE's acceptance probability (Theorem 2). The greedy draft tree gives the
// node reached after a verified prefix the L children the drafter ranks highest, Top_L(q),
// and the target accepts one of them with probability gamma = sum_{v in Top_L(q)} p(v).
//
// Two launches:
//   1. hs_topl_slice_kernel: every logit is read once. A work unit is one slice (2048 bf16 or
//      1024 fp32 logits) of one row of one (query, position), and one wave does it alone:
//      for the target row, the slice's softmax statistics (max, lowest argmax, exp2 sum);
//      for a drafter row, the slice's local Top_L as exact integer keys. The waves of a
//      workgroup share nothing (no barrier), and the target row is read once per slice.
//   2. hs_topl_merge_kernel, one wave per (query, drafter, position): the global Top_L among
//      the slices' candidates, the target's normaliser from the slice statistics, the target
//      logits of the L winners (gathered from the logits), and gamma, the greedy hit and the
//      ranked children.
//
// Ranking keys. A logit becomes a signed integer that orders like its value (-0 and +0 map to
// the same integer), and its token index is appended so that equal logits rank lower index
// first. Keys are therefore distinct: the L-th largest of a set of keys is the one with
// exactly L - 1 larger ones, found by counting (or, for long lists, by a bitwise search with
// wave ballots over the bits in which the keys differ).
#include "hs_wave.h"

namespace hs {

namespace {

constexpr int kMaxTopL = HS_MAX_TOPL;
constexpr int kMergeCap = 512;  // candidates per wave held in LDS by the merge

struct TopArgs {
  int B, N, K, S, L;
  int64_t V, nvec;
  uint32_t units;  // B * K * (N + 1) * S work units of the first launch
  FastDiv divS, divR, divK, divNK;  // by S, N + 1, K and N * K
  float c;         // log2(e) / T; 0 when no mass is wanted
  int want_sum;    // target exp2 sums (the mass needs them)
  int want_arg;    // target argmax (the greedy hit needs it)
  int64_t* ckey;   // [B*N*K][S][L] candidate keys of each slice (kNone64: no candidate)
  float4* tstat;   // [B*K][S]: slice max, exp2 offset, exp2 sum, argmax (bits)
  float* gamma;    // [B][N][K]
  uint8_t* hit;    // [B][N][K]
  int32_t* idx;    // [B][N][K][L]
  RowTable rows;  // last: the scalars above sit in the first scalar-cache lines
};


constexpr int64_t kNone64 = INT64_MIN;
constexpr uint64_t kFlip64 = 0x8000000000000000ull;

// ---- integer images of logits --------------------------------------------------------------

// Two 16-bit sign-magnitude logits (bf16 or fp16; one 32-bit word) to two int16 that order
// like the values, -0 as +0: magnitude for a positive value, minus the magnitude for a
// negative one.
__device__ inline uint32_t bf16x2_ordered(uint32_t w) {
  typedef short s2 __attribute__((ext_vector_type(2)));
  s2 x;
  __builtin_memcpy(&x, &w, 4);
  const s2 m = x >> (s2)15;  // -1 in each negative half
  const s2 sv = (x ^ (m & (s2)0x7FFF)) - m;
  uint32_t r;
  __builtin_memcpy(&r, &sv, 4);
  return r;
}
// One fp32 logit to an int32 that orders like the value, -0 as +0.
__device__ inline int32_t f32_ordered(float f) {
  const int32_t x = __float_as_int(f);
  const int32_t m = x >> 31;
  return (x ^ (m & 0x7FFFFFFF)) - m;
}

// Key layout per storage type. A lane's E logits of a row slice are vectors i * 64 + lane
// (i = 0..3) of the slice, so element e of vector i has slice index
// j = i * 64 * VE + lane * VE + e. The key is (ordered value, 0xFF..F - j); it is built from a
// lane-independent part (0xFF..F - i * 64 * VE - e) and the lane's share lane * VE is
// subtracted once from the lane maximum, or added to a threshold.
template <int DT>
struct KeyOf;
template <>
struct KeyOf<HS_BF16> {
  using K = int32_t;
  using U = uint32_t;
  static constexpr int VE = 8;
  static constexpr int E = 4 * VE;
  static constexpr K kNone = INT32_MIN + 1024;  // stays below every real key after - lane * VE
  static constexpr K kMin = INT32_MIN;
  static constexpr K kValidMin = INT32_MIN + 65536;
  static constexpr U kFlip = 0x80000000u;
  // Both keys of a word by byte permutes: lo = (value of element 2h, index part of 2h),
  // hi = (value of 2h + 1, index part of 2h + 1); the index parts are constants kept in scalar
  // registers (a vector op cannot take a 32-bit literal here).
  __device__ static inline void build(const uint4& x, int i, K (&k)[E]) {
    const uint32_t w[4] = {x.x, x.y, x.z, x.w};
    uint32_t sel_lo, sel_hi;
    asm volatile("s_mov_b32 %0, 0x05040100" : "=s"(sel_lo));
    asm volatile("s_mov_b32 %0, 0x07060302" : "=s"(sel_hi));
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      const uint32_t o = bf16x2_ordered(w[h]);
      const uint32_t j0 = (uint32_t)(i * 64 * VE + 2 * h);
      uint32_t cc;  // (0xFFFF - j0 - 1) << 16 | (0xFFFF - j0)
      asm volatile("s_mov_b32 %0, %1"
                   : "=s"(cc)
                   : "i"((int32_t)(((0xFFFFu - j0 - 1) << 16) | (0xFFFFu - j0))));
      k[i * VE + 2 * h] = (K)__builtin_amdgcn_perm(o, cc, sel_lo);
      k[i * VE + 2 * h + 1] = (K)__builtin_amdgcn_perm(o, cc, sel_hi);
    }
  }
  // slice index and global key of a true (lane share removed) key
  __device__ static inline int slice_index(K k) { return 0xFFFF - (int)((uint32_t)k & 0xFFFFu); }
  __device__ static inline int64_t global_key(K k, int64_t g) {
    return (int64_t)((uint64_t)(int64_t)(k >> 16) << 48) | (int64_t)(0xFFFFFFFFu - (uint32_t)g);
  }
};
// fp16 (IEEE binary16) is sign-magnitude in 16 bits like bf16: the same keys order it.
template <>
struct KeyOf<HS_F16> : KeyOf<HS_BF16> {};
template <>
struct KeyOf<HS_F32> {
  using K = int64_t;
  using U = uint64_t;
  static constexpr int VE = 4;
  static constexpr int E = 4 * VE;
  static constexpr K kNone = INT64_MIN + 1024;
  static constexpr K kMin = INT64_MIN;
  static constexpr K kValidMin = INT64_MIN + ((int64_t)1 << 32);
  static constexpr U kFlip = 0x8000000000000000ull;
  __device__ static inline void build(const float4& x, int i, K (&k)[E]) {
    const float f[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int e = 0; e < 4; ++e)
      k[i * VE + e] = (K)(((uint64_t)(int64_t)f32_ordered(f[e]) << 32) |
                          (uint64_t)(0xFFFFFFFFu - (uint32_t)(i * 64 * VE + e)));
  }
  __device__ static inline int slice_index(K k) { return (int)(0xFFFFFFFFu - (uint32_t)k); }
  __device__ static inline int64_t global_key(K k, int64_t g) {
    return (int64_t)(((uint64_t)k & 0xFFFFFFFF00000000ull) | (uint64_t)(0xFFFFFFFFu - (uint32_t)g));
  }
};

// ---- wave-wide selection ---------------------------------------------------------------------

__device__ inline uint32_t wave_or32(uint32_t x) {
  x |= (uint32_t)dpp_i<0xB1>((int)x);
  x |= (uint32_t)dpp_i<0x4E>((int)x);
  x |= (uint32_t)dpp_i<0x141>((int)x);
  x |= (uint32_t)dpp_i<0x140>((int)x);
  return (uint32_t)(__builtin_amdgcn_readlane((int)x, 0) | __builtin_amdgcn_readlane((int)x, 16) |
                    __builtin_amdgcn_readlane((int)x, 32) | __builtin_amdgcn_readlane((int)x, 48));
}
__device__ inline uint32_t wave_or(uint32_t x) { return wave_or32(x); }
__device__ inline uint64_t wave_or(uint64_t x) {
  return ((uint64_t)wave_or32((uint32_t)(x >> 32)) << 32) | wave_or32((uint32_t)x);
}
__device__ inline uint32_t first_lane(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_readfirstlane((int)x);
}
__device__ inline uint64_t first_lane(uint64_t x) {
  return ((uint64_t)first_lane((uint32_t)(x >> 32)) << 32) | first_lane((uint32_t)x);
}
__device__ inline int highest_bit(uint32_t x) { return 31 - __builtin_clz(x); }
__device__ inline int highest_bit(uint64_t x) { return 63 - __builtin_clzll(x); }
__device__ inline int32_t bcast(int32_t x, int l) { return __builtin_amdgcn_readlane(x, l); }
__device__ inline int64_t bcast(int64_t x, int l) {
  return (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)((uint64_t)x >> 32), l) << 32) |
                   (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(uint64_t)x, l));
}
__device__ inline int mbcnt(uint64_t m) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}
// LDS written by some lanes of the wave, then read by others.
__device__ inline void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}
// The key of the neighbouring lane (lanes 2i and 2i + 1 swap).
__device__ inline int32_t lane_swap(int32_t x) { return __builtin_amdgcn_mov_dpp(x, 0xB1, 0xF, 0xF, true); }
__device__ inline int64_t lane_swap(int64_t x) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)(uint64_t)x, 0xB1, 0xF, 0xF, true);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)((uint64_t)x >> 32), 0xB1, 0xF, 0xF, true);
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// The largest x with #{u >= x} >= L over the keys u (unsigned images, 0 = no key) spread over
// the wave: u[j] for j < nu (wave-uniform) in every lane. The keys are distinct, so with at
// least L of them x is the L-th largest; with fewer it is at most their minimum. Bits on which
// every key agrees are fixed first and only the others are searched, highest first. All lanes
// must be active.
template <typename U, int NU>
__device__ inline U wave_kth(const U (&u)[NU], int nu, int L) {
  const uint64_t who = __ballot(u[0] != 0);
  if (who == 0) return 0;
  const int src = __builtin_ctzll(who);  // a lane whose first key exists
  U ref;
  if (sizeof(U) == 8)
    ref = (U)(((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)u[0] >> 32), src) << 32) |
              (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u[0], src));
  else
    ref = (U)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u[0], src);
  U diff = 0;
#pragma unroll
  for (int j = 0; j < NU; ++j) {
    if (j >= nu) break;
    if (u[j] != 0) diff |= u[j] ^ ref;
  }
  U vary = first_lane(wave_or(diff));
  U cur = ref & ~vary;
  while (vary) {
    const U b = (U)1 << highest_bit(vary);
    vary &= ~b;
    const U cand = cur | b;  // > 0, so absent keys never count
    int cnt = 0;
#pragma unroll
    for (int j = 0; j < NU; ++j) {
      if (j >= nu) break;
      cnt += __builtin_popcountll(__ballot(u[j] >= cand));
    }
    if (cnt >= L) cur = cand;
  }
  return cur;
}

// How many of the keys buf[0..n) exceed `mine`, n <= 64 wave-uniform. buf is 16-byte aligned
// and holds the smallest key value from n up to the next multiple of 16 (so no key needs a
// bounds test). All lanes read the same addresses (broadcasts), 16 keys per batch.
template <typename K>
__device__ inline int rank_in(const K* buf, int n, K mine) {
  constexpr int P = 16 / sizeof(K), CH = 16 / P;
  typedef K KP __attribute__((ext_vector_type(P)));
  int r = 0;
#pragma unroll
  for (int c0 = 0; c0 < 64; c0 += 16) {
    if (c0 >= n) break;  // wave-uniform
    KP v[CH];
#pragma unroll
    for (int i = 0; i < CH; ++i) v[i] = *reinterpret_cast<const KP*>(buf + c0 + i * P);
#pragma unroll
    for (int i = 0; i < CH; ++i)
#pragma unroll
      for (int p = 0; p < P; ++p) r += v[i][p] > mine ? 1 : 0;
  }
  return r;
}

// A 16-byte vector of a row: one global load away from the row end; near it, only the
// logits before V (the rest read as -inf) and nothing past the last vector.
template <int DT>
__device__ inline typename Vec<DT>::Raw load_vec(const char* rowp, int64_t vi, int64_t nvec,
                                                 int64_t V, bool tail) {
  using Vt = Vec<DT>;
  if (!tail) {
    // nontemporal for 16-bit logits (every logit is read once): 4% faster on large_pool_stream
    // and 7% on the single query than plain loads (bf16)
    typename Vt::Raw r;
    typedef unsigned int u4 __attribute__((ext_vector_type(4)));
    typedef const __attribute__((address_space(1))) u4* gp4;
    const u4 v = DT != HS_F32 ? __builtin_nontemporal_load((gp4)(rowp + vi * 16))
                              : *(gp4)(rowp + vi * 16);
    __builtin_memcpy(&r, &v, 16);
    return r;
  }
  if (vi >= nvec) return Vt::neg_raw();
  return Vt::load_raw(rowp, vi, V);
}

// ---- launch 1: per-slice statistics and candidates -------------------------------------------

// One work unit, decoded: slice s of row `row` (0 = target, 1 + i = drafter i) of group grp
// = b * K + k. Every field is uniform over the wave.
struct Unit {
  int s, row, grp, b, k;
  bool tail;
  int64_t v0;        // first 16-byte vector of the slice
  const char* rowp;  // the row's first logit
};

template <int DT>
__device__ inline Unit decode_unit(const TopArgs& A, uint32_t u) {
  Unit q;
  const uint32_t rs = fdiv(u, A.divS);
  q.s = (int)(u - rs * (uint32_t)A.S);
  const uint32_t grp = fdiv(rs, A.divR);
  q.row = (int)(rs - grp * (uint32_t)(A.N + 1));
  q.grp = (int)grp;
  q.b = (int)fdiv(grp, A.divK);
  q.k = q.grp - q.b * A.K;
  q.tail = q.s == A.S - 1;
  q.v0 = (int64_t)q.s * kThreads;
  q.rowp = reinterpret_cast<const char*>(A.rows.ptr[q.row]) +
           ((int64_t)q.b * A.rows.sb[q.row] + (int64_t)q.k * A.rows.sk[q.row]) * Vec<DT>::kBytes;
  return q;
}

template <int DT>
__device__ inline void load_unit(const TopArgs& A, const Unit& q, int lane,
                                 typename Vec<DT>::Raw (&x)[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) x[i] = load_vec<DT>(q.rowp, q.v0 + i * 64 + lane, A.nvec, A.V, q.tail);
}

// The target's slice statistics: max, lowest argmax (when the greedy hit is wanted), exp2
// offset (exp_offset_of) and the sum of exp2(z c - offset).
template <int DT>
__device__ inline void target_unit(const TopArgs& A, const Unit& q, const typename Vec<DT>::Raw (&x)[4],
                                   int lane) {
  using Vt = Vec<DT>;
  constexpr int VE = Vt::kElems;
  float z[4 * VE];
#pragma unroll
  for (int i = 0; i < 4; ++i) Vt::unpack(x[i], z + i * VE);
  float m = -INFINITY;
  int idx = INT_MAX;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t e0 = (q.v0 + i * 64 + lane) * VE;
#pragma unroll
    for (int e = 0; e < VE; ++e) {
      const float v = z[i * VE + e];
      if (A.want_arg) {
        if (e0 + e < A.V && (idx == INT_MAX || v > m)) {  // lowest index of the max
          m = v;
          idx = (int)(e0 + e);
        }
      } else if (e0 + e < A.V) {
        m = fmaxf(m, v);
      }
    }
  }
  // offset o = exp_offset_of(m, c), at or above m c; a lane whose max scaled by c is -inf (no
  // finite logit, or only ones below the fp32 range after scaling) sums against 0 instead,
  // where each of its logits gives exp2(-inf) = 0 or, for a NaN logit, NaN; the combine
  // carries such a sum as s * 0
  float o = -INFINITY, sum = 0.0f;
  if (A.want_sum) {
    o = exp_offset_of(m, A.c);
    const float off = o != -INFINITY ? o : 0.0f;
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t e0 = (q.v0 + i * 64 + lane) * VE;
#pragma unroll
      for (int e = 0; e < VE; ++e)
        if (e0 + e < A.V) acc[e & 3] += __builtin_amdgcn_exp2f(fmaf(z[i * VE + e], A.c, -off));
    }
    sum = (acc[0] + acc[1]) + (acc[2] + acc[3]);
  }
  if (A.want_arg) wave_max<true>(m, idx);
  else wave_max<false>(m, idx);
  if (A.want_sum) wave_lse(o, sum);
  if (lane == 0) A.tstat[(int64_t)q.grp * A.S + q.s] = make_float4(m, o, sum, __int_as_float(idx));
}

// A drafter row slice's local Top_L, as global keys in rank order (kNone64 past the slice's
// tokens). cand and lm are this wave's LDS.
template <int DT>
__device__ inline void drafter_unit(const TopArgs& A, const Unit& q, typename Vec<DT>::Raw (&x)[4],
                                    int lane, typename KeyOf<DT>::K* cand,
                                    typename KeyOf<DT>::K* lm) {
  using KO = KeyOf<DT>;
  using Key = typename KO::K;
  using UKey = typename KO::U;
  constexpr int VE = KO::VE, E = KO::E;
  constexpr int kCap = kMaxTopL * E;  // candidates of one row slice held in LDS
  // the lane's keys (tokens at or past V get kNone)
  auto row_keys = [&](Key (&key)[E]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) KO::build(x[i], i, key);
    if (q.tail) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int e = 0; e < VE; ++e)
          if ((q.v0 + i * 64 + lane) * VE + e >= A.V) key[i * VE + e] = KO::kNone;
    }
  };
  const Key lane_share = (Key)(lane * VE);
  Key thr;
  int C = 0;
  {
    Key key[E];
    row_keys(key);
    Key mk = key[0];
#pragma unroll
    for (int e = 1; e < E; ++e) mk = max(mk, key[e]);
    mk -= lane_share;

    // theta: the L-th largest of the 32 maxima of lane pairs, by rank counting (they are
    // distinct: exactly one pair has L - 1 larger ones; L <= 32). Every key >= theta lies in
    // one of those L pairs, so at most 2 L E keys of the slice reach it (usually about L),
    // and the slice's Top_L is among them.
    const Key pm = max(mk, lane_swap(mk));
    if ((lane & 1) == 0) lm[lane >> 1] = pm;
    wave_lds_sync();
    const uint64_t sel = __ballot((lane & 1) == 0 && rank_in(lm, 32, pm) == A.L - 1);
    Key theta = sel ? bcast(pm, __builtin_ctzll(sel)) : KO::kValidMin;
    if (theta < KO::kValidMin) theta = KO::kValidMin;

    // the candidates, compacted to LDS one element position at a time
    const Key kMaxKey = (Key)(~(UKey)0 >> 1);
    thr = theta > kMaxKey - lane_share ? kMaxKey : theta + lane_share;  // saturating
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const bool c = key[e] >= thr;
      const uint64_t m = __ballot(c);
      if (m != 0) {  // wave-uniform
        const int pos = C + mbcnt(m);
        if (c && pos < kCap) cand[pos] = key[e] - lane_share;
        C += __builtin_popcountll(m);
      }
    }
    if (C <= kCap && lane < 16) cand[C + lane] = KO::kMin;  // padding for the rank counts
    wave_lds_sync();
  }

  // exact Top_L among the C candidates (C >= L unless the slice holds fewer tokens)
  const int64_t orow = (((int64_t)q.b * A.N + (q.row - 1)) * A.K + q.k) * A.S + q.s;
  int64_t* okey = A.ckey + orow * A.L;
  const int64_t g0 = (int64_t)q.s * kThreads * VE;  // first token of the slice
  if (C <= 64) {  // ranks by counting, written in rank order
    const bool have = lane < C;
    const Key mine = have ? cand[lane] : (Key)0;
    const int rk = rank_in(cand, C, mine);
    if (have && rk < A.L) okey[rk] = KO::global_key(mine, g0 + KO::slice_index(mine));
  } else {
    // many candidates (long runs of equal logits): a bitwise search, output in scan order
    constexpr int NU = kCap / 64;
    constexpr int NR = NU > E ? NU : E;
    const bool in_lds = C <= kCap;
    // the candidates' unsigned images (0: none): u[j] = entry j * 64 + lane of the LDS list,
    // or, when the list overflowed, u[e] = the lane's element e (the row slice is read again:
    // a rare path, its loads are not overlapped)
    UKey u[NR];
    int nu;
    if (in_lds) {
      nu = (C + 63) / 64;
#pragma unroll
      for (int j = 0; j < NR; ++j) {
        const int xx = j * 64 + lane;
        u[j] = j < nu && xx < C ? (UKey)cand[xx] ^ KO::kFlip : 0;
      }
    } else {
      nu = E;
      load_unit<DT>(A, q, lane, x);
      Key key[E];
      row_keys(key);
#pragma unroll
      for (int j = 0; j < NR; ++j)
        u[j] = j < E && key[j < E ? j : 0] >= thr ? (UKey)(key[j < E ? j : 0] - lane_share) ^ KO::kFlip : 0;
    }
    const UKey kth = wave_kth<UKey, NR>(u, nu, A.L);
    int base = 0;
#pragma unroll
    for (int j = 0; j < NR; ++j) {
      if (j >= nu) break;  // wave-uniform
      const bool win = u[j] != 0 && u[j] >= kth;
      const uint64_t wm = __ballot(win);
      const int slot = base + mbcnt(wm);
      if (win && slot < A.L) {
        const Key kk = (Key)(u[j] ^ KO::kFlip);
        okey[slot] = KO::global_key(kk, g0 + KO::slice_index(kk));
      }
      base += __builtin_popcountll(wm);
    }
  }
  for (int slot = C + lane; slot < A.L; slot += 64) okey[slot] = kNone64;  // fewer than L tokens
  wave_lds_sync();  // the LDS lists are rewritten by the next unit
}

template <int DT>
__global__ __launch_bounds__(kThreads) void hs_topl_slice_kernel(TopArgs A) {
  using Vt = Vec<DT>;
  using KO = KeyOf<DT>;
  using Key = typename KO::K;
  constexpr int kCap = kMaxTopL * KO::E;
  __shared__ __attribute__((aligned(16))) Key s_cand[kWaves][kCap + 16];  // + room for the padding
  __shared__ __attribute__((aligned(16))) Key s_lmax[kWaves][32];
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform over the wave
  const uint32_t u = blockIdx.x * kWaves + wv;
  if (u >= A.units) return;  // wave-uniform; the waves share no barrier
  typename Vt::Raw x[4];
  const Unit q = decode_unit<DT>(A, u);
  load_unit<DT>(A, q, lane, x);
  if (q.row == 0) target_unit<DT>(A, q, x, lane);
  else drafter_unit<DT>(A, q, x, lane, s_cand[wv], s_lmax[wv]);
}

// ---- launch 2: global Top_L and the mass ----------------------------------------------------
// One wave per (query, drafter, position).

template <int DT>
__global__ __launch_bounds__(kThreads) void hs_topl_merge_kernel(TopArgs A) {
  constexpr int R = 16;   // candidates per lane held in registers
  constexpr int RS = 8;   // slice statistics records per lane loaded up front
  __shared__ __attribute__((aligned(16))) int64_t s_key[kWaves][kMergeCap + 16];  // + padding
  __shared__ __attribute__((aligned(16))) int64_t s_lmax[kWaves][64];
  __shared__ __attribute__((aligned(16))) int64_t s_wkey[kWaves][64];
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform over the wave
  const int64_t rows = (int64_t)A.B * A.N * A.K;
  const int64_t r = (int64_t)blockIdx.x * kWaves + wv;
  if (r >= rows) return;  // wave-uniform; no workgroup barrier below
  const uint32_t r32 = (uint32_t)r;  // rows < 2^31
  const int k = (int)(r32 - fdiv(r32, A.divK) * (uint32_t)A.K);
  const int b = (int)fdiv(r32, A.divNK);
  const int grp = b * A.K + k;
  const int L = A.L;
  const int nc = A.S * L;
  const int64_t* ck = A.ckey + r * nc;

  // loads up front: the target's statistics records, then the candidates (unconditional
  // loads at a clamped index, then a select: no branch between the loads)
  const int nst = A.S;
  const float4* ts = A.tstat + (int64_t)grp * nst;
  const float4 none_st = make_float4(-INFINITY, -INFINITY, 0.0f, __int_as_float(INT_MAX));
  float4 st[RS];
#pragma unroll
  for (int j = 0; j < RS; ++j) st[j] = ts[min(j * 64 + lane, nst - 1)];
#pragma unroll
  for (int j = 0; j < RS; ++j)
    if (j * 64 + lane >= nst) st[j] = none_st;
  const bool resident = nc <= 64 * R;
  int64_t kr[R];
  int64_t mk = kNone64;
  for (int x0 = 0; x0 < nc; x0 += 64 * R) {
#pragma unroll
    for (int j = 0; j < R; ++j) kr[j] = ck[min(x0 + j * 64 + lane, nc - 1)];
#pragma unroll
    for (int j = 0; j < R; ++j) {
      if (x0 + j * 64 + lane >= nc) kr[j] = kNone64;
      mk = max(mk, kr[j]);
    }
  }

  // the target's softmax statistics
  float m = -INFINITY, o = -INFINITY, sm = 0.0f;
  int am = INT_MAX;
#pragma unroll
  for (int j = 0; j < RS; ++j) {
    argmax_combine(m, am, st[j].x, __float_as_int(st[j].w));
    if (A.want_sum) lse2_combine(o, sm, st[j].y, st[j].z);
  }
  for (int x = RS * 64 + lane; x < nst; x += 64) {
    const float4 q = ts[x];
    argmax_combine(m, am, q.x, __float_as_int(q.w));
    if (A.want_sum) lse2_combine(o, sm, q.y, q.z);
  }
  wave_max<true>(m, am);
  if (A.gamma) wave_lse(o, sm);

  // theta: the L-th largest lane maximum, by rank counting. The lanes holding a real
  // candidate are distinct and at least L (slice 0 lists L real tokens in L consecutive
  // entries); lanes without one hold kNone64 and rank below all of them.
  int64_t* lm = s_lmax[wv];
  lm[lane] = mk;
  wave_lds_sync();
  const uint64_t sel = __ballot(mk != kNone64 && rank_in(lm, 64, mk) == L - 1);
  const int64_t theta = sel ? bcast(mk, __builtin_ctzll(sel)) : kNone64 + 1;

  // the candidates >= theta (at most L lanes hold any), compacted to LDS
  int64_t* key = s_key[wv];
  int C = 0;
  for (int x0 = 0; x0 < nc; x0 += 64 * R) {
    if (!resident) {
#pragma unroll
      for (int j = 0; j < R; ++j) kr[j] = ck[min(x0 + j * 64 + lane, nc - 1)];
#pragma unroll
      for (int j = 0; j < R; ++j)
        if (x0 + j * 64 + lane >= nc) kr[j] = kNone64;
    }
#pragma unroll
    for (int j = 0; j < R; ++j) {
      const bool c = kr[j] >= theta;
      const uint64_t mm = __ballot(c);
      if (mm != 0) {  // wave-uniform
        const int pos = C + mbcnt(mm);
        if (c && pos < kMergeCap) key[pos] = kr[j];
        C += __builtin_popcountll(mm);
      }
    }
  }
  if (C <= kMergeCap && lane < 16) key[C + lane] = kNone64;  // padding for the rank counts
  wave_lds_sync();

  // exact Top_L: per lane a winner flag, its key and its rank
  bool win;
  int64_t wkey;
  int rank;
  if (C <= 64) {
    const bool have = lane < C;
    wkey = have ? key[lane] : kNone64;
    rank = rank_in(key, C, wkey);
    win = have && rank < L;
  } else {
    int64_t kth;
    if (C <= kMergeCap) {
      constexpr int NU = kMergeCap / 64;
      const int nu = (C + 63) / 64;
      uint64_t u[NU];
#pragma unroll
      for (int j = 0; j < NU; ++j) {
        const int x = j * 64 + lane;
        u[j] = j < nu && x < C ? (uint64_t)key[x] ^ kFlip64 : 0;
      }
      kth = (int64_t)(wave_kth<uint64_t, NU>(u, nu, L) ^ kFlip64);
    } else {
      // more candidates than the LDS holds: search the lists in place (same result, slower)
      const uint64_t ref = (uint64_t)theta ^ kFlip64;
      uint64_t diff = 0;
      for (int x = lane; x < nc; x += 64)
        if (ck[x] >= theta) diff |= ((uint64_t)ck[x] ^ kFlip64) ^ ref;
      uint64_t vary = first_lane(wave_or(diff));
      uint64_t cur = ref & ~vary;
      while (vary) {
        const uint64_t bb = 1ull << highest_bit(vary);
        vary &= ~bb;
        const uint64_t cnd = cur | bb;
        int c = 0;
        for (int x0 = 0; x0 < nc; x0 += 64) {
          const int x = x0 + lane;
          c += __builtin_popcountll(
              __ballot(x < nc && ck[x] >= theta && ((uint64_t)ck[x] ^ kFlip64) >= cnd));
        }
        if (c >= L) cur = cnd;
      }
      kth = (int64_t)(cur ^ kFlip64);
    }
    // the L winners to LDS in scan order, then ranked among themselves
    int64_t* wk = s_wkey[wv];
    const bool in_lds = C <= kMergeCap;
    const int nscan = in_lds ? C : nc;
    int base = 0;
    for (int x0 = 0; x0 < nscan; x0 += 64) {
      const int x = x0 + lane;
      int64_t kv = kNone64;
      if (x < nscan) kv = in_lds ? key[x] : ck[x];
      const bool w = x < nscan && kv >= kth;
      const uint64_t wm = __ballot(w);
      const int slot = base + mbcnt(wm);
      if (w && slot < kMaxTopL) wk[slot] = kv;
      base += __builtin_popcountll(wm);
    }
    if (lane < 16) wk[min(base, kMaxTopL) + lane] = kNone64;  // padding for the rank counts
    wave_lds_sync();
    const int W = min(base, L);
    win = lane < W;
    wkey = win ? wk[lane] : kNone64;
    rank = rank_in(wk, W, wkey);
  }

  // the target logits of the winners, gathered from the target row
  const int gidx = (int)(0xFFFFFFFFu - (uint32_t)(uint64_t)wkey);
  float zt = 0.0f;
  if (win) {
    const char* trow = reinterpret_cast<const char*>(A.rows.ptr[0]) +
                       ((int64_t)b * A.rows.sb[0] + (int64_t)k * A.rows.sk[0]) * Vec<DT>::kBytes;
    if constexpr (DT == HS_F32)
      zt = reinterpret_cast<const float*>(trow)[gidx];
    else
      zt = Vec<DT>::lo(reinterpret_cast<const uint16_t*>(trow)[gidx]);
  }
  if (A.gamma) {
    const float e = win ? __builtin_amdgcn_exp2f(fmaf(zt, A.c, -o)) : 0.0f;
    const float tot = wave_sum_f(e);
    if (lane == 0) A.gamma[r] = fminf(tot / sm, 1.0f);
  }
  if (A.hit) {
    const bool h = __ballot(win && gidx == am) != 0;
    if (lane == 0) A.hit[r] = h ? 1 : 0;
  }
  if (A.idx && win) A.idx[r * L + rank] = gidx;
}

// One wave per unit. (A resident grid looping over the units with the next unit's logits in
// registers was measured slower: the extra registers halve the waves a SIMD holds.)
template <int DT>
void launch_t(const TopArgs& A, int64_t nrows, hipStream_t st) {
  const int64_t wgs = ((int64_t)A.units + kWaves - 1) / kWaves;
  hs_topl_slice_kernel<DT><<<(unsigned)wgs, kThreads, 0, st>>>(A);
  if (hipGetLastError() != hipSuccess) return;
  hs_topl_merge_kernel<DT><<<(unsigned)((nrows + kWaves - 1) / kWaves), kThreads, 0, st>>>(A);
}

}  // namespace


size_t topl_ws_bytes(const TeamGeom& g, int L) {
  const size_t rows = (size_t)g.B * g.N * g.K;
  return align256(rows * g.S * L * 8) + align256((size_t)g.G * g.S * 16);
}

bool topl_fits(const TeamGeom& g) {
  return (int64_t)g.G * (g.N + 1) * g.S < ((int64_t)1 << 31) &&
         (int64_t)g.B * g.N * g.K < ((int64_t)1 << 31);
}

int launch_topl(const TeamGeom& g, const RowTable& rows, int L, float c, bool want_sum,
                float* gamma, uint8_t* hit, int32_t* idx, char* ws, hipStream_t stream) {
  TopArgs A;
  A.rows = rows;
  A.B = g.B;
  A.N = g.N;
  A.K = g.K;
  A.S = g.S;
  A.L = L;
  A.V = g.V;
  A.nvec = g.nvec;
  A.units = (uint32_t)((int64_t)g.G * (g.N + 1) * g.S);
  A.divS = make_fastdiv((uint32_t)g.S);
  A.divR = make_fastdiv((uint32_t)(g.N + 1));
  A.divK = make_fastdiv((uint32_t)g.K);
  A.divNK = make_fastdiv((uint32_t)(g.N * g.K));
  A.c = c;
  A.want_sum = want_sum ? 1 : 0;
  A.want_arg = hit != nullptr ? 1 : 0;
  const size_t nrows = (size_t)g.B * g.N * g.K;
  A.ckey = reinterpret_cast<int64_t*>(ws);
  A.tstat = reinterpret_cast<float4*>(ws + align256(nrows * g.S * L * 8));
  A.gamma = gamma;
  A.hit = hit;
  A.idx = idx;
  if (g.dtype == HS_BF16) launch_t<HS_BF16>(A, (int64_t)nrows, stream);
  else if (g.dtype == HS_F16) launch_t<HS_F16>(A, (int64_t)nrows, stream);
  else launch_t<HS_F32>(A, (int64_t)nrows, stream);
  return hipGetLastError() == hipSuccess ? HS_OK : HS_ERR_HIP;
}

}  // namespace hs
