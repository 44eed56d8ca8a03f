// hs_eval_topl: EAGLE's acceptance probability (Theorem 2). The greedy draft tree gives the
// node reached after a verified prefix the L children the drafter ranks highest, Top_L(q),
// and the target accepts one of them with probability gamma = sum_{v in Top_L(q)} p(v).
//
// Two launches:
//   1. hs_topl_slice_kernel, one workgroup per (query, position, row set, slice): every logit
//      is read once. The target's slice goes to LDS and, for the first row set, into its
//      softmax statistics (max, lowest argmax, exp2 sum). Each wave owns whole drafter-row
//      slices and writes the slice's local Top_L as exact integer keys, with the target
//      logit at each candidate gathered from LDS.
//   2. hs_topl_merge_kernel, one wave per (query, drafter, position): the global Top_L among
//      the slices' candidates, the target's normaliser from the slice statistics, and gamma,
//      the greedy hit and the ranked children.
//
// Ranking keys. A logit becomes a signed integer that orders like its value (-0 and +0 map to
// the same integer), and its token index is appended so that equal logits rank lower index
// first. Keys are therefore distinct, and "the L-th largest key" is found by a bitwise search
// with wave ballots over just the bits in which the keys differ.
#include "hs_rowstats.h"
#include "hs_wave.h"

namespace hs {

namespace {

constexpr int kMaxTopL = HS_MAX_TOPL;
constexpr int kMergeCap = 512;  // candidates per wave held in LDS by the merge

struct TopArgs {
  RowTable rows;
  int B, N, K, D, nsub, S, L;
  int64_t V, nvec;
  float c;       // log2(e) / T; 0 when no mass is wanted
  int want_sum;  // target exp2 sums (the mass needs them)
  int64_t* ckey; // [B*N*K][S][L] candidate keys of each slice (kNone64: no candidate)
  float* czt;    // [B*N*K][S][L] target logit at the candidate's token
  float4* tstat; // [B*K][S]: slice max, exp2 offset, exp2 sum, argmax (bits)
  float* gamma;  // [B][N][K]
  uint8_t* hit;  // [B][N][K]
  int32_t* idx;  // [B][N][K][L]
};

constexpr int64_t kNone64 = INT64_MIN;

// ---- integer images of logits --------------------------------------------------------------

// Two bf16 logits (one 32-bit word) to two int16 that order like the values, -0 as +0:
// magnitude for a positive value, minus the magnitude for a negative one.
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

// Key layout per storage type. A lane's E logits of a row slice are vectors
// q * 64 + lane (q = 0..3) of the slice, so element e of vector q has slice index
// j = q * 64 * VE + lane * VE + e. The key is (ordered value, 0xFF..F - j); it is built
// from a lane-independent part (0xFF..F - q * 64 * VE - e) and the lane's share lane * VE is
// subtracted once from the lane maximum, or added to a threshold.
template <int DT>
struct KeyOf;
template <>
struct KeyOf<HS_BF16> {
  using K = int32_t;
  using U = uint32_t;
  static constexpr int VE = 8;
  static constexpr int E = 4 * VE;
  static constexpr int kBits = 16;            // index bits
  static constexpr K kNone = INT32_MIN + 1024;  // stays below every real key after - lane * VE
  static constexpr K kValidMin = INT32_MIN + 65536;
  static constexpr U kFlip = 0x80000000u;
  __device__ static inline void build(const uint4& x, int q, K (&k)[E]) {
    const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      const uint32_t o = bf16x2_ordered(w[h]);
      const uint32_t j0 = (uint32_t)(q * 64 * VE + 2 * h);
      k[q * VE + 2 * h] = (K)((o << 16) | (0xFFFFu - j0));
      k[q * VE + 2 * h + 1] = (K)((o & 0xFFFF0000u) | (0xFFFFu - j0 - 1));
    }
  }
  // slice index and global key of a true (lane share removed) key
  __device__ static inline int slice_index(K k) { return 0xFFFF - (int)((uint32_t)k & 0xFFFFu); }
  __device__ static inline int64_t global_key(K k, int64_t g) {
    return (int64_t)((uint64_t)(int64_t)(k >> 16) << 48) | (int64_t)(0xFFFFFFFFu - (uint32_t)g);
  }
};
template <>
struct KeyOf<HS_F32> {
  using K = int64_t;
  using U = uint64_t;
  static constexpr int VE = 4;
  static constexpr int E = 4 * VE;
  static constexpr int kBits = 32;
  static constexpr K kNone = INT64_MIN + 1024;
  static constexpr K kValidMin = INT64_MIN + ((int64_t)1 << 32);
  static constexpr U kFlip = 0x8000000000000000ull;
  __device__ static inline void build(const float4& x, int q, K (&k)[E]) {
    const float f[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int e = 0; e < 4; ++e)
      k[q * VE + e] = (K)(((uint64_t)(int64_t)f32_ordered(f[e]) << 32) |
                          (uint64_t)(0xFFFFFFFFu - (uint32_t)(q * 64 * VE + e)));
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

// Inclusive prefix sum over the wave (lane l gets sum of lanes 0..l).
__device__ inline int wave_incl_scan(int x) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int y = __shfl_up(x, d, 64);
    if (lane >= d) x += y;
  }
  return x;
}

template <int DT>
__device__ inline typename Vec<DT>::Raw load_vec(const char* rowp, int64_t vi, int64_t nvec,
                                                 int64_t V, bool tail) {
  using Vt = Vec<DT>;
  if (!tail) {
    typename Vt::Raw r;
    typedef unsigned int u4 __attribute__((ext_vector_type(4)));
    const u4 v = *(const __attribute__((address_space(1))) u4*)(rowp + vi * 16);
    __builtin_memcpy(&r, &v, 16);
    return r;
  }
  if (vi >= nvec) return Vt::neg_raw();
  return Vt::load_raw(rowp, vi, V);
}

__device__ inline float raw_logit(const void* lds_row, int dtype_bf16, int j) {
  if (dtype_bf16) return __uint_as_float((uint32_t)reinterpret_cast<const uint16_t*>(lds_row)[j] << 16);
  return reinterpret_cast<const float*>(lds_row)[j];
}

// ---- launch 1: per-slice statistics and candidates -------------------------------------------

template <int DT, int D>
__global__ __launch_bounds__(kThreads) void hs_topl_slice_kernel(TopArgs A) {
  using Vt = Vec<DT>;
  using KO = KeyOf<DT>;
  using Key = typename KO::K;
  using UKey = typename KO::U;
  constexpr int VE = KO::VE, E = KO::E;
  constexpr int kCap = kMaxTopL * E;  // candidates of one row slice (see below)
  constexpr int kRowsPerWave = (D + kWaves - 1) / kWaves;
  __shared__ __attribute__((aligned(16))) char s_target[kThreads * 16];
  __shared__ Key s_cand[kWaves][kCap];

  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  const int64_t item = blockIdx.x;
  const int s = (int)(item % A.S);
  const int64_t gs = item / A.S;
  const int set = (int)(gs % A.nsub);
  const int grp = (int)(gs / A.nsub);
  const int b = grp / A.K, k = grp % A.K;
  const int n = min(D, A.N - set * D);
  const bool tail = s == A.S - 1;
  const int64_t v0 = (int64_t)s * kThreads;  // first vector of the slice

  // loads: the target's vector first (it is waited for first), then this wave's rows
  const char* trow = reinterpret_cast<const char*>(A.rows.ptr[0]) +
                     ((int64_t)b * A.rows.sb[0] + (int64_t)k * A.rows.sk[0]) * Vt::kBytes;
  const typename Vt::Raw tv = load_vec<DT>(trow, v0 + t, A.nvec, A.V, tail);
  typename Vt::Raw dv[kRowsPerWave][4];
#pragma unroll
  for (int h = 0; h < kRowsPerWave; ++h) {
    const int r = wv + kWaves * h;
    if (r < n) {
      const int row = 1 + set * D + r;
      const char* p = reinterpret_cast<const char*>(A.rows.ptr[row]) +
                      ((int64_t)b * A.rows.sb[row] + (int64_t)k * A.rows.sk[row]) * Vt::kBytes;
#pragma unroll
      for (int q = 0; q < 4; ++q) dv[h][q] = load_vec<DT>(p, v0 + q * 64 + lane, A.nvec, A.V, tail);
    }
  }

  // target slice: to LDS for the gathers, and its statistics (first row set only)
  *reinterpret_cast<typename Vt::Raw*>(s_target + t * 16) = tv;
  if (set == 0) {
    float z[VE];
    Vt::unpack(tv, z);
    float m = -INFINITY;
    int idx = INT_MAX;
    const int64_t e0 = (v0 + t) * VE;
#pragma unroll
    for (int e = 0; e < VE; ++e)
      if (e0 + e < A.V && (idx == INT_MAX || z[e] > m)) {  // lowest index of the max
        m = z[e];
        idx = (int)(e0 + e);
      }
    float o = -INFINITY, sum = 0.0f;
    if (A.want_sum && m != -INFINITY) {
      o = m * A.c;
#pragma unroll
      for (int e = 0; e < VE; ++e)
        if (e0 + e < A.V) sum += __builtin_amdgcn_exp2f(fmaf(z[e], A.c, -o));
    }
    const SliceStat st = A.want_sum ? block_reduce_stat<true, true>(m, idx, o, sum)
                                    : block_reduce_stat<false, true>(m, idx, o, sum);
    if (t == 0)
      A.tstat[(int64_t)grp * A.S + s] = make_float4(st.m, st.o, st.s, __int_as_float(st.idx));
  }
  __syncthreads();

  const Key lane_share = (Key)(lane * VE);
  Key* cand = s_cand[wv];
#pragma unroll
  for (int h = 0; h < kRowsPerWave; ++h) {
    const int r = wv + kWaves * h;
    if (r >= n) break;  // wave-uniform
    Key key[E];
#pragma unroll
    for (int q = 0; q < 4; ++q) KO::build(dv[h][q], q, key);
    if (tail) {  // tokens at or past V are no candidates
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int e = 0; e < VE; ++e)
          if ((v0 + q * 64 + lane) * VE + e >= A.V) key[q * VE + e] = KO::kNone;
    }
    Key mk = key[0];
#pragma unroll
    for (int e = 1; e < E; ++e) mk = max(mk, key[e]);
    mk -= lane_share;

    // theta: the L-th largest lane maximum. Exactly L lanes hold a key >= theta (fewer when
    // theta is clamped to the valid range), so at most L * E keys of the slice reach it, and
    // the slice's Top_L is among them.
    const UKey um[1] = {(UKey)mk ^ KO::kFlip};  // > 0: mk >= kNone - lane share
    Key theta = (Key)(wave_kth<UKey, 1>(um, 1, A.L) ^ KO::kFlip);
    if (theta < KO::kValidMin) theta = KO::kValidMin;
    // per-lane threshold on the lane-independent key part (saturating)
    const Key thr = theta > (Key)(~(UKey)0 >> 1) - lane_share ? (Key)(~(UKey)0 >> 1) : theta + lane_share;
    int cnt = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) cnt += key[e] >= thr ? 1 : 0;
    const int incl = wave_incl_scan(cnt);
    const int C = __builtin_amdgcn_readlane(incl, 63);
    int pos = incl - cnt;
#pragma unroll
    for (int e = 0; e < E; ++e)
      if (key[e] >= thr) {
        if (pos < kCap) cand[pos] = key[e] - lane_share;
        ++pos;
      }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    // exact Top_L among the C <= kCap candidates (C >= L unless the slice holds fewer tokens)
    const int Cc = min(C, kCap);
    constexpr int NU = kCap / 64;
    const int nu = (Cc + 63) / 64;
    UKey u[NU];  // candidate keys, 0 past the end (real keys are >= kValidMin, so never 0)
#pragma unroll
    for (int j = 0; j < NU; ++j) {
      const int x = j * 64 + lane;
      u[j] = j < nu && x < Cc ? (UKey)cand[x] ^ KO::kFlip : 0;
    }
    const UKey kth = wave_kth<UKey, NU>(u, nu, A.L);
    const int64_t orow = (((int64_t)b * A.N + set * D + r) * A.K + k) * A.S + s;
    int64_t* okey = A.ckey + orow * A.L;
    float* ozt = A.czt + orow * A.L;
    int base = 0;
#pragma unroll
    for (int j = 0; j < NU; ++j) {
      if (j >= nu) break;  // wave-uniform
      const bool win = u[j] != 0 && u[j] >= kth;
      const uint64_t wm = __ballot(win);
      const int slot = base + __builtin_popcountll(wm & ((1ull << lane) - 1));
      if (win && slot < A.L) {
        const Key kk = (Key)(u[j] ^ KO::kFlip);
        const int jj = KO::slice_index(kk) & (kThreads * VE - 1);  // < kThreads * VE by construction
        okey[slot] = KO::global_key(kk, (int64_t)s * kThreads * VE + jj);
        ozt[slot] = raw_logit(s_target, DT == HS_BF16, jj);
      }
      base += __builtin_popcountll(wm);
    }
    for (int slot = base + lane; slot < A.L; slot += 64) {
      okey[slot] = kNone64;
      ozt[slot] = 0.0f;
    }
    __builtin_amdgcn_wave_barrier();  // the candidate buffer is reused by the next row
  }
}

// ---- launch 2: global Top_L and the mass ----------------------------------------------------

__device__ inline bool ge_u64(uint64_t a, uint64_t b) { return a >= b; }

__global__ __launch_bounds__(kThreads) void hs_topl_merge_kernel(TopArgs A) {
  __shared__ int64_t s_key[kWaves][kMergeCap];
  __shared__ int32_t s_ent[kWaves][kMergeCap];
  __shared__ int64_t s_wkey[kWaves][kMaxTopL];
  __shared__ int32_t s_went[kWaves][kMaxTopL];
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  const int64_t rows = (int64_t)A.B * A.N * A.K;
  const int64_t r = (int64_t)blockIdx.x * kWaves + wv;
  if (r >= rows) return;  // wave-uniform; no workgroup barrier below
  const int k = (int)(r % A.K);
  const int b = (int)(r / ((int64_t)A.N * A.K));
  const int grp = b * A.K + k;
  const int L = A.L;
  const int nc = A.S * L;
  const int64_t* ck = A.ckey + r * nc;
  const float* cz = A.czt + r * nc;
  constexpr uint64_t kFlip = 0x8000000000000000ull;

  // pass 1: lane maxima, theta = the L-th largest of them (clamped to real keys)
  int64_t mk = kNone64;
  for (int x = lane; x < nc; x += 64) mk = max(mk, ck[x]);
  const uint64_t um[1] = {(uint64_t)mk ^ kFlip};  // 0 for a lane without candidates
  int64_t theta = (int64_t)(wave_kth<uint64_t, 1>(um, 1, L) ^ kFlip);
  if (theta < kNone64 + 1) theta = kNone64 + 1;

  // pass 2: the candidates >= theta (at most L lanes hold any), compacted in LDS
  int cnt = 0;
  for (int x = lane; x < nc; x += 64) cnt += ck[x] >= theta ? 1 : 0;
  const int incl = wave_incl_scan(cnt);
  const int C = __builtin_amdgcn_readlane(incl, 63);
  int64_t kth;
  int64_t* key = s_key[wv];
  int32_t* ent = s_ent[wv];
  if (C <= kMergeCap) {
    int pos = incl - cnt;
    for (int x = lane; x < nc; x += 64) {
      const int64_t v = ck[x];
      if (v >= theta) {
        key[pos] = v;
        ent[pos] = x;
        ++pos;
      }
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    constexpr int NU = kMergeCap / 64;
    const int nu = (C + 63) / 64;
    uint64_t u[NU];
#pragma unroll
    for (int j = 0; j < NU; ++j) {
      const int x = j * 64 + lane;
      u[j] = j < nu && x < C ? (uint64_t)key[x] ^ kFlip : 0;
    }
    kth = (int64_t)(wave_kth<uint64_t, NU>(u, nu, L) ^ kFlip);
  } else {
    // more candidates than the LDS holds: search the lists in place (same result, slower)
    uint64_t ref = (uint64_t)theta ^ kFlip;
    uint64_t diff = 0;
    for (int x = lane; x < nc; x += 64)
      if (ck[x] >= theta) diff |= ((uint64_t)ck[x] ^ kFlip) ^ ref;
    uint64_t vary = first_lane(wave_or(diff));
    uint64_t cur = ref & ~vary;
    while (vary) {
      const int bit = highest_bit(vary);
      const uint64_t bb = 1ull << bit;
      vary &= ~bb;
      const uint64_t cand = cur | bb;
      int c = 0;
      for (int x0 = 0; x0 < nc; x0 += 64) {
        const int x = x0 + lane;
        c += __builtin_popcountll(__ballot(x < nc && ck[x] >= theta && ((uint64_t)ck[x] ^ kFlip) >= cand));
      }
      if (c >= L) cur = cand;
    }
    kth = (int64_t)(cur ^ kFlip);
  }
  __builtin_amdgcn_wave_barrier();

  // the winners (exactly L: V >= L real tokens), moved to lanes 0 .. L-1
  int64_t* wk = s_wkey[wv];
  int32_t* we = s_went[wv];
  int base = 0;
  const bool in_lds = C <= kMergeCap;
  const int nscan = in_lds ? C : nc;
  for (int x0 = 0; x0 < nscan; x0 += 64) {
    const int x = x0 + lane;
    int64_t kv = kNone64;
    int ev = 0;
    if (x < nscan) {
      kv = in_lds ? key[x] : ck[x];
      ev = in_lds ? ent[x] : x;
    }
    const bool win = x < nscan && kv >= kth;
    const uint64_t wm = __ballot(win);
    const int slot = base + __builtin_popcountll(wm & ((1ull << lane) - 1));
    if (win && slot < kMaxTopL) {
      wk[slot] = kv;
      we[slot] = ev;
    }
    base += __builtin_popcountll(wm);
  }
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  const int W = min(base, L);
  const bool mine = lane < W;
  const int64_t wkey = mine ? wk[lane] : kNone64;
  const float zt = mine ? cz[we[lane]] : 0.0f;
  const int gidx = (int)(0xFFFFFFFFu - (uint32_t)(uint64_t)wkey);

  // the target's softmax statistics from its slices
  const float4* ts = A.tstat + (int64_t)grp * A.S;
  float m = -INFINITY, o = -INFINITY, sm = 0.0f;
  int am = INT_MAX;
  for (int x = lane; x < A.S; x += 64) {
    const float4 st = ts[x];
    argmax_combine(m, am, st.x, __float_as_int(st.w));
    if (A.want_sum) lse2_combine(o, sm, st.y, st.z);
  }
  wave_max<true>(m, am);
  if (A.gamma) {
    wave_lse(o, sm);
    const float e = mine ? __builtin_amdgcn_exp2f(fmaf(zt, A.c, -o)) : 0.0f;
    const float tot = wave_sum_f(e);
    if (lane == 0) A.gamma[r] = fminf(tot / sm, 1.0f);
  }
  if (A.hit) {
    const bool h = __ballot(mine && gidx == am) != 0;
    if (lane == 0) A.hit[r] = h ? 1 : 0;
  }
  if (A.idx) {
    int rank = 0;
    for (int q = 0; q < W; ++q) {
      const int64_t kq = (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readlane(
                                        (int)(uint32_t)((uint64_t)wkey >> 32), q) << 32) |
                                   (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)wkey, q));
      rank += kq > wkey ? 1 : 0;
    }
    if (mine) A.idx[r * L + rank] = gidx;
  }
}

template <int DT, int D>
void launch_slice(const TopArgs& A, int64_t items, hipStream_t st) {
  hs_topl_slice_kernel<DT, D><<<(unsigned)items, kThreads, 0, st>>>(A);
}

}  // namespace

size_t topl_ws_bytes(const TeamGeom& g, int L) {
  const size_t rows = (size_t)g.B * g.N * g.K;
  size_t off = align256(rows * g.S * L * 8);
  off += align256(rows * g.S * L * 4);
  off += align256((size_t)g.G * g.S * 16);
  return off;
}

int launch_topl(const TeamGeom& g, const RowTable& rows, int L, float c, bool want_sum,
                float* gamma, uint8_t* hit, int32_t* idx, char* ws, hipStream_t stream) {
  TopArgs A;
  A.rows = rows;
  A.B = g.B;
  A.N = g.N;
  A.K = g.K;
  A.D = g.D;
  A.nsub = g.nsub;
  A.S = g.S;
  A.L = L;
  A.V = g.V;
  A.nvec = g.nvec;
  A.c = c;
  A.want_sum = want_sum ? 1 : 0;
  const size_t nrows = (size_t)g.B * g.N * g.K;
  size_t off = 0;
  A.ckey = reinterpret_cast<int64_t*>(ws + off);
  off += align256(nrows * g.S * L * 8);
  A.czt = reinterpret_cast<float*>(ws + off);
  off += align256(nrows * g.S * L * 4);
  A.tstat = reinterpret_cast<float4*>(ws + off);
  A.gamma = gamma;
  A.hit = hit;
  A.idx = idx;
  const int64_t items = g.items;
  if (g.dtype == HS_BF16) {
    switch (g.D) {
      case 1: launch_slice<HS_BF16, 1>(A, items, stream); break;
      case 2: launch_slice<HS_BF16, 2>(A, items, stream); break;
      case 4: launch_slice<HS_BF16, 4>(A, items, stream); break;
      default: launch_slice<HS_BF16, 8>(A, items, stream); break;
    }
  } else {
    switch (g.D) {
      case 1: launch_slice<HS_F32, 1>(A, items, stream); break;
      case 2: launch_slice<HS_F32, 2>(A, items, stream); break;
      case 4: launch_slice<HS_F32, 4>(A, items, stream); break;
      default: launch_slice<HS_F32, 8>(A, items, stream); break;
    }
  }
  if (hipGetLastError() != hipSuccess) return HS_ERR_HIP;
  const int64_t wgs = ((int64_t)nrows + kWaves - 1) / kWaves;
  hs_topl_merge_kernel<<<(unsigned)wgs, kThreads, 0, stream>>>(A);
  return hipGetLastError() == hipSuccess ? HS_OK : HS_ERR_HIP;
}

}  // namespace hs
