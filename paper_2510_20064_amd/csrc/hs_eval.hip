// Drafter evaluation: softmax statistics, alpha = sum_v min(p, q_i) for every drafter
// (Theorem 1), greedy agreement and argmax.
//
// A (query, position) group holds N + 1 logits rows: row 0 is the target, rows 1..N the
// drafters. Rows are cut into S slices of up to 1024 16-byte vectors (8192 bf16 or 4096
// fp32 logits). Every work item is one wave (64 lanes), which streams its slice as up to 4
// sub-slices of 256 vectors (4 per lane), double-buffered, reduces across lanes on the DPP
// network and publishes with one lane. No wave ever waits for another one to make progress:
//   kernel 1, item (g, r, s) : max / lowest argmax / exp2 sum of slice s of row r. The row's
//                              last finisher folds its S slices into the row's log2
//                              normaliser (as hi + lo) and argmax; with argmax outputs, the
//                              group's last row writes argmax and agreement.
//   kernel 2, item (g, c, s) : for the drafters of row set c (CH drafters), the sum over
//                              slice s of exp2(min(e_t, e_i)), e = z c - log2(normaliser),
//                              c = log2(e) / T. The group's last finisher sums each
//                              drafter's S partials in slice order into alpha, clamped to [0, 1].
// Kernel 2 re-reads the slices kernel 1 streamed (two passes over the logits: both row
// normalisers are needed before any min can be taken). Slice s is processed on XCD s % 8 in
// both kernels (workgroups are dispatched to the 8 XCDs round-robin); the waves of one
// (group, slice) run together, so the target slice they share is read once per XCD.
//
// Words that cross waves are 64-bit relaxed atomics whose low half is a non-zero tag. A
// consumer reads them only after a completion counter says every producer has finished, so
// any wait is for visibility alone (bounded all the same: NaN / argmax -2 on expiry, never
// a hang). Consumers zero the words and counters they were the last to use, so a completed
// call leaves the workspace zero-filled for the next one.
#include <algorithm>
#include <climits>

#include "hs_internal.h"

namespace hs {

constexpr int kXcds = 8;
constexpr int kBlockWaves = kThreads / 64;
constexpr int kSubVec = 4;              // 16-byte vectors per lane per sub-slice
constexpr int kSubVecs = 64 * kSubVec;  // vectors per sub-slice
constexpr int kMaxSubs = kSliceVecs / kSubVecs;  // sub-slices per slice
constexpr int kMaxCH = 8;               // drafters per row set
constexpr uint32_t kSpinLimit = 1u << 20;

struct EvalArgs {
  RowTable rows;
  Geom g;
  float c;
  int g0, gn;  // this launch covers groups [g0, g0 + gn)
  int CH, nch;
  float* alpha;
  uint8_t* agree;
  int32_t* argmax_t;
  int32_t* argmax_d;
  uint64_t* sstat;  // [G][R][S][2]: (max, argmax + 1), (sum, 1)
  uint64_t* rstat;  // [G][R][3]   : (Xhi, 1), (Xlo, 1), (argmax + 1)
  uint64_t* parts;  // [G][N][S]   : (partial sum, 1)
  uint32_t* ctr;    // [G][R] slices done per row; [G] rows done (kernel 1), then row sets
                    // done (kernel 2); [G][nch] minsum items done per row set
#ifdef HS_TRACE
  uint64_t* trace;  // per wave: 8 timestamps
#endif
};
#ifdef HS_TRACE
#define HS_STAMP_AT(base, i)                                                             \
  if (lane == 0 && A.trace)                                                              \
  A.trace[((size_t)(base) + blockIdx.x * kBlockWaves + (threadIdx.x >> 6)) * 8 + (i)] = \
      __builtin_amdgcn_s_memrealtime()
#define HS_STAMP(i) HS_STAMP_AT(0, i)
#define HS_STAMP1(i) HS_STAMP_AT(200000, i)
#else
#define HS_STAMP(i)
#define HS_STAMP1(i)
#endif

// ---- cross-wave words and counters -------------------------------------------------------

__device__ inline void put_word(uint64_t* w, uint64_t v) {
  __hip_atomic_store(w, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline uint64_t get_word(uint64_t* w) {
  return __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// v if it is tagged, else w polled until it is (bounded: NaN / -2 on expiry).
__device__ inline uint64_t settle_word(uint64_t* w, uint64_t v) {
  uint32_t n = 0;
  while ((uint32_t)v == 0u) {
    __builtin_amdgcn_s_sleep(4);
    v = get_word(w);
    if (++n > kSpinLimit) return ((uint64_t)0x7FC00000u << 32) | 0xFFFFFFFFu;
  }
  return v;
}
__device__ inline uint64_t tag_f(float x) { return ((uint64_t)__float_as_uint(x) << 32) | 1u; }
__device__ inline float word_f(uint64_t w) { return __uint_as_float((uint32_t)(w >> 32)); }
__device__ inline void ctr_zero(uint32_t* p) {
  __hip_atomic_store(p, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// One increment for the wave; true in every lane if it was the last of `total`.
__device__ inline bool wave_count_last(uint32_t* ctr, uint32_t total, int lane) {
  int last = 0;
  if (lane == 0)
    last = __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
           total - 1;
  return __builtin_amdgcn_readfirstlane(last) != 0;
}

struct Counters {
  uint32_t* row;    // [G][R]
  uint32_t* rows;   // [G]
  uint32_t* items;  // [G][nch]
};
__device__ inline Counters counters(const EvalArgs& A) {
  Counters C;
  C.row = A.ctr;
  C.rows = A.ctr + (size_t)A.g.G * A.g.R;
  C.items = C.rows + A.g.G;
  return C;
}

// ---- wave reductions on the DPP network ----------------------------------------------------
// Pairs and quads by quad_perm, 8- and 16-lane groups by the half-row and row mirrors, then
// the four row results are combined in a fixed order; every lane gets the same value. All
// 64 lanes must be active.

template <int CTRL>
__device__ inline float dpp_f(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xF, 0xF, false));
}
template <int CTRL>
__device__ inline int dpp_i(int x) {
  return __builtin_amdgcn_mov_dpp(x, CTRL, 0xF, 0xF, false);
}
__device__ inline float lane_f(float x, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), l));
}

__device__ inline float wave_sum_f(float v) {
  v += dpp_f<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp_f<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp_f<0x141>(v);  // row_half_mirror
  v += dpp_f<0x140>(v);  // row_mirror
  return (lane_f(v, 0) + lane_f(v, 16)) + (lane_f(v, 32) + lane_f(v, 48));
}

template <int CTRL>
__device__ inline void argmax_step(float& m, int& idx) {
  const float m2 = dpp_f<CTRL>(m);
  const int i2 = dpp_i<CTRL>(idx);
  argmax_combine(m, idx, m2, i2);
}
template <bool NEED_ARG>
__device__ inline void wave_max(float& m, int& idx) {
  if (NEED_ARG) {
    argmax_step<0xB1>(m, idx);
    argmax_step<0x4E>(m, idx);
    argmax_step<0x141>(m, idx);
    argmax_step<0x140>(m, idx);
    float r = lane_f(m, 0);
    int ri = __builtin_amdgcn_readlane(idx, 0);
#pragma unroll
    for (int l = 16; l < 64; l += 16)
      argmax_combine(r, ri, lane_f(m, l), __builtin_amdgcn_readlane(idx, l));
    m = r;
    idx = ri;
  } else {
    m = fmaxf(m, dpp_f<0xB1>(m));
    m = fmaxf(m, dpp_f<0x4E>(m));
    m = fmaxf(m, dpp_f<0x141>(m));
    m = fmaxf(m, dpp_f<0x140>(m));
    m = fmaxf(fmaxf(lane_f(m, 0), lane_f(m, 16)), fmaxf(lane_f(m, 32), lane_f(m, 48)));
  }
}

template <int CTRL>
__device__ inline void lse_step(float& o, float& s) {
  const float o2 = dpp_f<CTRL>(o);
  const float s2 = dpp_f<CTRL>(s);
  lse2_combine(o, s, o2, s2);
}
__device__ inline void wave_lse(float& o, float& s) {
  lse_step<0xB1>(o, s);
  lse_step<0x4E>(o, s);
  lse_step<0x141>(o, s);
  lse_step<0x140>(o, s);
  float ro = lane_f(o, 0), rs = lane_f(s, 0);
#pragma unroll
  for (int l = 16; l < 64; l += 16) lse2_combine(ro, rs, lane_f(o, l), lane_f(s, l));
  o = ro;
  s = rs;
}

// ---- loads -----------------------------------------------------------------------------------

template <int DT>
__device__ inline const char* row_base(const EvalArgs& A, int r, int b, int k) {
  return reinterpret_cast<const char*>(A.rows.ptr[r]) +
         ((int64_t)b * A.rows.sb[r] + (int64_t)k * A.rows.sk[r]) * Vec<DT>::kBytes;
}

// The lane's kSubVec vectors of sub-slice `sub` of the slice [v0, v1); -inf beyond it.
template <int DT>
__device__ inline void load_sub(const char* rowp, int64_t v0, int64_t v1, int sub, int64_t V,
                                int lane, typename Vec<DT>::Raw* raw) {
#pragma unroll
  for (int j = 0; j < kSubVec; ++j) {
    const int64_t vi = v0 + (int64_t)sub * kSubVecs + j * 64 + lane;
    raw[j] = vi < v1 ? Vec<DT>::load_raw(rowp, vi, V) : Vec<DT>::neg_raw();
  }
}

// Item index -> (slice s, index within its XCD class): waves of workgroup b serve XCD b % 8
// and take slices s with s % 8 == b % 8. Returns false past the end of the class.
__device__ inline bool xcd_item(int per_slice, int S, int& s, int& rest) {
  const int x = blockIdx.x % kXcds;
  const int nx = S > x ? (S - x + kXcds - 1) / kXcds : 0;
  const int idx = (blockIdx.x / kXcds) * kBlockWaves + (threadIdx.x >> 6);
  if (idx >= per_slice * nx) return false;
  s = x + kXcds * (idx % nx);
  rest = idx / nx;
  return true;
}

// ---- kernel 1: row statistics ------------------------------------------------------------------

// Per-lane running statistics of one row: max / lowest argmax, and the sum of exp2(z c - o)
// against o = fl(max * c).
struct LaneStat {
  float m, o, s;
  int idx;
};

template <int DT, bool NEED_SUM, bool NEED_ARG>
__device__ inline void lane_stat_sub(LaneStat& st, const typename Vec<DT>::Raw* raw, int64_t vb,
                                     int lane, float c) {
  using Vt = Vec<DT>;
  constexpr int E = Vt::kElems;
  float z[kSubVec][E];
#pragma unroll
  for (int j = 0; j < kSubVec; ++j) Vt::unpack(raw[j], z[j]);
  float mk = -INFINITY;
  int ik = INT_MAX;
#pragma unroll
  for (int j = 0; j < kSubVec; ++j)
#pragma unroll
    for (int e = 0; e < E; ++e) {
      if (NEED_ARG) {
        if (z[j][e] > mk) {
          mk = z[j][e];
          ik = (int)((vb + j * 64 + lane) * E + e);
        }
      } else {
        mk = fmaxf(mk, z[j][e]);
      }
    }
  if (NEED_ARG) argmax_combine(st.m, st.idx, mk, ik);
  else st.m = fmaxf(st.m, mk);
  if (NEED_SUM && st.m != -INFINITY) {
    const float on = st.m * c;  // rounded product; the row fold recomputes exactly this value
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < kSubVec; ++j)
#pragma unroll
      for (int e = 0; e < E; ++e) acc[e & 3] += __builtin_amdgcn_exp2f(fmaf(z[j][e], c, -on));
    const float add = (acc[0] + acc[1]) + (acc[2] + acc[3]);
    st.s = (st.s > 0.0f ? st.s * __builtin_amdgcn_exp2f(st.o - on) : 0.0f) + add;
    st.o = on;
  }
}

// Fold the S slice statistics of row r of group grp: lane j takes slices j, j + 64, ... in
// order, then the wave reduces; publishes the row's log2 normaliser and argmax.
template <bool NEED_SUM, bool NEED_ARG>
__device__ inline void fold_row(const EvalArgs& A, int grp, int r, int lane) {
  const Geom& g = A.g;
  uint64_t* base = A.sstat + ((int64_t)grp * g.R + r) * g.S * 2;
  LaneStat st{-INFINITY, -INFINITY, 0.0f, INT_MAX};
  for (int j = lane; j < g.S; j += 64) {
    uint64_t* w = base + 2 * j;
    const uint64_t w0 = settle_word(w, get_word(w));
    const float ms = word_f(w0);
    if (NEED_ARG) argmax_combine(st.m, st.idx, ms, (int)(uint32_t)w0 - 1);
    else st.m = fmaxf(st.m, ms);
    put_word(w, 0);
    if (NEED_SUM) {
      lse2_combine(st.o, st.s, ms * A.c, word_f(settle_word(w + 1, get_word(w + 1))));
      put_word(w + 1, 0);
    }
  }
  wave_max<NEED_ARG>(st.m, st.idx);
  if (NEED_SUM) wave_lse(st.o, st.s);
  if (lane == 0) {
    uint64_t* w = A.rstat + ((int64_t)grp * g.R + r) * 3;
    if (NEED_SUM) {
      // log2 normaliser O + log2(sum) as an unevaluated sum hi + lo (TwoSum)
      const float l2 = log2f(st.s);
      const float hi = st.o + l2;
      const float bb = hi - st.o;
      const float lo = (st.o - (hi - bb)) + (l2 - bb);
      put_word(w + 0, tag_f(hi));
      put_word(w + 1, tag_f(lo));
    }
    if (NEED_ARG) put_word(w + 2, (uint64_t)(uint32_t)(st.idx + 1));
  }
}

template <int DT, bool NEED_SUM, bool NEED_ARG>
__global__ __launch_bounds__(kThreads) void hs_rowstats_kernel(EvalArgs A) {
  using Raw = typename Vec<DT>::Raw;
  const Geom& g = A.g;
  const int lane = threadIdx.x & 63;
  int s, rest;
  if (!xcd_item(A.gn * g.R, g.S, s, rest)) return;
  HS_STAMP1(0);
  const int r = rest % g.R;
  const int grp = A.g0 + rest / g.R;
  const int b = grp / g.K, k = grp % g.K;
  const int64_t v0 = (int64_t)s * g.vps;
  const int64_t v1 = min(v0 + g.vps, g.nvec);
  const int nsub = (int)((v1 - v0 + kSubVecs - 1) / kSubVecs);
  const char* rowp = row_base<DT>(A, r, b, k);
  LaneStat st{-INFINITY, -INFINITY, 0.0f, INT_MAX};
  // every load of the slice is issued before the first is used: one memory round trip
  Raw raw[kMaxSubs][kSubVec];
#pragma unroll
  for (int sub = 0; sub < kMaxSubs; ++sub)
    if (sub < nsub) load_sub<DT>(rowp, v0, v1, sub, g.V, lane, raw[sub]);
#pragma unroll
  for (int sub = 0; sub < kMaxSubs; ++sub)
    if (sub < nsub)
      lane_stat_sub<DT, NEED_SUM, NEED_ARG>(st, raw[sub], v0 + (int64_t)sub * kSubVecs, lane, A.c);
  // a lane whose logits are all -inf still owns its lowest valid index
  if (NEED_ARG && st.idx == INT_MAX && v0 + lane < v1)
    st.idx = (int)((v0 + lane) * Vec<DT>::kElems);
  wave_max<NEED_ARG>(st.m, st.idx);
  if (NEED_SUM) wave_lse(st.o, st.s);
  if (lane == 0) {
    uint64_t* w = A.sstat + (((int64_t)grp * g.R + r) * g.S + s) * 2;
    put_word(w, ((uint64_t)__float_as_uint(st.m) << 32) | (uint32_t)(NEED_ARG ? st.idx + 1 : 1));
    if (NEED_SUM) put_word(w + 1, tag_f(st.s));
  }
  HS_STAMP1(1);
  const Counters C = counters(A);
  uint32_t* rc = C.row + (size_t)grp * g.R + r;
  if (!wave_count_last(rc, (uint32_t)g.S, lane)) { HS_STAMP1(2); return; }
  HS_STAMP1(3);
  if (lane == 0) ctr_zero(rc);
  fold_row<NEED_SUM, NEED_ARG>(A, grp, r, lane);
  HS_STAMP1(4);
  if (!NEED_ARG) return;
  if (!wave_count_last(C.rows + grp, (uint32_t)g.R, lane)) return;
  if (lane == 0) ctr_zero(C.rows + grp);
  // argmax outputs and agreement of the group
  const int bq = grp / g.K, kq = grp % g.K;
  int idx[2] = {-2, -2};
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int rr = lane + 64 * h;
    if (rr < g.R) {
      uint64_t* w = A.rstat + ((int64_t)grp * g.R + rr) * 3 + 2;
      idx[h] = (int)(uint32_t)settle_word(w, get_word(w)) - 1;
      put_word(w, 0);
    }
  }
  const int idx0 = __builtin_amdgcn_readlane(idx[0], 0);
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int rr = lane + 64 * h;
    if (rr < g.R) {
      if (rr == 0) {
        if (A.argmax_t) A.argmax_t[(int64_t)bq * g.K + kq] = idx[h];
      } else {
        const int64_t o = ((int64_t)bq * g.N + (rr - 1)) * g.K + kq;
        if (A.argmax_d) A.argmax_d[o] = idx[h];
        if (A.agree) A.agree[o] = (uint8_t)(idx[h] == idx0);
      }
    }
  }
}

// ---- kernel 2: min-sum -----------------------------------------------------------------------

template <int DT>
__global__ __launch_bounds__(kThreads) void hs_minsum_kernel(EvalArgs A) {
  using Vt = Vec<DT>;
  using Raw = typename Vt::Raw;
  constexpr int E = Vt::kElems;
  const Geom& g = A.g;
  const int lane = threadIdx.x & 63;
  int s, rest;
  if (!xcd_item(A.gn * A.nch, g.S, s, rest)) return;
  HS_STAMP(0);
  const int rs = rest % A.nch;
  const int grp = A.g0 + rest / A.nch;
  const int b = grp / g.K, k = grp % g.K;
  const int64_t v0 = (int64_t)s * g.vps;
  const int64_t v1 = min(v0 + g.vps, g.nvec);
  const int nsub = (int)((v1 - v0 + kSubVecs - 1) / kSubVecs);
  const int r0 = 1 + rs * A.CH;
  const int n = min(A.CH, g.N - rs * A.CH);
  // normalisers (hi, lo) of the target and the drafters, one word per lane
  float xw = 0.0f;
  if (lane < 2 * (n + 1)) {
    const int row = (lane < 2) ? 0 : r0 + (lane / 2 - 1);
    uint64_t* w = A.rstat + ((int64_t)grp * g.R + row) * 3 + (lane & 1);
    xw = word_f(settle_word(w, get_word(w)));
  }
  const float xth = lane_f(xw, 0), xtl = lane_f(xw, 1);
  HS_STAMP(1);
  const char* tp = row_base<DT>(A, 0, b, k);
  // Steps t = 0 .. nsub*n - 1 visit (sub-slice t / n, drafter t % n); loads run one step
  // ahead (two drafter buffers), and the target's next sub-slice is loaded as soon as the
  // current one has been turned into exponents.
  float acc[kMaxCH];
#pragma unroll
  for (int d = 0; d < kMaxCH; ++d) acc[d] = 0.0f;
  Raw ra[kSubVec], rb[kSubVec], rt[kSubVec];
  float et[kSubVec][E];
  const int steps = nsub * n;
  auto load_d = [&](int t, Raw* dst) {
    load_sub<DT>(row_base<DT>(A, r0 + t % n, b, k), v0, v1, t / n, g.V, lane, dst);
  };
  auto step = [&](int t, const Raw* cur) {
    const int sub = t / n, d = t % n;
    if (d == 0) {
#pragma unroll
      for (int j = 0; j < kSubVec; ++j) {
        Vt::unpack(rt[j], et[j]);
#pragma unroll
        for (int e = 0; e < E; ++e) et[j][e] = fmaf(et[j][e], A.c, -xth) - xtl;
      }
      if (sub + 1 < nsub) load_sub<DT>(tp, v0, v1, sub + 1, g.V, lane, rt);
    }
    const float xh = lane_f(xw, 2 * (d + 1)), xl = lane_f(xw, 2 * (d + 1) + 1);
    float a4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < kSubVec; ++j) {
      float z[E];
      Vt::unpack(cur[j], z);
#pragma unroll
      for (int e = 0; e < E; ++e)
        a4[e & 3] += __builtin_amdgcn_exp2f(fminf(et[j][e], fmaf(z[e], A.c, -xh) - xl));
    }
    const float v = (a4[0] + a4[1]) + (a4[2] + a4[3]);
#pragma unroll
    for (int dd = 0; dd < kMaxCH; ++dd) acc[dd] += (dd == d) ? v : 0.0f;
  };
  load_sub<DT>(tp, v0, v1, 0, g.V, lane, rt);
  load_d(0, ra);
  for (int t = 0; t < steps; t += 2) {
    if (t + 1 < steps) load_d(t + 1, rb);
    step(t, ra);
    if (t + 2 < steps) load_d(t + 2, ra);
    if (t + 1 < steps) step(t + 1, rb);
  }
#pragma unroll
  for (int d = 0; d < kMaxCH; ++d) {
    if (d < n) {
      const float v = wave_sum_f(acc[d]);
      if (lane == 0) put_word(A.parts + ((int64_t)grp * g.N + (r0 - 1) + d) * g.S + s, tag_f(v));
    }
  }
  HS_STAMP(2);
  // The row set's last wave folds its drafters' S partials (slice order) into alpha; the
  // group's last row set then clears the row statistics.
  const Counters C = counters(A);
  uint32_t* rc = C.items + (size_t)grp * A.nch + rs;
  if (!wave_count_last(rc, (uint32_t)g.S, lane)) { HS_STAMP(3); return; }
  HS_STAMP(4);
  if (lane == 0) ctr_zero(rc);
  for (int d = lane; d < n; d += 64) {
    uint64_t* base = A.parts + ((int64_t)grp * g.N + (r0 - 1) + d) * g.S;
    float a = 0.0f;
    for (int s0 = 0; s0 < g.S; s0 += 32) {
      uint64_t w[32];
#pragma unroll
      for (int j = 0; j < 32; ++j)
        if (s0 + j < g.S) w[j] = get_word(base + s0 + j);
#pragma unroll
      for (int j = 0; j < 32; ++j)
        if (s0 + j < g.S) {
          a += word_f(settle_word(base + s0 + j, w[j]));
          put_word(base + s0 + j, 0);
        }
    }
    A.alpha[((int64_t)b * g.N + (r0 - 1) + d) * g.K + k] = fminf(fmaxf(a, 0.0f), 1.0f);
  }
  if (!wave_count_last(C.rows + grp, (uint32_t)A.nch, lane)) return;
  if (lane == 0) ctr_zero(C.rows + grp);
  for (int r = lane; r < g.R; r += 64) {
    uint64_t* w = A.rstat + ((int64_t)grp * g.R + r) * 3;
    put_word(w + 0, 0);
    put_word(w + 1, 0);
  }
  HS_STAMP(5);
}

// ---- launcher ------------------------------------------------------------------------------------

template <int DT, bool NEED_SUM, bool NEED_ARG>
static void launch_rowstats(const EvalArgs& A, hipStream_t stream) {
  const int n0 = (A.g.S + kXcds - 1) / kXcds;  // slices of XCD class 0 (the largest)
  const int64_t waves = (int64_t)A.gn * A.g.R * n0;
  const int64_t blocks = kXcds * ((waves + kBlockWaves - 1) / kBlockWaves);
  hs_rowstats_kernel<DT, NEED_SUM, NEED_ARG><<<(unsigned)blocks, kThreads, 0, stream>>>(A);
}

template <int DT>
static void launch_minsum(const EvalArgs& A, hipStream_t stream) {
  const int n0 = (A.g.S + kXcds - 1) / kXcds;
  const int64_t waves = (int64_t)A.gn * A.nch * n0;
  const int64_t blocks = kXcds * ((waves + kBlockWaves - 1) / kBlockWaves);
  hs_minsum_kernel<DT><<<(unsigned)blocks, kThreads, 0, stream>>>(A);
}

template <int DT>
static void launch_chunk(const EvalArgs& A, bool need_sum, bool need_arg, hipStream_t stream) {
  if (need_sum && need_arg) launch_rowstats<DT, true, true>(A, stream);
  else if (need_sum) launch_rowstats<DT, true, false>(A, stream);
  else launch_rowstats<DT, false, true>(A, stream);
  if (need_sum) launch_minsum<DT>(A, stream);
}

#ifdef HS_TRACE
uint64_t* g_trace = nullptr;  // per-wave timestamps of the next launch (debug builds only)
#endif

int launch_round(const Geom& g, const RowTable& rows, float c, bool need_sum, bool need_arg,
                 float* alpha, uint8_t* agree, int32_t* argmax_t, int32_t* argmax_d, char* ws,
                 const TailArgs* tail, hipStream_t stream) {
  const WsLayout L = ws_layout(g);
  EvalArgs A{};
  A.rows = rows;
  A.g = g;
  A.c = c;
  A.alpha = alpha;
  A.agree = agree;
  A.argmax_t = argmax_t;
  A.argmax_d = argmax_d;
  A.sstat = reinterpret_cast<uint64_t*>(ws + L.slice_stats);
  A.rstat = reinterpret_cast<uint64_t*>(ws + L.row_stats);
  A.parts = reinterpret_cast<uint64_t*>(ws + L.parts);
  A.ctr = reinterpret_cast<uint32_t*>(ws + L.counters);
  // One launch pair covers every group. (Splitting the groups into chunks that fit the
  // 256 MB Infinity Cache does not help: its read bandwidth is no higher than HBM's.)
  A.g0 = 0;
  A.gn = g.G;
  // drafters per minsum item: one, so every wave's chain of dependent loads stays short and
  // the kernel has the most waves; the target slice the drafters share is re-read by waves
  // that run together and hits the L2
  A.CH = 1;
  A.nch = g.N;
#ifdef HS_TRACE
  A.trace = g_trace;
#endif
  if (g.dtype == HS_F32) launch_chunk<HS_F32>(A, need_sum, need_arg, stream);
  else launch_chunk<HS_BF16>(A, need_sum, need_arg, stream);
  if (hipGetLastError() != hipSuccess) return HS_ERR_HIP;
  if (tail) return launch_tail(*tail, stream);
  return HS_OK;
}

}  // namespace hs
