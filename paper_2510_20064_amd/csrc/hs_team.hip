// Drafter evaluation with one read of every logit: softmax statistics, alpha =
// sum_v min(p, q_i) for every drafter (Theorem 1), greedy argmax and agreement.
//
// min(p_v, q_v) needs both rows' normalisers, which depend on the whole row, so the
// slices of a row have to meet before any min can be taken. Here they meet on chip: a
// work item is (row set, slice) = the target slice and the slices of up to D drafters of
// one (query, position) group, 256 16-byte vectors each, held in the registers of one
// 256-thread workgroup (thread t owns vector t of every row). The S items of a row set form
// a team that is resident at the same time:
//   1. every item reduces its rows (max, lowest argmax, exp2 sum) and publishes them;
//      it keeps e_v = exp2(z_v c - o) against its lane's offset o = fl(m_lane c),
//      c = log2(e) / T;
//   2. item s folds the S slice statistics of row s (rows s, s + S, ... when S is smaller
//      than the row count) into the row's log2 normaliser L = hi + lo and publishes it;
//   3. every item reads the normalisers and takes, per drafter,
//      sum_v min(p_v, q_v) = F_d sum_v min(e_t,v G, e_d,v), with a_x = o_x - L_x,
//      F_d = 2^(a_d) and G = 2^(a_t - a_d): one multiply, one min and one add per drafter
//      logit, no second exponential;
//   4. a second launch sums each drafter's S slice partials in slice order into alpha.
// The loads of an item's successor are issued before its exchange (step 2 - 3), so HBM stays
// busy while the team waits.
//
// Items are dealt to workgroups round-robin, item i to workgroup i mod P, where P is a
// multiple of S no larger than what the device holds at once: every team lies inside one
// round and all of its members are resident, so waiting on a team member cannot deadlock.
// Words crossing workgroups carry the call's epoch as tag; the fold launch advances the
// epoch. Every wait is bounded: a word that never arrives yields NaN (argmax -2), no hang.
#include <algorithm>
#include <atomic>
#include <cstdio>

#include "hs_wave.h"

namespace hs {

constexpr uint32_t kSpinLimit = 1u << 18;  // polls before a wait gives up (~0.5 s)

struct TeamArgs {
  RowTable rows;
  int N, K, nsub, S, items;
  int64_t V, nvec;
  float c;
  const uint32_t* epoch;
  uint64_t* fail;  // set, with the call's tag, by the first wait that gives up
  uint64_t* stat;  // [sets][D + 1][S][3]
  uint64_t* norm;  // [sets][D + 1][3]
  float* part;     // [G][N][S]
  int32_t* argmax_t;
  int32_t* argmax_d;
  uint8_t* agree;
#ifdef HS_TRACE
  uint64_t* trace;  // [items][8] phase timestamps of workgroup thread 0
#endif
};

#ifdef HS_TRACE
uint64_t* g_trace = nullptr;
extern "C" __attribute__((visibility("default"))) void hs_debug_set_trace(void* p) {
  g_trace = reinterpret_cast<uint64_t*>(p);
}
#define HS_STAMP(i) \
  if (t == 0 && A.trace) A.trace[(size_t)it * 8 + (i)] = __builtin_amdgcn_s_memrealtime()
#else
#define HS_STAMP(i)
#endif

// Tag of this call's words: never 0, the content of a zero-filled workspace.
__device__ inline uint32_t call_tag(const uint32_t* epoch) { return (*epoch % 0xFFFFFFFFu) + 1u; }

// The word at w once it carries tag. Bounded: after kSpinLimit polls, or as soon as another
// wait of this call has given up, the value is 0xFFFFFFFE (a NaN as float, -2 as int); the
// first wait to give up raises the call's fail flag, so one lost word costs one time-out,
// not one per wait.
__device__ inline uint64_t await_word(const uint64_t* w, uint32_t tag, uint64_t* fail) {
  constexpr uint64_t kLost = 0xFFFFFFFEull << 32;
  uint64_t v = get_word(w);
  for (uint32_t n = 1; (uint32_t)v != tag; ++n) {
    if (n == kSpinLimit) {
      put_word(fail, word_of(1, tag));
      return kLost | tag;
    }
    if ((n & 255) == 0 && (uint32_t)get_word(fail) == tag) return kLost | tag;
    __builtin_amdgcn_s_sleep(2);
    v = get_word(w);
  }
  return v;
}

// Fold of row rr of row set `set`: the S slice statistics, two slices per lane per pass
// (lane j takes slices j, j + 64, ... in order), then the wave. Publishes the row's log2
// normaliser as hi + lo and its argmax; writes the argmax and agreement outputs.
template <int D, bool NEED_SUM, bool NEED_ARG>
__device__ __forceinline__ void fold_row(const TeamArgs& A, int set, int rr, int b, int k, int sub,
                                uint32_t tag, int lane) {
  constexpr int RM = D + 1;
  const int S = A.S;
  const uint64_t* base = A.stat + ((int64_t)set * RM + rr) * S * 3;
  float m = -INFINITY, o = -INFINITY, sum = 0.0f;
  int idx = INT_MAX;
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
        if ((uint32_t)w[h][0] != tag) w[h][0] = await_word(base + 3 * j, tag, A.fail);
        const float ms = word_f(w[h][0]);
        if (NEED_ARG) {
          if ((uint32_t)w[h][2] != tag) w[h][2] = await_word(base + 3 * j + 2, tag, A.fail);
          argmax_combine(m, idx, ms, word_i(w[h][2]));
        } else {
          m = fmaxf(m, ms);
        }
        if (NEED_SUM) {
          if ((uint32_t)w[h][1] != tag) w[h][1] = await_word(base + 3 * j + 1, tag, A.fail);
          lse2_combine(o, sum, ms * A.c, word_f(w[h][1]));
        }
      }
    }
  }
  wave_max<NEED_ARG>(m, idx);
  if (NEED_SUM) wave_lse(o, sum);
  if (lane != 0) return;
  uint64_t* nw = A.norm + ((int64_t)set * RM + rr) * 3;
  if (NEED_SUM) {
    // log2 normaliser o + log2(sum) as an unevaluated sum hi + lo (TwoSum)
    const float l2 = log2f(sum);
    const float hi = o + l2;
    const float bb = hi - o;
    const float lo = (o - (hi - bb)) + (l2 - bb);
    put_word(nw, word_of(hi, tag));
    put_word(nw + 1, word_of(lo, tag));
  }
  if (NEED_ARG) {
    put_word(nw + 2, word_of(idx, tag));
    if (rr == 0) {
      if (sub == 0 && A.argmax_t) A.argmax_t[(int64_t)b * A.K + k] = idx;
    } else {
      const int64_t oi = ((int64_t)b * A.N + sub * D + rr - 1) * A.K + k;
      if (A.argmax_d) A.argmax_d[oi] = idx;
      if (A.agree) {
        const int it = word_i(await_word(A.norm + (int64_t)set * RM * 3 + 2, tag, A.fail));
        A.agree[oi] = (uint8_t)(idx == it);
      }
    }
  }
}

// Position of work item `it`: row set, slice, group (b, k), drafters n in the set, and the
// calling thread's vector index within the row.
struct ItemPos {
  int set, s, g, sub, b, k, n;
  int vi;  // a row holds fewer than 2^31 logits
};
__device__ inline ItemPos item_pos(const TeamArgs& A, int it, int D) {
  ItemPos q;
  q.set = it / A.S;
  q.s = it - q.set * A.S;
  q.g = q.set / A.nsub;
  q.sub = q.set - q.g * A.nsub;
  q.b = q.g / A.K;
  q.k = q.g - q.b * A.K;
  q.n = min(D, A.N - q.sub * D);
  q.vi = q.s * kThreads + (int)threadIdx.x;
  return q;
}

template <int DT, int D, bool NEED_SUM, bool NEED_ARG>
__global__ __launch_bounds__(kThreads, 3) void hs_team_kernel(TeamArgs A) {
  using Vt = Vec<DT>;
  using Raw = typename Vt::Raw;
  constexpr int E = Vt::kElems;
  constexpr int RM = D + 1;
  constexpr int XR = NEED_SUM ? RM : 1;  // rows of kept e_v
  __shared__ float sh_m[kWaves][RM];
  __shared__ float sh_s[kWaves][RM];
  __shared__ int sh_i[kWaves][RM];
  __shared__ float sh_hi[RM];
  __shared__ float sh_lo[RM];
  __shared__ float sh_p[kWaves][D];

  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  const uint32_t tag = call_tag(A.epoch);
  const int S = A.S;
  const int P = gridDim.x;
  Raw nxt[RM];

  // Issue the loads of item `it` into nxt: one unconditional 16-byte load per row, from an
  // address clamped into the row's complete vectors (lanes past the row end are masked to -inf
  // before use), so the loads of all rows are in flight together. The one partial vector at
  // the end of a row (V not a multiple of the vector width) is then re-read element by
  // element, in a branch taken only by the slice that holds it.
  const int64_t vfull = A.V / E;  // complete 16-byte vectors per row
  auto fetch = [&](int it) __attribute__((always_inline)) {
    const ItemPos q = item_pos(A, it, D);
    const char* rp[RM];
#pragma unroll
    for (int r = 0; r < RM; ++r) {
      const int row = r == 0 ? 0 : q.sub * D + min(r, q.n);
      rp[r] = reinterpret_cast<const char*>(A.rows.ptr[row]) +
              ((int64_t)q.b * A.rows.sb[row] + (int64_t)q.k * A.rows.sk[row]) * Vt::kBytes;
    }
    if (vfull > 0) {
      // uniform row base + 32-bit lane offset (a row holds < 2^31 logits)
      const uint32_t off = (uint32_t)((q.vi < vfull ? q.vi : vfull - 1) * 16);
#pragma unroll
      for (int r = 0; r < RM; ++r)
        if (r <= q.n) nxt[r] = *reinterpret_cast<const Raw*>(rp[r] + off);
    }
    if (vfull < A.nvec && (int64_t)(q.s + 1) * kThreads > vfull) {  // this slice holds the tail
#pragma unroll
      for (int r = 0; r < RM; ++r)
        if (r <= q.n && q.vi == vfull) nxt[r] = Vt::load_raw(rp[r], q.vi, A.V);
    }
  };

  float ex[XR][E];  // e_v of the current item, against the wave's offset of its row
  float ow[RM];     // that offset (wave-uniform), -inf for a wave with no finite logit

  int it = blockIdx.x;
  if (it < A.items) fetch(it);
  for (; it < A.items; it += P) {
    const ItemPos q = item_pos(A, it, D);
    HS_STAMP(0);

    // ---- 1. slice statistics of every row; e_v kept for step 3 ----
    // Per row: the wave's max m_w (and lowest argmax), then e_v = exp2(z_v c - o_w) against
    // o_w = fl(m_w c), and their wave sum; lane 0 leaves (m_w, sum, argmax) in LDS.
    if ((int64_t)(q.s + 1) * kThreads > A.nvec) {  // the slice that runs past the row end
#pragma unroll
      for (int r = 0; r < RM; ++r)
        if (q.vi >= A.nvec) nxt[r] = Vt::neg_raw();
    }
#pragma unroll
    for (int r = 0; r < RM; ++r) {
      if (r > q.n) continue;
      float z[E];
      Vt::unpack(nxt[r], z);
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
      // a lane whose logits are all -inf still owns its lowest valid index
      if (NEED_ARG && idx == INT_MAX && q.vi < A.nvec) idx = q.vi * E;
      wave_max<NEED_ARG>(m, idx);
      float sw = 0.0f;
      if constexpr (NEED_SUM) {
        // rounded product (no contraction), recomputed alike by every reader; a wave with
        // no finite logit takes offset 0 and gets exp2(-inf) = 0 throughout
        const float oc = m != -INFINITY ? m * A.c : 0.0f;
        float a0 = 0.0f, a1 = 0.0f;
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const float x = __builtin_amdgcn_exp2f(fmaf(z[e], A.c, -oc));
          ex[r][e] = x;
          if (e & 1) a1 += x;
          else a0 += x;
        }
        sw = wave_sum_f(a0 + a1);
        // wave-uniform: keep it in a scalar register
        ow[r] = __int_as_float(
            __builtin_amdgcn_readfirstlane(__float_as_int(m != -INFINITY ? oc : -INFINITY)));
      }
      if (lane == 0) {
        sh_m[wv][r] = m;
        sh_s[wv][r] = sw;
        if (NEED_ARG) sh_i[wv][r] = idx;
      }
    }
    HS_STAMP(1);
    if (it + P < A.items) fetch(it + P);  // the successor's loads fly during the exchange
    __syncthreads();
    HS_STAMP(2);

    // workgroup statistics of each row, published by lane r of wave 0
    if (wv == 0 && lane <= q.n) {
      const int r = lane;
      float m = sh_m[0][r];
      int idx = NEED_ARG ? sh_i[0][r] : 0;
#pragma unroll
      for (int w = 1; w < kWaves; ++w) {
        if (NEED_ARG) argmax_combine(m, idx, sh_m[w][r], sh_i[w][r]);
        else m = fmaxf(m, sh_m[w][r]);
      }
      uint64_t* wp = A.stat + (((int64_t)q.set * RM + r) * S + q.s) * 3;
      put_word(wp, word_of(m, tag));
      if (NEED_SUM) {
        const float o = m * A.c;
        float sum = 0.0f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
          const float mw = sh_m[w][r];
          if (mw != -INFINITY) sum += sh_s[w][r] * __builtin_amdgcn_exp2f(mw * A.c - o);
        }
        put_word(wp + 1, word_of(sum, tag));
      }
      if (NEED_ARG) put_word(wp + 2, word_of(idx, tag));
    }
    __syncthreads();
    HS_STAMP(3);

    // ---- 2. fold duty: rows s, s + S, ... of the row set, spread over the waves ----
    for (int rr = q.s + wv * S; rr <= q.n; rr += kWaves * S)
      fold_row<D, NEED_SUM, NEED_ARG>(A, q.set, rr, q.b, q.k, q.sub, tag, lane);
    HS_STAMP(4);

    // ---- 3. normalisers, then the min-sum of every drafter ----
    if constexpr (NEED_SUM) {
      if (wv == 0 && lane < 2 * (q.n + 1)) {
        const int r = lane >> 1;
        const float x =
            word_f(await_word(A.norm + ((int64_t)q.set * RM + r) * 3 + (lane & 1), tag, A.fail));
        if (lane & 1) sh_lo[r] = x;
        else sh_hi[r] = x;
      }
      HS_STAMP(5);
      __syncthreads();
      // p_v = e_t,v 2^(a_t), q_v = e_d,v 2^(a_d) with a_x = (o_x - hi_x) - lo_x, all
      // wave-uniform: min(p_v, q_v) = 2^(a_d) min(e_t,v 2^(a_t - a_d), e_d,v)
      const float at = (ow[0] - sh_hi[0]) - sh_lo[0];
#pragma unroll
      for (int d = 0; d < D; ++d) {
        if (d >= q.n) continue;
        const int r = d + 1;
        const float ad = (ow[r] - sh_hi[r]) - sh_lo[r];
        const float G = __builtin_amdgcn_exp2f(at - ad);
        float a0 = 0.0f, a1 = 0.0f;
#pragma unroll
        for (int e = 0; e < E; ++e) {
          // both >= 0 or +NaN (0 * inf): unsigned order of the bits is their order and a
          // NaN loses, as with fminf, without fminf's canonicalising of the operands
          const float y =
              __uint_as_float(min(__float_as_uint(ex[0][e] * G), __float_as_uint(ex[r][e])));
          if (e & 1) a1 += y;
          else a0 += y;
        }
        const float v = wave_sum_f(a0 + a1) * __builtin_amdgcn_exp2f(ad);
        if (lane == 0) sh_p[wv][d] = v;
      }
      __syncthreads();
      HS_STAMP(6);
      if (wv == 0 && lane < q.n)
        A.part[((int64_t)q.g * A.N + q.sub * D + lane) * S + q.s] =
            (sh_p[0][lane] + sh_p[1][lane]) + (sh_p[2][lane] + sh_p[3][lane]);
      HS_STAMP(7);
    }
  }
}

// ---- 4. alpha from the slice partials; advances the epoch ----------------------------------

struct FoldArgs {
  const float* part;  // NULL: epoch only
  float* alpha;
  int B, N, K, S;
  uint32_t* epoch;
};

// One wave per output alpha[b][i][k]: lane j sums slices j, j + 64, ... in order, then the
// wave in a fixed order; clamped to [0, 1] (NaN passes through).
__global__ __launch_bounds__(kThreads) void hs_fold_kernel(FoldArgs A) {
  if (blockIdx.x == 0 && threadIdx.x == 0) A.epoch[0] = A.epoch[0] + 1u;
  if (!A.part) return;
  const int lane = threadIdx.x & 63;
  const int64_t o = (int64_t)blockIdx.x * kWaves + (threadIdx.x >> 6);
  if (o >= (int64_t)A.B * A.N * A.K) return;
  const int k = (int)(o % A.K);
  const int64_t bi = o / A.K;
  const int i = (int)(bi % A.N);
  const int64_t b = bi / A.N;
  const float* src = A.part + ((b * A.K + k) * A.N + i) * A.S;
  float v = 0.0f;
  for (int j = lane; j < A.S; j += 64) v += src[j];
  v = wave_sum_f(v);
  if (lane == 0) A.alpha[o] = v != v ? v : fminf(fmaxf(v, 0.0f), 1.0f);
}

// ---- host side -------------------------------------------------------------------------------

namespace {

template <int DT, int D, bool NS, bool NA>
int capacity_t() {
  static std::atomic<int> cached[64];  // per device; 0 = not yet known
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  int v = cached[dev].load(std::memory_order_relaxed);
  if (v > 0) return v;
  int per_cu = 0, cus = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, hs_team_kernel<DT, D, NS, NA>,
                                                   kThreads, 0) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return 0;
  v = per_cu * cus;
  cached[dev].store(v, std::memory_order_relaxed);
  return v;
}

template <int DT, int D, bool NS, bool NA>
int launch_t(const TeamArgs& A, const TeamGeom& g, hipStream_t stream) {
  // a round: a multiple of S that the device holds at once
  const int64_t per_round = (int64_t)(capacity_t<DT, D, NS, NA>() / g.S) * g.S;
  if (per_round == 0) return HS_ERR_LIMIT;
  const int64_t P = std::min<int64_t>(g.items, per_round);
  hs_team_kernel<DT, D, NS, NA><<<(unsigned)P, kThreads, 0, stream>>>(A);
#ifdef HS_TRACE
  fprintf(stderr, "team grid %lld S %d items %lld\n", (long long)P, g.S, (long long)g.items);
#endif
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
  return by_set<F, HS_BF16>(g.D, ns, na, args...);
}

template <int DT, int D, bool NS, bool NA>
struct Capacity {
  static int run() { return capacity_t<DT, D, NS, NA>(); }
};
template <int DT, int D, bool NS, bool NA>
struct Launch {
  static int run(const TeamArgs& A, const TeamGeom& g, hipStream_t s) {
    return launch_t<DT, D, NS, NA>(A, g, s);
  }
};

}  // namespace

int team_capacity(const TeamGeom& g, bool need_sum, bool need_arg) {
  return dispatch<Capacity>(g, need_sum, need_arg);
}

int launch_round(const TeamGeom& g, const RowTable& rows, float c, bool need_sum, bool need_arg,
                 float* alpha, uint8_t* agree, int32_t* argmax_t, int32_t* argmax_d, char* ws,
                 const TailArgs* tail, hipStream_t stream) {
  const TeamWs L = team_ws(g);
  TeamArgs A{};
  A.rows = rows;
  A.N = g.N;
  A.K = g.K;
  A.nsub = g.nsub;
  A.S = g.S;
  A.items = (int)g.items;
  A.V = g.V;
  A.nvec = g.nvec;
  A.c = c;
  A.epoch = reinterpret_cast<const uint32_t*>(ws + L.epoch);
  A.fail = reinterpret_cast<uint64_t*>(ws + L.epoch + 8);
  A.stat = reinterpret_cast<uint64_t*>(ws + L.stat);
  A.norm = reinterpret_cast<uint64_t*>(ws + L.norm);
  A.part = need_sum ? reinterpret_cast<float*>(ws + L.part) : nullptr;
  A.argmax_t = argmax_t;
  A.argmax_d = argmax_d;
  A.agree = agree;
#ifdef HS_TRACE
  A.trace = g_trace;
#endif
  int rc = dispatch<Launch>(g, need_sum, need_arg, A, g, stream);
  if (rc) return rc;
  if (hipGetLastError() != hipSuccess) return HS_ERR_HIP;

  FoldArgs F{A.part, alpha, g.B, g.N, g.K, g.S, reinterpret_cast<uint32_t*>(ws + L.epoch)};
  const int64_t outs = need_sum ? (int64_t)g.B * g.N * g.K : 0;
  const unsigned blocks = outs ? (unsigned)((outs + kWaves - 1) / kWaves) : 1u;
  hs_fold_kernel<<<blocks, kThreads, 0, stream>>>(F);
  if (hipGetLastError() != hipSuccess) return HS_ERR_HIP;
  if (tail) return launch_tail(*tail, stream);
  return HS_OK;
}

}  // namespace hs
