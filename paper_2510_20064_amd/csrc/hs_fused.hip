// One verification round in one launch: softmax statistics, alpha for every drafter
// (Theorem 1), greedy agreement, and optionally the per-query learner step.
//
// Work decomposition. A (query, position) group holds N + 1 logits rows: row 0 is the
// target, rows 1..N the drafters. Rows are cut into S slices (<= 8192 logits each). The
// target row forms row set 0; the drafters form row sets 1..nch of CH drafters each.
//   stats item (rs, s)  : max / argmax / exp2 sum of slice s of every row in row set rs.
//                         The row set's last stats item combines its S slices into the
//                         row's log2 normaliser and argmax ("row stats").
//   minsum item (rs, s) : sum_v exp2(min(e_t, e_i)) over slice s for the drafters of row set
//                         rs >= 1, e = z c - log2(normaliser), c = log2(e) / T. It waits for
//                         the row stats of row 0 and of row set rs.
//   group final         : the group's last item sums the S slice partials of each drafter in
//                         order (alpha, clamped to [0, 1]) and writes argmax / agreement.
//   query final         : the last group of a query runs the learner step (fused round only).
// Items of group g sit on queue g % 8 in the order stats(0), stats(1), then
// [stats(c), minsum(c-1)] for c >= 2, then minsum(nch): a minsum item re-reads slices that
// the same queue streamed shortly before, and the workgroups of one XCD (blockIdx % 8 on a
// round-robin dispatch) serve the same queue, so the re-read hits that XCD's L2. Each HBM
// byte is read once.
//
// Progress. Every wait is on items fetched earlier from the same queue, and a stats item
// never waits, so the kernel completes with any number of resident workgroups. Data that
// crosses workgroups is published as 64-bit relaxed atomic words whose low half is a
// non-zero validity tag; consumers poll them (bounded spin: on expiry the result is NaN /
// argmax -2 instead of a hang) and reset them to zero after the last read, and the last
// workgroup to exit resets the queue counters, so a completed launch leaves the workspace
// zero-filled for the next one.
#include "hs_learner.h"
#include "hs_rowstats.h"

namespace hs {

constexpr int kQueues = 8;
constexpr uint32_t kSpinLimit = 1u << 21;
constexpr int kFoldChunk = 32;  // slices folded per pass in the combine steps

struct FusedArgs {
  RowTable rows;
  Geom g;
  float c;
  int CH, nch, lag, Lg;
  int tail;
  float* alpha;
  uint8_t* agree;
  int32_t* argmax_t;
  int32_t* argmax_d;
  uint64_t* sstat;  // [G][R][S][2]: (m, argmax + 1), (sum, 1)
  uint64_t* rstat;  // [G][R][3]   : (Xhi, 1), (Xlo, 1), (argmax + 1)
  uint64_t* parts;  // [G][N][S]   : (partial sum, 1)
  uint32_t* ctr;    // [kQueues] fetch, [1] exit, pad to 16, [G][1 + nch] row-set stats,
                    // [G][nch] row-set minsum, [G] group, [B] query
  TailArgs ta;
#ifdef HS_TRACE
  uint64_t* trace;  // per workgroup: [64 records][4 words]
#endif
};

__device__ inline void put_word(uint64_t* w, uint64_t v) {
  __hip_atomic_store(w, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline uint64_t wait_word(uint64_t* w) {
  uint64_t v = __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  uint32_t n = 0;
  while ((uint32_t)v == 0u) {
    __builtin_amdgcn_s_sleep(2);
    v = __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (++n > kSpinLimit) return ((uint64_t)0x7FC00000u << 32) | 0xFFFFFFFFu;
  }
  return v;
}
__device__ inline uint64_t tag_f(float x) { return ((uint64_t)__float_as_uint(x) << 32) | 1u; }
__device__ inline float word_f(uint64_t w) { return __uint_as_float((uint32_t)(w >> 32)); }
__device__ inline uint32_t ctr_add(uint32_t* p) {
  return __hip_atomic_fetch_add(p, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline void ctr_zero(uint32_t* p) {
  __hip_atomic_store(p, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Increments a completion counter once for the workgroup; true in every thread if this was
// the last of `total` increments.
__device__ inline bool block_count_last(uint32_t* ctr, uint32_t total) {
  __shared__ int s_last;
  __syncthreads();
  if (threadIdx.x == 0) s_last = (ctr_add(ctr) == total - 1);
  __syncthreads();
  return s_last != 0;
}

struct Counters {
  uint32_t* fetch;
  uint32_t* exitc;
  uint32_t* rowset;  // [G][1 + nch]: stats items done per row set
  uint32_t* minsum;  // [G][nch]: minsum items done per drafter row set
  uint32_t* group;   // [G]: row sets completed (stats and minsum)
  uint32_t* query;   // [B]: groups completed
};
__device__ inline Counters counters(const FusedArgs& A) {
  Counters C;
  C.fetch = A.ctr;
  C.exitc = A.ctr + kQueues;
  C.rowset = A.ctr + 16;
  C.minsum = C.rowset + (size_t)A.g.G * (1 + A.nch);
  C.group = C.minsum + (size_t)A.g.G * A.nch;
  C.query = C.group + A.g.G;
  return C;
}
// Completions a group needs: one per row-set combine, plus one per finished minsum row set.
__device__ inline uint32_t group_total(const FusedArgs& A, bool need_sum) {
  return (uint32_t)(1 + A.nch + (need_sum ? A.nch : 0));
}

__device__ inline void rowset_rows(const FusedArgs& A, int rs, int& r0, int& r1) {
  if (rs == 0) {
    r0 = 0;
    r1 = 1;
  } else {
    r0 = 1 + (rs - 1) * A.CH;
    r1 = 1 + min(rs * A.CH, A.g.N);
  }
}

// ---- row stats of a row set: fold the S slice statistics of each row in slice order -------

template <bool NEED_SUM, bool NEED_ARG>
__device__ __forceinline__ void combine_rowset(const FusedArgs& A, int grp, int rs) {
  __shared__ float sh_m[8][kFoldChunk];
  __shared__ float sh_s[8][kFoldChunk];
  __shared__ int sh_i[8][kFoldChunk];
  const Geom& g = A.g;
  int r0, r1;
  rowset_rows(A, rs, r0, r1);
  const int nr = r1 - r0;
  const int t = threadIdx.x;
  float m = -INFINITY, o = -INFINITY, ssum = 0.0f;
  int idx = INT_MAX;
  for (int s0 = 0; s0 < g.S; s0 += kFoldChunk) {
    const int ns = min(kFoldChunk, g.S - s0);
    for (int p = t; p < nr * ns; p += kThreads) {
      const int rr = p / ns, ss = p % ns;
      uint64_t* w = A.sstat + (((int64_t)grp * g.R + r0 + rr) * g.S + s0 + ss) * 2;
      const uint64_t w0 = wait_word(w);
      sh_m[rr][ss] = word_f(w0);
      sh_i[rr][ss] = (int)(uint32_t)w0 - 1;
      put_word(w, 0);
      if (NEED_SUM) {
        sh_s[rr][ss] = word_f(wait_word(w + 1));
        put_word(w + 1, 0);
      }
    }
    __syncthreads();
    if (t < nr) {
      for (int ss = 0; ss < ns; ++ss) {
        const float ms = sh_m[t][ss];
        if (NEED_ARG) argmax_combine(m, idx, ms, sh_i[t][ss]);
        else m = fmaxf(m, ms);
        // the offset is the rounded product the slice sums were taken against (the library
        // is built without multiply-add contraction, which would use the exact product)
        if (NEED_SUM) lse2_combine(o, ssum, ms * A.c, sh_s[t][ss]);
      }
    }
    __syncthreads();
  }
  if (t < nr) {
    uint64_t* w = A.rstat + ((int64_t)grp * g.R + r0 + t) * 3;
    if (NEED_SUM) {
      // log2 normaliser O + log2(sum) as an unevaluated sum hi + lo (TwoSum)
      const float ls = log2f(ssum);
      const float hi = o + ls;
      const float bb = hi - o;
      const float lo = (o - (hi - bb)) + (ls - bb);
      put_word(w + 0, tag_f(hi));
      put_word(w + 1, tag_f(lo));
    }
    if (NEED_ARG) put_word(w + 2, (uint64_t)(uint32_t)(idx + 1));
  }
}

// ---- group final: alpha, argmax, agreement; resets the group's words and counters --------

template <bool NEED_SUM, bool NEED_ARG>
__device__ __forceinline__ void group_final(const FusedArgs& A, const Counters& C, int grp) {
  __shared__ float sh_p[8][kFoldChunk];
  __shared__ int sh_idx[kMaxRows];
  const Geom& g = A.g;
  const int t = threadIdx.x;
  const int b = grp / g.K, k = grp % g.K;
  if (NEED_SUM) {
    for (int i0 = 0; i0 < g.N; i0 += 8) {
      const int ni = min(8, g.N - i0);
      float acc = 0.0f;
      for (int s0 = 0; s0 < g.S; s0 += kFoldChunk) {
        const int ns = min(kFoldChunk, g.S - s0);
        for (int p = t; p < ni * ns; p += kThreads) {
          const int ii = p / ns, ss = p % ns;
          uint64_t* w = A.parts + ((int64_t)grp * g.N + i0 + ii) * g.S + s0 + ss;
          sh_p[ii][ss] = word_f(wait_word(w));
          put_word(w, 0);
        }
        __syncthreads();
        if (t < ni)
          for (int ss = 0; ss < ns; ++ss) acc += sh_p[t][ss];
        __syncthreads();
      }
      if (t < ni) A.alpha[((int64_t)b * g.N + i0 + t) * g.K + k] = fminf(fmaxf(acc, 0.0f), 1.0f);
    }
  }
  if (t < g.R) {
    uint64_t* w = A.rstat + ((int64_t)grp * g.R + t) * 3;
    if (NEED_ARG) sh_idx[t] = (int)(uint32_t)wait_word(w + 2) - 1;
    put_word(w + 0, 0);
    put_word(w + 1, 0);
    put_word(w + 2, 0);
  }
  if (t <= A.nch) ctr_zero(C.rowset + (size_t)grp * (1 + A.nch) + t);
  if (t < A.nch) ctr_zero(C.minsum + (size_t)grp * A.nch + t);
  if (t == 0) ctr_zero(C.group + grp);
  __syncthreads();
  if (NEED_ARG && t < g.R) {
    const int idx = sh_idx[t];
    if (t == 0) {
      if (A.argmax_t) A.argmax_t[(int64_t)b * g.K + k] = idx;
    } else {
      const int64_t o = ((int64_t)b * g.N + (t - 1)) * g.K + k;
      if (A.argmax_d) A.argmax_d[o] = idx;
      if (A.agree) A.agree[o] = (uint8_t)(idx == sh_idx[0]);
    }
  }
}

// ---- query final: the learner step once all K groups of the query are done ---------------

__device__ __forceinline__ void query_final(const FusedArgs& A, const Counters& C, int b, double* lds) {
  // outputs of the K group finals (other workgroups) must be visible before the learner
  // reads them: release them here, acquire after the count
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  if (!block_count_last(C.query + b, (uint32_t)A.g.K)) return;
  if (threadIdx.x == 0) ctr_zero(C.query + b);
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  if (threadIdx.x < 64) tail_query(A.ta, b, lds);
}

// ---- stats item ----------------------------------------------------------------------------

template <int DT, bool NEED_SUM, bool NEED_ARG>
__device__ __forceinline__ void stats_item(const FusedArgs& A, const Counters& C, int grp, int rs, int s,
                           double* lds) {
  const Geom& g = A.g;
  const int b = grp / g.K, k = grp % g.K;
  const int64_t v0 = (int64_t)s * g.vps;
  const int64_t v1 = min(v0 + g.vps, g.nvec);
  int r0, r1;
  rowset_rows(A, rs, r0, r1);
  for (int r = r0; r < r1; ++r) {
    const char* rowp = reinterpret_cast<const char*>(A.rows.ptr[r]) +
                       ((int64_t)b * A.rows.sb[r] + (int64_t)k * A.rows.sk[r]) * Vec<DT>::kBytes;
    const SliceStat st = row_slice_stats<DT, NEED_SUM, NEED_ARG>(rowp, v0, v1, g.V, A.c);
    if (threadIdx.x == 0) {
      uint64_t* w = A.sstat + (((int64_t)grp * g.R + r) * g.S + s) * 2;
      put_word(w, ((uint64_t)__float_as_uint(st.m) << 32) |
                      (uint32_t)(NEED_ARG ? st.idx + 1 : 1));
      if (NEED_SUM) put_word(w + 1, tag_f(st.s));
    }
  }
  if (!block_count_last(C.rowset + (size_t)grp * (1 + A.nch) + rs, (uint32_t)g.S)) return;
  combine_rowset<NEED_SUM, NEED_ARG>(A, grp, rs);
  if (!block_count_last(C.group + grp, group_total(A, NEED_SUM))) return;
  group_final<NEED_SUM, NEED_ARG>(A, C, grp);
  if (A.tail) query_final(A, C, b, lds);
}

// ---- minsum item ---------------------------------------------------------------------------

template <int DT, bool NEED_ARG>
__device__ __forceinline__ void minsum_item(const FusedArgs& A, const Counters& C, int grp, int rs, int s,
                            double* lds) {
  using Vt = Vec<DT>;
  constexpr int E = Vt::kElems, U = Vt::kU;
  __shared__ float sh_x[2 * (kMinsumChunk + 1)];
  __shared__ float sh_acc[kWaves][kMinsumChunk];
  const Geom& g = A.g;
  const int t = threadIdx.x;
  const int b = grp / g.K, k = grp % g.K;
  int r0, r1;
  rowset_rows(A, rs, r0, r1);
  const int n = r1 - r0;
  // normalisers of the target and of this row set's drafters
  if (t < 2 * (n + 1)) {
    const int row = (t < 2) ? 0 : r0 + (t / 2 - 1);
    sh_x[t] = word_f(wait_word(A.rstat + ((int64_t)grp * g.R + row) * 3 + (t & 1)));
  }
  __syncthreads();
  const int64_t v0 = (int64_t)s * g.vps;
  const int64_t v1 = min(v0 + g.vps, g.nvec);
  float et[U][E];
  {
    const float xh = sh_x[0], xl = sh_x[1];
    const char* rowp = reinterpret_cast<const char*>(A.rows.ptr[0]) +
                       ((int64_t)b * A.rows.sb[0] + (int64_t)k * A.rows.sk[0]) * Vt::kBytes;
#pragma unroll
    for (int j = 0; j < U; ++j) {
      const int64_t vi = v0 + (int64_t)j * kThreads + t;
      if (vi < v1) {
        Vt::load(rowp, vi, g.V, et[j]);
#pragma unroll
        for (int e = 0; e < E; ++e) et[j][e] = fmaf(et[j][e], A.c, -xh) - xl;
      } else {
#pragma unroll
        for (int e = 0; e < E; ++e) et[j][e] = -INFINITY;
      }
    }
  }
  // drafters one at a time; the next drafter's slice is in flight while this one is summed
  using Raw = typename Vt::Raw;
  const int lane = t & 63, wv = t >> 6;
  Raw cur[U], nxt[U];
  auto load_raw = [&](int jj, Raw* dst) {
    const int r = r0 + jj;
    const char* rowp = reinterpret_cast<const char*>(A.rows.ptr[r]) +
                       ((int64_t)b * A.rows.sb[r] + (int64_t)k * A.rows.sk[r]) * Vt::kBytes;
#pragma unroll
    for (int j = 0; j < U; ++j) {
      const int64_t vi = v0 + (int64_t)j * kThreads + t;
      dst[j] = vi < v1 ? Vt::load_raw(rowp, vi, g.V) : Vt::zero_raw();
    }
  };
  load_raw(0, cur);
#pragma unroll 1
  for (int jj = 0; jj < n; ++jj) {
    if (jj + 1 < n) load_raw(jj + 1, nxt);
    const float xh = sh_x[2 * (jj + 1)], xl = sh_x[2 * (jj + 1) + 1];
    float a4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < U; ++j) {
      float zd[E];
      Vt::unpack(cur[j], zd);
#pragma unroll
      for (int e = 0; e < E; ++e)
        a4[e & 3] += __builtin_amdgcn_exp2f(fminf(et[j][e], fmaf(zd[e], A.c, -xh) - xl));
    }
    const float v = wave_sum((a4[0] + a4[1]) + (a4[2] + a4[3]));
    if (lane == 0) sh_acc[wv][jj] = v;
#pragma unroll
    for (int j = 0; j < U; ++j) cur[j] = nxt[j];
  }
  __syncthreads();
  if (t < n) {
    float v = sh_acc[0][t];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) v += sh_acc[w][t];
    put_word(A.parts + ((int64_t)grp * g.N + (r0 - 1) + t) * g.S + s, tag_f(v));
  }
  if (!block_count_last(C.minsum + (size_t)grp * A.nch + (rs - 1), (uint32_t)g.S)) return;
  if (!block_count_last(C.group + grp, group_total(A, true))) return;
  group_final<true, NEED_ARG>(A, C, grp);
  if (A.tail) query_final(A, C, b, lds);
}

// ---- the persistent kernel -------------------------------------------------------------------

template <int DT, bool NEED_SUM, bool NEED_ARG>
__global__ __launch_bounds__(kThreads) void hs_round_kernel(FusedArgs A) {
  extern __shared__ double lds[];
  __shared__ int s_item, s_q;
  const Counters C = counters(A);
  const int S = A.g.S;
  const int q0 = blockIdx.x & (kQueues - 1);
  // Thread 0 claims items from queue q0 first, then from the following queues once q0 is
  // exhausted. The claim of the next item is issued before the current item is processed,
  // so the atomic's round trip overlaps the work; claims stay in queue order, so every
  // wait still points at an item claimed earlier and the dependency graph stays acyclic.
  int qi = 0;
  uint32_t pend = 0;
  auto qlen = [&](int q) -> uint32_t {
    const int ng = A.g.G > q ? (A.g.G - q + kQueues - 1) / kQueues : 0;
    return (uint32_t)ng * (uint32_t)A.Lg;
  };
  if (threadIdx.x == 0) pend = ctr_add(C.fetch + q0);
#ifdef HS_TRACE
  int nrec = 0;
#endif
  for (;;) {
#ifdef HS_TRACE
    const uint64_t t_fetch = __builtin_amdgcn_s_memrealtime();
#endif
    if (threadIdx.x == 0) {
      int item = -1, qq = 0;
      for (;;) {
        const int q = (q0 + qi) & (kQueues - 1);
        if (pend < qlen(q)) {
          item = (int)pend;
          qq = q;
          break;
        }
        if (++qi >= kQueues) break;
        pend = ctr_add(C.fetch + ((q0 + qi) & (kQueues - 1)));
      }
      if (item >= 0) pend = ctr_add(C.fetch + qq);
      s_item = item;
      s_q = qq;
    }
    __syncthreads();
    const int item = s_item, q = s_q;
    __syncthreads();
    if (item < 0) break;
    const int grp = q + kQueues * (item / A.Lg);
    int pos = item % A.Lg;
    int type = 0, rs = 0, s = 0;
    if (pos < S) {
      type = 1;
      s = pos;
    } else {
      pos -= S;
      for (int c = 1; c <= A.nch && type == 0; ++c) {
        if (pos < S) {
          type = 1;
          rs = c;
          s = pos;
        } else {
          pos -= S;
          if (NEED_SUM && c - A.lag >= 1) {
            if (pos < S) {
              type = 2;
              rs = c - A.lag;
              s = pos;
            } else {
              pos -= S;
            }
          }
        }
      }
      if (type == 0) {  // minsum items of the last `lag` row sets
        type = 2;
        rs = A.nch - A.lag + 1 + pos / S;
        s = pos % S;
      }
    }
#ifdef HS_TRACE
    const uint64_t t_start = __builtin_amdgcn_s_memrealtime();
#endif
    if (type == 1)
      stats_item<DT, NEED_SUM, NEED_ARG>(A, C, grp, rs, s, lds);
    else if (NEED_SUM)
      minsum_item<DT, NEED_ARG>(A, C, grp, rs, s, lds);
#ifdef HS_TRACE
    if (threadIdx.x == 0 && nrec < 64) {
      uint64_t* r = A.trace + ((size_t)blockIdx.x * 64 + nrec) * 4;
      r[0] = ((uint64_t)type << 56) | ((uint64_t)grp << 32) | ((uint64_t)rs << 16) | (uint64_t)s;
      r[1] = t_fetch;
      r[2] = t_start;
      r[3] = __builtin_amdgcn_s_memrealtime();
      ++nrec;
    }
#endif
  }
  // the last workgroup out resets the fetch counters for the next launch
  if (threadIdx.x == 0 && ctr_add(C.exitc) == gridDim.x - 1) {
    for (int q = 0; q < kQueues; ++q) ctr_zero(C.fetch + q);
    ctr_zero(C.exitc);
  }
}

// ---- launcher --------------------------------------------------------------------------------

size_t fused_counter_words(const Geom& g) { return 16 + (size_t)g.G * (2 + g.N) + g.B; }

template <int DT, bool NEED_SUM, bool NEED_ARG>
static int launch_fused_t(FusedArgs& A, size_t lds_bytes, hipStream_t stream) {
  auto kern = hs_round_kernel<DT, NEED_SUM, NEED_ARG>;
  static int cus = 0;
  static int occ[2] = {0, 0};
  if (cus == 0) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return HS_ERR_HIP;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      return HS_ERR_HIP;
  }
  int per_cu = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, kThreads, lds_bytes) !=
      hipSuccess)
    return HS_ERR_HIP;
  (void)occ;
  if (per_cu < 1) per_cu = 1;
  const int64_t items = (int64_t)A.g.G * A.Lg;
  int64_t grid = (int64_t)cus * per_cu;
  if (grid > items) grid = items;
  kern<<<(unsigned)grid, kThreads, lds_bytes, stream>>>(A);
  return hipGetLastError() == hipSuccess ? HS_OK : HS_ERR_HIP;
}

#ifdef HS_TRACE
uint64_t* g_trace = nullptr;  // trace buffer of the next launch (debug builds only)
#endif

int launch_round(const Geom& g, const RowTable& rows, float c, bool need_sum, bool need_arg,
                 float* alpha, uint8_t* agree, int32_t* argmax_t, int32_t* argmax_d, char* ws,
                 const TailArgs* tail, hipStream_t stream) {
  const WsLayout L = ws_layout(g);
  FusedArgs A;
  A.rows = rows;
  A.g = g;
  A.c = c;
  // drafters per row set: the largest of 8, 4, 2, 1 that still leaves >= 2048 minsum items
  int CH = 8;
  while (CH > 1 && (int64_t)g.G * g.S * ((g.N + CH - 1) / CH) < 2048) CH >>= 1;
  A.CH = CH;
  A.nch = (g.N + CH - 1) / CH;
  A.lag = 1;
  A.Lg = g.S * (1 + A.nch) + (need_sum ? g.S * A.nch : 0);
  A.tail = tail != nullptr;
  A.alpha = alpha;
  A.agree = agree;
  A.argmax_t = argmax_t;
  A.argmax_d = argmax_d;
  A.sstat = reinterpret_cast<uint64_t*>(ws + L.slice_stats);
  A.rstat = reinterpret_cast<uint64_t*>(ws + L.row_stats);
  A.parts = reinterpret_cast<uint64_t*>(ws + L.parts);
  A.ctr = reinterpret_cast<uint32_t*>(ws + L.counters);
#ifdef HS_TRACE
  A.trace = g_trace;
#endif
  size_t lds = 0;
  if (tail) {
    A.ta = *tail;
    lds = sizeof(double) * (size_t)tail_lds_doubles(*tail);
  } else {
    A.ta = TailArgs{};
  }
  if (g.dtype == HS_F32) {
    if (need_sum && need_arg) return launch_fused_t<HS_F32, true, true>(A, lds, stream);
    if (need_sum) return launch_fused_t<HS_F32, true, false>(A, lds, stream);
    return launch_fused_t<HS_F32, false, true>(A, lds, stream);
  }
  if (need_sum && need_arg) return launch_fused_t<HS_BF16, true, true>(A, lds, stream);
  if (need_sum) return launch_fused_t<HS_BF16, true, false>(A, lds, stream);
  return launch_fused_t<HS_BF16, false, true>(A, lds, stream);
}

}  // namespace hs
