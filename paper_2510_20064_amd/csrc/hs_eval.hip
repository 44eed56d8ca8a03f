// Drafter evaluation kernels (Theorem 1 for every drafter, Section 3.2).
//
// alpha[b][i][k] = sum_v min(p_v, q_v) with p = softmax(z_t / T), q = softmax(z_i / T).
// Both normalisers are needed before any min can be taken, so the work splits in two
// sweeps over a (query, position) group of N + 1 rows:
//   stats  : per row slice, max / argmax / sum of exp2(z c - o)   (c = log2(e) / T)
//   combine: per row, the slice statistics -> log2 normaliser and argmax; greedy outputs
//   minsum : per slice, sum_v exp2(min(e_t, e_i)) with e = z c - log2(normaliser)
//   final  : per (group, drafter), ordered sum of the slice partials -> alpha in [0, 1]
// Every exponent is formed by one fused multiply-add and exp2 runs on the hardware
// transcendental unit; one exp per drafter logit per sweep, no rescaling exps.
#include <climits>

#include "hs_internal.h"

namespace hs {

// ---- block reductions --------------------------------------------------------------------

template <bool NEED_SUM, bool NEED_ARG>
__device__ inline SliceStat block_reduce_stat(float m, int idx, float o, float s) {
  __shared__ SliceStat sh[kWaves];
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    float m2 = __shfl_xor(m, off, 64);
    if (NEED_ARG) {
      int i2 = __shfl_xor(idx, off, 64);
      argmax_combine(m, idx, m2, i2);
    } else {
      m = fmaxf(m, m2);
    }
    if (NEED_SUM) {
      float o2 = __shfl_xor(o, off, 64);
      float s2 = __shfl_xor(s, off, 64);
      lse2_combine(o, s, o2, s2);
    }
  }
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  if (lane == 0) sh[wv] = SliceStat{m, idx, o, s};
  __syncthreads();
  SliceStat r = sh[0];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) {
    SliceStat x = sh[w];
    if (NEED_ARG) argmax_combine(r.m, r.idx, x.m, x.idx);
    else r.m = fmaxf(r.m, x.m);
    if (NEED_SUM) lse2_combine(r.o, r.s, x.o, x.s);
  }
  __syncthreads();
  return r;
}

// Statistics of one row slice: vectors [v0, v1) of a row whose first logit is at rowp.
template <int DT, bool NEED_SUM, bool NEED_ARG>
__device__ inline SliceStat row_slice_stats(const char* rowp, int64_t v0, int64_t v1, int64_t V,
                                            float c) {
  using Vt = Vec<DT>;
  constexpr int E = Vt::kElems, U = Vt::kU;
  const int t = threadIdx.x;
  float z[U][E];
#pragma unroll
  for (int j = 0; j < U; ++j) {
    int64_t vi = v0 + (int64_t)j * kThreads + t;
    if (vi < v1) {
      Vt::load(rowp, vi, V, z[j]);
    } else {
#pragma unroll
      for (int e = 0; e < E; ++e) z[j][e] = -INFINITY;
    }
  }
  float m = -INFINITY;
  int idx = INT_MAX;
#pragma unroll
  for (int j = 0; j < U; ++j) {
#pragma unroll
    for (int e = 0; e < E; ++e) {
      float x = z[j][e];
      if (NEED_ARG) {
        if (x > m) {
          m = x;
          idx = (int)((v0 + (int64_t)j * kThreads + t) * E + e);
        }
      } else {
        m = fmaxf(m, x);
      }
    }
  }
  // a thread whose logits are all -inf still owns its lowest valid index
  if (NEED_ARG && idx == INT_MAX && v0 + t < v1) idx = (int)((v0 + t) * E);
  float o = -INFINITY, s = 0.0f;
  if (NEED_SUM && m != -INFINITY) {
    o = m * c;
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < U; ++j)
#pragma unroll
      for (int e = 0; e < E; ++e) acc[e & 3] += __builtin_amdgcn_exp2f(fmaf(z[j][e], c, -o));
    s = (acc[0] + acc[1]) + (acc[2] + acc[3]);
  }
  return block_reduce_stat<NEED_SUM, NEED_ARG>(m, idx, o, s);
}

__device__ inline const char* row_ptr(const RowTable& rows, int r, int b, int k, int es) {
  return reinterpret_cast<const char*>(rows.ptr[r]) +
         ((int64_t)b * rows.sb[r] + (int64_t)k * rows.sk[r]) * es;
}

// ---- stats sweep: one workgroup per (group, row, slice) ----------------------------------

template <int DT, bool NEED_SUM, bool NEED_ARG>
__global__ __launch_bounds__(kThreads) void hs_eval_stats_kernel(RowTable rows, Geom g, float c,
                                                                 SliceStat* out) {
  const int64_t item = blockIdx.x;
  const int s = (int)(item % g.S);
  const int64_t t = item / g.S;
  const int r = (int)(t % g.R);
  const int grp = (int)(t / g.R);
  const int b = grp / g.K, k = grp % g.K;
  const char* rowp = row_ptr(rows, r, b, k, Vec<DT>::kBytes);
  const int64_t v0 = (int64_t)s * g.vps;
  const int64_t v1 = v0 + g.vps < g.nvec ? v0 + g.vps : g.nvec;
  SliceStat st = row_slice_stats<DT, NEED_SUM, NEED_ARG>(rowp, v0, v1, g.V, c);
  if (threadIdx.x == 0) out[item] = st;
}

// ---- combine: one workgroup per group, one thread per row ---------------------------------

__global__ __launch_bounds__(128) void hs_eval_combine_kernel(Geom g, const SliceStat* ss,
                                                              RowStat* rs, int32_t* argmax_t,
                                                              int32_t* argmax_d, uint8_t* agree) {
  const int grp = blockIdx.x;
  const int r = threadIdx.x;
  __shared__ int idx0;
  RowStat out{0.f, 0.f, 0, -INFINITY};
  if (r < g.R) {
    const SliceStat* p = ss + ((int64_t)grp * g.R + r) * g.S;
    float m = -INFINITY, o = -INFINITY, s = 0.0f;
    int idx = INT_MAX;
    for (int j = 0; j < g.S; ++j) {
      SliceStat x = p[j];
      argmax_combine(m, idx, x.m, x.idx);
      lse2_combine(o, s, x.o, x.s);
    }
    // log2 normaliser O + log2(s) as an unevaluated double-float sum (TwoSum)
    float ls = log2f(s);
    float hi = o + ls;
    float bb = hi - o;
    float lo = (o - (hi - bb)) + (ls - bb);
    out = RowStat{hi, lo, idx, m};
    rs[(int64_t)grp * g.R + r] = out;
    if (r == 0) idx0 = idx;
  }
  __syncthreads();
  if (r < g.R) {
    const int b = grp / g.K, k = grp % g.K;
    if (r == 0) {
      if (argmax_t) argmax_t[(int64_t)b * g.K + k] = out.idx;
    } else {
      const int64_t o = ((int64_t)b * g.N + (r - 1)) * g.K + k;
      if (argmax_d) argmax_d[o] = out.idx;
      if (agree) agree[o] = (uint8_t)(out.idx == idx0);
    }
  }
}

// ---- min-sum sweep: one workgroup per (group, drafter chunk, slice) -----------------------

template <int DT>
__global__ __launch_bounds__(kThreads) void hs_eval_minsum_kernel(RowTable rows, Geom g, float c,
                                                                  const RowStat* rs, float* parts) {
  using Vt = Vec<DT>;
  constexpr int E = Vt::kElems, U = Vt::kU;
  const int nch = (g.N + kMinsumChunk - 1) / kMinsumChunk;
  const int64_t item = blockIdx.x;
  const int s = (int)(item % g.S);
  const int64_t tt = item / g.S;
  const int ch = (int)(tt % nch);
  const int grp = (int)(tt / nch);
  const int b = grp / g.K, k = grp % g.K;
  const int i0 = ch * kMinsumChunk;
  const int n = (g.N - i0) < kMinsumChunk ? (g.N - i0) : kMinsumChunk;
  const int64_t v0 = (int64_t)s * g.vps;
  const int64_t v1 = v0 + g.vps < g.nvec ? v0 + g.vps : g.nvec;
  const int t = threadIdx.x;
  const RowStat* rsg = rs + (int64_t)grp * g.R;

  // target log2-probabilities of this slice, -inf outside it
  float et[U][E];
  {
    const RowStat r0 = rsg[0];
    const char* rowp = row_ptr(rows, 0, b, k, Vt::kBytes);
#pragma unroll
    for (int j = 0; j < U; ++j) {
      int64_t vi = v0 + (int64_t)j * kThreads + t;
      if (vi < v1) {
        Vt::load(rowp, vi, g.V, et[j]);
#pragma unroll
        for (int e = 0; e < E; ++e) et[j][e] = fmaf(et[j][e], c, -r0.Xhi) - r0.Xlo;
      } else {
#pragma unroll
        for (int e = 0; e < E; ++e) et[j][e] = -INFINITY;
      }
    }
  }
  float acc[kMinsumChunk];
#pragma unroll
  for (int ii = 0; ii < kMinsumChunk; ++ii) {
    acc[ii] = 0.0f;
    if (ii < n) {
      const RowStat ri = rsg[1 + i0 + ii];
      const char* rowp = row_ptr(rows, 1 + i0 + ii, b, k, Vt::kBytes);
      float zd[U][E];
#pragma unroll
      for (int j = 0; j < U; ++j) {
        int64_t vi = v0 + (int64_t)j * kThreads + t;
        if (vi < v1) {
          Vt::load(rowp, vi, g.V, zd[j]);
        } else {
#pragma unroll
          for (int e = 0; e < E; ++e) zd[j][e] = 0.0f;
        }
      }
      float a4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < U; ++j)
#pragma unroll
        for (int e = 0; e < E; ++e) {
          float ei = fmaf(zd[j][e], c, -ri.Xhi) - ri.Xlo;
          a4[e & 3] += __builtin_amdgcn_exp2f(fminf(et[j][e], ei));
        }
      acc[ii] = (a4[0] + a4[1]) + (a4[2] + a4[3]);
    }
  }
  __shared__ float sh[kWaves][kMinsumChunk];
  const int lane = t & 63, wv = t >> 6;
#pragma unroll
  for (int ii = 0; ii < kMinsumChunk; ++ii) {
    float v = wave_sum(acc[ii]);
    if (lane == 0) sh[wv][ii] = v;
  }
  __syncthreads();
  if (t < n) {
    float v = sh[0][t];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) v += sh[w][t];
    parts[((int64_t)grp * g.N + i0 + t) * g.S + s] = v;
  }
}

// ---- final: ordered sum of the slice partials ----------------------------------------------

__global__ __launch_bounds__(64) void hs_eval_final_kernel(Geom g, const float* parts,
                                                           float* alpha) {
  const int grp = blockIdx.x;
  const int i = threadIdx.x;
  if (i >= g.N) return;
  const float* p = parts + ((int64_t)grp * g.N + i) * g.S;
  float a = 0.0f;
  for (int j = 0; j < g.S; ++j) a += p[j];
  a = fminf(fmaxf(a, 0.0f), 1.0f);
  const int b = grp / g.K, k = grp % g.K;
  alpha[((int64_t)b * g.N + i) * g.K + k] = a;
}

// ---- hs_softmax_stats: one workgroup per row, looping over its slices ----------------------

template <int DT>
__global__ __launch_bounds__(kThreads) void hs_softmax_stats_kernel(const char* x, int64_t ld,
                                                                    int64_t V, int64_t nvec,
                                                                    int64_t vps, int S, float c,
                                                                    float* rmax, float* rlse,
                                                                    int32_t* ramax) {
  const int64_t row = blockIdx.x;
  const char* rowp = x + row * ld * Vec<DT>::kBytes;
  float m = -INFINITY, o = -INFINITY, s = 0.0f;
  int idx = INT_MAX;
  for (int j = 0; j < S; ++j) {
    const int64_t v0 = (int64_t)j * vps;
    const int64_t v1 = v0 + vps < nvec ? v0 + vps : nvec;
    SliceStat st = row_slice_stats<DT, true, true>(rowp, v0, v1, V, c);
    argmax_combine(m, idx, st.m, st.idx);
    lse2_combine(o, s, st.o, st.s);
  }
  if (threadIdx.x == 0) {
    if (rmax) rmax[row] = m;
    if (ramax) ramax[row] = idx;
    if (rlse) rlse[row] = (o == -INFINITY) ? NAN : (o + log2f(s)) * 0.69314718055994530942f;
  }
}

// ---- launchers ----------------------------------------------------------------------------

template <int DT>
static int launch_eval_dt(const Geom& g, const RowTable& rows, float c, bool need_sum,
                          bool need_argmax, float* alpha, uint8_t* agree, int32_t* argmax_t,
                          int32_t* argmax_d, char* ws, hipStream_t stream) {
  const WsLayout L = ws_layout(g);
  SliceStat* ss = reinterpret_cast<SliceStat*>(ws + L.slice_stats);
  RowStat* rs = reinterpret_cast<RowStat*>(ws + L.row_stats);
  float* parts = reinterpret_cast<float*>(ws + L.parts);
  const unsigned n1 = (unsigned)((int64_t)g.G * g.R * g.S);
  if (need_sum && need_argmax)
    hs_eval_stats_kernel<DT, true, true><<<n1, kThreads, 0, stream>>>(rows, g, c, ss);
  else if (need_sum)
    hs_eval_stats_kernel<DT, true, false><<<n1, kThreads, 0, stream>>>(rows, g, c, ss);
  else
    hs_eval_stats_kernel<DT, false, true><<<n1, kThreads, 0, stream>>>(rows, g, c, ss);
  hs_eval_combine_kernel<<<g.G, 128, 0, stream>>>(g, ss, rs, argmax_t, argmax_d, agree);
  if (need_sum) {
    const int nch = (g.N + kMinsumChunk - 1) / kMinsumChunk;
    const unsigned n2 = (unsigned)((int64_t)g.G * nch * g.S);
    hs_eval_minsum_kernel<DT><<<n2, kThreads, 0, stream>>>(rows, g, c, rs, parts);
    hs_eval_final_kernel<<<g.G, 64, 0, stream>>>(g, parts, alpha);
  }
  return hipGetLastError() == hipSuccess ? HS_OK : HS_ERR_HIP;
}

int launch_eval(const Geom& g, const RowTable& rows, float c, bool need_sum, bool need_argmax,
                float* alpha, uint8_t* agree, int32_t* argmax_t, int32_t* argmax_d, char* ws,
                hipStream_t stream) {
  if (g.dtype == HS_F32)
    return launch_eval_dt<HS_F32>(g, rows, c, need_sum, need_argmax, alpha, agree, argmax_t,
                                  argmax_d, ws, stream);
  return launch_eval_dt<HS_BF16>(g, rows, c, need_sum, need_argmax, alpha, agree, argmax_t,
                                 argmax_d, ws, stream);
}

int launch_softmax_stats(const void* x, int dtype, int64_t rows, int64_t V, int64_t ld, float c,
                         float* row_max, float* row_lse, int32_t* row_argmax,
                         hipStream_t stream) {
  const int E = dtype == HS_F32 ? Vec<HS_F32>::kElems : Vec<HS_BF16>::kElems;
  const int64_t nvec = (V + E - 1) / E;
  const int64_t per = (int64_t)kThreads * (dtype == HS_F32 ? Vec<HS_F32>::kU : Vec<HS_BF16>::kU);
  const int S = (int)((nvec + per - 1) / per);
  const int64_t vps = (nvec + S - 1) / S;
  const char* xp = reinterpret_cast<const char*>(x);
  if (dtype == HS_F32)
    hs_softmax_stats_kernel<HS_F32><<<(unsigned)rows, kThreads, 0, stream>>>(
        xp, ld, V, nvec, vps, S, c, row_max, row_lse, row_argmax);
  else
    hs_softmax_stats_kernel<HS_BF16><<<(unsigned)rows, kThreads, 0, stream>>>(
        xp, ld, V, nvec, vps, S, c, row_max, row_lse, row_argmax);
  return hipGetLastError() == hipSuccess ? HS_OK : HS_ERR_HIP;
}

}  // namespace hs
