// hs_softmax_stats: max, lowest-index argmax and natural-log normaliser of `rows` temperature
// softmaxes. One workgroup per row.
#include "hs_rowstats.h"

namespace hs {

// Each thread walks its vectors of the row (stride kThreads, U per chunk) keeping a running max,
// lowest argmax and an exp2 sum against its own integer-valued offset o = exp_offset_of(m, c)
// (at or above m c, so no exponent is positive): a larger max rescales the sum by
// 2^(o_old - o_new) exactly, and the next chunk's loads are in flight while the current one is
// reduced. One block reduction per row at the end.
template <int DT>
__global__ __launch_bounds__(kThreads) void hs_softmax_stats_kernel(const char* x, int64_t ld,
                                                                    int64_t V, int64_t nvec,
                                                                    float c, float* rmax,
                                                                    float* rlse,
                                                                    int32_t* ramax) {
  using Vt = Vec<DT>;
  using Raw = typename Vt::Raw;
  constexpr int E = Vt::kElems, U = Vt::kU;
  constexpr int64_t kStep = (int64_t)U * kThreads;  // vectors per chunk of the workgroup
  const int t = threadIdx.x;
  const int64_t row = blockIdx.x;
  const char* rowp = x + row * ld * Vt::kBytes;
  // branch-free 16-byte loads at an index clamped into the row's complete vectors, nontemporal
  // for 16-bit logits (every logit is read once: 6% faster than plain loads on both bf16 workloads
  // measured); the one partial vector at the row end, and vectors past it, are then replaced
  // in the lanes that hold them
  const int64_t vfull = V / E;  // complete 16-byte vectors of the row
  auto fetch = [&](int64_t v0, Raw (&r)[U]) __attribute__((always_inline)) {
    typedef unsigned int u4 __attribute__((ext_vector_type(4)));
    typedef const __attribute__((address_space(1))) u4* gp4;
    if (vfull > 0) {
#pragma unroll
      for (int j = 0; j < U; ++j) {
        const int64_t vi = v0 + (int64_t)j * kThreads + t;
        const gp4 a = (gp4)(rowp + (vi < vfull ? vi : vfull - 1) * 16);
        const u4 v = DT != HS_F32 ? __builtin_nontemporal_load(a) : *a;
        __builtin_memcpy(&r[j], &v, 16);
      }
    }
#pragma unroll
    for (int j = 0; j < U; ++j) {
      const int64_t vi = v0 + (int64_t)j * kThreads + t;
      if (vi >= vfull) r[j] = vi < nvec ? Vt::load_raw(rowp, vi, V) : Vt::neg_raw();
    }
  };
  float m = -INFINITY, o = -INFINITY, s = 0.0f;
  int idx = INT_MAX;
  Raw cur[U], nxt[U];
  fetch(0, cur);
  for (int64_t v0 = 0; v0 < nvec; v0 += kStep) {
    if (v0 + kStep < nvec) fetch(v0 + kStep, nxt);
    float z[U][E];
#pragma unroll
    for (int j = 0; j < U; ++j) Vt::unpack(cur[j], z[j]);
    // the chunk's max first (NaN ignored); only a chunk that raises the running max is searched
    // for the index, in increasing index order, so the first element equal to the chunk max is
    // the lowest index attaining it, and the strict compare keeps an earlier chunk's on a tie
    float cm = z[0][0];
#pragma unroll
    for (int j = 0; j < U; ++j)
#pragma unroll
      for (int e = (j == 0 ? 1 : 0); e < E; ++e) cm = fmaxf(cm, z[j][e]);
    if (cm > m) {
      bool found = false;
#pragma unroll
      for (int j = 0; j < U; ++j)
#pragma unroll
        for (int e = 0; e < E; ++e)
          if (!found && z[j][e] == cm) {
            found = true;
            m = z[j][e];
            idx = (int)((v0 + (int64_t)j * kThreads + t) * E + e);
          }
    }
    // o = -inf until the running max scaled by c is finite; until then the sum is taken
    // against offset 0, where every logit seen so far gives exp2(-inf) = 0 (a -inf logit, or a
    // finite one whose product with c is below the fp32 range) or NaN (a NaN logit), so the
    // sum is 0 or NaN and is carried into the first finite offset as s * 0
    const float on = exp_offset_of(m, c);
    if (on != o) {
      s = (o == -INFINITY) ? s * 0.0f : ldexpf(s, (int)fmaxf(o - on, -256.0f));
      o = on;
    }
    const float off = o != -INFINITY ? o : 0.0f;
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < U; ++j)
#pragma unroll
      for (int e = 0; e < E; ++e) acc[e & 3] += __builtin_amdgcn_exp2f(fmaf(z[j][e], c, -off));
    s += (acc[0] + acc[1]) + (acc[2] + acc[3]);
#pragma unroll
    for (int j = 0; j < U; ++j) cur[j] = nxt[j];
  }
  // a thread whose logits are all -inf still owns its lowest valid index
  if (idx == INT_MAX && t < nvec) idx = t * E;
  const SliceStat r = block_reduce_stat<true, true>(m, idx, o, s);
  if (t == 0) {
    if (rmax) rmax[row] = r.m;
    if (ramax) ramax[row] = r.idx;
    if (rlse) rlse[row] = (r.o == -INFINITY) ? NAN : (r.o + log2f(r.s)) * 0.69314718055994530942f;
  }
}

int launch_softmax_stats(const void* x, int dtype, int64_t rows, int64_t V, int64_t ld, float c,
                         float* row_max, float* row_lse, int32_t* row_argmax,
                         hipStream_t stream) {
  const int E = dtype == HS_F32 ? Vec<HS_F32>::kElems : Vec<HS_BF16>::kElems;
  const int64_t nvec = (V + E - 1) / E;
  const char* xp = reinterpret_cast<const char*>(x);
  if (dtype == HS_F32)
    hs_softmax_stats_kernel<HS_F32><<<(unsigned)rows, kThreads, 0, stream>>>(
        xp, ld, V, nvec, c, row_max, row_lse, row_argmax);
  else if (dtype == HS_F16)
    hs_softmax_stats_kernel<HS_F16><<<(unsigned)rows, kThreads, 0, stream>>>(
        xp, ld, V, nvec, c, row_max, row_lse, row_argmax);
  else
    hs_softmax_stats_kernel<HS_BF16><<<(unsigned)rows, kThreads, 0, stream>>>(
        xp, ld, V, nvec, c, row_max, row_lse, row_argmax);
  return hipGetLastError() == hipSuccess ? HS_OK : HS_ERR_HIP;
}

}  // namespace hs
