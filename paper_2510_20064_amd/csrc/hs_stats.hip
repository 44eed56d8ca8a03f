// hs_softmax_stats: max, lowest-index argmax and natural-log normaliser of `rows` temperature
// softmaxes. One workgroup per row, looping over the row's slices.
#include "hs_rowstats.h"

namespace hs {

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
    const SliceStat st = row_slice_stats<DT, true, true>(rowp, v0, v1, V, c);
    argmax_combine(m, idx, st.m, st.idx);
    lse2_combine(o, s, st.o, st.s);
  }
  if (threadIdx.x == 0) {
    if (rmax) rmax[row] = m;
    if (ramax) ramax[row] = idx;
    if (rlse) rlse[row] = (o == -INFINITY) ? NAN : (o + log2f(s)) * 0.69314718055994530942f;
  }
}

int launch_softmax_stats(const void* x, int dtype, int64_t rows, int64_t V, int64_t ld, float c,
                         float* row_max, float* row_lse, int32_t* row_argmax,
                         hipStream_t stream) {
  const int E = dtype == HS_F32 ? Vec<HS_F32>::kElems : Vec<HS_BF16>::kElems;
  const int64_t nvec = (V + E - 1) / E;
  const int64_t per = kSliceElems / E;
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
