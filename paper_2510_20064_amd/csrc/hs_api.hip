// C ABI of libhedgespec: host-side validation, launch geometry, workspace sizing.
// Every argument is checked before the first HIP call; on an error nothing is enqueued.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>

#include "hs_internal.h"

#define HS_API extern "C" __attribute__((visibility("default")))

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}

int ok() {
  g_err[0] = 0;
  return HS_OK;
}

int elem_bytes(int dtype) { return dtype == HS_F32 ? 4 : 2; }

int check_shape(int B, int N, int K, int64_t V) {
  if (B < 1 || N < 1 || K < 1 || V < 1)
    return fail(HS_ERR_SHAPE, "B, N, K and V must be >= 1 (got B=%d N=%d K=%d V=%lld)", B, N, K,
                (long long)V);
  if (B > HS_MAX_QUERIES || N > HS_MAX_DRAFTERS || K > HS_MAX_POSITIONS || V > INT32_MAX)
    return fail(HS_ERR_LIMIT, "limits: B <= %d, N <= %d, K <= %d, V <= 2^31-1 (got B=%d N=%d K=%d)",
                HS_MAX_QUERIES, HS_MAX_DRAFTERS, HS_MAX_POSITIONS, B, N, K);
  return HS_OK;
}

int check_view(const hs_view* v, int dtype, const char* what) {
  if (!v || !v->ptr) return fail(HS_ERR_NULL, "%s: NULL view or pointer", what);
  if (v->stride_b < 0 || v->stride_k < 0) return fail(HS_ERR_SHAPE, "%s: negative stride", what);
  const int64_t es = elem_bytes(dtype);
  if (((uintptr_t)v->ptr & 15) != 0 || ((v->stride_b * es) & 15) != 0 ||
      ((v->stride_k * es) & 15) != 0)
    return fail(HS_ERR_ALIGN, "%s: rows must start on 16-byte boundaries", what);
  return HS_OK;
}

int check_parent(const int32_t* parent, int M) {
  if (!parent) return HS_OK;
  if (parent[0] != -1) return fail(HS_ERR_TREE, "parent[0] must be -1 (the root)");
  for (int n = 1; n < M; ++n)
    if (parent[n] < 0 || parent[n] >= n)
      return fail(HS_ERR_TREE, "parent[%d] = %d: a parent must precede its child", n, parent[n]);
  return HS_OK;
}

struct EvalReq {
  const hs_view* target;
  const hs_view* drafters;
  int N, B, K;
  int64_t V;
  int dtype;
  float T;
  int mode;
  float* alpha;
  uint8_t* agree;
  int32_t* argmax_t;
  int32_t* argmax_d;
  void* ws;
  size_t ws_bytes;
};

int validate_eval(const EvalReq& q, hs::TeamGeom* g, hs::RowTable* rows) {
  int rc = check_shape(q.B, q.N, q.K, q.V);
  if (rc) return rc;
  if (q.dtype != HS_F32 && q.dtype != HS_BF16 && q.dtype != HS_F16)
    return fail(HS_ERR_DTYPE, "unknown dtype %d", q.dtype);
  if (q.mode != HS_SAMPLE && q.mode != HS_GREEDY) return fail(HS_ERR_ARG, "unknown mode %d", q.mode);
  if (!q.drafters) return fail(HS_ERR_NULL, "drafters_host is NULL");
  if ((rc = check_view(q.target, q.dtype, "target"))) return rc;
  for (int i = 0; i < q.N; ++i) {
    char what[32];
    snprintf(what, sizeof(what), "drafter %d", i);
    if ((rc = check_view(&q.drafters[i], q.dtype, what))) return rc;
  }
  if (q.mode == HS_SAMPLE && !q.alpha) return fail(HS_ERR_NULL, "sample mode needs alpha");
  if (q.mode == HS_GREEDY && !q.agree) return fail(HS_ERR_NULL, "greedy mode needs agree");
  if (q.alpha && !(isfinite(q.T) && q.T > 0.0f))
    return fail(HS_ERR_TEMPERATURE, "temperature must be finite and > 0 (got %g)", (double)q.T);
  if (!hs::team_geom(q.B, q.N, q.K, q.V, q.dtype, g))
    return fail(HS_ERR_LIMIT, "V = %lld is beyond the evaluation limit of %lld logits per row",
                (long long)q.V, (long long)hs::kMaxTeamSlices * hs::kThreads * (16 / elem_bytes(q.dtype)));
  const size_t need = hs::team_ws(*g).total;
  if (!q.ws) return fail(HS_ERR_WORKSPACE, "workspace is NULL (need %zu bytes)", need);
  if (q.ws_bytes < need)
    return fail(HS_ERR_WORKSPACE, "workspace too small: %zu < %zu bytes", q.ws_bytes, need);
  if (((uintptr_t)q.ws & 255) != 0) return fail(HS_ERR_ALIGN, "workspace must be 256-byte aligned");
  rows->ptr[0] = q.target->ptr;
  rows->sb[0] = q.target->stride_b;
  rows->sk[0] = q.target->stride_k;
  for (int i = 0; i < q.N; ++i) {
    rows->ptr[1 + i] = q.drafters[i].ptr;
    rows->sb[1 + i] = q.drafters[i].stride_b;
    rows->sk[1 + i] = q.drafters[i].stride_k;
  }
  for (int r = q.N + 1; r < hs::kMaxRows; ++r) {
    rows->ptr[r] = nullptr;
    rows->sb[r] = rows->sk[r] = 0;
  }
  return HS_OK;
}

// The one check that asks the device, made after every host-side check: a team of S
// workgroups must fit on the device at once.
int check_capacity(const EvalReq& q, const hs::TeamGeom& g) {
  const int cap = hs::team_capacity(g, q.alpha != nullptr, q.agree || q.argmax_t || q.argmax_d);
  if (cap < g.S)
    return fail(HS_ERR_LIMIT, "the device holds %d evaluation workgroups at once, %d are needed",
                cap, g.S);
  return HS_OK;
}

int run_eval(const EvalReq& q, const hs::TeamGeom& g, const hs::RowTable& rows,
             const hs::TailArgs* tail, hipStream_t s) {
  const bool need_sum = q.alpha != nullptr;
  const bool need_arg = q.agree || q.argmax_t || q.argmax_d;
  const float c = need_sum ? (float)(1.4426950408889634 / (double)q.T) : 1.0f;
  int rc = hs::launch_round(g, rows, c, need_sum, need_arg, q.alpha, q.agree, q.argmax_t,
                            q.argmax_d, reinterpret_cast<char*>(q.ws), tail, s);
  if (rc) return fail(rc, "kernel launch failed: %s", hipGetErrorString(hipGetLastError()));
  return HS_OK;
}

struct TailReq {
  const float* alpha;
  const uint8_t* agree;
  int mode, B, N, K;
  const int32_t* parent;
  const int32_t* path_end;
  double* eal;
  double* prefix;
  int loss_kind;
  double* loss;
};

int validate_tail(const TailReq& q, hs::TailArgs* a) {
  int rc = check_shape(q.B, q.N, q.K, 1);
  if (rc) return rc;
  if (q.mode != HS_SAMPLE && q.mode != HS_GREEDY) return fail(HS_ERR_ARG, "unknown mode %d", q.mode);
  if (q.mode == HS_SAMPLE && !q.alpha) return fail(HS_ERR_NULL, "sample mode needs alpha");
  if (q.mode == HS_GREEDY && !q.agree) return fail(HS_ERR_NULL, "greedy mode needs agree");
  if (!q.eal) return fail(HS_ERR_NULL, "eal is NULL");
  if (q.loss_kind < HS_LOSS_LENGTH || q.loss_kind > HS_LOSS_ACCEPT_CHUNK)
    return fail(HS_ERR_ARG, "unknown loss kind %d", q.loss_kind);
  if ((rc = check_parent(q.parent, q.K))) return rc;
  if (q.parent && q.loss_kind == HS_LOSS_ACCEPT_TOKEN)
    return fail(HS_ERR_TREE, "token-level acceptance loss is defined for chains only");
  memset(a, 0, sizeof(*a));
  a->alpha = q.alpha;
  a->agree = q.agree;
  a->gamma_src = q.mode == HS_SAMPLE ? 1 : 2;
  a->B = q.B;
  a->N = q.N;
  a->M = q.K;
  a->tree = q.parent != nullptr;
  for (int n = 0; n < HS_MAX_POSITIONS; ++n) a->parent[n] = (q.parent && n < q.K) ? q.parent[n] : n - 1;
  a->path_end = q.path_end;
  a->eal = q.eal;
  a->prefix = q.prefix;
  a->loss_kind = q.loss_kind;
  a->loss_out = q.loss;
  a->L = q.loss_kind == HS_LOSS_ACCEPT_TOKEN ? q.K : 1;
  return HS_OK;
}

}  // namespace

HS_API const char* hs_status_string(int status) {
  switch (status) {
    case HS_OK: return "HS_OK";
    case HS_ERR_NULL: return "HS_ERR_NULL";
    case HS_ERR_SHAPE: return "HS_ERR_SHAPE";
    case HS_ERR_DTYPE: return "HS_ERR_DTYPE";
    case HS_ERR_ALIGN: return "HS_ERR_ALIGN";
    case HS_ERR_TEMPERATURE: return "HS_ERR_TEMPERATURE";
    case HS_ERR_TREE: return "HS_ERR_TREE";
    case HS_ERR_WORKSPACE: return "HS_ERR_WORKSPACE";
    case HS_ERR_LIMIT: return "HS_ERR_LIMIT";
    case HS_ERR_HIP: return "HS_ERR_HIP";
    case HS_ERR_ARG: return "HS_ERR_ARG";
    default: return "HS_ERR_UNKNOWN";
  }
}

HS_API const char* hs_last_error(void) { return g_err; }

HS_API int hs_version(void) { return 100; }

HS_API void hs_set_wait_limit(int polls) { hs::set_wait_polls(polls); }

namespace hs {
// Streaming-read probe (hs_probe.hip): `vectors` 16-byte vectors of x read once by `grid`
// workgroups of 256 threads with `unroll` (1, 2, 4 or 8) loads in flight per thread; one word
// per wave to out (grid * 4 words).
int launch_stream_read(const void* x, uint64_t vectors, int grid, int unroll, bool nontemporal,
                       uint32_t* out, hipStream_t s);
}  // namespace hs

HS_API int hs_stream_read(const void* x, size_t bytes, int grid, int unroll, int nontemporal,
                          uint32_t* out, void* stream) {
  if (!x || !out) return fail(HS_ERR_NULL, "hs_stream_read: NULL buffer");
  if (((uintptr_t)x & 15) != 0 || (bytes & 15) != 0)
    return fail(HS_ERR_ALIGN, "hs_stream_read: buffer and size must be multiples of 16 bytes");
  if (bytes == 0 || grid < 1 || grid > 65536)
    return fail(HS_ERR_SHAPE, "hs_stream_read: need bytes > 0 and 1 <= grid <= 65536");
  if (unroll != 1 && unroll != 2 && unroll != 4 && unroll != 8)
    return fail(HS_ERR_ARG, "hs_stream_read: unroll must be 1, 2, 4 or 8 (got %d)", unroll);
  const int rc = hs::launch_stream_read(x, bytes / 16, grid, unroll, nontemporal != 0, out,
                                        (hipStream_t)stream);
  return rc == HS_OK ? HS_OK : fail(rc, "hs_stream_read: launch failed");
}

HS_API int hs_softmax_stats(const void* logits, int dtype, int64_t rows, int64_t V, int64_t ld,
                            float temperature, float* row_max, float* row_lse,
                            int32_t* row_argmax, void* stream) {
  if (!logits) return fail(HS_ERR_NULL, "logits is NULL");
  if (dtype != HS_F32 && dtype != HS_BF16 && dtype != HS_F16)
    return fail(HS_ERR_DTYPE, "unknown dtype %d", dtype);
  if (rows < 1 || V < 1 || ld < V) return fail(HS_ERR_SHAPE, "need rows >= 1, 1 <= V <= ld");
  if (rows > INT32_MAX || V > INT32_MAX) return fail(HS_ERR_LIMIT, "rows and V must be < 2^31");
  if (!(isfinite(temperature) && temperature > 0.0f))
    return fail(HS_ERR_TEMPERATURE, "temperature must be finite and > 0");
  const int64_t es = elem_bytes(dtype);
  if (((uintptr_t)logits & 15) != 0 || ((ld * es) & 15) != 0)
    return fail(HS_ERR_ALIGN, "rows must start on 16-byte boundaries");
  if (!row_max && !row_lse && !row_argmax) return ok();
  const float c = (float)(1.4426950408889634 / (double)temperature);
  int rc = hs::launch_softmax_stats(logits, dtype, rows, V, ld, c, row_max, row_lse, row_argmax,
                                    (hipStream_t)stream);
  if (rc) return fail(rc, "kernel launch failed: %s", hipGetErrorString(hipGetLastError()));
  return ok();
}

HS_API size_t hs_eval_alpha_workspace_size(int B, int N, int K, int64_t V, int dtype) {
  hs::TeamGeom g;
  if (!hs::team_geom(B, N, K, V, dtype, &g)) return 0;
  return hs::team_ws(g).total;
}

HS_API int hs_eval_alpha(const hs_view* target, const hs_view* drafters_host, int N, int B, int K,
                         int64_t V, int dtype, float temperature, int mode, float* alpha,
                         uint8_t* agree, int32_t* argmax_t, int32_t* argmax_d, void* workspace,
                         size_t workspace_bytes, void* stream) {
  EvalReq q{target, drafters_host, N, B, K, V, dtype, temperature, mode, alpha, agree, argmax_t,
            argmax_d, workspace, workspace_bytes};
  hs::TeamGeom g;
  hs::RowTable rows;
  int rc = validate_eval(q, &g, &rows);
  if (rc) return rc;
  if ((rc = check_capacity(q, g))) return rc;
  rc = run_eval(q, g, rows, nullptr, (hipStream_t)stream);
  return rc ? rc : ok();
}

namespace {

// ---- the evaluation workspace of hs_eval_alpha_noalloc ----------------------------------------
// A file-scope device array, zero-initialised when the code object is loaded; every device the
// library runs on holds its own copy for the life of the process. In host code its name is only
// a stand-in: the device address of each device's copy comes from hipGetSymbolAddress, looked
// up once per device (with that device current) and kept here.
constexpr size_t kStaticWsBytes = (size_t)64 << 20;
__device__ __align__(256) unsigned char scratch[kStaticWsBytes];

std::mutex g_scratch_mu;
void* g_scratch_ptr[64];  // per device ordinal; nullptr until looked up

// This device's copy of `scratch` (nullptr with an error message if it cannot be found).
void* static_workspace() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) {
    fail(HS_ERR_HIP, "hs_eval_alpha_noalloc: no current HIP device");
    return nullptr;
  }
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t rc = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (rc != hipSuccess || !p) {
      fail(HS_ERR_HIP, "hs_eval_alpha_noalloc: hipGetSymbolAddress failed on device %d: %s", dev,
           hipGetErrorString(rc));
      return nullptr;
    }
    g_scratch_ptr[dev] = p;
  }
  return g_scratch_ptr[dev];
}

}  // namespace

HS_API size_t hs_eval_alpha_noalloc_max_workspace(void) { return kStaticWsBytes; }

HS_API int hs_eval_alpha_noalloc(const hs_view* target, const hs_view* drafters_host, int N,
                                 int B, int K, int64_t V, int dtype, float temperature, int mode,
                                 float* alpha, uint8_t* agree, int32_t* argmax_t,
                                 int32_t* argmax_d, void* stream) {
  // the shape's workspace must fit in the fixed array: checked before any HIP call
  hs::TeamGeom g;
  if (!hs::team_geom(B, N, K, V, dtype, &g)) {
    EvalReq probe{target, drafters_host, N, B, K, V, dtype, temperature, mode, alpha, agree,
                  argmax_t, argmax_d, reinterpret_cast<void*>(256), kStaticWsBytes};
    hs::RowTable rows;
    return validate_eval(probe, &g, &rows);  // the shape's own error code and message
  }
  const size_t need = hs::team_ws(g).total;
  if (need > kStaticWsBytes)
    return fail(HS_ERR_WORKSPACE,
                "hs_eval_alpha_noalloc: this shape needs %zu bytes of workspace, more than the "
                "fixed %zu (use hs_eval_alpha with a workspace of its own)",
                need, kStaticWsBytes);
  EvalReq q{target, drafters_host, N, B, K, V, dtype, temperature, mode, alpha, agree, argmax_t,
            argmax_d, reinterpret_cast<void*>(256), kStaticWsBytes};
  hs::RowTable rows;
  int rc = validate_eval(q, &g, &rows);  // every host-side check, before the first HIP call
  if (rc) return rc;
  q.ws = static_workspace();
  if (!q.ws) return HS_ERR_HIP;
  if ((rc = check_capacity(q, g))) return rc;
  rc = run_eval(q, g, rows, nullptr, (hipStream_t)stream);
  return rc ? rc : ok();
}

namespace {

struct TopReq {
  const hs_view* target;
  const hs_view* drafters;
  int N, B, K;
  int64_t V;
  int dtype, L;
  float T;
  int mode;
  float* gamma;
  uint8_t* hit;
  int32_t* children;
  void* ws;
  size_t ws_bytes;
};

int validate_topl(const TopReq& q, hs::TeamGeom* g, hs::RowTable* rows) {
  int rc = check_shape(q.B, q.N, q.K, q.V);
  if (rc) return rc;
  if (q.dtype != HS_F32 && q.dtype != HS_BF16 && q.dtype != HS_F16)
    return fail(HS_ERR_DTYPE, "unknown dtype %d", q.dtype);
  if (q.mode != HS_SAMPLE && q.mode != HS_GREEDY) return fail(HS_ERR_ARG, "unknown mode %d", q.mode);
  if (q.L < 1 || q.L > HS_MAX_TOPL || q.L > q.V)
    return fail(HS_ERR_SHAPE, "need 1 <= L <= min(V, %d) (got L=%d, V=%lld)", HS_MAX_TOPL, q.L,
                (long long)q.V);
  if (!q.drafters) return fail(HS_ERR_NULL, "drafters_host is NULL");
  if ((rc = check_view(q.target, q.dtype, "target"))) return rc;
  for (int i = 0; i < q.N; ++i) {
    char what[32];
    snprintf(what, sizeof(what), "drafter %d", i);
    if ((rc = check_view(&q.drafters[i], q.dtype, what))) return rc;
  }
  if (q.mode == HS_SAMPLE && !q.gamma) return fail(HS_ERR_NULL, "sample mode needs gamma");
  if (q.mode == HS_GREEDY && !q.hit) return fail(HS_ERR_NULL, "greedy mode needs hit");
  if (q.gamma && !(isfinite(q.T) && q.T > 0.0f))
    return fail(HS_ERR_TEMPERATURE, "temperature must be finite and > 0 (got %g)", (double)q.T);
  if (!hs::team_geom(q.B, q.N, q.K, q.V, q.dtype, g))
    return fail(HS_ERR_LIMIT, "V = %lld is beyond the evaluation limit of %lld logits per row",
                (long long)q.V, (long long)hs::kMaxTeamSlices * hs::kThreads * (16 / elem_bytes(q.dtype)));
  if (!hs::topl_fits(*g))
    return fail(HS_ERR_LIMIT, "B * K * (N + 1) * ceil(V / slice) must stay below 2^31");
  const size_t need = hs::topl_ws_bytes(*g, q.L);
  if (!q.ws) return fail(HS_ERR_WORKSPACE, "workspace is NULL (need %zu bytes)", need);
  if (q.ws_bytes < need)
    return fail(HS_ERR_WORKSPACE, "workspace too small: %zu < %zu bytes", q.ws_bytes, need);
  if (((uintptr_t)q.ws & 255) != 0) return fail(HS_ERR_ALIGN, "workspace must be 256-byte aligned");
  rows->ptr[0] = q.target->ptr;
  rows->sb[0] = q.target->stride_b;
  rows->sk[0] = q.target->stride_k;
  for (int i = 0; i < q.N; ++i) {
    rows->ptr[1 + i] = q.drafters[i].ptr;
    rows->sb[1 + i] = q.drafters[i].stride_b;
    rows->sk[1 + i] = q.drafters[i].stride_k;
  }
  for (int r = q.N + 1; r < hs::kMaxRows; ++r) {
    rows->ptr[r] = nullptr;
    rows->sb[r] = rows->sk[r] = 0;
  }
  return HS_OK;
}

}  // namespace

HS_API size_t hs_eval_topl_workspace_size(int B, int N, int K, int64_t V, int L, int dtype) {
  hs::TeamGeom g;
  if (L < 1 || L > HS_MAX_TOPL || L > V || !hs::team_geom(B, N, K, V, dtype, &g)) return 0;
  return hs::topl_ws_bytes(g, L);
}

HS_API int hs_eval_topl(const hs_view* target, const hs_view* drafters_host, int N, int B, int K,
                        int64_t V, int dtype, int L, float temperature, int mode, float* gamma,
                        uint8_t* hit, int32_t* children, void* workspace, size_t workspace_bytes,
                        void* stream) {
  TopReq q{target, drafters_host, N, B, K, V, dtype, L, temperature, mode, gamma, hit, children,
           workspace, workspace_bytes};
  hs::TeamGeom g;
  hs::RowTable rows;
  int rc = validate_topl(q, &g, &rows);
  if (rc) return rc;
  const float c = gamma ? (float)(1.4426950408889634 / (double)temperature) : 0.0f;
  rc = hs::launch_topl(g, rows, L, c, gamma != nullptr, gamma, hit, children,
                       reinterpret_cast<char*>(workspace), (hipStream_t)stream);
  if (rc) return fail(rc, "kernel launch failed: %s", hipGetErrorString(hipGetLastError()));
  return ok();
}

namespace hs {
// defined next to its kernel in hs_cmass.hip
int launch_candidate_mass(const void* tptr, int64_t sb, int64_t sk, int dtype, int B, int N,
                          int K, int64_t V, int C, float c, const float* lse,
                          const int32_t* cand, float* gamma, hipStream_t stream);
}  // namespace hs

HS_API int hs_candidate_mass(const hs_view* target, int N, int B, int K, int64_t V, int dtype,
                             float temperature, const float* target_lse, const int32_t* cand,
                             int C, float* gamma, void* stream) {
  int rc = check_shape(B, N, K, V);
  if (rc) return rc;
  if (dtype != HS_F32 && dtype != HS_BF16 && dtype != HS_F16)
    return fail(HS_ERR_DTYPE, "unknown dtype %d", dtype);
  if ((rc = check_view(target, dtype, "target"))) return rc;
  if (!target_lse || !cand || !gamma)
    return fail(HS_ERR_NULL, "target_lse, cand and gamma are required");
  if (C < 1 || C > HS_MAX_CANDIDATES)
    return fail(HS_ERR_LIMIT, "C must be in [1, %d] (got %d)", HS_MAX_CANDIDATES, C);
  if (!(isfinite(temperature) && temperature > 0.0f))
    return fail(HS_ERR_TEMPERATURE, "temperature must be finite and > 0 (got %g)",
                (double)temperature);
  const float c = (float)(1.4426950408889634 / (double)temperature);
  rc = hs::launch_candidate_mass(target->ptr, target->stride_b, target->stride_k, dtype, B, N, K,
                                 V, C, c, target_lse, cand, gamma, (hipStream_t)stream);
  if (rc) return fail(rc, "kernel launch failed: %s", hipGetErrorString(hipGetLastError()));
  return ok();
}

HS_API int hs_play(const double* weights, int B, int N, int how, const double* u,
                   int32_t* choice, void* stream) {
  int rc = check_shape(B, N, 1, 1);
  if (rc) return rc;
  if (how != HS_PLAY_ARGMAX && how != HS_PLAY_SAMPLE) return fail(HS_ERR_ARG, "unknown play rule %d", how);
  if (!weights || !choice) return fail(HS_ERR_NULL, "weights and choice are required");
  if (how == HS_PLAY_SAMPLE && !u) return fail(HS_ERR_NULL, "sampling needs the uniform draws u");
  rc = hs::launch_play(weights, B, N, how, u, choice, (hipStream_t)stream);
  if (rc) return fail(rc, "kernel launch failed: %s", hipGetErrorString(hipGetLastError()));
  return ok();
}

HS_API int hs_regret_update(const double* loss, int L, int B, int N, const int32_t* played,
                            double* cum_loss, double* played_loss, double* regret,
                            const double* eal, double* eal_sum, void* stream) {
  int rc = check_shape(B, N, 1, 1);
  if (rc) return rc;
  if (L < 1) return fail(HS_ERR_SHAPE, "L must be >= 1");
  if (!loss || !played || !cum_loss || !played_loss || !regret)
    return fail(HS_ERR_NULL, "loss, played, cum_loss, played_loss and regret are required");
  if ((eal == nullptr) != (eal_sum == nullptr))
    return fail(HS_ERR_NULL, "eal and eal_sum must be given together");
  rc = hs::launch_regret(loss, L, B, N, played, cum_loss, played_loss, regret, eal, eal_sum,
                         (hipStream_t)stream);
  if (rc) return fail(rc, "kernel launch failed: %s", hipGetErrorString(hipGetLastError()));
  return ok();
}

HS_API int hs_accept_len(const float* alpha, const uint8_t* agree, int mode, int B, int N, int K,
                         const int32_t* parent_host, const int32_t* path_end, double* eal,
                         double* prefix, int loss_kind, double* loss, void* stream) {
  TailReq q{alpha, agree, mode, B, N, K, parent_host, path_end, eal, prefix, loss_kind, loss};
  hs::TailArgs a{};
  int rc = validate_tail(q, &a);
  if (rc) return rc;
  rc = hs::launch_tail(a, (hipStream_t)stream);
  if (rc) return fail(rc, "kernel launch failed: %s", hipGetErrorString(hipGetLastError()));
  return ok();
}

static int learner_common(const double* loss, int L, int B, int N) {
  if (!loss) return fail(HS_ERR_NULL, "loss is NULL");
  if (L < 1 || B < 1 || N < 1) return fail(HS_ERR_SHAPE, "L, B and N must be >= 1");
  if (B > HS_MAX_QUERIES || N > HS_MAX_DRAFTERS)
    return fail(HS_ERR_LIMIT, "limits: B <= %d, N <= %d", HS_MAX_QUERIES, HS_MAX_DRAFTERS);
  return HS_OK;
}

HS_API int hs_hedge_update(double* logw, double* w, const double* loss, int L, int B, int N,
                           double eta, void* stream) {
  if (!logw || !w) return fail(HS_ERR_NULL, "logw and w are required");
  int rc = learner_common(loss, L, B, N);
  if (rc) return rc;
  if (!isfinite(eta)) return fail(HS_ERR_ARG, "eta must be finite");
  hs::TailArgs a{};
  memset(&a, 0, sizeof(a));
  a.gamma_src = 0;
  a.B = B;
  a.N = N;
  a.M = 1;
  a.loss_in = loss;
  a.L = L;
  a.logw = logw;
  a.w = w;
  a.eta = eta;
  rc = hs::launch_tail(a, (hipStream_t)stream);
  if (rc) return fail(rc, "kernel launch failed: %s", hipGetErrorString(hipGetLastError()));
  return ok();
}

HS_API int hs_normalhedge_update(double* R, double* p, double* c, const double* loss, int L,
                                 int B, int N, void* stream) {
  if (!R || !p || !c) return fail(HS_ERR_NULL, "R, p and c are required");
  int rc = learner_common(loss, L, B, N);
  if (rc) return rc;
  hs::TailArgs a{};
  memset(&a, 0, sizeof(a));
  a.gamma_src = 0;
  a.B = B;
  a.N = N;
  a.M = 1;
  a.loss_in = loss;
  a.L = L;
  a.R = R;
  a.p = p;
  a.c = c;
  rc = hs::launch_tail(a, (hipStream_t)stream);
  if (rc) return fail(rc, "kernel launch failed: %s", hipGetErrorString(hipGetLastError()));
  return ok();
}

HS_API int hs_delayed_update(const float* alpha, const uint8_t* agree, int mode, int B, int N,
                             int K, const int32_t* count, int64_t hybrid_tokens, float* hist,
                             int64_t* clock,
                             double* logw, double* w, double eta, double* R, double* p,
                             double* c, double* loss, int32_t* nloss, void* stream) {
  int rc = check_shape(B, N, K, 1);
  if (rc) return rc;
  if (mode != HS_SAMPLE && mode != HS_GREEDY) return fail(HS_ERR_ARG, "unknown mode %d", mode);
  if (mode == HS_SAMPLE && !alpha) return fail(HS_ERR_NULL, "sample mode needs alpha");
  if (mode == HS_GREEDY && !agree) return fail(HS_ERR_NULL, "greedy mode needs agree");
  if (!count || !hist || !clock) return fail(HS_ERR_NULL, "count, hist and clock are required");
  if ((logw == nullptr) != (w == nullptr))
    return fail(HS_ERR_NULL, "logw and w must be given together");
  if (!((R == nullptr) == (p == nullptr) && (R == nullptr) == (c == nullptr)))
    return fail(HS_ERR_NULL, "R, p and c must be given together");
  if (logw && !isfinite(eta)) return fail(HS_ERR_ARG, "eta must be finite");
  if (hybrid_tokens < 0) return fail(HS_ERR_ARG, "hybrid_tokens must be >= 0");
  hs::DelayArgs a{};
  a.alpha = alpha;
  a.agree = agree;
  a.gamma_src = mode == HS_SAMPLE ? 1 : 2;
  a.B = B;
  a.N = N;
  a.K = K;
  a.count = count;
  a.hybrid = hybrid_tokens;
  a.hist = hist;
  a.clock = clock;
  a.logw = logw;
  a.w = w;
  a.eta = eta;
  a.R = R;
  a.p = p;
  a.c = c;
  a.loss = loss;
  a.nloss = nloss;
  rc = hs::launch_delayed(a, (hipStream_t)stream);
  if (rc) return fail(rc, "kernel launch failed: %s", hipGetErrorString(hipGetLastError()));
  return ok();
}

HS_API int hs_round(const hs_round_args* r, void* stream) {
  if (!r) return fail(HS_ERR_NULL, "args is NULL");
  EvalReq q{&r->target, r->drafters_host, r->N, r->B, r->K, r->V, r->dtype, r->temperature,
            r->mode, r->alpha, r->agree, r->argmax_t, r->argmax_d, r->workspace,
            r->workspace_bytes};
  hs::TeamGeom g;
  hs::RowTable rows;
  int rc = validate_eval(q, &g, &rows);
  if (rc) return rc;
  TailReq t{r->alpha, r->agree, r->mode, r->B, r->N, r->K, r->parent_host, r->path_end, r->eal,
            r->prefix, r->loss_kind, r->loss};
  hs::TailArgs a{};
  if ((rc = validate_tail(t, &a))) return rc;
  if ((r->logw == nullptr) != (r->w == nullptr))
    return fail(HS_ERR_NULL, "logw and w must be given together");
  if (!((r->R == nullptr) == (r->p == nullptr) && (r->R == nullptr) == (r->c == nullptr)))
    return fail(HS_ERR_NULL, "R, p and c must be given together");
  if (r->logw && !isfinite(r->eta)) return fail(HS_ERR_ARG, "eta must be finite");
  a.logw = r->logw;
  a.w = r->w;
  a.eta = r->eta;
  a.R = r->R;
  a.p = r->p;
  a.c = r->c;
  if ((rc = check_capacity(q, g))) return rc;
  if ((rc = run_eval(q, g, rows, &a, (hipStream_t)stream))) return rc;
  return ok();
}
