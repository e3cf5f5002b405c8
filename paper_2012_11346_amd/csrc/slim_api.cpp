// Host side of the C ABI declared in include/slim.h: argument validation,
// workspace layout, segment planning and kernel dispatch.
#include <hip/hip_runtime.h>

#include <climits>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>

#include "../../include/slim.h"
#include "slim_common.hpp"
#include "slim_kernels.hpp"

namespace {

thread_local std::string g_last_error;

int fail(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return status;
}

int ok() {
  g_last_error.clear();
  return SLIM_OK;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(SLIM_EHIP, "%s: %s", what, hipGetErrorString(e));
}

constexpr int kTileRows = 32;

int check_problem(const slim_problem* p) {
  if (p == nullptr) return fail(SLIM_EINVAL, "problem is NULL");
  if (p->B < 1 || p->H < 1 || p->L < 1) return fail(SLIM_EINVAL, "B, H, L must be >= 1");
  if (p->C < 1) return fail(SLIM_EINVAL, "slice length C must be >= 1 (got %d)", (int)p->C);
  if (p->dtype != SLIM_F32 && p->dtype != SLIM_BF16) return fail(SLIM_EINVAL, "unknown dtype %d", (int)p->dtype);
  if (p->kind != SLIM_FAVOR_PLUS && p->kind != SLIM_RELU) return fail(SLIM_EINVAL, "unknown kind %d", (int)p->kind);
  if (p->d != 32 && p->d != 64) return fail(SLIM_EUNSUPPORTED, "head dim d=%d not supported (32 or 64)", (int)p->d);
  if (p->M != 64 && p->M != 128 && p->M != 256)
    return fail(SLIM_EUNSUPPORTED, "feature count M=%d not supported (64, 128 or 256)", (int)p->M);
  if (p->L > (int64_t)INT_MAX / 2) return fail(SLIM_EUNSUPPORTED, "L=%lld too long", (long long)p->L);
  if (p->B * p->H > 65535) return fail(SLIM_EUNSUPPORTED, "B*H=%lld too large", (long long)(p->B * p->H));
  if (p->B > 65535 || p->H > 65535) return fail(SLIM_EUNSUPPORTED, "B or H above 65535");
  if (p->kind == SLIM_RELU && !(p->relu_eps > 0.f)) return fail(SLIM_EINVAL, "relu_eps must be > 0");
  if (p->dtype == SLIM_F32 && (int64_t)p->d * p->M > 4096)
    return fail(SLIM_EUNSUPPORTED, "fp32 problems need d*M <= 4096 (got d=%d, M=%d)", (int)p->d, (int)p->M);
  return SLIM_OK;
}

int clamp_C(const slim_problem* p) { return (int)(p->C > p->L ? p->L : p->C); }

// Segments per head: 1 for now; the walk is sequential per head.
int plan_segments(const slim_problem* p) {
  (void)p;
  return 1;
}

size_t state_elems(const slim_problem* p) { return (size_t)p->M * (size_t)(p->d + 1); }

struct FwdWs {
  size_t bytes;
};

size_t fwd_ws_bytes(const slim_problem* p) {
  (void)p;
  return 0;
}

size_t bwd_ws_bytes(const slim_problem* p, int P) {
  // dW partials per workgroup
  const size_t heads = (size_t)p->B * (size_t)p->H;
  return heads * (size_t)P * (size_t)p->M * (size_t)p->d * sizeof(float);
}

typedef hipError_t (*fwd_fn)(const slim::FwdArgs&, hipStream_t);
typedef hipError_t (*feat_fn)(const slim::FeatArgs&, hipStream_t);
typedef hipError_t (*bwd_fn)(const slim::BwdArgs&, hipStream_t);

struct Dispatch {
  fwd_fn fwd;
  feat_fn feat;
  bwd_fn bwd;
};

template <class T, int D, int FW, int KIND>
Dispatch make_dispatch() {
  typedef slim::Cfg<T, D, FW, kTileRows, KIND> G;
  return Dispatch{&slim::launch_fwd_walk<G>, &slim::launch_featmap<G>, &slim::launch_bwd_walk<G>};
}

template <int KIND>
Dispatch pick_bf16(int d, int M) {
  if (d == 64) {
    if (M == 256) return make_dispatch<slim::bf16, 64, 64, KIND>();
    if (M == 128) return make_dispatch<slim::bf16, 64, 32, KIND>();
    return make_dispatch<slim::bf16, 64, 16, KIND>();
  }
  if (M == 256) return make_dispatch<slim::bf16, 32, 64, KIND>();
  if (M == 128) return make_dispatch<slim::bf16, 32, 32, KIND>();
  return make_dispatch<slim::bf16, 32, 16, KIND>();
}

template <int KIND>
Dispatch pick_f32(int d, int M) {
  if (d == 64) return make_dispatch<float, 64, 16, KIND>();
  if (M == 128) return make_dispatch<float, 32, 32, KIND>();
  return make_dispatch<float, 32, 16, KIND>();
}

// callers have checked supported(p)
Dispatch dispatch(const slim_problem* p) {
  if (p->dtype == SLIM_BF16) return p->kind == SLIM_FAVOR_PLUS ? pick_bf16<slim::kFavor>(p->d, p->M)
                                                               : pick_bf16<slim::kRelu>(p->d, p->M);
  return p->kind == SLIM_FAVOR_PLUS ? pick_f32<slim::kFavor>(p->d, p->M) : pick_f32<slim::kRelu>(p->d, p->M);
}

}  // namespace

extern "C" {

const char* slim_status_string(int status) {
  switch (status) {
    case SLIM_OK:
      return "ok";
    case SLIM_EINVAL:
      return "invalid argument";
    case SLIM_EUNSUPPORTED:
      return "unsupported problem";
    case SLIM_EWORKSPACE:
      return "workspace missing or too small";
    case SLIM_EHIP:
      return "HIP runtime error";
    default:
      return "unknown status";
  }
}

const char* slim_last_error(void) { return g_last_error.c_str(); }

int slim_num_segments(const slim_problem* p) {
  if (check_problem(p) != SLIM_OK) return 0;
  return plan_segments(p);
}

size_t slim_workspace_bytes(const slim_problem* p, int phase) {
  if (check_problem(p) != SLIM_OK) return 0;
  if (phase == SLIM_PHASE_FWD) return fwd_ws_bytes(p);
  if (phase == SLIM_PHASE_BWD) return bwd_ws_bytes(p, plan_segments(p));
  fail(SLIM_EINVAL, "unknown phase %d", phase);
  return 0;
}

int slim_featmap(const slim_problem* p, const void* X, const float* W, int role, float* phi, float* shift,
                 void* stream) {
  int st = check_problem(p);
  if (st != SLIM_OK) return st;
  if (X == nullptr || W == nullptr || phi == nullptr) return fail(SLIM_EINVAL, "X, W and phi must be non-NULL");
  if (role != SLIM_QUERY && role != SLIM_KEY) return fail(SLIM_EINVAL, "unknown role %d", role);
  if (p->kind == SLIM_FAVOR_PLUS && shift == nullptr) return fail(SLIM_EINVAL, "FAVOR+ needs a shift buffer");
  slim::FeatArgs a;
  a.X = X;
  a.W = W;
  a.phi = phi;
  a.shift = shift;
  a.B = (int)p->B;
  a.H = (int)p->H;
  a.L = (int)p->L;
  a.role = role;
  a.relu_eps = p->relu_eps;
  hipError_t e = dispatch(p).feat(a, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "feature-map launch");
  return ok();
}

int slim_fwd(const slim_problem* p, const void* Q, const void* K, const void* V, const float* W,
             const float* state_in, const float* kshift_in, void* Y, float* state_out, float* kshift_out, void* ws,
             size_t ws_bytes, void* stream) {
  int st = check_problem(p);
  if (st != SLIM_OK) return st;
  if (Q == nullptr || K == nullptr || V == nullptr || W == nullptr || Y == nullptr)
    return fail(SLIM_EINVAL, "Q, K, V, W and Y must be non-NULL");
  if (p->kind == SLIM_FAVOR_PLUS) {
    if (kshift_out == nullptr) return fail(SLIM_EINVAL, "FAVOR+ needs kshift_out");
    if (state_in != nullptr && kshift_in == nullptr) return fail(SLIM_EINVAL, "state_in needs kshift_in (FAVOR+)");
  }
  const size_t need = fwd_ws_bytes(p);
  if (need > 0 && (ws == nullptr || ws_bytes < need))
    return fail(SLIM_EWORKSPACE, "forward workspace needs %zu bytes, got %zu", need, ws == nullptr ? 0 : ws_bytes);
  const int P = plan_segments(p);
  slim::FwdArgs a;
  std::memset(&a, 0, sizeof(a));
  a.Q = Q;
  a.K = K;
  a.V = V;
  a.W = W;
  a.Y = Y;
  a.state_out = state_out;
  a.kshift_out = (p->kind == SLIM_FAVOR_PLUS) ? kshift_out : nullptr;
  a.seg_state = state_in;
  a.seg_shift = kshift_in;
  a.B = (int)p->B;
  a.H = (int)p->H;
  a.L = (int)p->L;
  a.C = clamp_C(p);
  a.P = P;
  a.relu_eps = p->relu_eps;
  hipError_t e = dispatch(p).fwd(a, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "forward launch");
  return ok();
}

int slim_bwd(const slim_problem* p, const void* Q, const void* K, const void* V, const float* W,
             const float* state_in, const float* kshift_in, const float* state_out, const float* kshift,
             const void* dY, const float* dstate_out, void* dQ, void* dK, void* dV, float* dW, float* dstate_in,
             void* ws, size_t ws_bytes, void* stream) {
  int st = check_problem(p);
  if (st != SLIM_OK) return st;
  if (Q == nullptr || K == nullptr || V == nullptr || W == nullptr || dY == nullptr || dQ == nullptr ||
      dK == nullptr || dV == nullptr || dW == nullptr)
    return fail(SLIM_EINVAL, "Q, K, V, W, dY, dQ, dK, dV and dW must be non-NULL");
  if (state_out == nullptr) return fail(SLIM_EINVAL, "state_out (B^(N) from slim_fwd) must be non-NULL");
  if (p->kind == SLIM_FAVOR_PLUS) {
    if (kshift == nullptr) return fail(SLIM_EINVAL, "FAVOR+ needs kshift (kshift_out of slim_fwd)");
    if (state_in != nullptr && kshift_in == nullptr) return fail(SLIM_EINVAL, "state_in needs kshift_in (FAVOR+)");
  }
  const int P = plan_segments(p);
  const size_t need = bwd_ws_bytes(p, P);
  if (ws == nullptr || ws_bytes < need)
    return fail(SLIM_EWORKSPACE, "backward workspace needs %zu bytes, got %zu", need, ws == nullptr ? 0 : ws_bytes);
  slim::BwdArgs a;
  std::memset(&a, 0, sizeof(a));
  a.Q = Q;
  a.K = K;
  a.V = V;
  a.dY = dY;
  a.W = W;
  a.kshift = (p->kind == SLIM_FAVOR_PLUS) ? kshift : nullptr;
  a.seg_start = state_in;
  a.start_shift = (p->kind == SLIM_FAVOR_PLUS) ? kshift_in : nullptr;
  a.seg_end = state_out;
  a.seg_gend = dstate_out;
  a.seg_gstart = dstate_in;
  a.dQ = dQ;
  a.dK = dK;
  a.dV = dV;
  a.dW_part = (float*)ws;
  a.dW = dW;
  a.B = (int)p->B;
  a.H = (int)p->H;
  a.L = (int)p->L;
  a.C = clamp_C(p);
  a.P = P;
  a.relu_eps = p->relu_eps;
  hipError_t e = dispatch(p).bwd(a, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "backward launch");
  return ok();
}

}  // extern "C"
