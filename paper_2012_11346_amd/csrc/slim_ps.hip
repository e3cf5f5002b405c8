// Explicit prefix-sum evaluation of a slice (slim_problem.within =
// SLIM_WITHIN_PS): the variant the paper benchmarks as "PS" (Sec. 3.2, the
// prefix sums of eq. 3 taken over the rows of one slice; Sec. 4.1).
//
// For every row l of a slice the state U_l = B + sum over the slice's rows
// l' <= l of g(K_l')^T [V_l' | 1] is written out in full, C M (d + 1) floats
// per head, and Y_l is U_l^T g(Q_l) normalised by its last entry.  The
// backward writes out the cotangents of the same states,
// Ghat_l = G_after + sum over the slice's rows l' >= l of g(Q_l') [dN_l' | dD_l']
// (the reverse prefix sum of the query terms), from which
// dg(K_l) = Ghat_l [V_l | 1] and dV_l = Ghat_l^T g(K_l); dg(Q_l) = U_l [dN_l | dD_l].
// Every kernel streams those states through HBM: the mode shows what
// materialising them costs (memory proportional to C), it is not meant to be
// fast.  It takes every dtype, map and shape of the problem description,
// float32 at d M = 16384 included.
//
// Layouts: a slice's states are [head][row][e][m] (e < d + 1 fastest-varying
// over m, so that one thread per feature reads a row of them with whole-wave
// accesses); the library's states are [head][m][e].  Features are computed
// in float32 from the float32 W held in LDS, [t][m] with rows padded by one
// float (the logits read it along m, the chain rule along t, both without
// bank conflicts).  One thread per feature (M <= 256).
#include "slim_common.hpp"
#include "slim_kernels.hpp"

namespace slim {

namespace {

constexpr int kPsThreads = 256;
// LDS floats of every kernel: W as [t][m] with pitch M + 1 (D <= 64, M <= 256),
// then the row buffers
constexpr int kPsLds = 64 * 257 + 2 * 64 + 4 * 256 + 3 * 65 + 16;

__device__ __forceinline__ float ps_wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float ps_wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
// over the workgroup; every thread gets the result (red: 4 floats of LDS)
__device__ __forceinline__ float ps_block_sum(float v, float* red) {
  v = ps_wave_sum(v);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return (red[0] + red[1]) + (red[2] + red[3]);
}
__device__ __forceinline__ float ps_block_max(float v, float* red) {
  v = ps_wave_max(v);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}

// W [M][D] (float32, global) -> Wt[t][m] with pitch M + 1
template <int D>
__device__ void ps_load_w(const float* W, int M, float* Wt) {
  for (int i = threadIdx.x; i < M * D; i += kPsThreads) Wt[(i % D) * (M + 1) + i / D] = W[i];
}

// one row of D elements of a [B,H,L,D] tensor into LDS as float
template <class T, int D>
__device__ __forceinline__ void ps_load_row(const T* X, size_t row, float* x) {
  if (threadIdx.x < D) x[threadIdx.x] = (float)X[row * D + threadIdx.x];
}

template <int D>
__device__ __forceinline__ float ps_logit(const float* Wt, int M, const float* x, int m) {
  float s = 0.f;
#pragma unroll 16
  for (int t = 0; t < D; ++t) s = fmaf(Wt[t * (M + 1) + m], x[t], s);
  return s;
}
template <int D>
__device__ __forceinline__ float ps_norm2(const float* x) {
  float s = 0.f;
#pragma unroll 16
  for (int t = 0; t < D; ++t) s = fmaf(x[t], x[t], s);
  return s;
}

// feature of a key row from its logit l (FAVOR+: exp(l - |k|^2 / 2 - shift) / sqrt(M))
__device__ __forceinline__ float ps_key_feature(int kind, float l, float nx, float shift, float inv_sqrt_m, float eps) {
  if (kind == kFavor) return __expf(l - 0.5f * nx - shift) * inv_sqrt_m;
  if (kind == kRelu) return fmaxf(l, 0.f) + eps;
  return l * l;
}
// d loss / d logit from d loss / d feature (the shifts are constants)
__device__ __forceinline__ float ps_coef(int kind, float dphi, float phi, float l) {
  if (kind == kFavor) return dphi * phi;
  if (kind == kRelu) return l > 0.f ? dphi : 0.f;
  return 2.f * l * dphi;
}

// dx[t] = sum_m coef[m] w_m[t] - x[t] csum (csum: FAVOR+'s norm term, else 0),
// thread t < D gets it; every thread takes part (red: kPsThreads floats)
template <int D>
__device__ __forceinline__ float ps_chain(const float* Wt, int M, const float* coef, float* red) {
  constexpr int PARTS = kPsThreads / D;
  const int t = threadIdx.x % D, part = threadIdx.x / D;
  const int per = (M + PARTS - 1) / PARTS, m0 = part * per, m1 = min(M, m0 + per);
  float s = 0.f;
  for (int m = m0; m < m1; ++m) s = fmaf(coef[m], Wt[t * (M + 1) + m], s);
  red[threadIdx.x] = s;
  __syncthreads();
  float r = 0.f;
  if (threadIdx.x < D)
    for (int q = 0; q < PARTS; ++q) r += red[q * D + threadIdx.x];
  return r;
}

}  // namespace

// ---- key shift: the largest w_m.k - |k|^2/2 of the rows a workgroup visits
template <class T, int D>
__global__ __launch_bounds__(kPsThreads) void ps_kmax_kernel(PsArgs a) {
  __shared__ float ps_lds[kPsLds];
  float* Wt = ps_lds;
  float* x = Wt + D * (a.M + 1);
  float* red = x + D;
  const size_t head = blockIdx.y;
  ps_load_w<D>(a.W, a.M, Wt);
  const int m = threadIdx.x;
  float mx = -INFINITY;
  for (int l = blockIdx.x; l < a.L; l += gridDim.x) {
    __syncthreads();
    ps_load_row<T, D>((const T*)a.K, head * a.L + l, x);
    __syncthreads();
    if (m < a.M) mx = fmaxf(mx, ps_logit<D>(Wt, a.M, x, m) - 0.5f * ps_norm2<D>(x));
  }
  mx = ps_block_max(mx, red);
  if (threadIdx.x == 0) a.part[head * gridDim.x + blockIdx.x] = mx;
}

// ---- terms: U[row][e][m] = g(k_row)_m [v_row | 1]_e for the slice's rows
template <class T, int D>
__global__ __launch_bounds__(kPsThreads) void ps_terms_kernel(PsArgs a) {
  __shared__ float ps_lds[kPsLds];
  float* Wt = ps_lds;
  float* x = Wt + D * (a.M + 1);
  float* v = x + D;
  const size_t head = blockIdx.y;
  const int M = a.M, E = D + 1;
  ps_load_w<D>(a.W, M, Wt);
  const int m = threadIdx.x;
  const float shift = a.kind == kFavor ? a.kshift[head] : 0.f, ism = rsqrtf((float)M);
  for (int i = blockIdx.x; i < a.rows; i += gridDim.x) {
    const size_t row = head * a.L + a.row0 + i;
    __syncthreads();
    ps_load_row<T, D>((const T*)a.K, row, x);
    if (threadIdx.x >= 64 && threadIdx.x < 64 + D) v[threadIdx.x - 64] = (float)((const T*)a.V)[row * D + threadIdx.x - 64];
    __syncthreads();
    if (m < M) {
      const float phi = ps_key_feature(a.kind, ps_logit<D>(Wt, M, x, m), ps_norm2<D>(x), shift, ism, a.relu_eps);
      float* u = a.U + ((size_t)head * a.C + i) * E * M + m;
      for (int e = 0; e < D; ++e) u[(size_t)e * M] = phi * v[e];
      u[(size_t)D * M] = phi;
    }
  }
}

// s += x with the rounding error carried in c (Kahan's compensated sum: the
// running sums over a slice's rows keep float32 accuracy instead of losing
// it in proportion to the row count)
__device__ __forceinline__ void kahan_add(float& s, float& c, float x) {
  const float y = x - c, t = s + y;
  c = (t - s) - y;
  s = t;
}

// ---- prefix sums over the slice's rows, one thread per state entry (e, m):
//   mode 0: u = S_in (zero if NULL), U[i] <- u += U[i], S_out = the last u
//   mode 1: S_out = S_in - sum_i U[i] (eq. 17: the state before the slice
//           from the state after it), then as mode 0 from S_out
//   mode 2: S_out = S_in (an exact state before the slice), then as mode 0
// S_in of head h at S_in + h in_stride (state layout [m][e]).
__global__ __launch_bounds__(kPsThreads) void ps_scan_kernel(PsArgs a, int mode) {
  const int E = a.d + 1, M = a.M;
  const int el = blockIdx.x * kPsThreads + threadIdx.x;  // e M + m
  if (el >= E * M) return;
  const size_t head = blockIdx.y;
  const int e = el / M, m = el - e * M;
  const size_t sidx = (size_t)m * E + e;
  float* U = a.U + (size_t)head * a.C * E * M + el;
  const size_t step = (size_t)E * M;
  float u = a.S_in != nullptr ? a.S_in[head * a.in_stride + sidx] : 0.f;
  constexpr int U8 = 8;  // rows whose loads are issued together
  if (mode == 1) {
    float s = 0.f, c = 0.f;
    int i = 0;
    for (; i + U8 <= a.rows; i += U8) {
      float t[U8];
#pragma unroll
      for (int j = 0; j < U8; ++j) t[j] = U[(size_t)(i + j) * step];
#pragma unroll
      for (int j = 0; j < U8; ++j) kahan_add(s, c, t[j]);
    }
    for (; i < a.rows; ++i) kahan_add(s, c, U[(size_t)i * step]);
    u -= s;
  }
  if (mode != 0) a.S_out[head * (size_t)M * E + sidx] = u;
  float c = 0.f;
  int i = 0;
  for (; i + U8 <= a.rows; i += U8) {
    float t[U8];
#pragma unroll
    for (int j = 0; j < U8; ++j) t[j] = U[(size_t)(i + j) * step];
#pragma unroll
    for (int j = 0; j < U8; ++j) {
      kahan_add(u, c, t[j]);
      U[(size_t)(i + j) * step] = u;
    }
  }
  for (; i < a.rows; ++i) {
    kahan_add(u, c, U[(size_t)i * step]);
    U[(size_t)i * step] = u;
  }
  if (mode == 0 && a.S_out != nullptr) a.S_out[head * (size_t)M * E + sidx] = u;
}

// ---- reverse prefix sums: g = G_in (zero if NULL), Gh[i] <- g += Gh[i] for
//      i from the last row down, G_out = the last g (the cotangent before the slice)
__global__ __launch_bounds__(kPsThreads) void ps_rscan_kernel(PsArgs a) {
  const int E = a.d + 1, M = a.M;
  const int el = blockIdx.x * kPsThreads + threadIdx.x;
  if (el >= E * M) return;
  const size_t head = blockIdx.y;
  const int e = el / M, m = el - e * M;
  const size_t sidx = head * (size_t)M * E + (size_t)m * E + e;
  float* Gh = a.Gh + (size_t)head * a.C * E * M + el;
  const size_t step = (size_t)E * M;
  float g = a.G_in != nullptr ? a.G_in[sidx] : 0.f, c = 0.f;
  constexpr int U8 = 8;  // rows whose loads are issued together
  int i = a.rows - 1;
  for (; i - U8 + 1 >= 0; i -= U8) {
    float t[U8];
#pragma unroll
    for (int j = 0; j < U8; ++j) t[j] = Gh[(size_t)(i - j) * step];
#pragma unroll
    for (int j = 0; j < U8; ++j) {
      kahan_add(g, c, t[j]);
      Gh[(size_t)(i - j) * step] = g;
    }
  }
  for (; i >= 0; --i) {
    kahan_add(g, c, Gh[(size_t)i * step]);
    Gh[(size_t)i * step] = g;
  }
  a.G_out[sidx] = g;
}

namespace {
// query features of one row (x in LDS) for thread m: the row's largest logit
// is the FAVOR+ shift (any per-row constant cancels); returns the feature,
// the logit in *lout
template <int D>
__device__ __forceinline__ float ps_query_feature(const PsArgs& a, const float* Wt, const float* x, float* red, float* lout) {
  const int m = threadIdx.x;
  const float l = m < a.M ? ps_logit<D>(Wt, a.M, x, m) : -INFINITY;
  *lout = l;
  if (a.kind == kFavor) {
    const float mx = ps_block_max(l, red);
    return m < a.M ? __expf(l - mx) : 0.f;
  }
  if (m >= a.M) return 0.f;
  return a.kind == kRelu ? fmaxf(l, 0.f) + a.relu_eps : l * l;
}
// out[e] = sum_m phi[m] X[e][m] for e < E (wave w takes e = w, w + 4, ...)
__device__ __forceinline__ void ps_contract(const float* X, const float* phi, int E, int M, float* out) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  for (int e = w; e < E; e += 4) {
    float s = 0.f;
    for (int m = lane; m < M; m += 64) s = fmaf(phi[m], X[(size_t)e * M + m], s);
    s = ps_wave_sum(s);
    if (lane == 0) out[e] = s;
  }
}
}  // namespace

// ---- outputs: Y_row = U_row^T g(q_row) / (last entry)
template <class T, int D>
__global__ __launch_bounds__(kPsThreads) void ps_out_kernel(PsArgs a) {
  __shared__ float ps_lds[kPsLds];
  float* Wt = ps_lds;
  float* x = Wt + D * (a.M + 1);
  float* phi = x + D;
  float* num = phi + kPsThreads;
  float* red = num + D + 1;
  const size_t head = blockIdx.y;
  const int M = a.M, E = D + 1;
  ps_load_w<D>(a.W, M, Wt);
  for (int i = blockIdx.x; i < a.rows; i += gridDim.x) {
    const size_t row = head * a.L + a.row0 + i;
    __syncthreads();
    ps_load_row<T, D>((const T*)a.Q, row, x);
    __syncthreads();
    float l;
    phi[threadIdx.x] = ps_query_feature<D>(a, Wt, x, red, &l);
    __syncthreads();
    ps_contract(a.U + ((size_t)head * a.C + i) * E * M, phi, E, M, num);
    __syncthreads();
    if (threadIdx.x < D) ((T*)a.Y)[row * D + threadIdx.x] = cvt<T>(num[threadIdx.x] / num[D]);
  }
}

// ---- queries' gradient: from the dY rows and the states U of the slice,
//      dq, dW (queries' share) and the query terms g(q) [dN | dD] -> Gh
template <class T, int D>
__global__ __launch_bounds__(kPsThreads) void ps_gq_kernel(PsArgs a) {
  __shared__ float ps_lds[kPsLds];
  float* Wt = ps_lds;
  float* x = Wt + D * (a.M + 1);
  float* dy = x + D;
  float* phi = dy + D;
  float* coef = phi + kPsThreads;
  float* num = coef + kPsThreads;
  float* ev = num + D + 1;
  float* red = ev + D + 1;
  float* red2 = red + kPsThreads;
  const size_t head = blockIdx.y;
  const int M = a.M, E = D + 1, m = threadIdx.x;
  ps_load_w<D>(a.W, M, Wt);
  float dw[D];
#pragma unroll
  for (int t = 0; t < D; ++t) dw[t] = 0.f;
  for (int i = blockIdx.x; i < a.rows; i += gridDim.x) {
    const size_t row = head * a.L + a.row0 + i;
    const float* U = a.U + ((size_t)head * a.C + i) * E * M;
    __syncthreads();
    ps_load_row<T, D>((const T*)a.Q, row, x);
    if (threadIdx.x >= 64 && threadIdx.x < 64 + D) dy[threadIdx.x - 64] = (float)((const T*)a.dY)[row * D + threadIdx.x - 64];
    __syncthreads();
    float l;
    const float ph = ps_query_feature<D>(a, Wt, x, red2, &l);
    phi[m] = ph;
    __syncthreads();
    ps_contract(U, phi, E, M, num);
    __syncthreads();
    // dN = dY / den, dD = -dY . Y / den = -dY . N / den^2
    const float den = num[D];
    const float t = threadIdx.x < D ? dy[threadIdx.x] * num[threadIdx.x] : 0.f;
    const float dyn = ps_block_sum(t, red2);
    if (threadIdx.x < D) ev[threadIdx.x] = dy[threadIdx.x] / den;
    if (threadIdx.x == 0) ev[D] = -dyn / (den * den);
    __syncthreads();
    float cf = 0.f;
    if (m < M) {
      float dphi = 0.f;
      for (int e = 0; e < E; ++e) dphi = fmaf(U[(size_t)e * M + m], ev[e], dphi);
      cf = ps_coef(a.kind, dphi, ph, l);
      float* gh = a.Gh + ((size_t)head * a.C + i) * E * M + m;
      for (int e = 0; e < E; ++e) gh[(size_t)e * M] = ph * ev[e];
#pragma unroll
      for (int tt = 0; tt < D; ++tt) dw[tt] = fmaf(cf, x[tt], dw[tt]);
    }
    coef[m] = cf;
    const float csum = a.kind == kFavor ? ps_block_sum(cf, red2) : 0.f;
    __syncthreads();
    const float dq = ps_chain<D>(Wt, M, coef, red);
    if (threadIdx.x < D) ((T*)a.dQ)[row * D + threadIdx.x] = cvt<T>(dq - x[threadIdx.x] * csum);
  }
  if (m < M) {
    float* p = a.dW_part + (((size_t)head * a.nslot + blockIdx.x) * M + m) * D;
#pragma unroll
    for (int tt = 0; tt < D; ++tt) p[tt] += dw[tt];
  }
}

// ---- keys' gradient: from the cotangent sums Gh of the slice, dk, dv and
//      dW (keys' share)
template <class T, int D>
__global__ __launch_bounds__(kPsThreads) void ps_gk_kernel(PsArgs a) {
  __shared__ float ps_lds[kPsLds];
  float* Wt = ps_lds;
  float* x = Wt + D * (a.M + 1);
  float* v = x + D;
  float* phi = v + D + 1;
  float* coef = phi + kPsThreads;
  float* dv = coef + kPsThreads;
  float* red = dv + D + 1;
  float* red2 = red + kPsThreads;
  const size_t head = blockIdx.y;
  const int M = a.M, E = D + 1, m = threadIdx.x;
  ps_load_w<D>(a.W, M, Wt);
  const float shift = a.kind == kFavor ? a.kshift[head] : 0.f, ism = rsqrtf((float)M);
  float dw[D];
#pragma unroll
  for (int t = 0; t < D; ++t) dw[t] = 0.f;
  for (int i = blockIdx.x; i < a.rows; i += gridDim.x) {
    const size_t row = head * a.L + a.row0 + i;
    const float* Gh = a.Gh + ((size_t)head * a.C + i) * E * M;
    __syncthreads();
    ps_load_row<T, D>((const T*)a.K, row, x);
    if (threadIdx.x >= 64 && threadIdx.x < 64 + D) v[threadIdx.x - 64] = (float)((const T*)a.V)[row * D + threadIdx.x - 64];
    if (threadIdx.x == 64 + D) v[D] = 1.f;
    __syncthreads();
    float l = 0.f, ph = 0.f;
    if (m < M) {
      l = ps_logit<D>(Wt, M, x, m);
      ph = ps_key_feature(a.kind, l, ps_norm2<D>(x), shift, ism, a.relu_eps);
    }
    phi[m] = ph;
    __syncthreads();
    ps_contract(Gh, phi, D, M, dv);  // dV = Gh^T g(k) over the value columns
    float cf = 0.f;
    if (m < M) {
      float dphi = 0.f;
      for (int e = 0; e < E; ++e) dphi = fmaf(Gh[(size_t)e * M + m], v[e], dphi);
      cf = ps_coef(a.kind, dphi, ph, l);
#pragma unroll
      for (int tt = 0; tt < D; ++tt) dw[tt] = fmaf(cf, x[tt], dw[tt]);
    }
    coef[m] = cf;
    const float csum = a.kind == kFavor ? ps_block_sum(cf, red2) : 0.f;
    __syncthreads();
    const float dk = ps_chain<D>(Wt, M, coef, red);
    if (threadIdx.x < D) {
      ((T*)a.dK)[row * D + threadIdx.x] = cvt<T>(dk - x[threadIdx.x] * csum);
      ((T*)a.dV)[row * D + threadIdx.x] = cvt<T>(dv[threadIdx.x]);
    }
  }
  if (m < M) {
    float* p = a.dW_part + (((size_t)head * a.nslot + blockIdx.x) * M + m) * D;
#pragma unroll
    for (int tt = 0; tt < D; ++tt) p[tt] += dw[tt];
  }
}

// ---- what the rows of each part add to the state: part r of a head covers
//      the slices [r NS / P2, (r + 1) NS / P2); written [head][part][m][e]
template <class T, int D>
__global__ __launch_bounds__(kPsThreads) void ps_sum_kernel(PsArgs a, int NS, int P2) {
  __shared__ float ps_lds[kPsLds];
  float* Wt = ps_lds;
  float* x = Wt + D * (a.M + 1);
  float* v = x + D;
  const size_t head = blockIdx.y;
  const int r = blockIdx.x, M = a.M, E = D + 1, m = threadIdx.x;
  ps_load_w<D>(a.W, M, Wt);
  const float shift = a.kind == kFavor ? a.kshift[head] : 0.f, ism = rsqrtf((float)M);
  const int s0 = (int)((int64_t)r * NS / P2), s1 = (int)((int64_t)(r + 1) * NS / P2);
  const int l0 = s0 * a.C, l1 = (int)min((int64_t)a.L, (int64_t)s1 * a.C);
  float acc[D + 1], cmp[D + 1];
#pragma unroll
  for (int e = 0; e <= D; ++e) acc[e] = cmp[e] = 0.f;
  for (int l = l0; l < l1; ++l) {
    const size_t row = head * a.L + l;
    __syncthreads();
    ps_load_row<T, D>((const T*)a.K, row, x);
    if (threadIdx.x >= 64 && threadIdx.x < 64 + D) v[threadIdx.x - 64] = (float)((const T*)a.V)[row * D + threadIdx.x - 64];
    __syncthreads();
    if (m < M) {
      const float phi = ps_key_feature(a.kind, ps_logit<D>(Wt, M, x, m), ps_norm2<D>(x), shift, ism, a.relu_eps);
#pragma unroll
      for (int e = 0; e < D; ++e) kahan_add(acc[e], cmp[e], phi * v[e]);
      kahan_add(acc[D], cmp[D], phi);
    }
  }
  if (m < M) {
    float* p = a.part + (((size_t)head * P2 + r) * M + m) * E;
#pragma unroll
    for (int e = 0; e <= D; ++e) p[e] = acc[e];
  }
}

// ---- launchers (grid: (workgroups per head, heads))
namespace {
template <class T, int D>
hipError_t ps_launch_t(int which, const PsArgs& a, int nwg, int extra, hipStream_t s) {
  const dim3 g(nwg, a.B * a.H);
  switch (which) {
    case kPsKmax: hipLaunchKernelGGL((ps_kmax_kernel<T, D>), g, dim3(kPsThreads), 0, s, a); break;
    case kPsTerms: hipLaunchKernelGGL((ps_terms_kernel<T, D>), g, dim3(kPsThreads), 0, s, a); break;
    case kPsOut: hipLaunchKernelGGL((ps_out_kernel<T, D>), g, dim3(kPsThreads), 0, s, a); break;
    case kPsGq: hipLaunchKernelGGL((ps_gq_kernel<T, D>), g, dim3(kPsThreads), 0, s, a); break;
    case kPsGk: hipLaunchKernelGGL((ps_gk_kernel<T, D>), g, dim3(kPsThreads), 0, s, a); break;
    case kPsSum: hipLaunchKernelGGL((ps_sum_kernel<T, D>), g, dim3(kPsThreads), 0, s, a, extra, nwg); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}
}  // namespace

hipError_t launch_ps(int which, const PsArgs& a, int nwg, int extra, hipStream_t s) {
  if (which == kPsScan0 || which == kPsScan1 || which == kPsScan2) {
    const dim3 g(((a.d + 1) * a.M + kPsThreads - 1) / kPsThreads, a.B * a.H);
    hipLaunchKernelGGL(ps_scan_kernel, g, dim3(kPsThreads), 0, s, a, which - kPsScan0);
    return hipGetLastError();
  }
  if (which == kPsRscan) {
    const dim3 g(((a.d + 1) * a.M + kPsThreads - 1) / kPsThreads, a.B * a.H);
    hipLaunchKernelGGL(ps_rscan_kernel, g, dim3(kPsThreads), 0, s, a);
    return hipGetLastError();
  }
  if (a.bf16) return a.d == 64 ? ps_launch_t<bf16, 64>(which, a, nwg, extra, s) : ps_launch_t<bf16, 32>(which, a, nwg, extra, s);
  return a.d == 64 ? ps_launch_t<float, 64>(which, a, nwg, extra, s) : ps_launch_t<float, 32>(which, a, nwg, extra, s);
}

}  // namespace slim
