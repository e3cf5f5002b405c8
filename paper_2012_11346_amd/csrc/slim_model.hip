// The low-memory training step of the s-layer Performer language model
// (include/slim_model.h): Algorithm 1 with Algorithm 2 (Sec. 3.2-3.3) over
// the model of Sec. 2.2 (eqs. 5-10), float32.
//
// Only the attention states cross slice boundaries: per layer r the state
// B_r = (sum g(K) V^T, sum g(K)) of every head (forward), and B_r with its
// cotangent G_r (backward).  Inside a slice every layer is row-wise except
// the attention, which is the library's own slim_fwd / slim_bwd (kind
// SLIM_SQUARE with W = I: the paper's element-wise square map, M = d = 64).
// The backward recovers the state before a slice by subtracting the
// slice's own sum from the state after it (eq. 17), recomputes the slice
// through all layers, and back-propagates through it with the state
// cotangents G_r carried from the later slices (eq. 18).
//
// Kernels here: a float32 matrix-core GEMM (v_mfma_f32_16x16x4_f32, 64 x 64
// tiles), row-wise layer normalisation and its backward, bias + GeLU,
// cross-entropy, the embedding and its deterministic backward, head
// split/merge copies and fixed-order column sums.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <vector>

#include "../../include/slim.h"
#include "../../include/slim_model.h"
#include "slim_kernels.hpp"

namespace slim {
namespace model {

typedef float f4 __attribute__((ext_vector_type(4)));
constexpr int kHead = 64;  // head dimension (d = M = 64)

// ---------------------------------------------------------------- GEMM
// C = alpha op(A) op(B) + beta C, row-major: op(A)[m][k] = TA ? A[k lda + m]
// : A[m lda + k], op(B)[k][n] = TB ? B[n ldb + k] : B[k ldb + n].  One
// workgroup per 64 x 64 tile of C; four waves of 32 x 32, each 2 x 2 matrix
// tiles of 16 x 16; K in steps of 16 through LDS ([k][m] and [k][n], rows
// padded so that the four k rows a product reads fall in distinct banks).
constexpr int GT = 64, GK = 16, GLD = GT + 16;

template <bool TA, bool TB>
__global__ __launch_bounds__(256) void gemm_kernel(int M, int N, int K, float alpha, const float* __restrict__ A,
                                                   int lda, const float* __restrict__ B, int ldb, float beta,
                                                   float* __restrict__ C, int ldc) {
  __shared__ float As[GK][GLD];
  __shared__ float Bs[GK][GLD];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int m0 = blockIdx.y * GT, n0 = blockIdx.x * GT;
  const int wm = (w >> 1) * 32, wn = (w & 1) * 32;
  f4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
  for (int k0 = 0; k0 < K; k0 += GK) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = tid + 256 * i;
      int m, ka;
      if (TA) {
        m = e % GT;
        ka = e / GT;
      } else {
        ka = e % GK;
        m = e / GK;
      }
      const int gm = m0 + m, gka = k0 + ka;
      float v = 0.f;
      if (gm < M && gka < K) v = TA ? A[(size_t)gka * lda + gm] : A[(size_t)gm * lda + gka];
      As[ka][m] = v;
      int n, kb;
      if (TB) {
        kb = e % GK;
        n = e / GK;
      } else {
        n = e % GT;
        kb = e / GT;
      }
      const int gn = n0 + n, gkb = k0 + kb;
      float u = 0.f;
      if (gn < N && gkb < K) u = TB ? B[(size_t)gn * ldb + gkb] : B[(size_t)gkb * ldb + gn];
      Bs[kb][n] = u;
    }
    __syncthreads();
    const int c = lane & 15, g = lane >> 4;
#pragma unroll
    for (int ks = 0; ks < GK; ks += 4) {
      float a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) a[i] = As[ks + g][wm + 16 * i + c];
#pragma unroll
      for (int j = 0; j < 2; ++j) b[j] = Bs[ks + g][wn + 16 * j + c];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
  }
  const int c = lane & 15, g = lane >> 4;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = m0 + wm + 16 * i + 4 * g + r, col = n0 + wn + 16 * j + c;
        if (row < M && col < N) {
          float* p = C + (size_t)row * ldc + col;
          *p = beta != 0.f ? alpha * acc[i][j][r] + beta * *p : alpha * acc[i][j][r];
        }
      }
}

hipError_t gemm(bool ta, bool tb, int M, int N, int K, float alpha, const float* A, int lda, const float* B, int ldb,
                float beta, float* C, int ldc, hipStream_t s) {
  if (M <= 0 || N <= 0) return hipSuccess;
  const dim3 grid((N + GT - 1) / GT, (M + GT - 1) / GT);
  if (ta && tb) hipLaunchKernelGGL((gemm_kernel<true, true>), grid, dim3(256), 0, s, M, N, K, alpha, A, lda, B, ldb, beta, C, ldc);
  else if (ta) hipLaunchKernelGGL((gemm_kernel<true, false>), grid, dim3(256), 0, s, M, N, K, alpha, A, lda, B, ldb, beta, C, ldc);
  else if (tb) hipLaunchKernelGGL((gemm_kernel<false, true>), grid, dim3(256), 0, s, M, N, K, alpha, A, lda, B, ldb, beta, C, ldc);
  else hipLaunchKernelGGL((gemm_kernel<false, false>), grid, dim3(256), 0, s, M, N, K, alpha, A, lda, B, ldb, beta, C, ldc);
  return hipGetLastError();
}

// ---------------------------------------------------------------- row-wise kernels

// sum over the 256 threads of a workgroup (every thread gets the result)
__device__ __forceinline__ float block_sum(float v, float* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  return (red[0] + red[1]) + (red[2] + red[3]);
}
__device__ __forceinline__ float block_max(float v, float* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  return fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}

// X0[i] = E[token] + PE(position): row i = (b, t) of the slice [a, a + n);
// the sinusoid angles in double precision (positions reach 1e4 and more)
__global__ __launch_bounds__(256) void embed_kernel(const int* tokens, int64_t L, int a, int n, const float* emb, int D,
                                                    int V, float* X) {
  const int i = blockIdx.x, b = i / n, t = i - b * n;
  const int64_t pos = a + t;
  const int tok = tokens[b * L + pos];
  if (tok < 0 || tok >= V) {  // outside the alphabet: the row (and the loss) becomes NaN
    for (int j = threadIdx.x; j < D; j += 256) X[(size_t)i * D + j] = __builtin_nanf("");
    return;
  }
  for (int j = threadIdx.x; j < D; j += 256) {
    const double ang = (double)pos / pow(10000.0, (double)(2 * (j / 2)) / (double)D);
    const double pe = (j & 1) ? cos(ang) : sin(ang);
    X[(size_t)i * D + j] = emb[(size_t)tok * D + j] + (float)pe;
  }
}

// out[i] = LN(x[i]) * g + b + res[i] (res may be null); stats[i] = (mean, rstd)
__global__ __launch_bounds__(256) void ln_fwd_kernel(const float* x, const float* g, const float* b, const float* res,
                                                     float* out, float* stats, int D, float eps) {
  __shared__ float red[4];
  const size_t row = (size_t)blockIdx.x * D;
  float s = 0.f;
  for (int j = threadIdx.x; j < D; j += 256) s += x[row + j];
  const float mu = block_sum(s, red) / (float)D;
  float q = 0.f;
  for (int j = threadIdx.x; j < D; j += 256) {
    const float c = x[row + j] - mu;
    q += c * c;
  }
  const float rstd = 1.f / sqrtf(block_sum(q, red) / (float)D + eps);
  for (int j = threadIdx.x; j < D; j += 256) {
    const float y = (x[row + j] - mu) * rstd * g[j] + b[j];
    out[row + j] = res ? y + res[row + j] : y;
  }
  if (threadIdx.x == 0) {
    stats[2 * blockIdx.x] = mu;
    stats[2 * blockIdx.x + 1] = rstd;
  }
}

// dx[i] = rstd / D (D dxh - sum dxh - xhat sum(dxh xhat)) + add[i], dxh = dy g;
// P[i] = dy xhat (for the gain's gradient)
__global__ __launch_bounds__(256) void ln_bwd_kernel(const float* x, const float* stats, const float* g, const float* dy,
                                                     const float* add, float* dx, float* P, int D) {
  __shared__ float red[4];
  const size_t row = (size_t)blockIdx.x * D;
  const float mu = stats[2 * blockIdx.x], rstd = stats[2 * blockIdx.x + 1];
  float s1 = 0.f, s2 = 0.f;
  for (int j = threadIdx.x; j < D; j += 256) {
    const float xh = (x[row + j] - mu) * rstd, d = dy[row + j] * g[j];
    s1 += d;
    s2 += d * xh;
  }
  s1 = block_sum(s1, red);
  s2 = block_sum(s2, red);
  for (int j = threadIdx.x; j < D; j += 256) {
    const float xh = (x[row + j] - mu) * rstd, d = dy[row + j] * g[j];
    float v = rstd / (float)D * ((float)D * d - s1 - xh * s2);
    if (add) v += add[row + j];
    dx[row + j] = v;
    P[row + j] = dy[row + j] * xh;
  }
}

// out[j] += sum_i P[i][j], rows in order (one thread per column)
__global__ __launch_bounds__(256) void colsum_kernel(const float* P, int rows, int n, float* out) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= n) return;
  float s = 0.f;
  for (int i = 0; i < rows; ++i) s += P[(size_t)i * n + j];
  out[j] += s;
}

__device__ __forceinline__ float gelu_f(float x) { return 0.5f * x * (1.f + erff(x * 0.70710678118654752f)); }
__device__ __forceinline__ float gelu_d(float x) {
  return 0.5f * (1.f + erff(x * 0.70710678118654752f)) + x * expf(-0.5f * x * x) * 0.39894228040143268f;
}

// Z += b (the pre-activation, kept), G = GeLU(Z)
__global__ __launch_bounds__(256) void bias_gelu_kernel(float* Z, const float* b, float* G, int n, size_t total) {
  const size_t e = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= total) return;
  const float z = Z[e] + b[e % n];
  Z[e] = z;
  G[e] = gelu_f(z);
}
// dZ = dG GeLU'(Z), in place of dG
__global__ __launch_bounds__(256) void gelu_bwd_kernel(float* dG, const float* Z, size_t total) {
  const size_t e = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= total) return;
  dG[e] *= gelu_d(Z[e]);
}
__global__ __launch_bounds__(256) void bias_add_kernel(float* Y, const float* b, int n, size_t total) {
  const size_t e = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= total) return;
  Y[e] += b[e % n];
}
__global__ __launch_bounds__(256) void copy_kernel(float* dst, const float* src, size_t total) {
  const size_t e = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (e < total) dst[e] = src[e];
}
__global__ __launch_bounds__(256) void identity_kernel(float* I, int n) {
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e < n * n) I[e] = (e / n == e % n) ? 1.f : 0.f;
}
__global__ __launch_bounds__(256) void fill_kernel(float* dst, float v, size_t total) {
  const size_t e = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (e < total) dst[e] = v;
}
// out = a - b
__global__ __launch_bounds__(256) void sub_kernel(float* out, const float* a, const float* b, size_t total) {
  const size_t e = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (e < total) out[e] = a[e] - b[e];
}

// Cross-entropy of row i = (b, t) against the next token (eq. 10): weight
// w = 1 / ((L - 1) B) on rows with position < L - 1, else 0; rowloss[i] =
// w (lse - logit[target]); logits become w (softmax - onehot) in place.
__global__ __launch_bounds__(256) void ce_kernel(float* logits, const int* tokens, int64_t L, int a, int n, int B,
                                                 int V, float* rowloss) {
  __shared__ float red[4];
  const int i = blockIdx.x, b = i / n, t = i - b * n;
  const int64_t pos = a + t;
  float* z = logits + (size_t)i * V;
  const bool has = pos < L - 1;
  int tgt = has ? tokens[b * L + pos + 1] : -1;
  const bool bad = has && (tgt < 0 || tgt >= V);  // outside the alphabet: NaN loss
  if (bad) tgt = -1;
  const float w = has ? 1.f / ((float)(L - 1) * (float)B) : 0.f;
  float mx = -INFINITY;
  for (int j = threadIdx.x; j < V; j += 256) mx = fmaxf(mx, z[j]);
  mx = block_max(mx, red);
  float se = 0.f;
  for (int j = threadIdx.x; j < V; j += 256) se += expf(z[j] - mx);
  se = block_sum(se, red);
  const float lse = mx + logf(se);
  float zt = 0.f;
  for (int j = threadIdx.x; j < V; j += 256) zt += (j == tgt) ? z[j] : 0.f;
  zt = block_sum(zt, red);
  for (int j = threadIdx.x; j < V; j += 256) z[j] = w * (expf(z[j] - lse) - (j == tgt ? 1.f : 0.f));
  if (threadIdx.x == 0) rowloss[i] = bad ? __builtin_nanf("") : w * (lse - zt);
}

// out[0] (+)= sum of v[0 .. n), in a fixed order (one workgroup)
__global__ __launch_bounds__(256) void sum_kernel(const float* v, int n, float* out, int accumulate) {
  __shared__ float red[4];
  float s = 0.f;
  for (int i = threadIdx.x; i < n; i += 256) s += v[i];
  s = block_sum(s, red);
  if (threadIdx.x == 0) out[0] = accumulate ? out[0] + s : s;
}

// heads [B, k, n, 64] <-> rows [B n, ld] at column offset col0 (head h at
// columns col0 + 64 h)
__global__ __launch_bounds__(256) void rows_to_heads_kernel(const float* src, int ld, int col0, float* dst, int k, int n,
                                                            size_t total) {
  const size_t e = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= total) return;
  const int c = (int)(e % kHead);
  size_t r = e / kHead;
  const int t = (int)(r % n);
  r /= n;
  const int h = (int)(r % k);
  const int b = (int)(r / k);
  dst[e] = src[((size_t)b * n + t) * ld + col0 + h * kHead + c];
}
__global__ __launch_bounds__(256) void heads_to_rows_kernel(const float* src, float* dst, int ld, int col0, int k, int n,
                                                            size_t total) {
  const size_t e = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= total) return;
  const int c = (int)(e % kHead);
  size_t r = e / kHead;
  const int t = (int)(r % n);
  r /= n;
  const int h = (int)(r % k);
  const int b = (int)(r / k);
  dst[((size_t)b * n + t) * ld + col0 + h * kHead + c] = src[e];
}

// dE[v] += sum over the slice's rows with token v of dX0[row], rows in
// order: workgroup (v, column block) compacts the matching rows of each
// 256-row chunk into LDS (ballot + prefix), then adds them column-wise
__global__ __launch_bounds__(256) void embed_bwd_kernel(const int* tokens, int64_t L, int a, int n, int rows,
                                                        const float* dX, int D, float* dE) {
  __shared__ int list[256];
  __shared__ int wcount[4];
  const int v = blockIdx.x, j = blockIdx.y * 256 + threadIdx.x;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  float acc = 0.f;
  for (int c0 = 0; c0 < rows; c0 += 256) {
    const int i = c0 + threadIdx.x;
    bool m = false;
    if (i < rows) {
      const int b = i / n, t = i - b * n;
      m = tokens[b * L + a + t] == v;
    }
    const unsigned long long bal = __ballot(m);
    const int before = __popcll(bal & ((1ull << lane) - 1ull));
    __syncthreads();  // the previous chunk's readers of list are done
    if (lane == 0) wcount[w] = __popcll(bal);
    __syncthreads();
    int off = 0;
    for (int ww = 0; ww < w; ++ww) off += wcount[ww];
    if (m) list[off + before] = i;
    const int total = wcount[0] + wcount[1] + wcount[2] + wcount[3];
    __syncthreads();
    if (j < D)
      for (int q = 0; q < total; ++q) acc += dX[(size_t)list[q] * D + j];
  }
  if (j < D) dE[(size_t)v * D + j] += acc;
}

inline dim3 grid1(size_t total) { return dim3((unsigned)((total + 255) / 256)); }

// ---------------------------------------------------------------- host side

size_t al(size_t n) { return (n + 255) & ~(size_t)255; }

struct Dims {
  int64_t B, L;
  int D, s, V, F, C, k, nmax;
  float eps;
  size_t rows_max() const { return (size_t)B * nmax; }
  size_t state_floats() const { return (size_t)B * k * kHead * (kHead + 1); }
};

slim_problem att_problem(const Dims& m, int n) {
  slim_problem p;
  std::memset(&p, 0, sizeof(p));
  p.B = m.B;
  p.H = m.k;
  p.L = n;
  p.d = kHead;
  p.M = kHead;
  p.C = n;
  p.dtype = SLIM_F32;
  p.kind = SLIM_SQUARE;
  p.relu_eps = 1e-3f;
  p.within = SLIM_WITHIN_ITER;
  return p;
}

// workspace regions (byte offsets)
struct Layout {
  size_t ident, attws, attws_bytes, states, gstates, bprev, delta, snew, wd;
  size_t X, QKV, Qh, Yh, A, st1, H, Z1, G1, Fo, st2;
  size_t logits, rowloss, dX, dH, dF, dG1, dA, dYh, dQh, dQKV, P;
  size_t total;
};

Layout layout(const Dims& m) {
  Layout l;
  std::memset(&l, 0, sizeof(l));
  size_t off = 0;
  auto take = [&](size_t& at, size_t bytes) {
    at = off;
    off += al(bytes);
  };
  const size_t R = m.rows_max(), D = m.D, F = m.F, S = m.state_floats(), s = m.s;
  const size_t HF = (size_t)m.B * m.k * m.nmax * kHead;  // floats of one [B, k, n, 64] tensor
  take(l.ident, kHead * kHead * 4);
  size_t aw = 0;
  const int last = (int)(m.L - (m.L - 1) / m.nmax * m.nmax);
  for (int n : {m.nmax, last}) {
    const slim_problem p = att_problem(m, n);
    aw = std::max(aw, std::max(slim_workspace_bytes(&p, SLIM_PHASE_FWD), slim_workspace_bytes(&p, SLIM_PHASE_BWD)));
  }
  l.attws_bytes = std::max<size_t>(aw, 256);
  take(l.attws, l.attws_bytes);
  take(l.states, s * S * 4);
  take(l.gstates, 2 * s * S * 4);
  take(l.bprev, s * S * 4);
  take(l.delta, S * 4);
  take(l.snew, S * 4);
  take(l.wd, kHead * kHead * 4);
  take(l.X, (s + 1) * R * D * 4);
  take(l.QKV, R * 3 * D * 4);
  take(l.Qh, s * 3 * HF * 4);
  take(l.Yh, HF * 4);
  take(l.A, s * R * D * 4);
  take(l.st1, s * R * 2 * 4);
  take(l.H, s * R * D * 4);
  take(l.Z1, s * R * F * 4);
  take(l.G1, s * R * F * 4);
  take(l.Fo, s * R * D * 4);
  take(l.st2, s * R * 2 * 4);
  take(l.logits, R * m.V * 4);
  take(l.rowloss, R * 4);
  take(l.dX, R * D * 4);
  take(l.dH, R * D * 4);
  take(l.dF, R * D * 4);
  take(l.dG1, R * F * 4);
  take(l.dA, R * D * 4);
  take(l.dYh, HF * 4);
  take(l.dQh, 3 * HF * 4);
  take(l.dQKV, R * 3 * D * 4);
  take(l.P, R * std::max(D, std::max(F, (size_t)m.V)) * 4);
  l.total = off;
  return l;
}

int check(const slim_model* mm, Dims* out) {
  if (mm == nullptr) return report(SLIM_EINVAL, "model description is NULL");
  Dims m;
  m.B = mm->B;
  m.L = mm->L;
  m.D = mm->D;
  m.s = mm->s;
  m.V = mm->vocab;
  m.F = mm->F;
  m.C = mm->C;
  m.eps = mm->ln_eps;
  if (m.B < 1 || m.L < 2 || m.s < 1 || m.C < 1) return report(SLIM_EINVAL, "B >= 1, L >= 2, s >= 1 and C >= 1 required");
  if (m.D < 64 || m.D % 64 != 0 || m.D > 4096) return report(SLIM_EUNSUPPORTED, "d_model must be a multiple of 64, at most 4096");
  if (m.V < 2 || m.V > 65536) return report(SLIM_EUNSUPPORTED, "vocab must be in [2, 65536]");
  if (m.F < 4 || m.F % 4 != 0 || m.F > (1 << 16)) return report(SLIM_EUNSUPPORTED, "d_ff must be a multiple of 4, at most 65536");
  if (!(m.eps > 0.f)) return report(SLIM_EINVAL, "ln_eps must be > 0");
  m.k = m.D / kHead;
  m.nmax = (int)std::min<int64_t>(m.C, m.L);
  if ((int64_t)m.B * m.nmax > (1 << 24) || m.L > ((int64_t)1 << 30) || m.B * m.L > ((int64_t)1 << 31) - 1)
    return report(SLIM_EUNSUPPORTED, "too many rows");
  if (m.B * m.k > 65535) return report(SLIM_EUNSUPPORTED, "B * heads above 65535");
  *out = m;
  return SLIM_OK;
}

// parameter slots
struct Params {
  const float *emb, *Wout, *bout;
  struct Layer {
    const float *Wq, *Wk, *Wv, *g1, *b1n, *W1, *b1, *W2, *b2, *g2, *b2n;
  };
  std::vector<Layer> l;
};
struct Grads {
  float *emb, *Wout, *bout;
  struct Layer {
    float *Wq, *Wk, *Wv, *g1, *b1n, *W1, *b1, *W2, *b2, *g2, *b2n;
  };
  std::vector<Layer> l;
};
template <class P, class T>
void unpack(P& p, T* const* a, int s) {
  p.emb = a[0];
  p.l.resize(s);
  for (int r = 0; r < s; ++r) {
    T* const* q = a + 1 + 11 * r;
    p.l[r] = {q[0], q[1], q[2], q[3], q[4], q[5], q[6], q[7], q[8], q[9], q[10]};
  }
  p.Wout = a[1 + 11 * s];
  p.bout = a[2 + 11 * s];
}

#define CHECK_HIP(x)                                            \
  do {                                                          \
    hipError_t e_ = (x);                                        \
    if (e_ != hipSuccess) return report(SLIM_EHIP, hipGetErrorString(e_)); \
  } while (0)
#define CHECK_SLIM(x)                          \
  do {                                         \
    int st_ = (x);                             \
    if (st_ != SLIM_OK) return st_;            \
  } while (0)

// One step of Algorithm 1.
int step(const Dims& m, const int* tokens, const Params& P, const Grads& G, float* loss, char* w, hipStream_t s) {
  const Layout lay = layout(m);
  const int D = m.D, F = m.F, V = m.V, k = m.k;
  const size_t S = m.state_floats();
  float* ident = (float*)(w + lay.ident);
  void* attws = w + lay.attws;
  float* states = (float*)(w + lay.states);
  float* gst = (float*)(w + lay.gstates);
  float* bprev = (float*)(w + lay.bprev);
  float* delta = (float*)(w + lay.delta);
  float* snew = (float*)(w + lay.snew);
  float* wd = (float*)(w + lay.wd);
  auto f = [&](size_t off) { return (float*)(w + off); };
  const size_t R = m.rows_max(), HF = (size_t)m.B * k * m.nmax * kHead;
  auto Xr = [&](int r) { return f(lay.X) + (size_t)r * R * D; };
  auto Ar = [&](int r) { return f(lay.A) + (size_t)r * R * D; };
  auto Hr = [&](int r) { return f(lay.H) + (size_t)r * R * D; };
  auto Z1r = [&](int r) { return f(lay.Z1) + (size_t)r * R * F; };
  auto G1r = [&](int r) { return f(lay.G1) + (size_t)r * R * F; };
  auto For = [&](int r) { return f(lay.Fo) + (size_t)r * R * D; };
  auto s1r = [&](int r) { return f(lay.st1) + (size_t)r * R * 2; };
  auto s2r = [&](int r) { return f(lay.st2) + (size_t)r * R * 2; };
  auto Qhr = [&](int r, int part) { return f(lay.Qh) + ((size_t)r * 3 + part) * HF; };
  float* QKV = f(lay.QKV);
  float* Yh = f(lay.Yh);
  float* logits = f(lay.logits);
  float* rowloss = f(lay.rowloss);
  float *dX = f(lay.dX), *dH = f(lay.dH), *dF = f(lay.dF), *dG1 = f(lay.dG1), *dA = f(lay.dA);
  float *dYh = f(lay.dYh), *dQh = f(lay.dQh), *dQKV = f(lay.dQKV), *Pp = f(lay.P);

  // identity W of the square map: g(x) = (x_i^2)
  hipLaunchKernelGGL(identity_kernel, grid1(kHead * kHead), dim3(256), 0, s, ident, kHead);
  CHECK_HIP(hipGetLastError());

  // queries, keys and values of layer r for the slice's rows, per head (the
  // activations of every layer stay in its buffers for the backward)
  auto layer_qkv = [&](int r, int n) -> int {
    const int rows = (int)(m.B * n);
    const size_t hf = (size_t)m.B * k * n * kHead;
    const float* X = Xr(r);
    CHECK_HIP(gemm(false, false, rows, D, D, 1.f, X, D, P.l[r].Wq, D, 0.f, QKV, 3 * D, s));
    CHECK_HIP(gemm(false, false, rows, D, D, 1.f, X, D, P.l[r].Wk, D, 0.f, QKV + D, 3 * D, s));
    CHECK_HIP(gemm(false, false, rows, D, D, 1.f, X, D, P.l[r].Wv, D, 0.f, QKV + 2 * D, 3 * D, s));
    for (int part = 0; part < 3; ++part)
      hipLaunchKernelGGL(rows_to_heads_kernel, grid1(hf), dim3(256), 0, s, QKV, 3 * D, part * D, Qhr(r, part), k, n, hf);
    CHECK_HIP(hipGetLastError());
    return SLIM_OK;
  };
  // the rest of layer r (eqs. 5-9) from the state before the slice
  auto layer_fwd = [&](int r, int a, int n, const float* state_in, float* state_out) -> int {
    const int rows = (int)(m.B * n);
    const size_t hf = (size_t)m.B * k * n * kHead;
    const float* X = Xr(r);
    const slim_problem p = att_problem(m, n);
    CHECK_SLIM(slim_fwd(&p, Qhr(r, 0), Qhr(r, 1), Qhr(r, 2), ident, state_in, nullptr, Yh, state_out, nullptr, nullptr,
                        attws, lay.attws_bytes, s));
    hipLaunchKernelGGL(heads_to_rows_kernel, grid1(hf), dim3(256), 0, s, Yh, Ar(r), D, 0, k, n, hf);
    hipLaunchKernelGGL(ln_fwd_kernel, dim3(rows), dim3(256), 0, s, Ar(r), P.l[r].g1, P.l[r].b1n, X, Hr(r), s1r(r), D,
                       m.eps);
    CHECK_HIP(gemm(false, false, rows, F, D, 1.f, Hr(r), D, P.l[r].W1, F, 0.f, Z1r(r), F, s));
    hipLaunchKernelGGL(bias_gelu_kernel, grid1((size_t)rows * F), dim3(256), 0, s, Z1r(r), P.l[r].b1, G1r(r), F,
                       (size_t)rows * F);
    CHECK_HIP(gemm(false, false, rows, D, F, 1.f, G1r(r), F, P.l[r].W2, D, 0.f, For(r), D, s));
    hipLaunchKernelGGL(bias_add_kernel, grid1((size_t)rows * D), dim3(256), 0, s, For(r), P.l[r].b2, D, (size_t)rows * D);
    hipLaunchKernelGGL(ln_fwd_kernel, dim3(rows), dim3(256), 0, s, For(r), P.l[r].g2, P.l[r].b2n, Hr(r), Xr(r + 1),
                       s2r(r), D, m.eps);
    CHECK_HIP(hipGetLastError());
    return SLIM_OK;
  };
  auto head_logits = [&](int a, int n) -> int {
    const int rows = (int)(m.B * n);
    CHECK_HIP(gemm(false, false, rows, V, D, 1.f, Xr(m.s), D, P.Wout, V, 0.f, logits, V, s));
    hipLaunchKernelGGL(bias_add_kernel, grid1((size_t)rows * V), dim3(256), 0, s, logits, P.bout, V, (size_t)rows * V);
    hipLaunchKernelGGL(ce_kernel, dim3(rows), dim3(256), 0, s, logits, tokens, m.L, a, n, (int)m.B, V, rowloss);
    CHECK_HIP(hipGetLastError());
    return SLIM_OK;
  };

  const int NS = (int)((m.L + m.nmax - 1) / m.nmax);
  // ---- forward: slices in order, layers inside; only the states cross
  hipLaunchKernelGGL(fill_kernel, grid1(m.s * S), dim3(256), 0, s, states, 0.f, (size_t)m.s * S);
  hipLaunchKernelGGL(fill_kernel, dim3(1), dim3(256), 0, s, loss, 0.f, (size_t)1);
  for (int q = 0; q < NS; ++q) {
    const int a = q * m.nmax, n = (int)std::min<int64_t>(m.nmax, m.L - a);
    hipLaunchKernelGGL(embed_kernel, dim3((unsigned)(m.B * n)), dim3(256), 0, s, tokens, m.L, a, n, P.emb, D, V, Xr(0));
    for (int r = 0; r < m.s; ++r) {
      CHECK_SLIM(layer_qkv(r, n));
      CHECK_SLIM(layer_fwd(r, a, n, states + r * S, snew));
      hipLaunchKernelGGL(copy_kernel, grid1(S), dim3(256), 0, s, states + r * S, snew, S);
    }
    CHECK_SLIM(head_logits(a, n));
    hipLaunchKernelGGL(sum_kernel, dim3(1), dim3(256), 0, s, rowloss, (int)(m.B * n), loss, 1);
    CHECK_HIP(hipGetLastError());
  }

  // ---- backward: slices in reverse
  auto zero = [&](float* p, size_t nflt) { hipLaunchKernelGGL(fill_kernel, grid1(nflt), dim3(256), 0, s, p, 0.f, nflt); };
  zero(G.emb, (size_t)V * D);
  zero(G.Wout, (size_t)D * V);
  zero(G.bout, V);
  for (int r = 0; r < m.s; ++r) {
    const Grads::Layer& g = G.l[r];
    for (float* p : {g.Wq, g.Wk, g.Wv}) zero(p, (size_t)D * D);
    for (float* p : {g.g1, g.b1n, g.b2, g.g2, g.b2n}) zero(p, D);
    zero(g.W1, (size_t)D * F);
    zero(g.b1, F);
    zero(g.W2, (size_t)F * D);
  }
  zero(gst, 2 * m.s * S);
  int gcur = 0;  // gst + (gcur * s + r) * S holds G_r
  for (int q = NS - 1; q >= 0; --q) {
    const int a = q * m.nmax, n = (int)std::min<int64_t>(m.nmax, m.L - a);
    const int rows = (int)(m.B * n);
    const size_t hf = (size_t)m.B * k * n * kHead;
    const slim_problem p = att_problem(m, n);
    // recompute the slice, each layer's state before the slice by eq. 17
    hipLaunchKernelGGL(embed_kernel, dim3((unsigned)rows), dim3(256), 0, s, tokens, m.L, a, n, P.emb, D, V, Xr(0));
    for (int r = 0; r < m.s; ++r) {
      CHECK_SLIM(layer_qkv(r, n));
      CHECK_SLIM(slim_fwd(&p, Qhr(r, 0), Qhr(r, 1), Qhr(r, 2), ident, nullptr, nullptr, Yh, delta, nullptr, nullptr,
                          attws, lay.attws_bytes, s));
      hipLaunchKernelGGL(sub_kernel, grid1(S), dim3(256), 0, s, bprev + r * S, states + r * S, delta, S);
      CHECK_HIP(hipGetLastError());
      CHECK_SLIM(layer_fwd(r, a, n, bprev + r * S, snew));
    }
    CHECK_SLIM(head_logits(a, n));
    // output layer
    CHECK_HIP(gemm(true, false, D, V, rows, 1.f, Xr(m.s), D, logits, V, 1.f, G.Wout, V, s));
    hipLaunchKernelGGL(colsum_kernel, grid1(V), dim3(256), 0, s, logits, rows, V, G.bout);
    CHECK_HIP(gemm(false, true, rows, D, V, 1.f, logits, V, P.Wout, V, 0.f, dX, D, s));
    for (int r = m.s - 1; r >= 0; --r) {
      const Params::Layer& pl = P.l[r];
      const Grads::Layer& gl = G.l[r];
      // X_{r+1} = LN2(Fo) + H
      hipLaunchKernelGGL(ln_bwd_kernel, dim3(rows), dim3(256), 0, s, For(r), s2r(r), pl.g2, dX, nullptr, dF, Pp, D);
      hipLaunchKernelGGL(colsum_kernel, grid1(D), dim3(256), 0, s, Pp, rows, D, gl.g2);
      hipLaunchKernelGGL(colsum_kernel, grid1(D), dim3(256), 0, s, dX, rows, D, gl.b2n);
      // Fo = GeLU(Z1) W2 + b2
      CHECK_HIP(gemm(true, false, F, D, rows, 1.f, G1r(r), F, dF, D, 1.f, gl.W2, D, s));
      hipLaunchKernelGGL(colsum_kernel, grid1(D), dim3(256), 0, s, dF, rows, D, gl.b2);
      CHECK_HIP(gemm(false, true, rows, F, D, 1.f, dF, D, pl.W2, D, 0.f, dG1, F, s));
      hipLaunchKernelGGL(gelu_bwd_kernel, grid1((size_t)rows * F), dim3(256), 0, s, dG1, Z1r(r), (size_t)rows * F);
      // Z1 = H W1 + b1; dH = dX (residual) + dZ1 W1^T
      CHECK_HIP(gemm(true, false, D, F, rows, 1.f, Hr(r), D, dG1, F, 1.f, gl.W1, F, s));
      hipLaunchKernelGGL(colsum_kernel, grid1(F), dim3(256), 0, s, dG1, rows, F, gl.b1);
      hipLaunchKernelGGL(copy_kernel, grid1((size_t)rows * D), dim3(256), 0, s, dH, dX, (size_t)rows * D);
      CHECK_HIP(gemm(false, true, rows, D, F, 1.f, dG1, F, pl.W1, F, 1.f, dH, D, s));
      // H = LN1(A) + X
      hipLaunchKernelGGL(ln_bwd_kernel, dim3(rows), dim3(256), 0, s, Ar(r), s1r(r), pl.g1, dH, nullptr, dA, Pp, D);
      hipLaunchKernelGGL(colsum_kernel, grid1(D), dim3(256), 0, s, Pp, rows, D, gl.g1);
      hipLaunchKernelGGL(colsum_kernel, grid1(D), dim3(256), 0, s, dH, rows, D, gl.b1n);
      CHECK_HIP(hipGetLastError());
      // attention: the slice's gradient with the state cotangent after it
      // (eq. 18 gives the one before it)
      hipLaunchKernelGGL(rows_to_heads_kernel, grid1(hf), dim3(256), 0, s, dA, D, 0, dYh, k, n, hf);
      float* gin = gst + ((size_t)gcur * m.s + r) * S;
      float* gout = gst + ((size_t)(1 - gcur) * m.s + r) * S;
      CHECK_SLIM(slim_bwd(&p, Qhr(r, 0), Qhr(r, 1), Qhr(r, 2), ident, bprev + r * S, nullptr, nullptr, dYh, gin, dQh,
                          dQh + hf, dQh + 2 * hf, wd, gout, nullptr, attws, lay.attws_bytes, s));
      for (int part = 0; part < 3; ++part)
        hipLaunchKernelGGL(heads_to_rows_kernel, grid1(hf), dim3(256), 0, s, dQh + part * hf, dQKV, 3 * D, part * D, k, n,
                           hf);
      CHECK_HIP(hipGetLastError());
      // Q, K, V = X Wq, X Wk, X Wv; dX = dH + sum dZ W^T
      const float* X = Xr(r);
      CHECK_HIP(gemm(true, false, D, D, rows, 1.f, X, D, dQKV, 3 * D, 1.f, gl.Wq, D, s));
      CHECK_HIP(gemm(true, false, D, D, rows, 1.f, X, D, dQKV + D, 3 * D, 1.f, gl.Wk, D, s));
      CHECK_HIP(gemm(true, false, D, D, rows, 1.f, X, D, dQKV + 2 * D, 3 * D, 1.f, gl.Wv, D, s));
      hipLaunchKernelGGL(copy_kernel, grid1((size_t)rows * D), dim3(256), 0, s, dX, dH, (size_t)rows * D);
      CHECK_HIP(gemm(false, true, rows, D, D, 1.f, dQKV, 3 * D, pl.Wq, D, 1.f, dX, D, s));
      CHECK_HIP(gemm(false, true, rows, D, D, 1.f, dQKV + D, 3 * D, pl.Wk, D, 1.f, dX, D, s));
      CHECK_HIP(gemm(false, true, rows, D, D, 1.f, dQKV + 2 * D, 3 * D, pl.Wv, D, 1.f, dX, D, s));
    }
    hipLaunchKernelGGL(embed_bwd_kernel, dim3(V, (D + 255) / 256), dim3(256), 0, s, tokens, m.L, a, n, rows, dX, D, G.emb);
    // the states before this slice become the states after the earlier one
    hipLaunchKernelGGL(copy_kernel, grid1(m.s * S), dim3(256), 0, s, states, bprev, (size_t)m.s * S);
    CHECK_HIP(hipGetLastError());
    gcur = 1 - gcur;
  }
  return report(SLIM_OK, "");
}

}  // namespace model
}  // namespace slim

extern "C" {

int slim_model_num_params(const slim_model* m) { return m == nullptr ? 0 : 11 * m->s + 3; }

size_t slim_model_workspace_bytes(const slim_model* mm) {
  slim::model::Dims m;
  if (slim::model::check(mm, &m) != SLIM_OK) return 0;
  return slim::model::layout(m).total;
}

int slim_model_step(const slim_model* mm, const int32_t* tokens, const float* const* params, float* const* grads,
                    float* loss, void* ws, size_t ws_bytes, void* stream) {
  slim::model::Dims m;
  int st = slim::model::check(mm, &m);
  if (st != SLIM_OK) return st;
  if (tokens == nullptr || params == nullptr || grads == nullptr || loss == nullptr)
    return slim::report(SLIM_EINVAL, "tokens, params, grads and loss must be non-NULL");
  const int np = 11 * m.s + 3;
  for (int i = 0; i < np; ++i)
    if (params[i] == nullptr || grads[i] == nullptr) return slim::report(SLIM_EINVAL, "a parameter or gradient pointer is NULL");
  const size_t need = slim::model::layout(m).total;
  if (ws == nullptr || ws_bytes < need) return slim::report(SLIM_EWORKSPACE, "model workspace too small");
  if (((uintptr_t)ws & 255) != 0) return slim::report(SLIM_EINVAL, "the workspace must be 256-byte aligned");
  slim::model::Params P;
  slim::model::Grads G;
  slim::model::unpack(P, params, m.s);
  slim::model::unpack(G, grads, m.s);
  return slim::model::step(m, (const int*)tokens, P, G, loss, (char*)ws, (hipStream_t)stream);
}

}  // extern "C"
