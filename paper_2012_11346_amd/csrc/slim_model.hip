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
// Kernels here: a float32 matrix-core GEMM (v_mfma_f32_16x16x4_f32, 128 x 128
// and 64 x 128 tiles, split K with a fixed-order reduction, epilogues for
// bias, bias + GeLU, GeLU's derivative and residual sums), row-wise layer
// normalisation and its backward, cross-entropy, the embedding and its
// deterministic backward, head split/merge copies and fixed-order column
// sums.
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

__device__ __forceinline__ float gelu_f(float x) { return 0.5f * x * (1.f + erff(x * 0.70710678118654752f)); }
__device__ __forceinline__ float gelu_d(float x) {
  return 0.5f * (1.f + erff(x * 0.70710678118654752f)) + x * expf(-0.5f * x * x) * 0.39894228040143268f;
}

// ---------------------------------------------------------------- GEMM
// C = epilogue(op(A) op(B)), row-major: op(A)[m][k] = TA ? A[k lda + m] :
// A[m lda + k], op(B)[k][n] = TB ? B[n ldb + k] : B[k ldb + n].
//
// Workgroup tile BM x 128 (BM = 128 or 64), four waves in 2 x 2, each wave
// (BM / 2) x 64 as (BM / 32) x 4 matrix tiles of 16 x 16 on
// v_mfma_f32_16x16x4_f32.  K runs in tiles of 16 through double-buffered
// LDS.  The summation index of the four products of one k tile is permuted
// so that lane group g (lane / 16) takes k = 4 g + j in product j.  An
// operand whose rows run along k in memory is held [m][k] (rows padded to 20
// floats): one 16-byte LDS read feeds a lane's four products.  An operand
// whose rows run along m (or n) is held as it is in memory, [k][m] (rows
// padded by 4 floats, so the four k rows a read touches fall in different
// banks), and a lane reads its four values one by one.  Either way the
// global tile lands in LDS with 16-byte writes.  Global loads are 16-byte
// vectors where the strides allow, prefetched one k tile ahead.  Long K is split over blockIdx.y; the
// partial products are summed in a fixed order by gemm_reduce_kernel, which
// then applies the epilogue (no atomics: results are reproducible).
constexpr int GBN = 128, GBK = 16, GKP = GBK + 4;

enum EpiOp { EPI_STORE = 0, EPI_ACC = 1, EPI_BIAS = 2, EPI_BIAS_GELU = 3, EPI_GELU_BWD = 4, EPI_ADD = 5 };
// STORE: C = v; ACC: C += v; BIAS: C = v + bias[n]; BIAS_GELU: C = z = v +
// bias[n], C2 = GeLU(z); GELU_BWD: C = v GeLU'(aux); ADD: C = v + aux.
// aux and C2 share C's leading dimension.
// Where C lives: one row-major matrix (layout 0); or the columns cut into
// groups of gcols, group g a row-major matrix of its own at Cg[g] (layout 1),
// or a [B][heads][hrows][64] head-split tensor at Cg[g] for row m = b hrows +
// t, column h 64 + c of the group (layout 2).  bias, aux and C2 serve layout 0.
struct Epi {
  int op;
  const float* bias;
  const float* aux;
  float* C2;
  int layout, gcols, hrows, heads;
  float *Cg0, *Cg1, *Cg2;  // separate members: an indexed array would go to scratch
};

// group of column (or row) i for groups of g: 0, 1 or 2 (selects, no divide)
__device__ __forceinline__ int group3(int i, int g) { return (i >= g) + (i >= 2 * g); }
template <typename T>
__device__ __forceinline__ T pick3(int grp, T a, T b, T c) {
  return grp == 0 ? a : (grp == 1 ? b : c);
}

// The epilogue's operation on element o of C (n: the column, for the bias),
// split into its read (C for EPI_ACC, the bias, aux) and its write, so that
// a tile's reads can all be issued before its first store (interleaved,
// each store might alias the next read and they would run one at a time).
__device__ __forceinline__ float epi_read(const Epi& e, const float* C, size_t o, int n) {
  switch (e.op) {
    case EPI_STORE: return 0.f;
    case EPI_ACC: return C[o];
    case EPI_BIAS:
    case EPI_BIAS_GELU: return e.bias[n];
    default: return e.aux[o];
  }
}
__device__ __forceinline__ void epi_write(const Epi& e, float* C, size_t o, float v, float x) {
  switch (e.op) {
    case EPI_STORE: C[o] = v; break;
    case EPI_ACC: C[o] = x + v; break;
    case EPI_BIAS: C[o] = v + x; break;
    case EPI_BIAS_GELU: {
      const float z = v + x;
      C[o] = z;
      e.C2[o] = gelu_f(z);
      break;
    }
    case EPI_GELU_BWD: C[o] = v * gelu_d(x); break;
    default: C[o] = v + x; break;
  }
}
__device__ __forceinline__ void epi_op(const Epi& e, float* C, size_t o, int n, float v) {
  epi_write(e, C, o, v, epi_read(e, C, o, n));
}
// where element (m, n) of the product goes: its matrix (C or a group's) and
// the offset in it; the row's and the column's parts of the offset add
__device__ __forceinline__ size_t epi_row(const Epi& e, int ldc, int m) {
  if (e.layout == 2) {
    const int b = m / e.hrows, t = m - b * e.hrows;
    return ((size_t)b * e.heads * e.hrows + t) * 64;
  }
  return (size_t)m * ldc;
}
__device__ __forceinline__ size_t epi_col(const Epi& e, float*& C, int n) {
  if (e.layout == 0) return n;
  const int grp = group3(n, e.gcols), col = n - grp * e.gcols;
  C = pick3(grp, e.Cg0, e.Cg1, e.Cg2);
  return e.layout == 1 ? (size_t)col : (size_t)(col >> 6) * e.hrows * 64 + (col & 63);
}
__device__ __forceinline__ void epi_store(const Epi& e, float* C, int ldc, int m, int n, float v) {
  const size_t ro = epi_row(e, ldc, m);
  const size_t co = epi_col(e, C, n);
  epi_op(e, C, ro + co, n, v);
}

struct GemmArgs {
  int M, N, K;
  const float* A;
  int lda;
  const float* B;
  int ldb;
  float* C;
  int ldc;
  Epi epi;
  int kchunk;   // k per split (a multiple of GBK)
  float* part;  // [splits][M][N] partial products when gridDim.y > 1
  int tiles_n;
  // grouped B (gN > 0: columns of op(B) in groups of gN, group g at Bg[g],
  // each with leading dimension ldb; gK > 0: rows of op(B) in groups of gK,
  // a multiple of GBK, likewise)
  const float *Bg0, *Bg1, *Bg2;
  int gN, gK;
};

// four consecutive floats, `avail` of them valid (zeros beyond)
template <bool VEC>
__device__ __forceinline__ float4 ld4(const float* p, int avail) {
  if (VEC && avail >= 4) return *reinterpret_cast<const float4*>(p);
  float4 r = make_float4(0.f, 0.f, 0.f, 0.f);
  if (avail > 0) r.x = p[0];
  if (avail > 1) r.y = p[1];
  if (avail > 2) r.z = p[2];
  if (avail > 3) r.w = p[3];
  return r;
}

// GRP: grouped B and grouped / head-split C (the kernels without it carry no
// code, and no registers, for either)
template <int BM, int BN, bool TA, bool TB, bool VEC, bool GRP>
__global__ __launch_bounds__(256) void gemm_kernel(GemmArgs g) {
  constexpr int AV = BM * GBK / 4 / 256;  // float4 loads per thread per k tile (A)
  constexpr int BV = BN * GBK / 4 / 256;  // (B)
  constexpr int TI = BM / 32;             // matrix tiles per wave along m
  constexpr int TJ = BN / 32;             // and along n
  // [m][k] (k-contiguous source) or [k][m] (m-contiguous source) per buffer
  constexpr int ALD = TA ? BM + 4 : GKP, BLD = TB ? GKP : BN + 4;
  constexpr int ASZ = TA ? GBK * ALD : BM * ALD, BSZ = TB ? BN * BLD : GBK * BLD;
  __shared__ __align__(16) float As[2][ASZ];
  __shared__ __align__(16) float Bs[2][BSZ];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  // XCD-aware order: consecutive tiles (sharing rows of A) on one XCD
  int tile = blockIdx.x;
  const int nt = gridDim.x;
  if ((nt & 7) == 0) tile = (tile & 7) * (nt >> 3) + (tile >> 3);
  const int m0 = (tile / g.tiles_n) * BM, n0 = (tile % g.tiles_n) * BN;
  const int kbeg = blockIdx.y * g.kchunk, kend = min(g.K, kbeg + g.kchunk);
  const int wm = (w >> 1) * (BM / 2), wn = (w & 1) * (BN / 2);
  const int M = g.M, N = g.N;

  // grouped B along n: each thread's columns are the same in every k tile,
  // so its group's base pointer is fixed before the loop
  const float* bcol[BV];
#pragma unroll
  for (int i = 0; i < BV; ++i) {
    const int n = n0 + 4 * ((tid + 256 * i) % (BN / 4));
    bcol[i] = g.B + n;
    if (GRP && !TB && g.gN > 0 && n < N) {
      const int grp = group3(n, g.gN);
      bcol[i] = pick3(grp, g.Bg0, g.Bg1, g.Bg2) + (n - grp * g.gN);
    }
  }

  float4 ra[AV], rb[BV];
  auto load = [&](int k0) {
#pragma unroll
    for (int i = 0; i < AV; ++i) {
      const int f = tid + 256 * i;
      if (!TA) {  // rows of A: 4 k per vector
        const int m = f >> 2, k = k0 + 4 * (f & 3);
        ra[i] = (m0 + m < M) ? ld4<VEC>(g.A + (size_t)(m0 + m) * g.lda + k, kend - k) : make_float4(0.f, 0.f, 0.f, 0.f);
      } else {  // rows of A^T: 4 m per vector
        const int k = k0 + f / (BM / 4), m = m0 + 4 * (f % (BM / 4));
        ra[i] = (k < kend) ? ld4<VEC>(g.A + (size_t)k * g.lda + m, M - m) : make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
#pragma unroll
    for (int i = 0; i < BV; ++i) {
      const int f = tid + 256 * i;
      if (TB) {  // rows of B^T: 4 k per vector
        const int n = f >> 2, k = k0 + 4 * (f & 3);
        const float* Bb = g.B;
        int kk = k;
        if (GRP && g.gK > 0) {  // the k tile lies in one group (k0 is uniform)
          const int grp = group3(k0, g.gK);
          Bb = pick3(grp, g.Bg0, g.Bg1, g.Bg2);
          kk = k - grp * g.gK;
        }
        rb[i] = (n0 + n < N) ? ld4<VEC>(Bb + (size_t)(n0 + n) * g.ldb + kk, kend - k) : make_float4(0.f, 0.f, 0.f, 0.f);
      } else {  // rows of B: 4 n per vector
        const int k = k0 + f / (BN / 4), n = n0 + 4 * (f % (BN / 4));
        rb[i] = (k < kend) ? ld4<VEC>(bcol[i] + (size_t)k * g.ldb, N - n) : make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int i = 0; i < AV; ++i) {
      const int f = tid + 256 * i;
      const int at = TA ? (f / (BM / 4)) * ALD + 4 * (f % (BM / 4)) : (f >> 2) * ALD + 4 * (f & 3);
      *reinterpret_cast<float4*>(&As[buf][at]) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < BV; ++i) {
      const int f = tid + 256 * i;
      const int at = TB ? (f >> 2) * BLD + 4 * (f & 3) : (f / (BN / 4)) * BLD + 4 * (f % (BN / 4));
      *reinterpret_cast<float4*>(&Bs[buf][at]) = rb[i];
    }
  };

  f4 acc[TI][TJ];
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
  const int c = lane & 15, q = lane >> 4;
  int buf = 0;
  if (kbeg < kend) {
    load(kbeg);
    store(0);
  }
  __syncthreads();
  for (int k0 = kbeg; k0 < kend; k0 += GBK) {
    const bool more = k0 + GBK < kend;
    if (more) load(k0 + GBK);
    float4 a[TI], b[TJ];
#pragma unroll
    for (int i = 0; i < TI; ++i) {
      if (TA) {
        const float* p = &As[buf][4 * q * ALD + wm + 16 * i + c];
        a[i] = make_float4(p[0], p[ALD], p[2 * ALD], p[3 * ALD]);
      } else {
        a[i] = *reinterpret_cast<const float4*>(&As[buf][(wm + 16 * i + c) * ALD + 4 * q]);
      }
    }
#pragma unroll
    for (int j = 0; j < TJ; ++j) {
      if (TB) {
        b[j] = *reinterpret_cast<const float4*>(&Bs[buf][(wn + 16 * j + c) * BLD + 4 * q]);
      } else {
        const float* p = &Bs[buf][4 * q * BLD + wn + 16 * j + c];
        b[j] = make_float4(p[0], p[BLD], p[2 * BLD], p[3 * BLD]);
      }
    }
    // each accumulator's four products are TI * 4 issues apart
#pragma unroll
    for (int i = 0; i < TI; ++i)
#pragma unroll
      for (int j = 0; j < TJ; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i].x, b[j].x, acc[i][j], 0, 0, 0);
#pragma unroll
    for (int i = 0; i < TI; ++i)
#pragma unroll
      for (int j = 0; j < TJ; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i].y, b[j].y, acc[i][j], 0, 0, 0);
#pragma unroll
    for (int i = 0; i < TI; ++i)
#pragma unroll
      for (int j = 0; j < TJ; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i].z, b[j].z, acc[i][j], 0, 0, 0);
#pragma unroll
    for (int i = 0; i < TI; ++i)
#pragma unroll
      for (int j = 0; j < TJ; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i].w, b[j].w, acc[i][j], 0, 0, 0);
    if (more) store(buf ^ 1);
    __syncthreads();
    buf ^= 1;
  }
  const bool split = gridDim.y > 1;
  if (GRP && !split) {
    // the tile's row offsets once, in LDS (the operand buffers are free
    // after the loop's last barrier), the column offsets once per j
    size_t* rowoff = reinterpret_cast<size_t*>(&As[0][0]);
    for (int i = tid; i < BM; i += 256) rowoff[i] = epi_row(g.epi, g.ldc, min(m0 + i, M - 1));
    __syncthreads();
    // (per 16 x 32 block: its reads, then its writes; the column offsets are
    // recomputed per block rather than held)
#pragma unroll
    for (int i = 0; i < TI; ++i)
#pragma unroll
      for (int j2 = 0; j2 < TJ; j2 += 2) {
        float x[2][4];
#pragma unroll
        for (int jj = 0; jj < 2; ++jj) {
          const int n = n0 + wn + 16 * (j2 + jj) + c;
          float* Cj = g.C;
          const size_t co = epi_col(g.epi, Cj, min(n, N - 1));
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int mm = wm + 16 * i + 4 * q + r;
            x[jj][r] = (m0 + mm < M && n < N) ? epi_read(g.epi, Cj, rowoff[mm] + co, n) : 0.f;
          }
        }
#pragma unroll
        for (int jj = 0; jj < 2; ++jj) {
          const int n = n0 + wn + 16 * (j2 + jj) + c;
          float* Cj = g.C;
          const size_t co = epi_col(g.epi, Cj, min(n, N - 1));
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int mm = wm + 16 * i + 4 * q + r;
            if (m0 + mm < M && n < N) epi_write(g.epi, Cj, rowoff[mm] + co, acc[i][j2 + jj][r], x[jj][r]);
          }
        }
      }
    return;
  }
  if (split) {
    float* part = g.part + (size_t)blockIdx.y * M * N;
#pragma unroll
    for (int i = 0; i < TI; ++i)
#pragma unroll
      for (int j = 0; j < TJ; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = m0 + wm + 16 * i + 4 * q + r, n = n0 + wn + 16 * j + c;
          if (m < M && n < N) part[(size_t)m * N + n] = acc[i][j][r];
        }
    return;
  }
  // the epilogue's reads first, then its writes: all of a lane's with the
  // 64-row tile, per 16-row block with the 128-row one (registers)
  constexpr int IB = TI <= 2 ? TI : 1;
#pragma unroll
  for (int i0 = 0; i0 < TI; i0 += IB) {
    float x[IB][TJ][4];
#pragma unroll
    for (int ii = 0; ii < IB; ++ii)
#pragma unroll
      for (int j = 0; j < TJ; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = m0 + wm + 16 * (i0 + ii) + 4 * q + r, n = n0 + wn + 16 * j + c;
          x[ii][j][r] = (m < M && n < N) ? epi_read(g.epi, g.C, (size_t)m * g.ldc + n, n) : 0.f;
        }
#pragma unroll
    for (int ii = 0; ii < IB; ++ii)
#pragma unroll
      for (int j = 0; j < TJ; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = m0 + wm + 16 * (i0 + ii) + 4 * q + r, n = n0 + wn + 16 * j + c;
          if (m < M && n < N) epi_write(g.epi, g.C, (size_t)m * g.ldc + n, acc[i0 + ii][j][r], x[ii][j][r]);
        }
  }
}

// C = epilogue(sum over splits of the partial products, in split order)
__global__ __launch_bounds__(256) void gemm_reduce_kernel(const float* part, int splits, int M, int N, float* C, int ldc,
                                                          Epi epi) {
  const size_t e = (size_t)blockIdx.x * 256 + threadIdx.x, MN = (size_t)M * N;
  if (e >= MN) return;
  // (eight, then four partials loaded at a time, added in split order)
  float v = 0.f;
  int s = 0;
  for (; s + 8 <= splits; s += 8) {
    float q[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) q[i] = part[(s + i) * MN + e];
#pragma unroll
    for (int i = 0; i < 8; ++i) v += q[i];
  }
  for (; s + 4 <= splits; s += 4) {
    const float p0 = part[s * MN + e], p1 = part[(s + 1) * MN + e], p2 = part[(s + 2) * MN + e],
                p3 = part[(s + 3) * MN + e];
    v = (((v + p0) + p1) + p2) + p3;
  }
  for (; s < splits; ++s) v += part[s * MN + e];
  epi_store(epi, C, ldc, (int)(e / N), (int)(e % N), v);
}

// Launch plan of one product: tile height, k per split and split count.
struct GemmPlan {
  int BM, BN, kchunk, splits, tiles_n, tiles;
};
inline GemmPlan gemm_plan(int M, int N, int K) {
  const int kt = (K + GBK - 1) / GBK;
  const int t128 = ((M + 127) / 128) * ((N + GBN - 1) / GBN);
  auto plan = [&](int BN) {
    GemmPlan p;
    // (a short reduction leaves the epilogue's reads and writes of C to set
    // the pace: the smaller tile gives twice the workgroups in flight)
    p.BM = (t128 >= 256 && kt > 8) ? 128 : 64;
    p.BN = BN;
    p.tiles_n = (N + BN - 1) / BN;
    p.tiles = ((M + p.BM - 1) / p.BM) * p.tiles_n;
    int s = 1;
    // split long K until about 512 workgroups run, keeping >= 8 k tiles each
    while (p.tiles * s < 512 && kt >= 16 * s && s < 64) s *= 2;  // next split keeps >= 8 k tiles
    const int per = std::max(1, (kt + s - 1) / s);
    p.kchunk = per * GBK;
    p.splits = (kt + per - 1) / per;
    return p;
  };
  const GemmPlan p = plan(GBN);
  // fewer workgroups than the split aims for (a short row count, or a
  // reduction too short to split further): 64-column tiles double them
  // (64-row tiles; 128-row ones only come with at least 256 tiles)
  if (p.BM == 64 && p.tiles * p.splits < 512) return plan(64);
  return p;
}
inline size_t gemm_part_bytes(int M, int N, int K) {
  const GemmPlan p = gemm_plan(M, N, K);
  return p.splits > 1 ? (size_t)p.splits * M * N * sizeof(float) : 0;
}

template <int BM, int BN, bool TA, bool TB, bool GRP>
void gemm_launch(const GemmArgs& a, dim3 grid, bool vec, hipStream_t s) {
  if (vec) hipLaunchKernelGGL((gemm_kernel<BM, BN, TA, TB, true, GRP>), grid, dim3(256), 0, s, a);
  else hipLaunchKernelGGL((gemm_kernel<BM, BN, TA, TB, false, GRP>), grid, dim3(256), 0, s, a);
}
template <int BM, int BN, bool GRP>
void gemm_launch(bool ta, bool tb, const GemmArgs& a, dim3 grid, bool vec, hipStream_t s) {
  if (ta && tb) gemm_launch<BM, BN, true, true, GRP>(a, grid, vec, s);
  else if (ta) gemm_launch<BM, BN, true, false, GRP>(a, grid, vec, s);
  else if (tb) gemm_launch<BM, BN, false, true, GRP>(a, grid, vec, s);
  else gemm_launch<BM, BN, false, false, GRP>(a, grid, vec, s);
}

// part: workspace for the partial products (gemm_part_bytes of the shape);
// grp: grouped B (Bg, gN, gK of GemmArgs), or nullptr
struct GroupB {
  const float* Bg[3];
  int gN, gK;
};
hipError_t gemm(bool ta, bool tb, int M, int N, int K, const float* A, int lda, const float* B, int ldb, float* C,
                int ldc, Epi epi, float* part, hipStream_t s, const GroupB* grp = nullptr) {
  if (M <= 0 || N <= 0) return hipSuccess;
  const GemmPlan p = gemm_plan(M, N, K);
  GemmArgs a;
  a.M = M;
  a.N = N;
  a.K = K;
  a.A = A;
  a.lda = lda;
  a.B = B;
  a.ldb = ldb;
  a.C = C;
  a.ldc = ldc;
  a.epi = epi;
  a.kchunk = p.kchunk;
  a.part = part;
  a.tiles_n = p.tiles_n;
  a.gN = a.gK = 0;
  a.Bg0 = a.Bg1 = a.Bg2 = nullptr;
  bool bal = ((uintptr_t)B & 15) == 0;
  if (grp != nullptr) {
    // a float4 of B, or a k tile, must not straddle two groups
    if (grp->gN % 4 != 0 || grp->gK % GBK != 0) return hipErrorInvalidValue;
    a.gN = grp->gN;
    a.gK = grp->gK;
    a.Bg0 = grp->Bg[0];
    a.Bg1 = grp->Bg[1];
    a.Bg2 = grp->Bg[2];
    for (int i = 0; i < 3; ++i) bal = bal && ((uintptr_t)grp->Bg[i] & 15) == 0;
  }
  const bool vec = lda % 4 == 0 && ldb % 4 == 0 && ((uintptr_t)A & 15) == 0 && bal;
  const dim3 grid(p.tiles, p.splits);
  const bool grouped = a.gN > 0 || a.gK > 0 || epi.layout != 0;
  // (128-row tiles only come with 128-column ones: they need 256 tiles)
  if (p.BM == 128) {
    if (grouped) gemm_launch<128, 128, true>(ta, tb, a, grid, vec, s);
    else gemm_launch<128, 128, false>(ta, tb, a, grid, vec, s);
  } else if (p.BN == 128) {
    if (grouped) gemm_launch<64, 128, true>(ta, tb, a, grid, vec, s);
    else gemm_launch<64, 128, false>(ta, tb, a, grid, vec, s);
  } else {
    if (grouped) gemm_launch<64, 64, true>(ta, tb, a, grid, vec, s);
    else gemm_launch<64, 64, false>(ta, tb, a, grid, vec, s);
  }
  if (p.splits > 1) {
    const size_t MN = (size_t)M * N;
    hipLaunchKernelGGL(gemm_reduce_kernel, dim3((unsigned)((MN + 255) / 256)), dim3(256), 0, s, part, p.splits, M, N, C,
                       ldc, epi);
  }
  return hipGetLastError();
}

inline Epi epi(int op, const float* bias = nullptr, const float* aux = nullptr, float* C2 = nullptr) {
  Epi e;
  std::memset(&e, 0, sizeof(e));
  e.op = op;
  e.bias = bias;
  e.aux = aux;
  e.C2 = C2;
  return e;
}
// C in column groups of gcols: row-major matrices (ldc of the call), or
// head-split tensors of hrows rows and `heads` heads
inline Epi epi_groups(int op, float* C0, float* C1, float* C2_, int gcols, int hrows = 0, int heads = 0) {
  Epi e = epi(op);
  e.layout = hrows > 0 ? 2 : 1;
  e.gcols = gcols;
  e.hrows = hrows;
  e.heads = heads;
  e.Cg0 = C0;
  e.Cg1 = C1;
  e.Cg2 = C2_;
  return e;
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

// Column sums in a fixed order.  A workgroup takes 64 columns; its four
// waves take interleaved quarters of the rows (wave q: rows q, q + 4, ...
// of the range, eight loads in flight per lane), and the four partial sums
// are added in wave order through LDS.  One stage when the rows fit one
// chunk of 64 (out_z[j] += the sum); else part[z][c][j] = the sum of chunk c
// and a second stage adds the chunks the same way (wave q: chunks q, q + 4,
// ...).  z selects one of two independent sums.
constexpr int kColChunk = 64;
struct ColsumArgs {
  const float* src[2];
  float* out[2];
};
// sum of rows r0, r0 + 4, r0 + 8, ... < r1 of column j (stride n), in order
__device__ __forceinline__ float colsum_strided(const float* src, int r0, int r1, size_t n, int j) {
  float s = 0.f;
  int r = r0;
  for (; r + 28 < r1; r += 32) {
    float v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = src[(size_t)(r + 4 * k) * n + j];
#pragma unroll
    for (int k = 0; k < 8; ++k) s += v[k];
  }
  for (; r < r1; r += 4) s += src[(size_t)r * n + j];
  return s;
}
// the four waves' sums of each column, added in wave order
__device__ __forceinline__ float colsum_waves(float v, float (*red)[64], int q, int jj) {
  red[q][jj] = v;
  __syncthreads();
  return ((red[0][jj] + red[1][jj]) + red[2][jj]) + red[3][jj];
}
__global__ __launch_bounds__(256) void colsum_part_kernel(ColsumArgs a, int rows, int n, float* part) {
  __shared__ float red[4][64];
  const int q = threadIdx.x >> 6, jj = threadIdx.x & 63;
  const int j = blockIdx.x * 64 + jj, c = blockIdx.y, z = blockIdx.z;
  const int r1 = min(rows, (c + 1) * kColChunk);
  const float v = j < n ? colsum_strided(a.src[z], c * kColChunk + q, r1, n, j) : 0.f;
  const float t = colsum_waves(v, red, q, jj);
  if (q == 0 && j < n) {
    if (gridDim.y == 1) a.out[z][j] += t;  // one chunk: the sum itself
    else part[((size_t)z * gridDim.y + c) * n + j] = t;
  }
}
__global__ __launch_bounds__(256) void colsum_final_kernel(ColsumArgs a, int chunks, int n, const float* part) {
  __shared__ float red[4][64];
  const int q = threadIdx.x >> 6, jj = threadIdx.x & 63;
  const int j = blockIdx.x * 64 + jj, z = blockIdx.y;
  const float v = j < n ? colsum_strided(part + (size_t)z * chunks * n, q, chunks, n, j) : 0.f;
  const float t = colsum_waves(v, red, q, jj);
  if (q == 0 && j < n) a.out[z][j] += t;
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
// parts consecutive head tensors of `per` floats each: part p goes to the
// columns from col0 + p colstep
__global__ __launch_bounds__(256) void heads_to_rows_kernel(const float* src, float* dst, int ld, int col0, int colstep,
                                                            int k, int n, size_t per, size_t total) {
  const size_t e = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= total) return;
  const int p = (int)(e / per);
  const size_t ep = e - (size_t)p * per;
  const int c = (int)(ep % kHead);
  size_t r = ep / kHead;
  const int t = (int)(r % n);
  r /= n;
  const int h = (int)(r % k);
  const int b = (int)(r / k);
  dst[((size_t)b * n + t) * ld + col0 + p * colstep + h * kHead + c] = src[e];
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
  size_t X, Qh, Yh, A, st1, H, Z1, G1, Fo, st2;
  size_t logits, rowloss, dX, dH, dF, dG1, dA, dYh, dQh, dQKV, P, part, part_bytes, red;
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
  // split-K partial products: the largest over the step's products, for
  // the full slice and the ragged last one
  size_t pb = 0;
  for (int n : {m.nmax, last}) {
    const int rows = (int)(m.B * n), d = m.D, f = m.F, v = m.V;
    const int shapes[][3] = {{rows, 3 * d, d}, {rows, f, d}, {rows, d, f}, {rows, v, d}, {rows, d, v},
                             {d, v, rows}, {f, d, rows}, {d, f, rows}, {d, 3 * d, rows}, {rows, d, 3 * d}};
    for (const auto& sh : shapes) pb = std::max(pb, gemm_part_bytes(sh[0], sh[1], sh[2]));
  }
  l.part_bytes = pb;
  take(l.part, std::max<size_t>(pb, 256));
  take(l.red, 2 * ((R + kColChunk - 1) / kColChunk) * std::max(D, std::max(F, (size_t)m.V)) * 4);
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
  // (rows of a slice: the column sums run one workgroup row per 64 rows, at most 65535 of them)
  if ((int64_t)m.B * m.nmax > (int64_t)65535 * kColChunk || m.L > ((int64_t)1 << 30) || m.B * m.L > ((int64_t)1 << 31) - 1)
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
  float* Yh = f(lay.Yh);
  float* logits = f(lay.logits);
  float* rowloss = f(lay.rowloss);
  float *dX = f(lay.dX), *dH = f(lay.dH), *dF = f(lay.dF), *dG1 = f(lay.dG1), *dA = f(lay.dA);
  float *dYh = f(lay.dYh), *dQh = f(lay.dQh), *dQKV = f(lay.dQKV), *Pp = f(lay.P);
  float* part = f(lay.part);
  float* red = f(lay.red);
  auto mm = [&](bool ta, bool tb, int M_, int N_, int K_, const float* A_, int lda, const float* B_, int ldb, float* C_,
                int ldc, Epi e, const GroupB* grp = nullptr) {
    return gemm(ta, tb, M_, N_, K_, A_, lda, B_, ldb, C_, ldc, e, part, s, grp);
  };
  // the three projection weights of layer r as one operand: columns (or
  // rows) D g .. D g + D - 1 of the grouped operand are those of Wq, Wk, Wv
  auto wqkv = [&](const float* Wq, const float* Wk, const float* Wv, bool along_k) {
    GroupB gb;
    gb.Bg[0] = Wq;
    gb.Bg[1] = Wk;
    gb.Bg[2] = Wv;
    gb.gN = along_k ? 0 : D;
    gb.gK = along_k ? D : 0;
    return gb;
  };
  // out0 += column sums of src0 (and out1 += those of src1), rows in order
  auto colsum = [&](int rows, int n, const float* src0, float* out0, const float* src1 = nullptr,
                    float* out1 = nullptr) {
    ColsumArgs ca;
    ca.src[0] = src0;
    ca.out[0] = out0;
    ca.src[1] = src1;
    ca.out[1] = out1;
    const int nz = src1 ? 2 : 1, chunks = (rows + kColChunk - 1) / kColChunk;
    hipLaunchKernelGGL(colsum_part_kernel, dim3((n + 63) / 64, chunks, nz), dim3(256), 0, s, ca, rows, n, red);
    if (chunks > 1)
      hipLaunchKernelGGL(colsum_final_kernel, dim3((n + 63) / 64, nz), dim3(256), 0, s, ca, chunks, n, red);
  };

  // identity W of the square map: g(x) = (x_i^2)
  hipLaunchKernelGGL(identity_kernel, grid1(kHead * kHead), dim3(256), 0, s, ident, kHead);
  CHECK_HIP(hipGetLastError());

  // queries, keys and values of layer r for the slice's rows, per head (the
  // activations of every layer stay in its buffers for the backward)
  auto layer_qkv = [&](int r, int n) -> int {
    const int rows = (int)(m.B * n);
    // [Q K V] = X [Wq Wk Wv], stored straight into the per-head tensors
    const GroupB gb = wqkv(P.l[r].Wq, P.l[r].Wk, P.l[r].Wv, false);
    CHECK_HIP(mm(false, false, rows, 3 * D, D, Xr(r), D, nullptr, D, nullptr, 0,
                 epi_groups(EPI_STORE, Qhr(r, 0), Qhr(r, 1), Qhr(r, 2), D, n, k), &gb));
    return SLIM_OK;
  };
  // the rest of layer r (eqs. 5-9) from the state before the slice
  auto layer_fwd = [&](int r, int a, int n, const float* state_in, float* state_out) -> int {
    const int rows = (int)(m.B * n);
    const size_t hf = (size_t)m.B * k * n * kHead;
    const float* X = Xr(r);
    const slim_problem p = att_problem(m, n);
    CHECK_SLIM(slim_fwd(&p, Qhr(r, 0), Qhr(r, 1), Qhr(r, 2), ident, state_in, nullptr, Yh, nullptr, state_out, nullptr,
                        nullptr, attws, lay.attws_bytes, s));
    hipLaunchKernelGGL(heads_to_rows_kernel, grid1(hf), dim3(256), 0, s, Yh, Ar(r), D, 0, 0, k, n, hf, hf);
    hipLaunchKernelGGL(ln_fwd_kernel, dim3(rows), dim3(256), 0, s, Ar(r), P.l[r].g1, P.l[r].b1n, X, Hr(r), s1r(r), D,
                       m.eps);
    CHECK_HIP(mm(false, false, rows, F, D, Hr(r), D, P.l[r].W1, F, Z1r(r), F, epi(EPI_BIAS_GELU, P.l[r].b1, nullptr, G1r(r))));
    CHECK_HIP(mm(false, false, rows, D, F, G1r(r), F, P.l[r].W2, D, For(r), D, epi(EPI_BIAS, P.l[r].b2)));
    hipLaunchKernelGGL(ln_fwd_kernel, dim3(rows), dim3(256), 0, s, For(r), P.l[r].g2, P.l[r].b2n, Hr(r), Xr(r + 1),
                       s2r(r), D, m.eps);
    CHECK_HIP(hipGetLastError());
    return SLIM_OK;
  };
  auto head_logits = [&](int a, int n) -> int {
    const int rows = (int)(m.B * n);
    CHECK_HIP(mm(false, false, rows, V, D, Xr(m.s), D, P.Wout, V, logits, V, epi(EPI_BIAS, P.bout)));
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
      CHECK_SLIM(slim_fwd(&p, Qhr(r, 0), Qhr(r, 1), Qhr(r, 2), ident, nullptr, nullptr, Yh, nullptr, delta, nullptr,
                          nullptr, attws, lay.attws_bytes, s));
      hipLaunchKernelGGL(sub_kernel, grid1(S), dim3(256), 0, s, bprev + r * S, states + r * S, delta, S);
      CHECK_HIP(hipGetLastError());
      CHECK_SLIM(layer_fwd(r, a, n, bprev + r * S, snew));
    }
    CHECK_SLIM(head_logits(a, n));
    // output layer
    CHECK_HIP(mm(true, false, D, V, rows, Xr(m.s), D, logits, V, G.Wout, V, epi(EPI_ACC)));
    colsum(rows, V, logits, G.bout);
    CHECK_HIP(mm(false, true, rows, D, V, logits, V, P.Wout, V, dX, D, epi(EPI_STORE)));
    for (int r = m.s - 1; r >= 0; --r) {
      const Params::Layer& pl = P.l[r];
      const Grads::Layer& gl = G.l[r];
      // X_{r+1} = LN2(Fo) + H
      hipLaunchKernelGGL(ln_bwd_kernel, dim3(rows), dim3(256), 0, s, For(r), s2r(r), pl.g2, dX, nullptr, dF, Pp, D);
      colsum(rows, D, Pp, gl.g2, dX, gl.b2n);
      // Fo = GeLU(Z1) W2 + b2
      CHECK_HIP(mm(true, false, F, D, rows, G1r(r), F, dF, D, gl.W2, D, epi(EPI_ACC)));
      colsum(rows, D, dF, gl.b2);
      CHECK_HIP(mm(false, true, rows, F, D, dF, D, pl.W2, D, dG1, F, epi(EPI_GELU_BWD, nullptr, Z1r(r))));
      // Z1 = H W1 + b1; dH = dX (residual) + dZ1 W1^T
      CHECK_HIP(mm(true, false, D, F, rows, Hr(r), D, dG1, F, gl.W1, F, epi(EPI_ACC)));
      colsum(rows, F, dG1, gl.b1);
      CHECK_HIP(mm(false, true, rows, D, F, dG1, F, pl.W1, F, dH, D, epi(EPI_ADD, nullptr, dX)));
      // H = LN1(A) + X
      hipLaunchKernelGGL(ln_bwd_kernel, dim3(rows), dim3(256), 0, s, Ar(r), s1r(r), pl.g1, dH, nullptr, dA, Pp, D);
      colsum(rows, D, Pp, gl.g1, dH, gl.b1n);
      CHECK_HIP(hipGetLastError());
      // attention: the slice's gradient with the state cotangent after it
      // (eq. 18 gives the one before it)
      hipLaunchKernelGGL(rows_to_heads_kernel, grid1(hf), dim3(256), 0, s, dA, D, 0, dYh, k, n, hf);
      float* gin = gst + ((size_t)gcur * m.s + r) * S;
      float* gout = gst + ((size_t)(1 - gcur) * m.s + r) * S;
      CHECK_SLIM(slim_bwd(&p, Qhr(r, 0), Qhr(r, 1), Qhr(r, 2), ident, bprev + r * S, nullptr, nullptr, dYh, nullptr,
                          nullptr, gin, dQh, dQh + hf, dQh + 2 * hf, wd, gout, nullptr, attws, lay.attws_bytes, s));
      hipLaunchKernelGGL(heads_to_rows_kernel, grid1(3 * hf), dim3(256), 0, s, dQh, dQKV, 3 * D, 0, D, k, n, hf, 3 * hf);
      CHECK_HIP(hipGetLastError());
      // [Q K V] = X [Wq Wk Wv]: [dWq dWk dWv] += X^T [dQ dK dV];
      // dX = dH + [dQ dK dV] [Wq Wk Wv]^T
      CHECK_HIP(mm(true, false, D, 3 * D, rows, Xr(r), D, dQKV, 3 * D, nullptr, D,
                   epi_groups(EPI_ACC, gl.Wq, gl.Wk, gl.Wv, D)));
      const GroupB gb = wqkv(pl.Wq, pl.Wk, pl.Wv, true);
      CHECK_HIP(mm(false, true, rows, D, 3 * D, dQKV, 3 * D, nullptr, D, dX, D, epi(EPI_ADD, nullptr, dH), &gb));
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
