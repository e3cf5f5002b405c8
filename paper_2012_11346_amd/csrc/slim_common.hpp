// Shared compile-time geometry and tile helpers for the forward, backward and
// feature-map kernels.
#pragma once

#include <climits>

#include "slim_device.hpp"

namespace slim {

enum Kind { kFavor = 0, kRelu = 1, kSquare = 2 };

// Features of the maps without shifts, from the logit l = w_m . x:
// ReLU max(l, 0) + eps, square l^2.
// (FAVOR+ has shifts and is formed by its callers; l is returned for it)
template <int KIND>
__device__ __forceinline__ float plain_feature(float l, float eps) {
  if constexpr (KIND == kRelu) return fmaxf(l, 0.f) + eps;
  else if constexpr (KIND == kSquare) return l * l;
  else return l;
}
// The chain-rule factor of a feature's cotangent dphi: FAVOR+ dphi * phi
// (then times (w - x)), ReLU dphi * [l > 0] (decided from phi > eps), square
// dphi * 2 l (the logit l itself is needed: phi = l^2 has lost its sign).
template <int KIND>
__device__ __forceinline__ float vjp_factor(float dphi, float phi, float l, float eps) {
  if constexpr (KIND == kFavor) return dphi * phi;
  else if constexpr (KIND == kRelu) return phi > eps ? dphi : 0.f;
  else return 2.f * l * dphi;
}

// Work split: a workgroup of 4 waves owns one (batch, head, segment); wave w
// owns features [w FW, (w + 1) FW) of the M = 4 FW features and keeps its
// share of the running state in registers.  The sequence is walked in tiles
// of at most TR rows that never straddle a slice boundary.
template <typename T_, int D_, int FW_, int TR_, int KIND_>
struct Cfg {
  typedef T_ T;
  static constexpr int D = D_;
  static constexpr int FW = FW_;
  static constexpr int M = 4 * FW_;
  static constexpr int TR = TR_;
  static constexpr int KIND = KIND_;
  static constexpr int MT = FW / 16;       // 16-row feature tiles per wave
  static constexpr int MB = (MT + 1) / 2;  // 32-deep feature blocks per wave
  static constexpr int ET = D / 16;        // 16-column value tiles (the ones column is tile ET)
  static constexpr int EB = D / 32;        // 32-deep head-dim blocks
  static constexpr int RT = TR / 16;       // 16-row tiles per sequence tile
  static constexpr int RB = TR / 32;       // 32-deep row blocks per sequence tile
  static constexpr int LDQ = D + 8;        // LDS pitch of the Q/K/V/dY/dN tiles (elements)
  static constexpr int LDZ = TR + 8;       // LDS pitch of per-wave [feature][row] buffers
  static constexpr int ZR = MB * 32;       // rows of per-wave [feature][row] buffers
  static constexpr int LDF = FW + 8;       // LDS pitch of per-wave [row][feature] buffers
  static constexpr int LDR = D + 4;        // LDS pitch (floats) of the reduction rows
  static constexpr int NT = 256;           // threads per workgroup
  static_assert(D == 32 || D == 64, "head dim");
  static_assert(FW == 16 || FW == 32 || FW == 64, "features per wave");
  static_assert(TR == 32 || TR == 64, "tile rows");
};

// Fragment-ordered copy of W, prepared once per call (wfrag_kernel): every
// operand fragment of W a wave uses is 64 lanes x 8 elements, contiguous, so
// a lane fetches it with one 16-byte (bf16) load.
//   block A  [wave][mt][kb]: slot s = W[w FW + 16 mt + c][32 kb + kp(g, s)]   (contracting over d)
//   block B  [wave][kb][et]: slot s = W[w FW + 32 kb + kp(g, s)][16 et + c]   (contracting over features)
//   block C  [kb][et], after the waves' blocks: slot s = W[32 kb + kp(g, s)][16 et + c]
//            (contracting over all M features)
//   block A' [wave][mt][kb], after block C (bf16 only): the low parts w_lo of
//            block A's entries, for the second product of the logits
template <class G>
struct WFragLayout {
  static constexpr int NA = G::MT * G::EB;  // fragments of block A per wave
  static constexpr int NB = G::MB * G::ET;  // fragments of block B per wave
  static constexpr int PER_WAVE = NA + NB;
  static constexpr int NC = (G::M / 32) * G::ET;  // fragments of block C
  static constexpr int NLO = kSplitW<typename G::T> ? 4 * NA : 0;  // fragments of block A'
  static constexpr int TOTAL = 4 * PER_WAVE + NC + NLO;  // fragments
  __device__ static int a(int w, int mt, int kb) { return w * PER_WAVE + mt * G::EB + kb; }
  __device__ static int b(int w, int kb, int et) { return w * PER_WAVE + NA + kb * G::ET + et; }
  __device__ static int c(int kb, int et) { return 4 * PER_WAVE + kb * G::ET + et; }
  __device__ static int alo(int w, int mt, int kb) { return 4 * PER_WAVE + NC + w * NA + mt * G::EB + kb; }
};

// Row range of tile j of a head, for slices of length C (already clamped to
// [1, L]).  Slices longer than TR are cut into TR-row tiles from the slice
// start; the last slice may be ragged.
struct TileMap {
  int L, C, TR, tps;  // tps: tiles per slice (1 when C <= TR)
  __host__ __device__ TileMap(int L_, int C_, int TR_) : L(L_), C(C_), TR(TR_) {
    tps = (C <= TR) ? 1 : (C + TR - 1) / TR;
  }
  __host__ __device__ int count_tiles() const {
    if (C <= TR) return (L + C - 1) / C;
    const int n_full = (L - 1) / C;  // slices before the last one
    const int last = L - n_full * C;
    return n_full * tps + (last + TR - 1) / TR;
  }
  __host__ __device__ void tile(int j, int& start, int& count) const {
    if (C <= TR) {
      start = j * C;
      count = min(C, L - start);
      return;
    }
    const int n = j / tps, tau = j - n * tps;
    const int s0 = n * C;
    const int s1 = min(s0 + C, L);
    start = s0 + tau * TR;
    count = min(TR, s1 - start);
  }
};

// 16-byte chunk copy of a [count x D] row block from global memory into an
// LDS tile of pitch LD, zero-filling rows [count, TR).  Optionally stores the
// squared row norms (float) into norms[TR].
template <typename T, int D, int TR, int LD, int NT>
__device__ __forceinline__ void load_rows(T* dst, const T* src, int count, float* norms) {
  constexpr int VEC = 16 / sizeof(T);
  constexpr int CPR = D / VEC;  // chunks per row
  constexpr int NCH = TR * CPR;
  static_assert(NCH % CPR == 0, "");
  for (int ch = threadIdx.x; ch < ((NCH + NT - 1) / NT) * NT; ch += NT) {
    const bool active = ch < NCH;
    const int r = ch / CPR, cc = ch - (ch / CPR) * CPR;
    uint4 v = {0u, 0u, 0u, 0u};
    if (active && r < count) v = *reinterpret_cast<const uint4*>(src + (size_t)r * D + cc * VEC);
    if (active) *reinterpret_cast<uint4*>(dst + r * LD + cc * VEC) = v;
    if (norms != nullptr) {
      float s = 0.f;
      const T* e = reinterpret_cast<const T*>(&v);
#pragma unroll
      for (int i = 0; i < VEC; ++i) {
        const float x = to_f32(e[i]);
        s += x * x;
      }
      s = sum_lane_group<CPR>(s);
      if (active && cc == 0) norms[r] = s;
    }
  }
}

constexpr size_t al16(size_t n) { return (n + 15) & ~(size_t)15; }

// ---------------------------------------------------------------------------
// Value dropout with per-slice seeds (Sec. 5): element (b, h, l, e) of V is
// kept when 16-bit field e % 16 of Philox4x64-10 (counter (r, e / 16,
// b H + h, 0), key (seed, n); n = l / C the slice of row l, r = l - n C) is
// >= t; the output is scaled by 1 / (1 - p) elsewhere.  t = 0: no dropout.
struct Drop {
  uint64_t seed;
  uint32_t t;
  int C;
  uint64_t head;  // b H + h
};

// Philox4x64-10 (Salmon et al., SC 2011): ten rounds of two 64 x 64 -> 128
// bit products, the key bumped by the Weyl constants between rounds
__device__ __forceinline__ void philox4x64_10(uint64_t (&c)[4], uint64_t k0, uint64_t k1) {
  constexpr uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
  constexpr uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
  for (int i = 0; i < 10; ++i) {
    const uint64_t hi0 = __umul64hi(M0, c[0]), lo0 = M0 * c[0];
    const uint64_t hi1 = __umul64hi(M1, c[2]), lo1 = M1 * c[2];
    const uint64_t n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
    c[0] = n0;
    c[1] = lo1;
    c[2] = n2;
    c[3] = lo0;
    k0 += W0;
    k1 += W1;
  }
}

// keep bits of the N consecutive elements e0 .. e0 + N - 1 of row l (N = 2,
// 4 or 8, e0 a multiple of N): bit i set when element e0 + i is kept
template <int N>
__device__ __forceinline__ unsigned drop_keep_bits(const Drop& dp, int l, int e0) {
  const int n = l / dp.C;
  uint64_t c[4] = {(uint64_t)(l - n * dp.C), (uint64_t)(e0 >> 4), dp.head, 0ull};
  philox4x64_10(c, dp.seed, (uint64_t)n);
  unsigned bits = 0;
#pragma unroll
  for (int i = 0; i < N; ++i) {
    const int j = (e0 & 15) + i;
    // (word j / 4 of the four outputs, selected with constant indices)
    const uint64_t wj = (j >> 2) == 0 ? c[0] : (j >> 2) == 1 ? c[1] : (j >> 2) == 2 ? c[2] : c[3];
    const unsigned f = (unsigned)(wj >> (16 * (j & 3))) & 0xFFFFu;
    bits |= (f >= dp.t ? 1u : 0u) << i;
  }
  return bits;
}

// zero the dropped elements of a 16-byte row chunk (8 bf16 or 4 floats)
// holding row l, columns e0 .. e0 + 16 / sizeof(T) - 1
template <typename T>
__device__ __forceinline__ void drop_chunk(uint4& v, const Drop& dp, int l, int e0) {
  constexpr int N = 16 / sizeof(T);
  const unsigned bits = drop_keep_bits<N>(dp, l, e0);
  unsigned w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    if constexpr (N == 8) {
      const unsigned m = ((bits >> (2 * q)) & 1u ? 0x0000FFFFu : 0u) | ((bits >> (2 * q + 1)) & 1u ? 0xFFFF0000u : 0u);
      w[q] &= m;
    } else {
      w[q] = (bits >> q) & 1u ? w[q] : 0u;
    }
  }
  v = uint4{w[0], w[1], w[2], w[3]};
}

// Raw buffer resource over [base, base + bytes): the hardware's range check
// makes loads past the end read zero and drops stores past the end, so
// accesses to a ragged last row block need no branch (and the compiler can
// count outstanding memory operations exactly).  bytes < 2^31.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t range_rsrc(const void* base, size_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
// N bytes (8 or 16) at byte offset off of a range resource
template <int N>
struct BufIO {
  static_assert(N == 8 || N == 16, "8- or 16-byte accesses");
  typedef unsigned u32v __attribute__((ext_vector_type(N / 4)));
  template <class V>
  __device__ __forceinline__ static V load(__amdgpu_buffer_rsrc_t rs, int off) {
    static_assert(sizeof(V) == N, "size");
    if constexpr (N == 8) return __builtin_bit_cast(V, __builtin_amdgcn_raw_buffer_load_b64(rs, off, 0, 0));
    else return __builtin_bit_cast(V, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
  }
  template <class V>
  __device__ __forceinline__ static void store(const V& v, __amdgpu_buffer_rsrc_t rs, int off) {
    static_assert(sizeof(V) == N, "size");
    if constexpr (N == 8) __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32v, v), rs, off, 0, 0);
    else __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32v, v), rs, off, 0, 0);
  }
};

// Register staging of a [count x D] row block (rows >= count read as zero)
// by NT threads numbered tid = 0 .. NT-1: fetch() issues the global loads,
// store() writes LDS (pitch LD) and optionally the squared row norms.
// Splitting the two lets the loads of the next tile overlap the compute of
// the current one.
template <typename T, int D, int TR, int NT>
struct RowStage {
  static constexpr int VEC = 16 / sizeof(T);
  static constexpr int CPR = D / VEC;  // 16-byte chunks per row
  static constexpr int NCH = TR * CPR;
  static constexpr int PER = (NCH + NT - 1) / NT;
  static_assert(CPR <= 16, "a row's chunks must sit in consecutive lanes of one wave");
  uint4 v[PER];

  __device__ __forceinline__ void fetch(const T* src, int count, int tid) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int ch = tid + i * NT;
      const int r = ch / CPR, cc = ch - (ch / CPR) * CPR;
      v[i] = uint4{0u, 0u, 0u, 0u};
      if (ch < NCH && r < count) v[i] = *reinterpret_cast<const uint4*>(src + (size_t)r * D + cc * VEC);
    }
  }
  // rows [row0, row0 + TR) of a range resource over whole rows; rows past
  // its end read as zero
  __device__ __forceinline__ void fetch(__amdgpu_buffer_rsrc_t rs, int row0, int tid) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int ch = tid + i * NT;
      const int r = ch / CPR, cc = ch - (ch / CPR) * CPR;
      // chunks past the block get an offset beyond any range
      const int off = ch < NCH ? ((row0 + r) * D + cc * VEC) * (int)sizeof(T) : INT_MAX - 15;
      v[i] = BufIO<16>::load<uint4>(rs, off);
    }
  }
  // value dropout of the staged rows: row r of the block is row l0 + r of
  // the head (rows past the block are zero already)
  __device__ __forceinline__ void drop(const Drop& dp, int l0, int tid) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int ch = tid + i * NT;
      const int r = ch / CPR, cc = ch - (ch / CPR) * CPR;
      if (ch < NCH) drop_chunk<T>(v[i], dp, l0 + r, cc * VEC);
    }
  }
  // into a row tile swizzled as kSwzRows (pitch LD): chunk cc of row r goes
  // to chunk cc ^ sw(r) / 2
  template <int LD>
  __device__ __forceinline__ void store_swz(T* dst, float* norms, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int ch = tid + i * NT;
      const bool active = ch < NCH;
      const int r = ch / CPR, cc = ch - (ch / CPR) * CPR;
      if (active) *reinterpret_cast<uint4*>(dst + r * LD + VEC * (cc ^ ((r >> 3) & 1))) = v[i];
      if (norms != nullptr) {
        float s = 0.f;
        const T* e = reinterpret_cast<const T*>(&v[i]);
#pragma unroll
        for (int k = 0; k < VEC; ++k) {
          const float x = to_f32(e[k]);
          s += x * x;
        }
        s = sum_lane_group<CPR>(s);
        if (active && cc == 0) norms[r] = s;
      }
    }
  }
  template <int LD>
  __device__ __forceinline__ void store(T* dst, float* norms, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int ch = tid + i * NT;
      const bool active = ch < NCH;
      const int r = ch / CPR, cc = ch - (ch / CPR) * CPR;
      if (active) *reinterpret_cast<uint4*>(dst + r * LD + cc * VEC) = v[i];
      if (norms != nullptr) {
        float s = 0.f;
        const T* e = reinterpret_cast<const T*>(&v[i]);
#pragma unroll
        for (int k = 0; k < VEC; ++k) {
          const float x = to_f32(e[k]);
          s += x * x;
        }
        s = sum_lane_group<CPR>(s);
        if (active && cc == 0) norms[r] = s;
      }
    }
  }
};

}  // namespace slim
