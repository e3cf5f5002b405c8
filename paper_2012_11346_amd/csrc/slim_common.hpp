// Shared compile-time geometry and tile helpers for the forward, backward and
// feature-map kernels.
#pragma once

#include "slim_device.hpp"

namespace slim {

enum Kind { kFavor = 0, kRelu = 1 };

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
#pragma unroll
      for (int o = 1; o < CPR; o <<= 1) s += __shfl_xor(s, o, 64);
      if (active && cc == 0) norms[r] = s;
    }
  }
}

}  // namespace slim
