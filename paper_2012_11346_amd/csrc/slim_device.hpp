// Device building blocks for the slice-wise causal linear attention kernels
// (gfx950, wave64).
//
// Matrix-core conventions.  A wave computes 16x16 fp32 result tiles with
// v_mfma_f32_16x16x32_bf16 (bf16 problems) or 8 chained
// v_mfma_f32_16x16x4_f32 (fp32 problems).  With lane = 16 g + c
// (g in 0..3, c in 0..15):
//
//   result tile  X[16 x 16]     lane (g, c), register r  <->  X[4g + r][c]
//   operand      "fragment"     lane (g, c), slot s      <->  row/col c, k = kp(g, s)
//
// where a fragment covers one 32-deep block of the contraction index k and
//
//   kp(g, s) = 16 (s / 4) + 4 g + (s % 4)
//
// is the slot order used everywhere in this library (A and B operands of one
// product must agree on it; the sum over k does not care about the order).
// With this order two result tiles stacked along their rows, X0 = rows
// [0, 16) and X1 = rows [16, 32), are directly an operand fragment that
// contracts over those 32 rows (tile_pair_frag), so results can feed the next
// product without leaving registers whenever the next contraction runs over
// the result's row index.  When it runs over the column index instead, the
// tile goes through LDS: store_tile_T writes X transposed (one 8-byte store
// per lane for bf16) and frag_tr reads it back with ds_read_b64_tr_b16, whose
// per-16-lane semantics (lane j supplies the address of 4 consecutive 16-bit
// values a_j; lane i receives slot r = mem[a_{4r + i/4} + i % 4]) turn a
// "k-major" LDS matrix (rows = contraction index, columns contiguous) into a
// fragment.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace slim {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));

#define SLIM_LDS __attribute__((address_space(3)))

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }
__device__ __forceinline__ int lane_g() { return (threadIdx.x & 63) >> 4; }
__device__ __forceinline__ int lane_c() { return threadIdx.x & 15; }

// Lane coordinates (g, c) as explicit values.  A kernel may rebuild them from
// an opaque copy of the thread index (fresh_lane) at the start of a phase, so
// that the compiler forms the lane-dependent addresses of that phase inside
// it instead of keeping every one of them live across a long loop.
struct Lane {
  int g, c;
};
__device__ __forceinline__ int fresh_tid() {
  int x = threadIdx.x;
  asm volatile("" : "+v"(x));
  return x;
}
__device__ __forceinline__ Lane fresh_lane() {
  const int x = fresh_tid();
  return Lane{(x & 63) >> 4, x & 15};
}
__device__ __forceinline__ Lane this_lane() { return Lane{lane_g(), lane_c()}; }
__device__ __forceinline__ int wave_id() { return threadIdx.x >> 6; }

// k offset of slot s of lane group g inside a 32-deep block
__device__ __forceinline__ int kp(int g, int s) { return 16 * (s >> 2) + 4 * g + (s & 3); }

template <typename T>
struct FragT;
template <>
struct FragT<bf16> {
  typedef bf16x8 type;
};
template <>
struct FragT<float> {
  typedef f32x8 type;
};

__device__ __forceinline__ f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }

// acc += A * B over one 32-deep block
__device__ __forceinline__ f32x4 mma(f32x4 acc, bf16x8 a, bf16x8 b) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma(f32x4 acc, f32x8 a, f32x8 b) {
#pragma unroll
  for (int j = 0; j < 8; ++j) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[j], b[j], acc, 0, 0, 0);
  return acc;
}

template <typename T>
__device__ __forceinline__ T cvt(float x);
template <>
__device__ __forceinline__ bf16 cvt<bf16>(float x) {
  return (bf16)x;
}
template <>
__device__ __forceinline__ float cvt<float>(float x) {
  return x;
}

template <typename T>
__device__ __forceinline__ float to_f32(T x) {
  return (float)x;
}

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
// floats to bf16 (round to nearest even) as whole vectors: the compiler then
// emits one v_cvt_pk_bf16_f32 per pair, where element-wise conversions into a
// vector can come out as one conversion per element plus byte permutes
__device__ __forceinline__ bf16x2 pk_bf16(float a, float b) { return __builtin_convertvector(f32x2{a, b}, bf16x2); }
__device__ __forceinline__ bf16x4 pk_bf16x4(const f32x4& x) { return __builtin_convertvector(x, bf16x4); }

// W enters the logits w_m . x as a pair of bf16 values, hi = RNE(w) and
// lo = RNE(w - hi), each with its own product against the bf16 row x: the
// pair carries about 16 significant bits of the float32 W, so the logits are
// those of the caller's W to ~2^-17 of sum_e |x_e w_e| instead of 2^-9 (an
// error that exp would turn into a relative error of the features).
// kSplitW<T> says whether the element type needs the second product.
template <typename T>
constexpr bool kSplitW = sizeof(T) == 2;
template <typename T>
__device__ __forceinline__ T w_lo(float x) {
  if constexpr (sizeof(T) == 2) return (T)(x - (float)(T)x);
  else return (T)0.f;
}

// ------------------------------------------------------------- fragments

template <typename T>
__device__ __forceinline__ typename FragT<T>::type frag_zero() {
  typename FragT<T>::type f;
#pragma unroll
  for (int s = 0; s < 8; ++s) f[s] = cvt<T>(0.f);
  return f;
}

// two result tiles (rows [0,16) and [16,32) of a 32-row block, same columns)
// as an operand contracting over those rows
template <typename T>
__device__ __forceinline__ typename FragT<T>::type tile_pair_frag(const f32x4& x0, const f32x4& x1) {
  typename FragT<T>::type f;
  if constexpr (sizeof(T) == 2) {
    const bf16x4 a = pk_bf16x4(x0), b = pk_bf16x4(x1);
    f = __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
  } else {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      f[r] = cvt<T>(x0[r]);
      f[4 + r] = cvt<T>(x1[r]);
    }
  }
  return f;
}
template <typename T>
__device__ __forceinline__ typename FragT<T>::type tile_half_frag(const f32x4& x0) {
  typename FragT<T>::type f;
  if constexpr (sizeof(T) == 2) {
    const bf16x4 a = pk_bf16x4(x0), z = {};
    f = __builtin_shufflevector(a, z, 0, 1, 2, 3, 4, 5, 6, 7);
  } else {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      f[r] = cvt<T>(x0[r]);
      f[4 + r] = cvt<T>(0.f);
    }
  }
  return f;
}

// Fragment from an LDS matrix stored with the contraction index contiguous:
// slot s = Z[row0 + c][k0 + kp(g, s)]  (pitch ld elements).
template <typename T>
__device__ __forceinline__ typename FragT<T>::type frag_rm(const Lane& L, const T* Z, int ld, int row0, int k0) {
  const int g = L.g, c = L.c;
  const T* p = Z + (row0 + c) * ld + k0 + 4 * g;
  typename FragT<T>::type f;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    f[r] = p[r];
    f[4 + r] = p[16 + r];
  }
  return f;
}
template <typename T>
__device__ __forceinline__ typename FragT<T>::type frag_rm(const T* Z, int ld, int row0, int k0) {
  return frag_rm(this_lane(), Z, ld, row0, k0);
}

// Fragment from an LDS matrix stored k-major (contraction index = row):
// slot s = Z[k0 + kp(g, s)][col0 + c]  (pitch ld elements).
__device__ __forceinline__ bf16x8 frag_tr(const Lane& L, const bf16* Z, int ld, int k0, int col0) {
  const int g = L.g, c = L.c;
  const bf16* p0 = Z + (k0 + 4 * g + (c >> 2)) * ld + col0 + 4 * (c & 3);
  const bf16* p1 = p0 + 16 * ld;
  typedef SLIM_LDS i16x4 lds_i16x4;
  i16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p0);
  i16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p1);
  bf16x8 f;
  bf16x4 av = __builtin_bit_cast(bf16x4, a);
  bf16x4 bv = __builtin_bit_cast(bf16x4, b);
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    f[r] = av[r];
    f[4 + r] = bv[r];
  }
  return f;
}
__device__ __forceinline__ f32x8 frag_tr(const Lane& L, const float* Z, int ld, int k0, int col0) {
  const int g = L.g, c = L.c;
  f32x8 f;
#pragma unroll
  for (int s = 0; s < 8; ++s) f[s] = Z[(k0 + kp(g, s)) * ld + col0 + c];
  return f;
}
__device__ __forceinline__ bf16x8 frag_tr(const bf16* Z, int ld, int k0, int col0) {
  return frag_tr(this_lane(), Z, ld, k0, col0);
}
__device__ __forceinline__ f32x8 frag_tr(const float* Z, int ld, int k0, int col0) {
  return frag_tr(this_lane(), Z, ld, k0, col0);
}

// Store result tile X[row0 + 4g + r][col0 + c] transposed: Z[col0 + c][row0 + 4g + r].
template <typename T>
__device__ __forceinline__ void store_tile_T(const Lane& L, T* Z, int ld, const f32x4& x, int row0, int col0) {
  T* p = Z + (col0 + L.c) * ld + row0 + 4 * L.g;
  if constexpr (sizeof(T) == 2) {
    *(bf16x4*)p = pk_bf16x4(x);
  } else {
#pragma unroll
    for (int r = 0; r < 4; ++r) p[r] = cvt<T>(x[r]);
  }
}
template <typename T>
__device__ __forceinline__ void store_tile_T(T* Z, int ld, const f32x4& x, int row0, int col0) {
  store_tile_T(this_lane(), Z, ld, x, row0, col0);
}

// halves of an operand fragment built by tile_pair_frag (the rounded values
// of its first and second result tile)
__device__ __forceinline__ bf16x4 frag_lo(const bf16x8& f) { return __builtin_shufflevector(f, f, 0, 1, 2, 3); }
__device__ __forceinline__ bf16x4 frag_hi(const bf16x8& f) { return __builtin_shufflevector(f, f, 4, 5, 6, 7); }
__device__ __forceinline__ f32x4 frag_lo(const f32x8& f) { return __builtin_shufflevector(f, f, 0, 1, 2, 3); }
__device__ __forceinline__ f32x4 frag_hi(const f32x8& f) { return __builtin_shufflevector(f, f, 4, 5, 6, 7); }

// store_tile_T of values already rounded (half of an operand fragment)
__device__ __forceinline__ void store_half_T(const Lane& L, bf16* Z, int ld, const bf16x4& v, int row0, int col0) {
  *(bf16x4*)(Z + (col0 + L.c) * ld + row0 + 4 * L.g) = v;
}
__device__ __forceinline__ void store_half_T(const Lane& L, float* Z, int ld, const f32x4& v, int row0, int col0) {
  *(f32x4*)(Z + (col0 + L.c) * ld + row0 + 4 * L.g) = v;
}

// bf16 operand fragment of ones over the rows of a 32-deep block: slot s is 1
// where k0 + kp(g, s) < count, else 0 (count wave-uniform).  A full block
// (the common case) is a constant.
__device__ __forceinline__ bf16x8 ones_rows_frag(const Lane& L, int k0, int count) {
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  constexpr unsigned one2 = 0x3F803F80u;  // two bf16 ones
  if (count >= k0 + 32) return __builtin_bit_cast(bf16x8, u32x4{one2, one2, one2, one2});
  const int rem = count - k0 - 4 * L.g;  // rows k0 + kp(g, s) < count
  bf16x8 f;
#pragma unroll
  for (int s = 0; s < 8; ++s) f[s] = (bf16)((s & 3) + 16 * (s >> 2) < rem ? 1.f : 0.f);
  return f;
}

// two stacked result tiles as an operand (has_b), or the first one with the
// second 16 entries of the 32-deep block zero
template <typename T>
__device__ __forceinline__ typename FragT<T>::type pair_or_half(const f32x4& a, const f32x4& b, bool has_b) {
  return has_b ? tile_pair_frag<T>(a, b) : tile_half_frag<T>(a);
}

// fragment slot s = Z[row0 + c][k0 + kp(g, s)], with slots 4..7 zero when the
// 32-deep block has only its first 16 entries
template <typename T>
__device__ __forceinline__ typename FragT<T>::type frag_rm_h(const T* Z, int ld, int row0, int k0, bool half) {
  if (!half) return frag_rm(Z, ld, row0, k0);
  const int g = lane_g(), c = lane_c();
  const T* p = Z + (row0 + c) * ld + k0 + 4 * g;
  typename FragT<T>::type f;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    f[r] = p[r];
    f[4 + r] = cvt<T>(0.f);
  }
  return f;
}

// result-tile values of a matrix stored transposed by store_tile_T:
// X[row0 + 4g + r][col0 + c] = Z[col0 + c][row0 + 4g + r]
template <typename T>
__device__ __forceinline__ f32x4 load_tile_T(const Lane& L, const T* Z, int ld, int row0, int col0) {
  const T* p = Z + (col0 + L.c) * ld + row0 + 4 * L.g;
  f32x4 x;
#pragma unroll
  for (int r = 0; r < 4; ++r) x[r] = to_f32(p[r]);
  return x;
}
template <typename T>
__device__ __forceinline__ f32x4 load_tile_T(const T* Z, int ld, int row0, int col0) {
  return load_tile_T(this_lane(), Z, ld, row0, col0);
}

// ------------------------------------------------------------- wave reductions

__device__ __forceinline__ float wave_max_over_g(float v) {
  // max over the 4 lanes that share c (lanes c, c+16, c+32, c+48)
  v = fmaxf(v, __shfl_xor(v, 16, 64));
  v = fmaxf(v, __shfl_xor(v, 32, 64));
  return v;
}
__device__ __forceinline__ float wave_sum_over_g(float v) {
  v += __shfl_xor(v, 16, 64);
  v += __shfl_xor(v, 32, 64);
  return v;
}
// x of another lane of the same row of 16 lanes (DPP control CTRL)
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}
// sum over aligned groups of N consecutive lanes (N = 1, 2, 4, 8 or 16),
// with DPP lane moves: quad permutations [1,0,3,2] and [2,3,0,1], then the
// mirror of each half row and of the row.  Each step adds the partial sum
// a butterfly over lane bits 0, 1, 2, 3 would add, so the results are the
// same, bit for bit.
template <int N>
__device__ __forceinline__ float sum_lane_group(float v) {
  static_assert(N == 1 || N == 2 || N == 4 || N == 8 || N == 16, "groups inside one row");
  if constexpr (N >= 2) v += dpp_f32<0xB1>(v);
  if constexpr (N >= 4) v += dpp_f32<0x4E>(v);
  if constexpr (N >= 8) v += dpp_f32<0x141>(v);
  if constexpr (N >= 16) v += dpp_f32<0x140>(v);
  return v;
}
// the same for the maximum
template <int N>
__device__ __forceinline__ float max_lane_group(float v) {
  static_assert(N == 1 || N == 2 || N == 4 || N == 8 || N == 16, "groups inside one row");
  if constexpr (N >= 2) v = fmaxf(v, dpp_f32<0xB1>(v));
  if constexpr (N >= 4) v = fmaxf(v, dpp_f32<0x4E>(v));
  if constexpr (N >= 8) v = fmaxf(v, dpp_f32<0x141>(v));
  if constexpr (N >= 16) v = fmaxf(v, dpp_f32<0x140>(v));
  return v;
}

// over the 16 lanes that share g (a row of the wave)
__device__ __forceinline__ float wave_max_over_c(float v) { return max_lane_group<16>(v); }
__device__ __forceinline__ float wave_sum_over_c(float v) { return sum_lane_group<16>(v); }
__device__ __forceinline__ float wave_max(float v) { return wave_max_over_c(wave_max_over_g(v)); }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

constexpr float kLog2e = 1.4426950408889634f;

// ------------------------------------------------------------- swizzled LDS tiles
//
// LDS of gfx950 serves reads from 64 four-byte banks (256 B per clock) and
// writes from 32 banks (128 B per clock).  A bf16 tile whose rows are read
// both as fragments (frag_rm: row c, k = 4g..) and transposed (frag_tr: rows
// 4g + c/4) and written by store_tile_T (row c, columns 4g..) cannot be
// conflict-free for all three patterns by padding alone.  The swizzled tile
// pads each row by 16 elements and XORs the 8-byte granule index (4 bf16)
// with a value sw(r) in [0, 4) taken from row bits 2..3:
//
//   element (r, e)  at  r * P + 4 * ((e >> 2) ^ sw(r)) + (e & 3),  P = row length + 16
//
// Row tiles staged from global memory in 16-byte chunks use sw(r) in {0, 2}
// (bit 3 of r), which keeps every chunk contiguous.  sw depends on r mod 16
// only and touches only the low two granule bits, so an access to rows
// starting at a multiple of 16 and columns starting at a multiple of 16 is a
// per-lane offset (SwzLane) plus a compile-time offset.
enum SwzMode { kSwzInter = 0, kSwzRows = 1 };

template <int MODE>
__device__ __forceinline__ int swz(int r) {
  return MODE == kSwzInter ? ((r >> 2) & 3) : (((r >> 3) & 1) << 1);
}

// per-lane element offsets of the three access patterns of a swizzled tile
template <int P, int MODE>
struct SwzLane {
  int a;  // row c, granule g (frag_rm, store_tile_T, load_tile_T)
  int b;  // row 4g + c/4, granule c % 4 (frag_tr)
  __device__ __forceinline__ explicit SwzLane(const Lane& L) {
    a = L.c * P + 4 * (L.g ^ swz<MODE>(L.c));
    const int r = 4 * L.g + (L.c >> 2);
    b = r * P + 4 * ((L.c & 3) ^ swz<MODE>(r));
  }
};

// element offset of (r, e) in a swizzled tile
template <int P, int MODE>
__device__ __forceinline__ int swz_off(int r, int e) {
  return r * P + 4 * ((e >> 2) ^ swz<MODE>(r)) + (e & 3);
}

// fragment slot s = Z[row0 + c][k0 + kp(g, s)]   (row0, k0 multiples of 16)
template <int P, int MODE>
__device__ __forceinline__ bf16x8 sfrag_rm(const SwzLane<P, MODE>& o, const bf16* Z, int row0, int k0) {
  const bf16* p = Z + o.a + row0 * P + k0;
  bf16x8 f;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    f[r] = p[r];
    f[4 + r] = p[16 + r];
  }
  return f;
}

// fragment slot s = Z[k0 + kp(g, s)][col0 + c]   (k0, col0 multiples of 16)
template <int P, int MODE>
__device__ __forceinline__ bf16x8 sfrag_tr(const SwzLane<P, MODE>& o, const bf16* Z, int k0, int col0) {
  typedef SLIM_LDS i16x4 lds_i16x4;
  const bf16* p0 = Z + o.b + k0 * P + col0;
  const i16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p0);
  const i16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p0 + 16 * P));
  const bf16x4 av = __builtin_bit_cast(bf16x4, a), bv = __builtin_bit_cast(bf16x4, b);
  bf16x8 f;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    f[r] = av[r];
    f[4 + r] = bv[r];
  }
  return f;
}

// result tile X[row0 + 4g + r][col0 + c] stored transposed: Z[col0 + c][row0 + 4g + r]
template <int P, int MODE>
__device__ __forceinline__ void sstore_tile_T(const SwzLane<P, MODE>& o, bf16* Z, const f32x4& x, int row0, int col0) {
  *(bf16x4*)(Z + o.a + col0 * P + row0) = pk_bf16x4(x);
}

// the same store for values already rounded (half of an operand fragment)
template <int P, int MODE>
__device__ __forceinline__ void sstore_half_T(const SwzLane<P, MODE>& o, bf16* Z, const bf16x4& v, int row0, int col0) {
  *(bf16x4*)(Z + o.a + col0 * P + row0) = v;
}
// X[row0 + 4g + r][col0 + c] of a tile stored transposed by sstore_tile_T
template <int P, int MODE>
__device__ __forceinline__ f32x4 sload_tile_T(const SwzLane<P, MODE>& o, const bf16* Z, int row0, int col0) {
  const bf16x4 v = *(const bf16x4*)(Z + o.a + col0 * P + row0);
  f32x4 x;
#pragma unroll
  for (int r = 0; r < 4; ++r) x[r] = (float)v[r];
  return x;
}

}  // namespace slim
