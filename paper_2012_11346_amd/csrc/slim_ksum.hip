// Key sums of contiguous row ranges: the state each part of a segmented
// sequence adds (eqs. 14-16 summed over the part), and the largest key
// exponent of each part.
//
// Each head's sequence is cut into P2 parts at the 32-row tile boundaries
// the walks use (part p holds tiles [p n / P2, (p + 1) n / P2), or whole
// slices when the caller asks for slice-aligned parts).  A part's
// contribution to the state is a plain sum over its rows,
//   [S | z] = sum_s K~[s]^T [V[s] | 1],
// with no causal structure, so this pass streams the part's rows in 64-row
// chunks with one barrier per chunk.  Four waves split the M features; per
// chunk a wave computes the key logits of its features on the matrix cores
// (W fragments in registers, or at 64 features per wave read per chunk),
// the features (FAVOR+: exp2 of the logit shifted by the
// head's fixed key shift and the row's -|k|^2/2; ReLU: max(., 0) + eps) and
// accumulates K~^T [V|1] into its share of the state in registers.  Rows
// move through double-buffered, swizzled LDS tiles; the rows two chunks
// ahead are fetched with range-checked loads (zero past the part).
//
// KS_MAX mode computes only the logits and returns, per part, the maximum of
// w_m.k - |k|^2/2 over its rows and all features: the maximum over a head's
// parts is the key shift of that head.
//
// kSumQuery mode (backward) sums the state cotangent a part's rows add
// (eq. 18 summed over the part), from the forward's outputs Y and logD:
//   G = sum_t u[t]^T [s dY[t] | -rowdot(dY[t], Y[t])],  u[t]_m = phi(q_t)_m / D_t,
// the row cotangents of eq. 2 (dN = s dY / D, dD = -rowdot(dY, Y) / D, s the
// dropout scale) with D known, so no state is needed: the same stream of
// 64-row chunks with the queries in place of the keys, dY in place of the
// values and the row dots in place of the ones column.  u comes from the
// query logits and logD (exp2(w_m.q log2(e) - logD) for FAVOR+, with the
// head's key shift folded in so that G is in the units of the walk's
// cotangent).
#include <type_traits>

#include "slim_common.hpp"
#include "slim_kernels.hpp"

namespace slim {

// DROP: value dropout on (its masks are generated only in that instantiation)
template <class G, int MODE, bool DROP>
__global__ __launch_bounds__(256, 2) void ksum_kernel(KsumArgs a) {
  typedef typename G::T T;
  typedef typename FragT<T>::type F;
  constexpr int D = G::D, FW = G::FW, M = G::M, MT = G::MT, ET = G::ET, EB = G::EB;
  constexpr int CR = 64;          // rows per chunk
  constexpr int CT = CR / 16;     // 16-row tiles per chunk
  constexpr int LDQ = D + 16;     // row tiles, swizzled (kSwzRows)
  constexpr int TQ = CR * LDQ;
  constexpr bool QRY = MODE == kSumQuery;
  constexpr bool SUMS = MODE != kSumMax;  // state sums (of keys, or of queries)
  typedef SwzLane<LDQ, kSwzRows> OR;
  static_assert(sizeof(T) == 2 && (MT % 2) == 0, "bf16, 32-feature blocks");

  __shared__ __attribute__((aligned(16))) T Kb[2 * TQ];
  __shared__ __attribute__((aligned(16))) T Vb[SUMS ? 2 * TQ : 8];
  // key row norms (kSumQuery: logD of the rows), read as 16-byte vectors
  __shared__ __attribute__((aligned(16))) float knb[2][CR];
  __shared__ float ddb[QRY ? 2 : 1][QRY ? CR : 1];  // kSumQuery: -rowdot(dY, Y) of the rows
  __shared__ float wmax[4];

  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int part = blockIdx.x, hd = blockIdx.y, b = blockIdx.z;
  const size_t head = (size_t)b * a.H + hd;
  const T* Kh = (const T*)a.K + head * (size_t)a.L * D;
  const T* Vh = (const T*)a.V + head * (size_t)a.L * D;

  // W fragments of this wave's features: slot s = W[w FW + 16 mt + c][32 kb + kp(g, s)],
  // with the low parts of a bf16 split (see w_lo).  With 64 features per
  // wave and sums (where registers are short) they are read at every chunk,
  // half of the feature tiles at a time: the high parts from a copy in LDS
  // (staged below), the low parts from the fragment table a.Wfrag;
  // otherwise they are held in registers.
  constexpr bool LO_TABLE = kSplitW<T> && MT == 4 && SUMS;
  constexpr int MR = LO_TABLE ? 1 : MT;
  F Wf[MR][EB], Wl[SUMS ? MR : 1][EB];
  if constexpr (!LO_TABLE) {
    const Lane L = this_lane();
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int kb = 0; kb < EB; ++kb)
#pragma unroll
        for (int s = 0; s < 8; ++s) {
          const float x = a.W[(size_t)(w * FW + 16 * mt + L.c) * D + 32 * kb + kp(L.g, s)];
          Wf[mt][kb][s] = cvt<T>(x);
          if constexpr (SUMS) Wl[mt][kb][s] = w_lo<T>(x);
        }
  }
  typedef WFragLayout<G> WL;
  const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(a.Wfrag), (short)0, LO_TABLE ? (int)(WL::TOTAL * 64 * sizeof(F)) : 0, 0x00020000);
  // With the fragment table, the high parts of the wave's fragments are
  // staged once into LDS (8 KiB per wave; each wave reads back only its
  // own), so each chunk fetches only the low parts from memory.
  __shared__ __attribute__((aligned(16))) F Wsh[LO_TABLE ? 4 * WL::NA * 64 : 1];
  if constexpr (LO_TABLE) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int i = 0; i < WL::NA; ++i)
      Wsh[(w * WL::NA + i) * 64 + lane] = __builtin_bit_cast(
          F, __builtin_amdgcn_raw_buffer_load_b128(wrs, lane * (int)sizeof(F),
                                                   WL::a(w, i / EB, i % EB) * 64 * (int)sizeof(F), 0));
  }

  // rows of this part
  const TileMap tm(a.L, a.C, 32);
  const int tb = a.tile_end > a.tile_begin ? a.tile_begin : 0;
  const int n_tiles = (a.tile_end > a.tile_begin ? a.tile_end : tm.count_tiles()) - tb;
  int j0, j1;
  if (a.align > 0) {
    // whole units of `align` tiles (slices) per part; the last unit may be short
    const int nu = (n_tiles + a.align - 1) / a.align;
    j0 = tb + min(n_tiles, a.align * (int)((int64_t)part * nu / a.P2));
    j1 = tb + min(n_tiles, a.align * (int)((int64_t)(part + 1) * nu / a.P2));
  } else {
    j0 = tb + (int)((int64_t)part * n_tiles / a.P2);
    j1 = tb + (int)((int64_t)(part + 1) * n_tiles / a.P2);
  }
  int r0 = 0, r1 = 0;
  if (j1 > j0) {
    int s_, c_;
    tm.tile(j0, r0, c_);
    tm.tile(j1 - 1, s_, c_);
    r1 = s_ + c_;
  }
  const int nrows = r1 - r0, nch = (nrows + CR - 1) / CR;
  const size_t nbytes = (size_t)nrows * D * sizeof(T);
  const __amdgpu_buffer_rsrc_t rK = range_rsrc(Kh + (size_t)r0 * D, nbytes);
  const __amdgpu_buffer_rsrc_t rV = range_rsrc(Vh + (size_t)r0 * D, nbytes);
  const __amdgpu_buffer_rsrc_t rY =
      range_rsrc(QRY ? (const T*)a.Y + head * (size_t)a.L * D + (size_t)r0 * D : nullptr, QRY ? nbytes : 0);
  const __amdgpu_buffer_rsrc_t rL = range_rsrc(QRY ? a.logD + head * (size_t)a.L + r0 : nullptr,
                                               QRY ? (size_t)nrows * sizeof(float) : 0);

  // row exponent offsets: keys exp2(x log2(e) - koff - 0.5 log2(e) |k|^2);
  // queries (kSumQuery) exp2(x log2(e) - (logD - kshift log2(e)))
  const float half_log2M = 0.5f * __log2f((float)M);
  float sh = 0.f;  // the head's key shift (FAVOR+)
  if constexpr (SUMS && G::KIND == kFavor) {
    if (!QRY && a.part_max != nullptr) {
      // the largest of the parts' key maxima and the initial state's shift
      // (every workgroup of the head takes the same maximum)
      sh = a.init_shift != nullptr ? a.init_shift[head] : -INFINITY;
      const float* pm = a.part_max + head * (size_t)a.n_part_max;
      int i = 0;
      for (; i + 8 <= a.n_part_max; i += 8) {
        float x[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) x[k] = pm[i + k];
#pragma unroll
        for (int k = 0; k < 8; ++k) sh = fmaxf(sh, x[k]);
      }
      for (; i < a.n_part_max; ++i) sh = fmaxf(sh, pm[i]);
      if (part == 0 && threadIdx.x == 0) a.shift_out[head] = sh;
    } else {
      sh = a.shift[head];
    }
  }
  const float koff = (SUMS && G::KIND == kFavor) ? (QRY ? -sh * kLog2e : sh * kLog2e + half_log2M) : 0.f;
  constexpr float kscale = QRY ? 1.f : 0.5f * kLog2e;

  f32x4 S[SUMS ? MT : 1][SUMS ? ET : 1], Sz[SUMS ? MT : 1];
  if constexpr (SUMS) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
      for (int et = 0; et < ET; ++et) S[mt][et] = zero4();
      Sz[mt] = zero4();
    }
  }
  float vmax = -INFINITY;

  RowStage<T, D, CR, 256> sk, sv, sy;
  const int tid = threadIdx.x;
  // (kSumQuery: no norms; knb holds the rows' logD)
  constexpr bool NORMS = G::KIND == kFavor && !QRY;
  float* const knorm = NORMS ? knb[0] : nullptr;
  // kSumQuery: the rows' logD and their dots rowdot(dY, Y), from the
  // staged dY and Y chunks (a row's chunks sit in consecutive lanes).
  // FAVOR+: logD enters the exponent of the features (threads 0 .. CR-1
  // hold one row each, for knb); ReLU: the staged dY rows and the dots are
  // divided by D instead (each thread holds the logD of its chunks' rows),
  // as the walk rounds dN = dY / D.
  typedef RowStage<T, D, CR, 256> RS;
  float lreg[G::KIND == kFavor ? 1 : RS::PER] = {};
  auto fetch_q = [&](int row0, int t) {
    if constexpr (QRY) {
      sy.fetch(rY, row0, t);
      if constexpr (G::KIND == kFavor) {
        lreg[0] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rL, t < CR ? (row0 + t) * 4 : INT_MAX - 3, 0, 0));
      } else {
#pragma unroll
        for (int i = 0; i < RS::PER; ++i) {
          const int ch = t + i * 256;
          lreg[i] = __uint_as_float(
              __builtin_amdgcn_raw_buffer_load_b32(rL, ch < RS::NCH ? (row0 + ch / RS::CPR) * 4 : INT_MAX - 3, 0, 0));
        }
      }
    }
  };
  // (before the dY chunks are written to LDS: with ReLU it scales them)
  auto store_q = [&](int buf, int t) {
    if constexpr (QRY) {
      if (G::KIND == kFavor && t < CR) knb[buf][t] = lreg[0];
#pragma unroll
      for (int i = 0; i < RS::PER; ++i) {
        const int ch = t + i * 256;
        const int r = ch / RS::CPR, cc = ch - r * RS::CPR;
        T* dy = reinterpret_cast<T*>(&sv.v[i]);
        const T* yy = reinterpret_cast<const T*>(&sy.v[i]);
        float d = 0.f;
#pragma unroll
        for (int k = 0; k < RS::VEC; ++k) d += to_f32(dy[k]) * to_f32(yy[k]);
        if constexpr (G::KIND != kFavor) {
          const float rd = fast_exp2(-lreg[i]);  // 1 / D
#pragma unroll
          for (int k = 0; k < RS::VEC; ++k) dy[k] = cvt<T>(to_f32(dy[k]) * rd);
          d *= rd;
        }
        d = sum_lane_group<RS::CPR>(d);
        if (ch < RS::NCH && cc == 0) ddb[buf][r] = -d;
      }
    }
  };
  // value dropout: dropped elements of the value rows are zeroed when staged
  const Drop drop{a.drop_seed, a.drop_t, a.C, head};
  sk.fetch(rK, 0, tid);
  if constexpr (SUMS) sv.fetch(rV, 0, tid);
  fetch_q(0, tid);
  sk.template store_swz<LDQ>(Kb, knorm, tid);
  store_q(0, tid);
  if constexpr (SUMS) {
    if (DROP) sv.drop(drop, r0, tid);
    sv.template store_swz<LDQ>(Vb, nullptr, tid);
  }
  sk.fetch(rK, CR, tid);
  if constexpr (SUMS) sv.fetch(rV, CR, tid);
  fetch_q(CR, tid);
  __syncthreads();

  for (int ci = 0; ci < nch; ++ci) {
    const int bf = ci & 1;
    const int cnt = min(CR, nrows - ci * CR);
    // rows of chunk ci + 1 into the other buffer (its readers, chunk ci - 1,
    // finished before the last barrier); rows of chunk ci + 2 into registers
    {
      const int t2 = fresh_tid();
      sk.template store_swz<LDQ>(Kb + (bf ^ 1) * TQ, NORMS ? knb[bf ^ 1] : nullptr, t2);
      store_q(bf ^ 1, t2);
      if constexpr (SUMS) {
        if (DROP) sv.drop(drop, r0 + (ci + 1) * CR, t2);
        sv.template store_swz<LDQ>(Vb + (bf ^ 1) * TQ, nullptr, t2);
      }
      sk.fetch(rK, (ci + 2) * CR, t2);
      if constexpr (SUMS) sv.fetch(rV, (ci + 2) * CR, t2);
      fetch_q((ci + 2) * CR, t2);
    }
    const T* Ks = Kb + bf * TQ;
    const T* Vs = Vb + bf * TQ;
    const float* kn = knb[bf];
    const Lane L = fresh_lane();
    const OR oR(L);

    // every operand of the chunk is read before the first product (the
    // fence keeps the compiler from putting a wait before each product):
    // key rows, row norms and (sums) the value rows
    F kf[CT][EB];
#pragma unroll
    for (int st = 0; st < CT; ++st)
#pragma unroll
      for (int kb = 0; kb < EB; ++kb) kf[st][kb] = sfrag_rm(oR, Ks, 16 * st, 32 * kb);
    f32x4 knv[CT];
#pragma unroll
    for (int st = 0; st < CT; ++st) knv[st] = *(const f32x4*)&kn[16 * st + 4 * L.g];
    F vf[SUMS ? CT / 2 : 1][SUMS ? ET : 1];
    if constexpr (SUMS) {
#pragma unroll
      for (int rb = 0; rb < CT / 2; ++rb)
#pragma unroll
        for (int et = 0; et < ET; ++et) vf[rb][et] = sfrag_tr(oR, Vs, 32 * rb, 16 * et);
    }
    __builtin_amdgcn_sched_barrier(0);

    // features of the feature tiles [m0, m1) (rows past the chunk: zero),
    // then [S | z] += K~^T [V | 1] over the chunk's rows, 32 rows per product
    auto feat_update = [&](f32x4 (&Lk)[CT][MT], auto m0c, auto m1c) {
      constexpr int m0 = decltype(m0c)::value, m1 = decltype(m1c)::value;
#pragma unroll
      for (int st = 0; st < CT; ++st) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const bool ok = 16 * st + 4 * L.g + r < cnt;
          const float kc = ok ? koff + kscale * knv[st][r] : INFINITY;
#pragma unroll
          for (int mt = m0; mt < m1; ++mt) {
            float x = Lk[st][mt][r];
            if (G::KIND == kFavor) x = fast_exp2(x * kLog2e - kc);
            else x = ok ? fmaxf(x, 0.f) + a.relu_eps : 0.f;
            Lk[st][mt][r] = x;
          }
        }
      }
#pragma unroll
      for (int rb = 0; rb < CT / 2; ++rb) {
        F ones;  // the ones column of [V | 1] (kSumQuery: -rowdot(dY, Y))
        const int rem = cnt - 32 * rb - 4 * L.g;  // rows 32 rb + kp(g, s) < cnt
#pragma unroll
        for (int s = 0; s < 8; ++s) {
          const int rr = (s & 3) + 16 * (s >> 2);
          const float one = QRY ? ddb[bf][32 * rb + 4 * L.g + rr] : 1.f;
          ones[s] = cvt<T>(rr < rem ? one : 0.f);
        }
#pragma unroll
        for (int mt = m0; mt < m1; ++mt) {
          const F kt = tile_pair_frag<T>(Lk[2 * rb][mt], Lk[2 * rb + 1][mt]);
#pragma unroll
          for (int et = 0; et < ET; ++et) S[mt][et] = mma(S[mt][et], kt, vf[rb][et]);
          Sz[mt] = mma(Sz[mt], kt, ones);
        }
      }
    };

    // logits: Lk[st][mt] rows s = 16 st + 4 g + r, columns m = w FW + 16 mt + c
    f32x4 Lk[CT][MT];
    if constexpr (LO_TABLE) {
      typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
      const int lane = fresh_tid() & 63, wlane = lane * (int)sizeof(F);
#pragma unroll
      for (int m2 = 0; m2 < MT; m2 += 2) {
        F Wh[2][EB], Wt[2][EB];
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int kb = 0; kb < EB; ++kb) {
            Wh[i][kb] = Wsh[(w * WL::NA + (m2 + i) * EB + kb) * 64 + lane];
            Wt[i][kb] = __builtin_bit_cast(
                F, __builtin_amdgcn_raw_buffer_load_b128(wrs, wlane, WL::alo(w, m2 + i, kb) * 64 * (int)sizeof(F), 0));
          }
#pragma unroll
        for (int st = 0; st < CT; ++st)
#pragma unroll
          for (int i = 0; i < 2; ++i) {
            f32x4 acc = zero4();
#pragma unroll
            for (int kb = 0; kb < EB; ++kb) acc = mma(acc, kf[st][kb], Wh[i][kb]);
#pragma unroll
            for (int kb = 0; kb < EB; ++kb) acc = mma(acc, kf[st][kb], Wt[i][kb]);
            Lk[st][m2 + i] = acc;
          }
        if (m2 == 0) feat_update(Lk, std::integral_constant<int, 0>(), std::integral_constant<int, 2>());
        else feat_update(Lk, std::integral_constant<int, 2>(), std::integral_constant<int, 4>());
      }
    } else {
#pragma unroll
      for (int st = 0; st < CT; ++st) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          f32x4 acc = zero4();
#pragma unroll
          for (int kb = 0; kb < EB; ++kb) acc = mma(acc, kf[st][kb], Wf[mt][kb]);
          // (the maxima take the bf16 W alone: the shift only has to be
          // near the maximum, any constant cancels)
          if constexpr (kSplitW<T> && SUMS) {
#pragma unroll
            for (int kb = 0; kb < EB; ++kb) acc = mma(acc, kf[st][kb], Wl[mt][kb]);
          }
          Lk[st][mt] = acc;
        }
      }
    }

    if constexpr (!SUMS) {
      // the key exponent w.k - |k|^2/2 of the chunk's rows
#pragma unroll
      for (int st = 0; st < CT; ++st) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          float v = -INFINITY;
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) v = fmaxf(v, Lk[st][mt][r]);
          vmax = fmaxf(vmax, 16 * st + 4 * L.g + r < cnt ? v - 0.5f * knv[st][r] : -INFINITY);
        }
      }
    } else if constexpr (!LO_TABLE) {
      feat_update(Lk, std::integral_constant<int, 0>(), std::integral_constant<int, MT>());
    }
    __syncthreads();
  }

  if constexpr (SUMS) {
    float* out = a.out + (head * a.P2 + part) * (size_t)M * (D + 1);
    const Lane L = this_lane();
    const float vs = QRY ? a.drop_scale : 1.f;  // dN = s dY / D
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const size_t row = (size_t)(w * FW + 16 * mt + 4 * L.g + r) * (D + 1);
#pragma unroll
        for (int et = 0; et < ET; ++et) out[row + 16 * et + L.c] = vs * S[mt][et][r];
        if (L.c == 0) out[row + D] = Sz[mt][r];
      }
  } else {
    vmax = wave_max(vmax);
    if ((threadIdx.x & 63) == 0) wmax[w] = vmax;
    __syncthreads();
    if (threadIdx.x == 0) a.out[head * a.P2 + part] = fmaxf(fmaxf(wmax[0], wmax[1]), fmaxf(wmax[2], wmax[3]));
  }
}

// kshift[head] = max over the head's parts (and over init_shift, when given)
__global__ void kshift_reduce_kernel(const float* part_max, int P2, const float* init_shift, float* kshift, int BH) {
  const int head = blockIdx.x * blockDim.x + threadIdx.x;
  if (head >= BH) return;
  float v = init_shift != nullptr ? init_shift[head] : -INFINITY;
  const float* pm = part_max + (size_t)head * P2;
  // (eight parts' loads issued together)
  int p = 0;
  for (; p + 8 <= P2; p += 8) {
    float x[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = pm[p + i];
#pragma unroll
    for (int i = 0; i < 8; ++i) v = fmaxf(v, x[i]);
  }
  for (; p < P2; ++p) v = fmaxf(v, pm[p]);
  kshift[head] = v;
}

template <class G>
hipError_t launch_ksum(const KsumArgs& a, int mode, hipStream_t s) {
  const dim3 grid(a.P2, a.H, a.B);
  if (mode == kSumStates) {
    if (a.drop_t != 0) hipLaunchKernelGGL((ksum_kernel<G, kSumStates, true>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((ksum_kernel<G, kSumStates, false>), grid, dim3(256), 0, s, a);
  } else if (mode == kSumQuery) {
    // (dY is not masked: the dropout scale enters the output, the masks the walk)
    hipLaunchKernelGGL((ksum_kernel<G, kSumQuery, false>), grid, dim3(256), 0, s, a);
  } else {
    hipLaunchKernelGGL((ksum_kernel<G, kSumMax, false>), grid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_kshift_reduce(const float* part_max, int P2, const float* init_shift, float* kshift, int BH,
                                hipStream_t s) {
  hipLaunchKernelGGL(kshift_reduce_kernel, dim3((BH + 63) / 64), dim3(64), 0, s, part_max, P2, init_shift, kshift, BH);
  return hipGetLastError();
}

#define SLIM_INST_KSUM(T, D, FW, TR, KIND) \
  template hipError_t launch_ksum<Cfg<T, D, FW, TR, KIND>>(const KsumArgs&, int, hipStream_t);
SLIM_FOR_EACH_BF16_CONFIG(SLIM_INST_KSUM)

}  // namespace slim
