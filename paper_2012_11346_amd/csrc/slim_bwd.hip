// Backward sweep (Algorithm 1, one layer).
//
// bwd_walk: one workgroup per (batch, head, segment) walks its tiles in
// reverse.  It holds, per wave (features F_w), the state B after the current
// tile and the state cotangent G after the tile, both in registers:
//   b1  downdate B -= K~^T [V|1] (eq. 17); on the first tile of a segment the
//       exact segment-start state is loaded instead, which bounds the drift
//       of repeated downdates to one segment
//   b2  recompute the tile: scores A^T, N, D, Y (eq. 2 inside the tile)
//   b3  dN = dY / D, dD = -(dY . Y) / D
//   b4  dA^T = tril(V dN^T + 1 dD^T)
//   b5  dQ~ = [dN|dD] [S|z]^T + dA K~
//   b6  dK~ = [V|1] G^T + dA^T Q~                        (G after the tile)
//   b7  dV = K~ dS + A^T dN
//   b8  G += Q~^T [dN|dD]                                (eq. 18)
//   b9  feature-map chain rule: dq = (dQ~ . Q~) W - q rowsum(dQ~ . Q~) for
//       FAVOR+ (masked for ReLU), same for keys; dW partial sums
// Cross-feature sums (N, D, dV, dq, dk) go through a cross-wave reduction in
// LDS.  dW partials of every workgroup are summed by dw_reduce in a fixed
// order, so results are deterministic.
#include "slim_common.hpp"
#include "slim_kernels.hpp"

namespace slim {

template <class G>
__device__ __forceinline__ void load_w_frags_b(typename FragT<typename G::T>::type (&Wf)[G::MT][G::EB],
                                               const float* W, int w) {
  const int g = lane_g(), c = lane_c();
#pragma unroll
  for (int mt = 0; mt < G::MT; ++mt)
#pragma unroll
    for (int kb = 0; kb < G::EB; ++kb)
#pragma unroll
      for (int s = 0; s < 8; ++s)
        Wf[mt][kb][s] = cvt<typename G::T>(W[(size_t)(w * G::FW + 16 * mt + c) * G::D + 32 * kb + kp(g, s)]);
}

// W fragments contracting over features: slot s = W[w FW + 32 kb + kp][16 et + c]
template <class G>
__device__ __forceinline__ void load_wt_frags(typename FragT<typename G::T>::type (&WT)[G::MB][G::ET],
                                              const float* W, int w) {
  const int g = lane_g(), c = lane_c();
#pragma unroll
  for (int kb = 0; kb < G::MB; ++kb)
#pragma unroll
    for (int et = 0; et < G::ET; ++et)
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const int m = 32 * kb + kp(g, s);
        WT[kb][et][s] = cvt<typename G::T>(m < G::FW ? W[(size_t)(w * G::FW + m) * G::D + 16 * et + c] : 0.f);
      }
}

template <class G>
__device__ __forceinline__ typename FragT<typename G::T>::type pair_or_half(const f32x4& a, const f32x4& b,
                                                                             bool has_b) {
  return has_b ? tile_pair_frag<typename G::T>(a, b) : tile_half_frag<typename G::T>(a);
}

template <class G>
__global__ __launch_bounds__(256, 1) void bwd_walk_kernel(BwdArgs a) {
  typedef typename G::T T;
  typedef typename FragT<T>::type F;
  constexpr int D = G::D, FW = G::FW, M = G::M, TR = G::TR, MT = G::MT, MB = G::MB, ET = G::ET, EB = G::EB,
                RT = G::RT, RB = G::RB, LDQ = G::LDQ, LDR = G::LDR;
  // per-wave buffers (element pitches)
  constexpr int LDZK = TR + 8;  // [m][s] and [m][s] for K~, (dK~.K~)
  constexpr int LDZF = FW + 8;  // [e][m], [t][m] buffers
  constexpr int LDZT = TR + 8;  // [t][s] buffers
  constexpr int ZR = G::ZR;
  constexpr int REG_A = (ZR * LDZK > D * LDZF) ? ZR * LDZK : D * LDZF;  // Zk | ZS | ZG
  constexpr int REG_B = (TR * LDZT > TR * LDZF) ? TR * LDZT : TR * LDZF;  // ZA | ZP | Zq
  constexpr int REG_C = TR * LDZT;                                        // ZdA
  constexpr int REG_D = ZR * LDZK;                                        // ZPk
  constexpr int REG = REG_A + REG_B + REG_C + REG_D;

  __shared__ __attribute__((aligned(16))) T Qs[TR * LDQ];
  __shared__ __attribute__((aligned(16))) T Ks[TR * LDQ];
  __shared__ __attribute__((aligned(16))) T Vs[TR * LDQ];
  __shared__ __attribute__((aligned(16))) T dNs[TR * LDQ];
  __shared__ __attribute__((aligned(16))) T Zw[4][REG];
  __shared__ __attribute__((aligned(16))) float Red[4][TR * LDR];
  __shared__ float qn[TR], kn[TR], qmx[4][TR], dDs[TR], rsum[4][TR], dzs[4][FW];
  __shared__ __attribute__((aligned(16))) T dDb[TR + 8];

  const int w = wave_id(), g = lane_g(), c = lane_c();
  const int p = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const size_t head = (size_t)b * a.H + h;
  const size_t hoff = head * (size_t)a.L * D;
  const T* Qh = (const T*)a.Q + hoff;
  const T* Kh = (const T*)a.K + hoff;
  const T* Vh = (const T*)a.V + hoff;
  const T* dYh = (const T*)a.dY + hoff;
  T* dQh = (T*)a.dQ + hoff;
  T* dKh = (T*)a.dK + hoff;
  T* dVh = (T*)a.dV + hoff;

  T* ZA_ = Zw[w];                     // region A
  T* ZB_ = Zw[w] + REG_A;             // region B
  T* ZC_ = Zw[w] + REG_A + REG_B;     // region C
  T* ZD_ = ZC_ + REG_C;               // region D

  F Wf[MT][EB];
  load_w_frags_b<G>(Wf, a.W, w);
  F WT[MB][ET];
  load_wt_frags<G>(WT, a.W, w);

  const size_t SZ = (size_t)M * (D + 1);
  const size_t sidx = (head * a.P + p) * SZ;                 // per-segment arrays
  const float* bstart = a.bounds + (head * (a.P + 1) + p) * SZ;  // state before the segment
  const float* bend = bstart + SZ;                            // state after the segment
  // dstate_in is relative to the caller's initial key shift
  float r0 = 1.f;
  if (G::KIND == kFavor && a.init_shift != nullptr) r0 = fast_exp2((a.init_shift[head] - a.kshift[head]) * kLog2e);

  f32x4 S[MT][ET + 1], Gs[MT][ET + 1], dWacc[MT][ET];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const size_t row = (size_t)(w * FW + 16 * mt + 4 * g + r) * (D + 1);
#pragma unroll
      for (int et = 0; et < ET; ++et) {
        S[mt][et][r] = bend[row + 16 * et + c];
        Gs[mt][et][r] = a.seg_gend ? a.seg_gend[sidx + row + 16 * et + c] : 0.f;
      }
      S[mt][ET][r] = bend[row + D];
      Gs[mt][ET][r] = a.seg_gend ? a.seg_gend[sidx + row + D] : 0.f;
    }
#pragma unroll
    for (int et = 0; et < ET; ++et) dWacc[mt][et] = zero4();
  }

  // zero all per-wave buffers once: pad rows must read as zero
  for (int i = lane_id(); i < REG; i += 64) Zw[w][i] = cvt<T>(0.f);

  const TileMap tm(a.L, a.C, TR);
  const int n_tiles = tm.count_tiles();
  const int j0 = (int)((int64_t)p * n_tiles / a.P), j1 = (int)((int64_t)(p + 1) * n_tiles / a.P);
  const float half_log2M = 0.5f * __log2f((float)M);
  const float koff = (G::KIND == kFavor) ? a.kshift[head] * kLog2e + half_log2M : 0.f;
  constexpr int TPR = 256 / TR, EPT = D / TPR;

  for (int j = j1 - 1; j >= j0; --j) {
    int start, count;
    tm.tile(j, start, count);
    load_rows<T, D, TR, LDQ, 256>(Qs, Qh + (size_t)start * D, count, G::KIND == kFavor ? qn : nullptr);
    load_rows<T, D, TR, LDQ, 256>(Ks, Kh + (size_t)start * D, count, G::KIND == kFavor ? kn : nullptr);
    load_rows<T, D, TR, LDQ, 256>(Vs, Vh + (size_t)start * D, count, nullptr);
    __syncthreads();

    // ---- b2 (features)
    f32x4 Lq[MT][RT], Lk[RT][MT];
    {
#pragma unroll
      for (int tt = 0; tt < RT; ++tt) {
        const float init = (G::KIND == kFavor) ? -0.5f * qn[16 * tt + c] : 0.f;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          f32x4 acc = {init, init, init, init};
#pragma unroll
          for (int kb = 0; kb < EB; ++kb) acc = mma(acc, Wf[mt][kb], frag_rm(Qs, LDQ, 16 * tt, 32 * kb));
          Lq[mt][tt] = acc;
        }
      }
#pragma unroll
      for (int st = 0; st < RT; ++st) {
        f32x4 init;
#pragma unroll
        for (int r = 0; r < 4; ++r) init[r] = (G::KIND == kFavor) ? -0.5f * kn[16 * st + 4 * g + r] : 0.f;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          f32x4 acc = init;
#pragma unroll
          for (int kb = 0; kb < EB; ++kb) acc = mma(acc, frag_rm(Ks, LDQ, 16 * st, 32 * kb), Wf[mt][kb]);
          Lk[st][mt] = acc;
        }
      }
    }
    if (G::KIND == kFavor) {
#pragma unroll
      for (int tt = 0; tt < RT; ++tt) {
        float v = -INFINITY;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int r = 0; r < 4; ++r) v = fmaxf(v, Lq[mt][tt][r]);
        v = wave_max_over_g(v);
        if (g == 0) qmx[w][16 * tt + c] = v;
      }
    }
    __syncthreads();
#pragma unroll
    for (int st = 0; st < RT; ++st)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const bool ok = 16 * st + 4 * g + r < count;
          const float x = Lk[st][mt][r];
          Lk[st][mt][r] = !ok ? 0.f : (G::KIND == kFavor) ? fast_exp2(x * kLog2e - koff) : fmaxf(x, 0.f) + a.relu_eps;
        }
#pragma unroll
    for (int tt = 0; tt < RT; ++tt) {
      const int t = 16 * tt + c;
      float qs = 0.f;
      if (G::KIND == kFavor) qs = fmaxf(fmaxf(qmx[0][t], qmx[1][t]), fmaxf(qmx[2][t], qmx[3][t])) * kLog2e;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float x = Lq[mt][tt][r];
          Lq[mt][tt][r] =
              (t >= count) ? 0.f : (G::KIND == kFavor) ? fast_exp2(x * kLog2e - qs) : fmaxf(x, 0.f) + a.relu_eps;
        }
    }

    F vf[RB][ET + 1];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int et = 0; et <= ET; ++et) {
        if (et < ET) {
          vf[rb][et] = frag_tr(Vs, LDQ, 32 * rb, 16 * et);
        } else {
#pragma unroll
          for (int s = 0; s < 8; ++s) vf[rb][et][s] = cvt<T>((32 * rb + kp(g, s) < count) ? 1.f : 0.f);
        }
      }

    // ---- b1: state before the tile
    if (j == j0) {
      // the exact state before the segment replaces the downdated one
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const size_t row = (size_t)(w * FW + 16 * mt + 4 * g + r) * (D + 1);
#pragma unroll
          for (int et = 0; et < ET; ++et) S[mt][et][r] = bstart[row + 16 * et + c];
          S[mt][ET][r] = bstart[row + D];
        }
    } else {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int et = 0; et <= ET; ++et)
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) {
            F kf = tile_pair_frag<T>(Lk[2 * rb][mt], Lk[2 * rb + 1][mt]);
#pragma unroll
            for (int s = 0; s < 8; ++s) kf[s] = -kf[s];
            S[mt][et] = mma(S[mt][et], kf, vf[rb][et]);
          }
    }

    // K~ transposed: Zk[m][s]
    T* Zk = ZA_;
#pragma unroll
    for (int st = 0; st < RT; ++st)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) store_tile_T<T>(Zk, LDZK, Lk[st][mt], 16 * st, 16 * mt);
    __syncthreads();

    F qf[MB][RT];
#pragma unroll
    for (int kb = 0; kb < MB; ++kb)
#pragma unroll
      for (int tt = 0; tt < RT; ++tt) qf[kb][tt] = pair_or_half<G>(Lq[2 * kb][tt], Lq[2 * kb + 1][tt], 2 * kb + 1 < MT);

    // ---- b2: scores A^T[s][t] (this wave's features), causal
    f32x4 At[RT][RT];
#pragma unroll
    for (int tt = 0; tt < RT; ++tt)
#pragma unroll
      for (int st = 0; st < RT; ++st) {
        At[st][tt] = zero4();
        if (st > tt) continue;
#pragma unroll
        for (int kb = 0; kb < MB; ++kb) At[st][tt] = mma(At[st][tt], frag_tr(Zk, LDZK, 32 * kb, 16 * st), qf[kb][tt]);
        if (st == tt) {
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (4 * g + r > c) At[st][tt][r] = 0.f;
        }
      }
    // A^T transposed: ZA[t][s]
    T* ZA = ZB_;
#pragma unroll
    for (int st = 0; st < RT; ++st)
#pragma unroll
      for (int tt = 0; tt < RT; ++tt) store_tile_T<T>(ZA, LDZT, At[st][tt], 16 * st, 16 * tt);

    // N^T[e][t] partial into Red as [t][e]
    {
      F sf[MB][ET + 1];
#pragma unroll
      for (int kb = 0; kb < MB; ++kb)
#pragma unroll
        for (int et = 0; et <= ET; ++et) sf[kb][et] = pair_or_half<G>(S[2 * kb][et], S[2 * kb + 1][et], 2 * kb + 1 < MT);
#pragma unroll
      for (int tt = 0; tt < RT; ++tt)
#pragma unroll
        for (int et = 0; et <= ET; ++et) {
          f32x4 acc = zero4();
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) {
            if (2 * rb > tt) continue;
            acc = mma(acc, vf[rb][et], pair_or_half<G>(At[2 * rb][tt], At[2 * rb + 1][tt], 2 * rb + 1 <= tt));
          }
#pragma unroll
          for (int kb = 0; kb < MB; ++kb) acc = mma(acc, sf[kb][et], qf[kb][tt]);
          if (et < ET) {
            store_tile_T<float>(Red[w], LDR, acc, 16 * et, 16 * tt);
          } else if (g == 0) {
            Red[w][(16 * tt + c) * LDR + D] = acc[0];
          }
        }
    }
    __syncthreads();

    // ---- b3: dN, dD per row (threads: TPR per row)
    {
      const int t = threadIdx.x / TPR, q = threadIdx.x % TPR;
      float dy[EPT], n[EPT];
      float den = 1.f, dot = 0.f;
      const bool ok = t < count;
      den = Red[0][t * LDR + D] + Red[1][t * LDR + D] + Red[2][t * LDR + D] + Red[3][t * LDR + D];
      const float inv = ok ? 1.f / den : 0.f;
#pragma unroll
      for (int i = 0; i < EPT; ++i) {
        const int e = q * EPT + i;
        dy[i] = ok ? to_f32(dYh[(size_t)(start + t) * D + e]) : 0.f;
        n[i] = Red[0][t * LDR + e] + Red[1][t * LDR + e] + Red[2][t * LDR + e] + Red[3][t * LDR + e];
        dot += dy[i] * (n[i] * inv);
      }
#pragma unroll
      for (int o = 1; o < TPR; o <<= 1) dot += __shfl_xor(dot, o, 64);
#pragma unroll
      for (int i = 0; i < EPT; ++i) dNs[t * LDQ + q * EPT + i] = cvt<T>(dy[i] * inv);
      if (q == 0) {
        const float dd = ok ? -dot * inv : 0.f;
        dDs[t] = dd;
        dDb[t] = cvt<T>(dd);
      }
    }
    __syncthreads();

    // ---- b4: dA^T[s][t] = sum_e V[s][e] dN[t][e] + dD[t], causal
    f32x4 dAt[RT][RT];
#pragma unroll
    for (int tt = 0; tt < RT; ++tt) {
      const float ddt = dDs[16 * tt + c];
#pragma unroll
      for (int st = 0; st < RT; ++st) {
        dAt[st][tt] = zero4();
        if (st > tt) continue;
        f32x4 acc = {ddt, ddt, ddt, ddt};
#pragma unroll
        for (int kb = 0; kb < EB; ++kb)
          acc = mma(acc, frag_rm(Vs, LDQ, 16 * st, 32 * kb), frag_rm(dNs, LDQ, 16 * tt, 32 * kb));
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int s = 16 * st + 4 * g + r;
          if (st == tt && 4 * g + r > c) acc[r] = 0.f;
          if (s >= count) acc[r] = 0.f;
        }
        dAt[st][tt] = acc;
      }
    }
    // dA^T transposed: ZdA[t][s]
    T* ZdA = ZC_;
#pragma unroll
    for (int st = 0; st < RT; ++st)
#pragma unroll
      for (int tt = 0; tt < RT; ++tt) store_tile_T<T>(ZdA, LDZT, dAt[st][tt], 16 * st, 16 * tt);

    // ---- b7: dV^T[e][s] = sum_m dS[m][e] K~[s][m] + sum_t dN[t][e] A^T[s][t]  (Red as [s][e])
    {
#pragma unroll
      for (int st = 0; st < RT; ++st)
#pragma unroll
        for (int et = 0; et < ET; ++et) {
          f32x4 acc = zero4();
#pragma unroll
          for (int kb = 0; kb < MB; ++kb)
            acc = mma(acc, pair_or_half<G>(Gs[2 * kb][et], Gs[2 * kb + 1][et], 2 * kb + 1 < MT),
                      frag_tr(Zk, LDZK, 32 * kb, 16 * st));
#pragma unroll
          for (int rb = 0; rb < RB; ++rb)
            acc = mma(acc, frag_tr(dNs, LDQ, 32 * rb, 16 * et), frag_tr(ZA, LDZT, 32 * rb, 16 * st));
          store_tile_T<float>(Red[w], LDR, acc, 16 * et, 16 * st);
        }
    }
    __syncthreads();
    {
      const int t = threadIdx.x / TPR, q = threadIdx.x % TPR;
      if (t < count) {
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
          const int e = q * EPT + i;
          const float v = Red[0][t * LDR + e] + Red[1][t * LDR + e] + Red[2][t * LDR + e] + Red[3][t * LDR + e];
          dVh[(size_t)(start + t) * D + e] = cvt<T>(v);
        }
      }
    }
    __syncthreads();

    // ---- b5: dQ~^T[m][t] = sum_e S[m][e] dN[t][e] + z[m] dD[t] + sum_s K~[s][m] dA^T[s][t]
    T* ZS = ZA_;  // S transposed [e][m] (Zk no longer needed)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int et = 0; et < ET; ++et) store_tile_T<T>(ZS, LDZF, S[mt][et], 16 * mt, 16 * et);
    __syncthreads();
    f32x4 Pq[MT][RT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int tt = 0; tt < RT; ++tt) {
        const float ddt = dDs[16 * tt + c];
        f32x4 acc;
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[r] = S[mt][ET][r] * ddt;
#pragma unroll
        for (int kb = 0; kb < EB; ++kb)
          acc = mma(acc, frag_tr(ZS, LDZF, 32 * kb, 16 * mt), frag_rm(dNs, LDQ, 16 * tt, 32 * kb));
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
          acc = mma(acc, tile_pair_frag<T>(Lk[2 * rb][mt], Lk[2 * rb + 1][mt]),
                    pair_or_half<G>(dAt[2 * rb][tt], dAt[2 * rb + 1][tt], 2 * rb + 1 <= tt));
        // chain rule through the feature map (shift treated as a constant)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float qv = Lq[mt][tt][r];
          acc[r] = (G::KIND == kFavor) ? acc[r] * qv : (qv > a.relu_eps ? acc[r] : 0.f);
        }
        Pq[mt][tt] = acc;
      }
    // row sums over features (FAVOR+ needs q * rowsum)
    if (G::KIND == kFavor) {
#pragma unroll
      for (int tt = 0; tt < RT; ++tt) {
        float v = 0.f;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int r = 0; r < 4; ++r) v += Pq[mt][tt][r];
        v = wave_sum_over_g(v);
        if (g == 0) rsum[w][16 * tt + c] = v;
      }
    }
    // dq^T[e][t] = sum_m W[m][e] Pq[m][t]  (Red as [t][e])
#pragma unroll
    for (int tt = 0; tt < RT; ++tt)
#pragma unroll
      for (int et = 0; et < ET; ++et) {
        f32x4 acc = zero4();
#pragma unroll
        for (int kb = 0; kb < MB; ++kb)
          acc = mma(acc, WT[kb][et], pair_or_half<G>(Pq[2 * kb][tt], Pq[2 * kb + 1][tt], 2 * kb + 1 < MT));
        store_tile_T<float>(Red[w], LDR, acc, 16 * et, 16 * tt);
      }
    // dW[m][e] += sum_t Pq[m][t] Q[t][e]: Pq transposed into ZP[t][m]
    T* ZP = ZB_;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int tt = 0; tt < RT; ++tt) store_tile_T<T>(ZP, LDZF, Pq[mt][tt], 16 * mt, 16 * tt);
    __syncthreads();
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int et = 0; et < ET; ++et)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
          dWacc[mt][et] = mma(dWacc[mt][et], frag_tr(ZP, LDZF, 32 * rb, 16 * mt), frag_tr(Qs, LDQ, 32 * rb, 16 * et));
    {
      const int t = threadIdx.x / TPR, q = threadIdx.x % TPR;
      if (t < count) {
        const float rs = (G::KIND == kFavor) ? rsum[0][t] + rsum[1][t] + rsum[2][t] + rsum[3][t] : 0.f;
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
          const int e = q * EPT + i;
          float v = Red[0][t * LDR + e] + Red[1][t * LDR + e] + Red[2][t * LDR + e] + Red[3][t * LDR + e];
          if (G::KIND == kFavor) v -= to_f32(Qs[t * LDQ + e]) * rs;
          dQh[(size_t)(start + t) * D + e] = cvt<T>(v);
        }
      }
    }
    __syncthreads();

    // ---- b6: dK~[s][m] = sum_e V[s][e] G[m][e] + dz[m] + sum_t dA^T[s][t] Q~[t][m]
    T* ZG = ZA_;  // G transposed [e][m]
    T* Zq = ZB_;  // Q~ as [t][m]
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
      for (int et = 0; et < ET; ++et) store_tile_T<T>(ZG, LDZF, Gs[mt][et], 16 * mt, 16 * et);
#pragma unroll
      for (int tt = 0; tt < RT; ++tt) store_tile_T<T>(Zq, LDZF, Lq[mt][tt], 16 * mt, 16 * tt);
      if (c == 0) {
#pragma unroll
        for (int r = 0; r < 4; ++r) dzs[w][16 * mt + 4 * g + r] = Gs[mt][ET][r];
      }
    }
    __syncthreads();
    f32x4 Pk[RT][MT];
#pragma unroll
    for (int st = 0; st < RT; ++st)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        f32x4 acc;
        const float dz = dzs[w][16 * mt + c];
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[r] = (16 * st + 4 * g + r < count) ? dz : 0.f;
#pragma unroll
        for (int kb = 0; kb < EB; ++kb)
          acc = mma(acc, frag_rm(Vs, LDQ, 16 * st, 32 * kb), frag_tr(ZG, LDZF, 32 * kb, 16 * mt));
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
          acc = mma(acc, frag_tr(ZdA, LDZT, 32 * rb, 16 * st), frag_tr(Zq, LDZF, 32 * rb, 16 * mt));
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float kv = Lk[st][mt][r];
          acc[r] = (G::KIND == kFavor) ? acc[r] * kv : (kv > a.relu_eps ? acc[r] : 0.f);
        }
        Pk[st][mt] = acc;
      }
    if (G::KIND == kFavor) {
#pragma unroll
      for (int st = 0; st < RT; ++st)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          float v = 0.f;
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) v += Pk[st][mt][r];
          v = wave_sum_over_c(v);
          if (c == 0) rsum[w][16 * st + 4 * g + r] = v;
        }
    }
    // Pk transposed: ZPk[m][s]
    T* ZPk = ZD_;
#pragma unroll
    for (int st = 0; st < RT; ++st)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) store_tile_T<T>(ZPk, LDZK, Pk[st][mt], 16 * st, 16 * mt);
    // dW[m][e] += sum_s Pk[s][m] K[s][e]
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int et = 0; et < ET; ++et)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
          dWacc[mt][et] = mma(dWacc[mt][et], tile_pair_frag<T>(Pk[2 * rb][mt], Pk[2 * rb + 1][mt]),
                              frag_tr(Ks, LDQ, 32 * rb, 16 * et));
    __syncthreads();
    // dk^T[e][s] = sum_m W[m][e] Pk[s][m]  (Red as [s][e])
#pragma unroll
    for (int st = 0; st < RT; ++st)
#pragma unroll
      for (int et = 0; et < ET; ++et) {
        f32x4 acc = zero4();
#pragma unroll
        for (int kb = 0; kb < MB; ++kb) acc = mma(acc, WT[kb][et], frag_tr(ZPk, LDZK, 32 * kb, 16 * st));
        store_tile_T<float>(Red[w], LDR, acc, 16 * et, 16 * st);
      }
    __syncthreads();
    {
      const int t = threadIdx.x / TPR, q = threadIdx.x % TPR;
      if (t < count) {
        const float rs = (G::KIND == kFavor) ? rsum[0][t] + rsum[1][t] + rsum[2][t] + rsum[3][t] : 0.f;
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
          const int e = q * EPT + i;
          float v = Red[0][t * LDR + e] + Red[1][t * LDR + e] + Red[2][t * LDR + e] + Red[3][t * LDR + e];
          if (G::KIND == kFavor) v -= to_f32(Ks[t * LDQ + e]) * rs;
          dKh[(size_t)(start + t) * D + e] = cvt<T>(v);
        }
      }
    }

    // ---- b8: G[m][e] += sum_t Q~[t][m] [dN|dD][t][e]
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int et = 0; et <= ET; ++et)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          F bfr;
          if (et < ET) {
            bfr = frag_tr(dNs, LDQ, 32 * rb, 16 * et);
          } else {
#pragma unroll
            for (int s = 0; s < 8; ++s) bfr[s] = dDb[32 * rb + kp(g, s)];
          }
          Gs[mt][et] = mma(Gs[mt][et], frag_tr(Zq, LDZF, 32 * rb, 16 * mt), bfr);
        }
    __syncthreads();
  }

  // per-workgroup dW partial, rows of this wave's features
  float* dwp = a.dW_part + (head * a.P + p) * (size_t)M * D;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int et = 0; et < ET; ++et)
#pragma unroll
      for (int r = 0; r < 4; ++r) dwp[(size_t)(w * FW + 16 * mt + 4 * g + r) * D + 16 * et + c] = dWacc[mt][et][r];
  // state cotangent before the sequence
  if (p == 0 && a.dstate_in != nullptr) {
    float* gout = a.dstate_in + head * SZ;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const size_t row = (size_t)(w * FW + 16 * mt + 4 * g + r) * (D + 1);
#pragma unroll
        for (int et = 0; et < ET; ++et) gout[row + 16 * et + c] = r0 * Gs[mt][et][r];
        if (c == 0) gout[row + D] = r0 * Gs[mt][ET][r];
      }
  }
}

// dW[m][e] = sum over workgroups of the partials, in a fixed order
__global__ __launch_bounds__(256) void dw_reduce_kernel(const float* part, int nparts, int n, float* dW) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  float s = 0.f;
  for (int k = 0; k < nparts; ++k) s += part[(size_t)k * n + i];
  dW[i] = s;
}

template <class G>
hipError_t launch_bwd_walk(const BwdArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(bwd_walk_kernel<G>, dim3(a.P, a.H, a.B), dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int n = G::M * G::D;
  hipLaunchKernelGGL(dw_reduce_kernel, dim3((n + 255) / 256), dim3(256), 0, s, a.dW_part, a.B * a.H * a.P, n, a.dW);
  return hipGetLastError();
}

#define SLIM_INST_BWD(T, D, FW, TR, KIND) \
  template hipError_t launch_bwd_walk<Cfg<T, D, FW, TR, KIND>>(const BwdArgs&, hipStream_t);
SLIM_FOR_EACH_CONFIG(SLIM_INST_BWD)

}  // namespace slim
