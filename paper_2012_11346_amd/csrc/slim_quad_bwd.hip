// Backward of the quadratic within-slice mode: Algorithm 1's reverse sweep
// with each slice's gradients taken from the masked quadratic form of eq. 2.
// For slice n, with [S|z] the state before it (eq. 17 downdates it from the
// state after it) and G the state cotangent after it (eq. 18), rows t, s of
// the slice and A[t][s] = Q~_t . K~_s (s <= t):
//
//   query pass  N_t, D_t recomputed as in the forward; dN_t = s dY_t / D_t,
//               dD_t = -(dY_t . Y_t) / D_t (stored with the row shift of Q~);
//               dQ~_t = [S|z] [dN_t|dD_t] + sum_{s <= t} dA[t][s] K~_s with
//               dA[t][s] = dN_t . V_s + dD_t; dQ and the query share of dW
//   key pass    dK~_s = [V_s|1] G^T + sum_{t >= s} dA[t][s] Q~_t,
//               dV_s = K~_s G + sum_{t >= s} A[t][s] dN_t; dK, dV and the
//               key share of dW
//   G sum       G before the slice = G + sum_t Q~_t^T [dN_t|dD_t]
//
// The passes take the 32-row tiles of the slice in parallel (one workgroup
// per tile, or several tiles per workgroup) and recompute the features of
// the other side for every tile pair.  The states enter as fragment tables
// (state_frag_kernel), so that neither pass holds a state in registers or
// LDS.  Each tile's dW share is added to its workgroup's own partial (one
// slot per workgroup, kept across the slices); the partials are summed in a
// fixed order at the end.
#include "slim_common.hpp"
#include "slim_kernels.hpp"

namespace slim {

// Fragment tables of a state X = [S|z] (M x (D + 1), fp32) as bf16 operands:
//   block T1 [w][mt][kb]: slot s = X[w FW + 16 mt + c][32 kb + kp(g, s)]           (rows m, contracting over e)
//   block T2 [w][kb][et]: slot s = X[w FW + 32 kb + kp(g, s)][16 et + c] for et < ET,
//                         X[w FW + 32 kb + kp(g, s)][D] for et == ET               (contracting over m)
template <class G>
struct StateFragLayout {
  static constexpr int N1 = G::MT * G::EB;
  static constexpr int N2 = G::MB * (G::ET + 1);
  static constexpr int TOTAL = 4 * (N1 + N2);  // fragments per head
  __device__ static int t1(int w, int mt, int kb) { return w * N1 + mt * G::EB + kb; }
  __device__ static int t2(int w, int kb, int et) { return 4 * N1 + w * N2 + kb * (G::ET + 1) + et; }
};

// grid (TOTAL, BH, n states), 64 threads: one fragment per wave
template <class G>
__global__ __launch_bounds__(64) void state_frag_kernel(const float* X0, bf16x8* F0, const float* X1, bf16x8* F1) {
  typedef StateFragLayout<G> SL;
  constexpr int D = G::D, FW = G::FW, M = G::M, EB = G::EB, ET = G::ET;
  const int f = blockIdx.x, head = blockIdx.y;
  const float* X = (blockIdx.z ? X1 : X0) + (size_t)head * M * (D + 1);
  bf16x8* F = (blockIdx.z ? F1 : F0) + (size_t)head * SL::TOTAL * 64;
  const int lane = threadIdx.x, g = lane >> 4, c = lane & 15;
  bf16x8 v;
  if (f < 4 * SL::N1) {
    const int w = f / SL::N1, rem = f - w * SL::N1, mt = rem / EB, kb = rem - mt * EB;
    const float* row = X + (size_t)(w * FW + 16 * mt + c) * (D + 1) + 32 * kb;
#pragma unroll
    for (int s = 0; s < 8; ++s) v[s] = cvt<bf16>(row[kp(g, s)]);
  } else {
    const int f2 = f - 4 * SL::N1, w = f2 / SL::N2, rem = f2 - w * SL::N2, kb = rem / (ET + 1), et = rem - kb * (ET + 1);
    const int col = et < ET ? 16 * et + c : D;
#pragma unroll
    for (int s = 0; s < 8; ++s) v[s] = cvt<bf16>(X[(size_t)(w * FW + 32 * kb + kp(g, s)) * (D + 1) + col]);
  }
  F[(size_t)f * 64 + lane] = v;
}

// W fragments of wave w's feature tile mt for the logits: the bf16 values and
// their low parts, from the fragment table
template <class G>
struct QuadWb {
  typedef typename FragT<typename G::T>::type F;
  const F* tab;
  int lane;
  __device__ explicit QuadWb(const void* table) : tab((const F*)table), lane(lane_id()) {}
  __device__ __forceinline__ void get(int w, int mt, F (&hi)[G::EB], F (&lo)[G::EB]) const {
#pragma unroll
    for (int kb = 0; kb < G::EB; ++kb) {
      hi[kb] = tab[WFragLayout<G>::a(w, mt, kb) * 64 + lane];
      lo[kb] = tab[WFragLayout<G>::alo(w, mt, kb) * 64 + lane];
    }
  }
  __device__ __forceinline__ F b(int w, int kb, int et) const { return tab[WFragLayout<G>::b(w, kb, et) * 64 + lane]; }
};

// Query features of a staged 32-row tile into Zq[t][m] (this wave's
// features; rows past `count` zero).  FAVOR+ rows are shifted by `qs` (log2
// units): the query pass takes the row maxima (qmx, over all waves), the
// key pass and the G sum the shifts the query pass stored.
template <class G>
__device__ __forceinline__ void query_logits(const Lane& L, const QuadWb<G>& wt, int w, const typename G::T* Qs,
                                             f32x4 (&Lq)[G::MT][G::RT]) {
  typedef typename FragT<typename G::T>::type F;
#pragma unroll
  for (int mt = 0; mt < G::MT; ++mt) {
    F hi[G::EB], lo[G::EB];
    wt.get(w, mt, hi, lo);
#pragma unroll
    for (int tt = 0; tt < G::RT; ++tt) {
      f32x4 acc = zero4();
#pragma unroll
      for (int kb = 0; kb < G::EB; ++kb) {
        const F qf = frag_rm(L, Qs, G::D + 8, 16 * tt, 32 * kb);
        acc = mma(acc, hi[kb], qf);
        acc = mma(acc, lo[kb], qf);
      }
      Lq[mt][tt] = acc;
    }
  }
}

// Key features of a staged 32-row tile into Zk[m][s] (this wave's features;
// rows past `count` zero), as the forward forms them
template <class G>
__device__ __forceinline__ void key_features(const Lane& L, const QuadWb<G>& wt, int w, const typename G::T* Ks,
                                             const float* kn, float koff, int count, float eps, typename G::T* Zk) {
  typedef typename FragT<typename G::T>::type F;
  constexpr int LDZ = G::TR + 8;
#pragma unroll
  for (int mt = 0; mt < G::MT; ++mt) {
    F hi[G::EB], lo[G::EB];
    wt.get(w, mt, hi, lo);
#pragma unroll
    for (int st = 0; st < G::RT; ++st) {
      f32x4 acc = zero4();
#pragma unroll
      for (int kb = 0; kb < G::EB; ++kb) {
        const F kf = frag_rm(L, Ks, G::D + 8, 16 * st, 32 * kb);
        acc = mma(acc, kf, hi[kb]);
        acc = mma(acc, kf, lo[kb]);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int s = 16 * st + 4 * L.g + r;
        if (G::KIND == kFavor) {
          const float kc = s < count ? koff + 0.5f * kLog2e * kn[s] : INFINITY;
          acc[r] = fast_exp2(acc[r] * kLog2e - kc);
        } else {
          acc[r] = s < count ? plain_feature<G::KIND>(acc[r], eps) : 0.f;
        }
      }
      store_tile_T<typename G::T>(L, Zk, LDZ, acc, 16 * st, 16 * mt);
    }
  }
}

// Value rows of a key tile into LDS, dropped elements zeroed (value dropout)
template <class G, bool DROP>
__device__ __forceinline__ void load_values(typename G::T* Vs, const typename G::T* Vh, int k0, int kcount,
                                            const Drop& drop) {
  typedef typename G::T T;
  constexpr int D = G::D, TR = G::TR, LDQ = D + 8;
  if constexpr (DROP) {
    constexpr int VEC = 16 / sizeof(T), CPR = D / VEC;
    for (int ch = threadIdx.x; ch < TR * CPR; ch += 256) {
      const int r = ch / CPR, cc = ch - (ch / CPR) * CPR;
      uint4 v = {0u, 0u, 0u, 0u};
      if (r < kcount) v = *reinterpret_cast<const uint4*>(Vh + (size_t)(k0 + r) * D + cc * VEC);
      drop_chunk<T>(v, drop, k0 + r, cc * VEC);
      *reinterpret_cast<uint4*>(Vs + r * LDQ + cc * VEC) = v;
    }
  } else {
    load_rows<T, D, TR, LDQ, 256>(Vs, Vh + (size_t)k0 * D, kcount, nullptr);
  }
}

// dN (as operands), dD and the query row shifts of a query tile from the
// query pass's rows; rows past `count` zero
template <class G>
__device__ __forceinline__ void load_dn(typename G::T* dNs, float* dDs, float* qsh, const float* DNt, int count) {
  constexpr int D = G::D, TR = G::TR, TPR = 256 / TR, EPT = D / TPR;
  const int tid = threadIdx.x, tr = tid / TPR, q = tid % TPR;
  const bool ok = tr < count;
  const float* src = DNt + (size_t)tr * (D + 4);
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const int e = q * EPT + i;
    dNs[tr * (D + 8) + e] = cvt<typename G::T>(ok ? src[e] : 0.f);
  }
  if (q == 0) {
    dDs[tr] = ok ? src[D] : 0.f;
    qsh[tr] = ok ? src[D + 1] : 0.f;
  }
}

// dW[m][e] += sum_t P[m][t] X[t][e] over a 32-row tile, this wave's features:
// P as operand fragments pf(mt) (rows m, contracting over t), X staged in
// LDS; added to the workgroup's own partial (no other workgroup writes it)
template <class G, class PF>
__device__ __forceinline__ void add_dw_tile(const Lane& L, PF pf, const typename G::T* Xs, float* slot, int w) {
#pragma unroll
  for (int mt = 0; mt < G::MT; ++mt) {
    const auto p = pf(mt);
    f32x4 acc[G::ET];
#pragma unroll
    for (int et = 0; et < G::ET; ++et) acc[et] = mma(zero4(), p, frag_tr(L, Xs, G::D + 8, 0, 16 * et));
#pragma unroll
    for (int et = 0; et < G::ET; ++et)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float* q = slot + (size_t)(w * G::FW + 16 * mt + 4 * L.g + r) * G::D + 16 * et + L.c;
        *q += acc[et][r];
      }
  }
}

// ---------------------------------------------------------------- query pass

template <class G>
struct QuadDqLds {
  typedef typename G::T T;
  static constexpr int D = G::D, FW = G::FW, TR = G::TR, M = G::M;
  static constexpr int LDQ = D + 8, LDZ = TR + 8, LDF = FW + 8, LDR = D + 4;
  static constexpr size_t TILE = al16((size_t)TR * LDQ * sizeof(T));
  static constexpr size_t oQ = 0, oK = TILE, oV = 2 * TILE, odN = 3 * TILE;
  static constexpr size_t oF = 4 * TILE;  // floats: kn, qmx[4], dDs, rsum[4], zs[M]
  static constexpr size_t oW = oF + al16((10 * TR + M) * sizeof(float));
  // per wave: Zq [t][m]; then Zk [m][s] + dA [t][s], or the reduction rows
  static constexpr size_t Z1 = al16((size_t)TR * LDF * sizeof(T));
  static constexpr size_t ZK = al16((size_t)FW * LDZ * sizeof(T));
  static constexpr size_t ZA = al16((size_t)TR * LDZ * sizeof(T));
  static constexpr size_t RD = al16((size_t)TR * LDR * sizeof(float));
  static constexpr size_t X = (ZK + ZA > RD) ? ZK + ZA : RD;
  static constexpr size_t WAVE = Z1 + X;
  static constexpr size_t TOTAL = oW + 4 * WAVE;
};

template <class G, bool DROP>
__global__ __launch_bounds__(256, 2) void quad_dq_kernel(QuadArgs a) {
  typedef typename G::T T;
  typedef typename FragT<T>::type F;
  typedef QuadDqLds<G> Lay;
  typedef StateFragLayout<G> SL;
  constexpr int D = G::D, FW = G::FW, M = G::M, TR = G::TR, MT = G::MT, MB = G::MB, ET = G::ET, EB = G::EB,
                RT = G::RT;
  constexpr int LDQ = Lay::LDQ, LDZ = Lay::LDZ, LDF = Lay::LDF, LDR = Lay::LDR;
  constexpr int TPR = 256 / TR, EPT = D / TPR;
  static_assert(RT == 2 && G::RB == 1 && MT % 2 == 0, "32-row tiles, whole 32-deep feature blocks");

  __shared__ __attribute__((aligned(16))) char arena[Lay::TOTAL];
  T* Qs = (T*)(arena + Lay::oQ);
  T* Ks = (T*)(arena + Lay::oK);
  T* Vs = (T*)(arena + Lay::oV);
  T* dNs = (T*)(arena + Lay::odN);  // dY, then dN in place
  float* kn = (float*)(arena + Lay::oF);
  float* qmx = kn + TR;       // [4][TR]
  float* dDs = qmx + 4 * TR;  // [TR]
  float* rsum = dDs + TR;     // [4][TR]
  float* zs = rsum + 4 * TR;  // [M]
  const int w = wave_id();
  char* wz = arena + Lay::oW + (size_t)w * Lay::WAVE;
  T* Zq = (T*)wz;                         // Q~ as [t][m]; then P = chain-rule factor of dQ~, in place
  T* Zk = (T*)(wz + Lay::Z1);             // K~ as [m][s]
  T* ZdA = (T*)(wz + Lay::Z1 + Lay::ZK);  // dA as [t][s]
  auto red = [&](int ww) -> float* { return (float*)(arena + Lay::oW + (size_t)ww * Lay::WAVE + Lay::Z1); };

  const int hd = blockIdx.y, b = blockIdx.z;
  const size_t head = (size_t)b * a.H + hd;
  const size_t hoff = head * (size_t)a.L * D;
  const T* Qh = (const T*)a.Q + hoff;
  const T* Kh = (const T*)a.K + hoff;
  const T* Vh = (const T*)a.V + hoff;
  const T* dYh = (const T*)a.dY + hoff;
  T* dQh = (T*)a.dQ + hoff;
  float* DNh = a.DN + head * (size_t)a.C * (D + 4);
  const QuadWb<G> wt(a.Wfrag);
  const F* Sf = (const F*)a.Sfrag + head * (size_t)SL::TOTAL * 64;
  const int lane = lane_id();
  const Drop drop{a.drop_seed, a.drop_t, a.C, head};
  const float half_log2M = 0.5f * __log2f((float)M);
  const float koff = (G::KIND == kFavor) ? a.kshift[head] * kLog2e + half_log2M : 0.f;

  for (int m = threadIdx.x; m < M; m += 256) zs[m] = a.S[(head * M + m) * (size_t)(D + 1) + D];
  float* dw_slot = a.dW_part + (head * gridDim.x + blockIdx.x) * (size_t)M * D;

  const int nt = (a.rows + TR - 1) / TR;
  for (int t = blockIdx.x; t < nt; t += gridDim.x) {
    const int q0 = a.row0 + t * TR, qcount = min(TR, a.rows - t * TR);
    __syncthreads();  // the previous tile's readers of every shared buffer are done
    load_rows<T, D, TR, LDQ, 256>(Qs, Qh + (size_t)q0 * D, qcount, nullptr);
    load_rows<T, D, TR, LDQ, 256>(dNs, dYh + (size_t)q0 * D, qcount, nullptr);
    __syncthreads();
    Lane L = fresh_lane();

    // (1) query features, Q~ -> Zq[t][m] (rows past the tile zero)
    f32x4 Lq[MT][RT];
    query_logits<G>(L, wt, w, Qs, Lq);
    if (G::KIND == kFavor) {
#pragma unroll
      for (int tt = 0; tt < RT; ++tt) {
        float v = -INFINITY;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int r = 0; r < 4; ++r) v = fmaxf(v, Lq[mt][tt][r]);
        v = wave_max_over_g(v);
        if (L.g == 0) qmx[w * TR + 16 * tt + L.c] = v;
      }
      __syncthreads();
    }
#pragma unroll
    for (int tt = 0; tt < RT; ++tt) {
      const int tr = 16 * tt + L.c;
      const float qs = (G::KIND == kFavor)
                           ? fmaxf(fmaxf(qmx[tr], qmx[TR + tr]), fmaxf(qmx[2 * TR + tr], qmx[3 * TR + tr])) * kLog2e
                           : 0.f;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float x = Lq[mt][tt][r];
          Lq[mt][tt][r] = tr >= qcount ? 0.f
                          : (G::KIND == kFavor) ? fast_exp2(x * kLog2e - qs)
                                                : plain_feature<G::KIND>(x, a.relu_eps);
        }
        store_tile_T<T>(L, Zq, LDF, Lq[mt][tt], 16 * mt, 16 * tt);
      }
    }
    F qf[MB][RT];
#pragma unroll
    for (int kb = 0; kb < MB; ++kb)
#pragma unroll
      for (int tt = 0; tt < RT; ++tt) qf[kb][tt] = tile_pair_frag<T>(Lq[2 * kb][tt], Lq[2 * kb + 1][tt]);

    // (2) this wave's share of N^T[e][t]: the state before the slice, then
    // every key tile of the slice up to the diagonal (as in the forward)
    f32x4 nacc[ET + 1][RT];
#pragma unroll
    for (int et = 0; et <= ET; ++et)
#pragma unroll
      for (int tt = 0; tt < RT; ++tt) {
        f32x4 acc = zero4();
#pragma unroll
        for (int kb = 0; kb < MB; ++kb) acc = mma(acc, Sf[SL::t2(w, kb, et) * 64 + lane], qf[kb][tt]);
        nacc[et][tt] = acc;
      }
    for (int u = 0; u <= t; ++u) {
      const int k0 = a.row0 + u * TR, kcount = min(TR, a.rows - u * TR);
      __syncthreads();
      load_rows<T, D, TR, LDQ, 256>(Ks, Kh + (size_t)k0 * D, kcount, G::KIND == kFavor ? kn : nullptr);
      load_values<G, DROP>(Vs, Vh, k0, kcount, drop);
      __syncthreads();
      L = fresh_lane();
      key_features<G>(L, wt, w, Ks, kn, koff, kcount, a.relu_eps, Zk);
      const bool diag = (u == t);
      f32x4 At[RT][RT];
#pragma unroll
      for (int tt = 0; tt < RT; ++tt)
#pragma unroll
        for (int st = 0; st < RT; ++st) {
          f32x4 acc = zero4();
          if (!(diag && st > tt)) {
#pragma unroll
            for (int kb = 0; kb < MB; ++kb) acc = mma(acc, frag_tr(L, Zk, LDZ, 32 * kb, 16 * st), qf[kb][tt]);
            if (diag && st == tt) {
#pragma unroll
              for (int r = 0; r < 4; ++r)
                if (4 * L.g + r > L.c) acc[r] = 0.f;
            }
          }
          At[st][tt] = acc;
        }
#pragma unroll
      for (int tt = 0; tt < RT; ++tt) {
        const F af = tile_pair_frag<T>(At[0][tt], At[1][tt]);
#pragma unroll
        for (int et = 0; et < ET; ++et) nacc[et][tt] = mma(nacc[et][tt], frag_tr(L, Vs, LDQ, 0, 16 * et), af);
        nacc[ET][tt] = mma(nacc[ET][tt], ones_rows_frag(L, 0, kcount), af);
      }
    }

    // (3) the waves' shares of N meet in LDS (rows [t][e], e = D: D_t)
    L = fresh_lane();
#pragma unroll
    for (int tt = 0; tt < RT; ++tt) {
#pragma unroll
      for (int et = 0; et < ET; ++et) store_tile_T<float>(L, red(w), LDR, nacc[et][tt], 16 * et, 16 * tt);
      if (L.g == 0) red(w)[(16 * tt + L.c) * LDR + D] = nacc[ET][tt][0];
    }
    __syncthreads();
    // (4) per row: Y = s N / D, dN = s dY / D, dD = -(dY . Y) / D (dN in place
    // of dY); the rows and the row shift go to the key pass
    {
      const int tid = fresh_tid();
      const int tr = tid / TPR, q = tid % TPR;
      const bool ok = tr < qcount;
      const float den = (red(0)[tr * LDR + D] + red(1)[tr * LDR + D]) + (red(2)[tr * LDR + D] + red(3)[tr * LDR + D]);
      const float inv = ok ? 1.f / den : 0.f;
      const float invs = inv * a.drop_scale;
      float dy[EPT];
      float dot = 0.f;
#pragma unroll
      for (int i = 0; i < EPT; ++i) {
        const int e = q * EPT + i;
        dy[i] = to_f32(dNs[tr * LDQ + e]);
        const float n = (red(0)[tr * LDR + e] + red(1)[tr * LDR + e]) + (red(2)[tr * LDR + e] + red(3)[tr * LDR + e]);
        dot += dy[i] * (n * invs);
      }
      dot = sum_lane_group<TPR>(dot);
      float* dst = DNh + (size_t)(t * TR + tr) * (D + 4);
#pragma unroll
      for (int i = 0; i < EPT; ++i) {
        const int e = q * EPT + i;
        const float dn = dy[i] * invs;
        dNs[tr * LDQ + e] = cvt<T>(dn);
        if (ok) dst[e] = dn;
      }
      if (q == 0) {
        const float dd = ok ? -dot * inv : 0.f;
        dDs[tr] = dd;
        if (ok) {
          dst[D] = dd;
          dst[D + 1] = (G::KIND == kFavor) ? fmaxf(fmaxf(qmx[tr], qmx[TR + tr]), fmaxf(qmx[2 * TR + tr], qmx[3 * TR + tr])) * kLog2e
                                           : 0.f;
        }
      }
    }
    __syncthreads();  // the reduction rows are read; dN and dD visible

    // (5) dQ~^T[m][t] = sum_e S[m][e] dN[t][e] + z[m] dD[t] + sum_s K~[s][m] dA[t][s]
    L = fresh_lane();
    f32x4 dq[MT][RT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int tt = 0; tt < RT; ++tt) {
        const float ddt = dDs[16 * tt + L.c];
        f32x4 acc;
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[r] = zs[w * FW + 16 * mt + 4 * L.g + r] * ddt;
#pragma unroll
        for (int kb = 0; kb < EB; ++kb)
          acc = mma(acc, Sf[SL::t1(w, mt, kb) * 64 + lane], frag_rm(L, dNs, LDQ, 16 * tt, 32 * kb));
        dq[mt][tt] = acc;
      }
    for (int u = 0; u <= t; ++u) {
      const int k0 = a.row0 + u * TR, kcount = min(TR, a.rows - u * TR);
      __syncthreads();
      load_rows<T, D, TR, LDQ, 256>(Ks, Kh + (size_t)k0 * D, kcount, G::KIND == kFavor ? kn : nullptr);
      load_values<G, DROP>(Vs, Vh, k0, kcount, drop);
      __syncthreads();
      L = fresh_lane();
      key_features<G>(L, wt, w, Ks, kn, koff, kcount, a.relu_eps, Zk);
      // dA[t][s] = V[s] . dN[t] + dD[t] (causal; key rows past the tile zero) -> ZdA[t][s]
      const bool diag = (u == t);
#pragma unroll
      for (int tt = 0; tt < RT; ++tt) {
        const float ddt = dDs[16 * tt + L.c];
#pragma unroll
        for (int st = 0; st < RT; ++st) {
          f32x4 acc = zero4();
          if (!(diag && st > tt)) {
            acc = f32x4{ddt, ddt, ddt, ddt};
#pragma unroll
            for (int kb = 0; kb < EB; ++kb)
              acc = mma(acc, frag_rm(L, Vs, LDQ, 16 * st, 32 * kb), frag_rm(L, dNs, LDQ, 16 * tt, 32 * kb));
#pragma unroll
            for (int r = 0; r < 4; ++r)
              if (16 * st + 4 * L.g + r >= kcount || (diag && st == tt && 4 * L.g + r > L.c)) acc[r] = 0.f;
          }
          store_tile_T<T>(L, ZdA, LDZ, acc, 16 * st, 16 * tt);
        }
      }
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int tt = 0; tt < RT; ++tt)
          dq[mt][tt] = mma(dq[mt][tt], frag_rm(L, Zk, LDZ, 16 * mt, 0), frag_rm(L, ZdA, LDZ, 16 * tt, 0));
    }

    // (6) chain rule of the features: P = dQ~ . Q~ (FAVOR+) or dQ~ masked
    // (ReLU) -> Zq in place; FAVOR+ row sums of P
    L = fresh_lane();
    {
      float rs[RT];
#pragma unroll
      for (int tt = 0; tt < RT; ++tt) rs[tt] = 0.f;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int tt = 0; tt < RT; ++tt) {
          const f32x4 qv = load_tile_T(L, Zq, LDF, 16 * mt, 16 * tt);
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            dq[mt][tt][r] = vjp_factor<G::KIND>(dq[mt][tt][r], qv[r], 0.f, a.relu_eps);
            rs[tt] += dq[mt][tt][r];
          }
          store_tile_T<T>(L, Zq, LDF, dq[mt][tt], 16 * mt, 16 * tt);
        }
      if (G::KIND == kFavor) {
#pragma unroll
        for (int tt = 0; tt < RT; ++tt) {
          const float v = wave_sum_over_g(rs[tt]);
          if (L.g == 0) rsum[w * TR + 16 * tt + L.c] = v;
        }
      }
    }
    // dq^T[e][t] = sum_m W[m][e] P[m][t] -> reduction rows [t][e]; dW[m][e] += sum_t P[m][t] Q[t][e]
#pragma unroll
    for (int tt = 0; tt < RT; ++tt)
#pragma unroll
      for (int et = 0; et < ET; ++et) {
        f32x4 acc = zero4();
#pragma unroll
        for (int kb = 0; kb < MB; ++kb) acc = mma(acc, wt.b(w, kb, et), frag_rm(L, Zq, LDF, 16 * tt, 32 * kb));
        store_tile_T<float>(L, red(w), LDR, acc, 16 * et, 16 * tt);
      }
    add_dw_tile<G>(L, [&](int mt) { return frag_tr(L, Zq, LDF, 0, 16 * mt); }, Qs, dw_slot, w);
    __syncthreads();
    {
      const int tid = fresh_tid();
      const int tr = tid / TPR, q = tid % TPR;
      if (tr < qcount) {
        const float rsv = (G::KIND == kFavor) ? (rsum[tr] + rsum[TR + tr]) + (rsum[2 * TR + tr] + rsum[3 * TR + tr]) : 0.f;
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
          const int e = q * EPT + i;
          float v = (red(0)[tr * LDR + e] + red(1)[tr * LDR + e]) + (red(2)[tr * LDR + e] + red(3)[tr * LDR + e]);
          if (G::KIND == kFavor) v -= to_f32(Qs[tr * LDQ + e]) * rsv;
          dQh[(size_t)(q0 + tr) * D + e] = cvt<T>(v);
        }
      }
    }
  }
}

// ---------------------------------------------------------------- key pass

template <class G>
struct QuadDkLds {
  typedef typename G::T T;
  static constexpr int D = G::D, FW = G::FW, TR = G::TR, M = G::M;
  static constexpr int LDQ = D + 8, LDZ = TR + 8, LDF = FW + 8, LDR = D + 4;
  static constexpr size_t TILE = al16((size_t)TR * LDQ * sizeof(T));
  static constexpr size_t oK = 0, oV = TILE, oQ = 2 * TILE, odN = 3 * TILE;
  static constexpr size_t oF = 4 * TILE;  // floats: kn, dDs, qsh, rsum[4], dzs[M]
  static constexpr size_t oW = oF + al16((7 * TR + M) * sizeof(float));
  // per wave: Zk [m][s]; then Zq [t][m], or the reduction rows
  static constexpr size_t ZK = al16((size_t)FW * LDZ * sizeof(T));
  static constexpr size_t Z1 = al16((size_t)TR * LDF * sizeof(T));
  static constexpr size_t RD = al16((size_t)TR * LDR * sizeof(float));
  static constexpr size_t X = Z1 > RD ? Z1 : RD;
  static constexpr size_t WAVE = ZK + X;
  static constexpr size_t TOTAL = oW + 4 * WAVE;
};

template <class G, bool DROP>
__global__ __launch_bounds__(256, 2) void quad_dk_kernel(QuadArgs a) {
  typedef typename G::T T;
  typedef typename FragT<T>::type F;
  typedef QuadDkLds<G> Lay;
  typedef StateFragLayout<G> SL;
  constexpr int D = G::D, FW = G::FW, M = G::M, TR = G::TR, MT = G::MT, MB = G::MB, ET = G::ET, EB = G::EB,
                RT = G::RT;
  constexpr int LDQ = Lay::LDQ, LDZ = Lay::LDZ, LDF = Lay::LDF, LDR = Lay::LDR;
  constexpr int TPR = 256 / TR, EPT = D / TPR;
  static_assert(RT == 2 && G::RB == 1 && MT % 2 == 0, "32-row tiles, whole 32-deep feature blocks");

  __shared__ __attribute__((aligned(16))) char arena[Lay::TOTAL];
  T* Ks = (T*)(arena + Lay::oK);
  T* Vs = (T*)(arena + Lay::oV);
  T* Qs = (T*)(arena + Lay::oQ);
  T* dNs = (T*)(arena + Lay::odN);
  float* kn = (float*)(arena + Lay::oF);
  float* dDs = kn + TR;        // [TR]
  float* qsh = dDs + TR;       // [TR]
  float* rsum = qsh + TR;      // [4][TR]
  float* dzs = rsum + 4 * TR;  // [M]
  const int w = wave_id();
  char* wz = arena + Lay::oW + (size_t)w * Lay::WAVE;
  T* Zk = (T*)wz;              // K~ as [m][s]; then P = chain-rule factor of dK~, in place
  T* Zq = (T*)(wz + Lay::ZK);  // Q~ as [t][m]
  auto red = [&](int ww) -> float* { return (float*)(arena + Lay::oW + (size_t)ww * Lay::WAVE + Lay::ZK); };

  const int hd = blockIdx.y, b = blockIdx.z;
  const size_t head = (size_t)b * a.H + hd;
  const size_t hoff = head * (size_t)a.L * D;
  const T* Qh = (const T*)a.Q + hoff;
  const T* Kh = (const T*)a.K + hoff;
  const T* Vh = (const T*)a.V + hoff;
  T* dKh = (T*)a.dK + hoff;
  T* dVh = (T*)a.dV + hoff;
  const float* DNh = a.DN + head * (size_t)a.C * (D + 4);
  const QuadWb<G> wt(a.Wfrag);
  const F* Gf = (const F*)a.Gfrag + head * (size_t)SL::TOTAL * 64;
  const int lane = lane_id();
  const Drop drop{a.drop_seed, a.drop_t, a.C, head};
  const float half_log2M = 0.5f * __log2f((float)M);
  const float koff = (G::KIND == kFavor) ? a.kshift[head] * kLog2e + half_log2M : 0.f;

  for (int m = threadIdx.x; m < M; m += 256) dzs[m] = a.Gc[(head * M + m) * (size_t)(D + 1) + D];
  float* dw_slot = a.dW_part + (head * gridDim.x + blockIdx.x) * (size_t)M * D;

  const int nt = (a.rows + TR - 1) / TR;
  for (int si = blockIdx.x; si < nt; si += gridDim.x) {
    const int k0 = a.row0 + si * TR, kcount = min(TR, a.rows - si * TR);
    __syncthreads();  // the previous tile's readers of every shared buffer are done
    load_rows<T, D, TR, LDQ, 256>(Ks, Kh + (size_t)k0 * D, kcount, G::KIND == kFavor ? kn : nullptr);
    load_values<G, DROP>(Vs, Vh, k0, kcount, drop);
    __syncthreads();
    Lane L = fresh_lane();
    key_features<G>(L, wt, w, Ks, kn, koff, kcount, a.relu_eps, Zk);

    // the cotangent after the slice: dK~[s][m] = sum_e V[s][e] G[m][e] + dz[m];
    // dV^T[e][s] = sum_m G[m][e] K~[s][m] (this wave's features)
    f32x4 dk[RT][MT], dv[ET][RT];
#pragma unroll
    for (int st = 0; st < RT; ++st)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const float dz = dzs[w * FW + 16 * mt + L.c];
        f32x4 acc;
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[r] = (16 * st + 4 * L.g + r < kcount) ? dz : 0.f;
#pragma unroll
        for (int kb = 0; kb < EB; ++kb)
          acc = mma(acc, frag_rm(L, Vs, LDQ, 16 * st, 32 * kb), Gf[SL::t1(w, mt, kb) * 64 + lane]);
        dk[st][mt] = acc;
      }
#pragma unroll
    for (int et = 0; et < ET; ++et)
#pragma unroll
      for (int st = 0; st < RT; ++st) {
        f32x4 acc = zero4();
#pragma unroll
        for (int kb = 0; kb < MB; ++kb) acc = mma(acc, Gf[SL::t2(w, kb, et) * 64 + lane], frag_tr(L, Zk, LDZ, 32 * kb, 16 * st));
        dv[et][st] = acc;
      }

    // every query tile of the slice from the diagonal on
    for (int t = si; t < nt; ++t) {
      const int q0 = a.row0 + t * TR, qcount = min(TR, a.rows - t * TR);
      __syncthreads();
      load_rows<T, D, TR, LDQ, 256>(Qs, Qh + (size_t)q0 * D, qcount, nullptr);
      load_dn<G>(dNs, dDs, qsh, DNh + (size_t)t * TR * (D + 4), qcount);
      __syncthreads();
      L = fresh_lane();
      // Q~ with the query pass's row shifts -> Zq[t][m]
      {
        f32x4 Lq[MT][RT];
        query_logits<G>(L, wt, w, Qs, Lq);
#pragma unroll
        for (int tt = 0; tt < RT; ++tt) {
          const int tr = 16 * tt + L.c;
          const float qs = qsh[tr];
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const float x = Lq[mt][tt][r];
              Lq[mt][tt][r] = tr >= qcount ? 0.f
                              : (G::KIND == kFavor) ? fast_exp2(x * kLog2e - qs)
                                                    : plain_feature<G::KIND>(x, a.relu_eps);
            }
            store_tile_T<T>(L, Zq, LDF, Lq[mt][tt], 16 * mt, 16 * tt);
          }
        }
      }
      // A[t][s] over this wave's features and dA[t][s] = dN[t] . V[s] + dD[t]
      // (causal on the diagonal tile; key rows past the tile zero); then
      // dV^T[e][s] += sum_t dN[t][e] A[t][s], dK~[s][m] += sum_t dA[t][s] Q~[t][m]
      const bool diag = (t == si);
#pragma unroll
      for (int st = 0; st < RT; ++st) {
        f32x4 aw[RT], da[RT];
#pragma unroll
        for (int tt = 0; tt < RT; ++tt) {
          f32x4 x = zero4(), y = zero4();
          if (!(diag && st > tt)) {
#pragma unroll
            for (int kb = 0; kb < MB; ++kb)
              x = mma(x, frag_rm(L, Zq, LDF, 16 * tt, 32 * kb), frag_tr(L, Zk, LDZ, 32 * kb, 16 * st));
#pragma unroll
            for (int r = 0; r < 4; ++r) y[r] = dDs[16 * tt + 4 * L.g + r];
#pragma unroll
            for (int kb = 0; kb < EB; ++kb)
              y = mma(y, frag_rm(L, dNs, LDQ, 16 * tt, 32 * kb), frag_rm(L, Vs, LDQ, 16 * st, 32 * kb));
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int sc = 16 * st + L.c;
              if (sc >= kcount || (diag && sc > 16 * tt + 4 * L.g + r)) {
                x[r] = 0.f;
                y[r] = 0.f;
              }
            }
          }
          aw[tt] = x;
          da[tt] = y;
        }
        const F awf = tile_pair_frag<T>(aw[0], aw[1]);
        const F daf = tile_pair_frag<T>(da[0], da[1]);
#pragma unroll
        for (int et = 0; et < ET; ++et) dv[et][st] = mma(dv[et][st], frag_tr(L, dNs, LDQ, 0, 16 * et), awf);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) dk[st][mt] = mma(dk[st][mt], daf, frag_tr(L, Zq, LDF, 0, 16 * mt));
      }
    }

    // chain rule of the key features: P = dK~ . K~ (FAVOR+) or masked (ReLU)
    // -> Zk in place; FAVOR+ row sums of P
    L = fresh_lane();
    {
      float rk[RT][4];
#pragma unroll
      for (int st = 0; st < RT; ++st)
#pragma unroll
        for (int r = 0; r < 4; ++r) rk[st][r] = 0.f;
#pragma unroll
      for (int st = 0; st < RT; ++st)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const f32x4 kv = load_tile_T(L, Zk, LDZ, 16 * st, 16 * mt);
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            dk[st][mt][r] = vjp_factor<G::KIND>(dk[st][mt][r], kv[r], 0.f, a.relu_eps);
            rk[st][r] += dk[st][mt][r];
          }
          store_tile_T<T>(L, Zk, LDZ, dk[st][mt], 16 * st, 16 * mt);
        }
      if (G::KIND == kFavor) {
#pragma unroll
        for (int st = 0; st < RT; ++st)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float v = wave_sum_over_c(rk[st][r]);
            if (L.c == 0) rsum[w * TR + 16 * st + 4 * L.g + r] = v;
          }
      }
    }
    // dk^T[e][s] = sum_m W[m][e] P[m][s] -> reduction rows [s][e]; dW[m][e] += sum_s P[m][s] K[s][e]
#pragma unroll
    for (int st = 0; st < RT; ++st)
#pragma unroll
      for (int et = 0; et < ET; ++et) {
        f32x4 acc = zero4();
#pragma unroll
        for (int kb = 0; kb < MB; ++kb) acc = mma(acc, wt.b(w, kb, et), frag_tr(L, Zk, LDZ, 32 * kb, 16 * st));
        store_tile_T<float>(L, red(w), LDR, acc, 16 * et, 16 * st);
      }
    add_dw_tile<G>(L, [&](int mt) { return frag_rm(L, Zk, LDZ, 16 * mt, 0); }, Ks, dw_slot, w);
    __syncthreads();
    {
      const int tid = fresh_tid();
      const int tr = tid / TPR, q = tid % TPR;
      if (tr < kcount) {
        const float rkv = (G::KIND == kFavor) ? (rsum[tr] + rsum[TR + tr]) + (rsum[2 * TR + tr] + rsum[3 * TR + tr]) : 0.f;
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
          const int e = q * EPT + i;
          float v = (red(0)[tr * LDR + e] + red(1)[tr * LDR + e]) + (red(2)[tr * LDR + e] + red(3)[tr * LDR + e]);
          if (G::KIND == kFavor) v -= to_f32(Ks[tr * LDQ + e]) * rkv;
          dKh[(size_t)(k0 + tr) * D + e] = cvt<T>(v);
        }
      }
    }
    __syncthreads();  // the reduction rows are read
    L = fresh_lane();
#pragma unroll
    for (int et = 0; et < ET; ++et)
#pragma unroll
      for (int st = 0; st < RT; ++st) store_tile_T<float>(L, red(w), LDR, dv[et][st], 16 * et, 16 * st);
    __syncthreads();
    {
      const int tid = fresh_tid();
      const int tr = tid / TPR, q = tid % TPR;
      if (tr < kcount) {
        const unsigned keep = DROP ? drop_keep_bits<EPT>(drop, k0 + tr, q * EPT) : ~0u;
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
          const int e = q * EPT + i;
          const float v = (red(0)[tr * LDR + e] + red(1)[tr * LDR + e]) + (red(2)[tr * LDR + e] + red(3)[tr * LDR + e]);
          dVh[(size_t)(k0 + tr) * D + e] = cvt<T>((keep >> i) & 1u ? v : 0.f);
        }
      }
    }
  }
}

// ---------------------------------------------------------------- G sum

template <class G>
struct QuadGsumLds {
  typedef typename G::T T;
  static constexpr int D = G::D, FW = G::FW, TR = G::TR;
  static constexpr int LDQ = D + 8, LDF = FW + 8, LDD = 24;
  static constexpr size_t TILE = al16((size_t)TR * LDQ * sizeof(T));
  static constexpr size_t oQ = 0, odN = TILE, odD = 2 * TILE;  // dD as column 0 of a [TR][16] tile
  static constexpr size_t oF = odD + al16((size_t)TR * LDD * sizeof(T));  // floats: dDs, qsh
  static constexpr size_t oW = oF + al16(2 * TR * sizeof(float));
  static constexpr size_t Z1 = al16((size_t)TR * LDF * sizeof(T));
  static constexpr size_t TOTAL = oW + 4 * Z1;
};

// part x of the slice's query tiles: sum_t Q~_t^T [dN_t|dD_t] -> out[B,H,x]
template <class G>
__global__ __launch_bounds__(256, 2) void quad_gsum_kernel(QuadArgs a) {
  typedef typename G::T T;
  typedef QuadGsumLds<G> Lay;
  constexpr int D = G::D, FW = G::FW, M = G::M, TR = G::TR, MT = G::MT, ET = G::ET, RT = G::RT;
  constexpr int LDQ = Lay::LDQ, LDF = Lay::LDF, LDD = Lay::LDD;
  static_assert(RT == 2 && G::RB == 1, "32-row tiles");

  __shared__ __attribute__((aligned(16))) char arena[Lay::TOTAL];
  T* Qs = (T*)(arena + Lay::oQ);
  T* dNs = (T*)(arena + Lay::odN);
  T* dDt = (T*)(arena + Lay::odD);
  float* dDs = (float*)(arena + Lay::oF);
  float* qsh = dDs + TR;
  const int w = wave_id();
  T* Zq = (T*)(arena + Lay::oW + (size_t)w * Lay::Z1);

  const int part = blockIdx.x, hd = blockIdx.y, b = blockIdx.z;
  const size_t head = (size_t)b * a.H + hd;
  const T* Qh = (const T*)a.Q + head * (size_t)a.L * D;
  const float* DNh = a.DN + head * (size_t)a.C * (D + 4);
  const QuadWb<G> wt(a.Wfrag);

  f32x4 Gp[MT][ET + 1];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int et = 0; et <= ET; ++et) Gp[mt][et] = zero4();

  const int nt = (a.rows + TR - 1) / TR;
  const int t0 = (int)((int64_t)part * nt / gridDim.x), t1 = (int)((int64_t)(part + 1) * nt / gridDim.x);
  for (int t = t0; t < t1; ++t) {
    const int q0 = a.row0 + t * TR, qcount = min(TR, a.rows - t * TR);
    __syncthreads();
    load_rows<T, D, TR, LDQ, 256>(Qs, Qh + (size_t)q0 * D, qcount, nullptr);
    load_dn<G>(dNs, dDs, qsh, DNh + (size_t)t * TR * (D + 4), qcount);
    __syncthreads();
    if (threadIdx.x < TR) {
#pragma unroll
      for (int j = 0; j < 16; ++j) dDt[threadIdx.x * LDD + j] = cvt<T>(j == 0 ? dDs[threadIdx.x] : 0.f);
    }
    Lane L = fresh_lane();
    {
      f32x4 Lq[MT][RT];
      query_logits<G>(L, wt, w, Qs, Lq);
#pragma unroll
      for (int tt = 0; tt < RT; ++tt) {
        const int tr = 16 * tt + L.c;
        const float qs = qsh[tr];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float x = Lq[mt][tt][r];
            Lq[mt][tt][r] = tr >= qcount ? 0.f
                            : (G::KIND == kFavor) ? fast_exp2(x * kLog2e - qs)
                                                  : plain_feature<G::KIND>(x, a.relu_eps);
          }
          store_tile_T<T>(L, Zq, LDF, Lq[mt][tt], 16 * mt, 16 * tt);
        }
      }
    }
    __syncthreads();  // dDt visible
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const auto qa = frag_tr(L, Zq, LDF, 0, 16 * mt);
#pragma unroll
      for (int et = 0; et < ET; ++et) Gp[mt][et] = mma(Gp[mt][et], qa, frag_tr(L, dNs, LDQ, 0, 16 * et));
      Gp[mt][ET] = mma(Gp[mt][ET], qa, frag_tr(L, dDt, LDD, 0, 0));
    }
  }
  float* o = a.out + (head * gridDim.x + part) * (size_t)M * (D + 1);
  const Lane L = this_lane();
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const size_t row = (size_t)(w * FW + 16 * mt + 4 * L.g + r) * (D + 1);
#pragma unroll
      for (int et = 0; et < ET; ++et) o[row + 16 * et + L.c] = Gp[mt][et][r];
      if (L.c == 0) o[row + D] = Gp[mt][ET][r];
    }
}

// ---------------------------------------------------------------- launchers

template <class G>
hipError_t launch_quad_dq(const QuadArgs& a, int nwg, hipStream_t s) {
  const dim3 grid(nwg, a.H, a.B);
  if (a.drop_t != 0) hipLaunchKernelGGL((quad_dq_kernel<G, true>), grid, dim3(256), 0, s, a);
  else hipLaunchKernelGGL((quad_dq_kernel<G, false>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

template <class G>
hipError_t launch_quad_dk(const QuadArgs& a, int nwg, hipStream_t s) {
  const dim3 grid(nwg, a.H, a.B);
  if (a.drop_t != 0) hipLaunchKernelGGL((quad_dk_kernel<G, true>), grid, dim3(256), 0, s, a);
  else hipLaunchKernelGGL((quad_dk_kernel<G, false>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

template <class G>
hipError_t launch_quad_gsum(const QuadArgs& a, int nwg, hipStream_t s) {
  hipLaunchKernelGGL((quad_gsum_kernel<G>), dim3(nwg, a.H, a.B), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <class G>
hipError_t launch_state_frag(const float* X0, void* F0, const float* X1, void* F1, int BH, hipStream_t s) {
  hipLaunchKernelGGL((state_frag_kernel<G>), dim3(StateFragLayout<G>::TOTAL, BH, X1 != nullptr ? 2 : 1), dim3(64), 0, s,
                     X0, (bf16x8*)F0, X1, (bf16x8*)F1);
  return hipGetLastError();
}

template <class G>
size_t state_frag_bytes() {
  return (size_t)StateFragLayout<G>::TOTAL * 64 * sizeof(bf16x8);
}

#define SLIM_INST_QUAD_BWD(T, D, FW, TR, KIND)                                                                  \
  template hipError_t launch_quad_dq<Cfg<T, D, FW, TR, KIND>>(const QuadArgs&, int, hipStream_t);             \
  template hipError_t launch_quad_dk<Cfg<T, D, FW, TR, KIND>>(const QuadArgs&, int, hipStream_t);             \
  template hipError_t launch_quad_gsum<Cfg<T, D, FW, TR, KIND>>(const QuadArgs&, int, hipStream_t);           \
  template hipError_t launch_state_frag<Cfg<T, D, FW, TR, KIND>>(const float*, void*, const float*, void*, int, \
                                                                 hipStream_t);                                \
  template size_t state_frag_bytes<Cfg<T, D, FW, TR, KIND>>();
SLIM_FOR_EACH_QUAD_CONFIG(SLIM_INST_QUAD_BWD)

}  // namespace slim
