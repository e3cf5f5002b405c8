// Carried state cotangent of the segmented reverse walk.
//
// The reverse walk of segment p starts from the cotangent G = 0 (segment
// P - 1: the caller's dstate_out), i.e. it leaves out G_end(p), the
// cotangent of the state after the segment that all later segments
// contribute (eq. 18 summed over them).  G enters the gradients of a row s
// only linearly, through
//   dV[s]  += K~[s] G                (the row's key feature against the state cotangent)
//   dK~[s] += [V[s] | 1] G^T         (and from there dk and dW through the feature map)
// so the missing part is added afterwards, row by row, once G_end(p) is known
// from a reverse scan of the per-segment totals:
//   dV[s]  += K~[s] G_end(p)
//   Pk[s]   = ([V[s] | 1] G_end(p)^T) . K~[s]          (FAVOR+; ReLU: masked where w.k <= 0)
//   dk[s]  += Pk[s] W - k[s] rowsum(Pk[s])              (FAVOR+; ReLU: Pk[s] W)
//   dW     += sum_s Pk[s]^T k[s]
// One workgroup per (segment p < P - 1, batch, head); wave w holds G_end(p)
// and W for its features as operand fragments and walks the segment's rows
// in 32-row tiles (no causal coupling between rows here).  Cross-feature sums
// go through per-wave reduction rows in LDS.
#include "slim_common.hpp"
#include "slim_kernels.hpp"

namespace slim {

template <class G>
__global__ __launch_bounds__(256, 1) void carry_kernel(CarryArgs a) {
  typedef typename G::T T;
  typedef typename FragT<T>::type F;
  typedef WFragLayout<G> WL;
  constexpr int D = G::D, FW = G::FW, M = G::M, TR = G::TR, MT = G::MT, MB = G::MB, ET = G::ET, EB = G::EB,
                RT = G::RT, LDQ = G::LDQ, LDR = G::LDR, LDF = G::LDF;
  constexpr bool ODD = (MT & 1) != 0;
  constexpr int NT = 256, TPR = NT / TR, EPT = D / TPR;
  static_assert(RT == 2 && G::RB == 1, "32-row tiles");
  static_assert(EPT % 4 == 0 && LDR % 4 == 0, "reduction rows are read as 16-byte vectors");

  __shared__ __attribute__((aligned(16))) T Ks[TR * LDQ];
  __shared__ __attribute__((aligned(16))) T Vs[TR * LDQ];
  __shared__ __attribute__((aligned(16))) float RedV[4][TR * LDR];
  __shared__ __attribute__((aligned(16))) float RedK[4][TR * LDR];
  __shared__ __attribute__((aligned(16))) T ZPk[4][TR * LDF];  // Pk as [s][m], per wave
  __shared__ float kn[TR];

  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane_g(), c = lane_c(), lane = lane_id();
  const int p = blockIdx.x, hd = blockIdx.y, b = blockIdx.z;
  const size_t head = (size_t)b * a.H + hd;
  const size_t hoff = head * (size_t)a.L * D;
  const T* Kh = (const T*)a.K + hoff;
  const T* Vh = (const T*)a.V + hoff;
  T* dKh = (T*)a.dK + hoff;
  T* dVh = (T*)a.dV + hoff;
  const size_t SZ = (size_t)M * (D + 1);
  const float* Ge = a.gend + (head * a.P + p) * SZ;  // G_end(p), rows m, columns e (column D: ones)
  const F* Wfr = reinterpret_cast<const F*>(a.Wfrag);

  // operand fragments of G_end and W for this wave's features
  F GA[MB][ET];  // slot s = G[w FW + 32 kb + kp][16 et + c]: contracts over features
  F GM[MT][EB];  // slot s = G[w FW + 16 mt + c][32 kb + kp]: contracts over value columns
  f32x4 gz[MT];  // ones column, rows m = w FW + 16 mt + 4 g + r
  F Wf[MT][EB], WB[MB][ET];
#pragma unroll
  for (int kb = 0; kb < MB; ++kb)
#pragma unroll
    for (int et = 0; et < ET; ++et) {
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const int m = 32 * kb + kp(g, s);
        GA[kb][et][s] = cvt<T>(m < FW ? Ge[(size_t)(w * FW + m) * (D + 1) + 16 * et + c] : 0.f);
      }
      WB[kb][et] = Wfr[WL::b(w, kb, et) * 64 + lane];
    }
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
    for (int kb = 0; kb < EB; ++kb) {
#pragma unroll
      for (int s = 0; s < 8; ++s) GM[mt][kb][s] = cvt<T>(Ge[(size_t)(w * FW + 16 * mt + c) * (D + 1) + 32 * kb + kp(g, s)]);
      Wf[mt][kb] = Wfr[WL::a(w, mt, kb) * 64 + lane];
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) gz[mt][r] = Ge[(size_t)(w * FW + 16 * mt + 4 * g + r) * (D + 1) + D];
  }
  f32x4 dWacc[MT][ET];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int et = 0; et < ET; ++et) dWacc[mt][et] = zero4();

  // rows of segment p
  const TileMap tm(a.L, a.C, TR);
  const int n_tiles = tm.count_tiles();
  const int j0 = (int)((int64_t)p * n_tiles / a.P), j1 = (int)((int64_t)(p + 1) * n_tiles / a.P);
  int row0 = 0, row1 = 0;
  if (j1 > j0) {
    int s_, c_;
    tm.tile(j0, row0, c_);
    tm.tile(j1 - 1, s_, c_);
    row1 = s_ + c_;
  }
  const float half_log2M = 0.5f * __log2f((float)M);
  const float koff = (G::KIND == kFavor) ? a.kshift[head] * kLog2e + half_log2M : 0.f;

  RowStage<T, D, TR, NT> sk, sv;
  // dV and dK rows of the next tile, in the reduction's thread mapping:
  // thread (t, q) holds entries [q EPT, q EPT + EPT) of row t
  typedef T tvec __attribute__((ext_vector_type(EPT)));
  const int rt = threadIdx.x / TPR, rq = threadIdx.x % TPR;
  tvec pdv, pdk;
  auto fetch_out = [&](int s0, int n) {
    if (rt < n) {
      const size_t o = (size_t)(s0 + rt) * D + rq * EPT;
      pdv = *(const tvec*)(dVh + o);
      pdk = *(const tvec*)(dKh + o);
    }
  };
  if (row1 > row0) {
    const int n0 = min(TR, row1 - row0);
    sk.fetch(Kh + (size_t)row0 * D, n0, threadIdx.x);
    sv.fetch(Vh + (size_t)row0 * D, n0, threadIdx.x);
    fetch_out(row0, n0);
  }
  for (int start = row0; start < row1; start += TR) {
    const int count = min(TR, row1 - start);
    sk.template store<LDQ>(Ks, G::KIND == kFavor ? kn : nullptr, threadIdx.x);
    sv.template store<LDQ>(Vs, nullptr, threadIdx.x);
    const tvec cdv = pdv, cdk = pdk;
    if (start + TR < row1) {
      const int nn = min(TR, row1 - start - TR);
      sk.fetch(Kh + (size_t)(start + TR) * D, nn, threadIdx.x);
      sv.fetch(Vh + (size_t)(start + TR) * D, nn, threadIdx.x);
      fetch_out(start + TR, nn);
    }
    __syncthreads();

#pragma unroll
    for (int st = 0; st < RT; ++st) {
      const bool col_ok = 16 * st + c < count;
      // K~^T[m][s] for this wave's features (columns s of the tile half st)
      f32x4 kt[MT];
      const float init = (G::KIND == kFavor) ? -0.5f * kn[16 * st + c] : 0.f;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        f32x4 acc = {init, init, init, init};
#pragma unroll
        for (int kb = 0; kb < EB; ++kb) acc = mma(acc, Wf[mt][kb], frag_rm(Ks, LDQ, 16 * st, 32 * kb));
#pragma unroll
        for (int r = 0; r < 4; ++r)
          acc[r] = !col_ok ? 0.f : (G::KIND == kFavor) ? fast_exp2(acc[r] * kLog2e - koff) : fmaxf(acc[r], 0.f) + a.relu_eps;
        kt[mt] = acc;
      }
      // dV^T[e][s] = sum_m G[m][e] K~^T[m][s] over this wave's features -> RedV[w][s][e]
#pragma unroll
      for (int et = 0; et < ET; ++et) {
        f32x4 acc = zero4();
#pragma unroll
        for (int kb = 0; kb < MB; ++kb) {
          const bool half = ODD && kb == MB - 1;
          acc = mma(acc, GA[kb][et], pair_or_half<T>(kt[2 * kb], kt[half ? 2 * kb : 2 * kb + 1], !half));
        }
        store_tile_T<float>(RedV[w], LDR, acc, 16 * et, 16 * st);
      }
      // dK~^T[m][s] = sum_e G[m][e] V[s][e] + z-cotangent[m]; Pk^T = dK~^T . K~^T (FAVOR+) or masked (ReLU)
      f32x4 pk[MT];
      float rs = 0.f;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        f32x4 acc = col_ok ? gz[mt] : zero4();
#pragma unroll
        for (int kb = 0; kb < EB; ++kb) acc = mma(acc, GM[mt][kb], frag_rm(Vs, LDQ, 16 * st, 32 * kb));
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          acc[r] = (G::KIND == kFavor) ? acc[r] * kt[mt][r] : (kt[mt][r] > a.relu_eps ? acc[r] : 0.f);
          rs += acc[r];
        }
        pk[mt] = acc;
        store_tile_T<T>(ZPk[w], LDF, acc, 16 * mt, 16 * st);
      }
      if (G::KIND == kFavor) rs = wave_sum_over_g(rs);
      // dk^T[e][s] = sum_m W[m][e] Pk^T[m][s] - k[s][e] rowsum(Pk[s]) over this wave's features -> RedK
#pragma unroll
      for (int et = 0; et < ET; ++et) {
        f32x4 acc;
        if (G::KIND == kFavor) {
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[r] = -to_f32(Ks[(16 * st + c) * LDQ + 16 * et + 4 * g + r]) * rs;
        } else {
          acc = zero4();
        }
#pragma unroll
        for (int kb = 0; kb < MB; ++kb) {
          const bool half = ODD && kb == MB - 1;
          acc = mma(acc, WB[kb][et], pair_or_half<T>(pk[2 * kb], pk[half ? 2 * kb : 2 * kb + 1], !half));
        }
        store_tile_T<float>(RedK[w], LDR, acc, 16 * et, 16 * st);
      }
    }
    // dW[m][e] += sum_s Pk[s][m] K[s][e] (this wave's rows m; Pk read back from its own buffer)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const F pf = frag_tr(ZPk[w], LDF, 0, 16 * mt);
#pragma unroll
      for (int et = 0; et < ET; ++et) dWacc[mt][et] = mma(dWacc[mt][et], pf, frag_tr(Ks, LDQ, 0, 16 * et));
    }
    __syncthreads();

    // dV, dK += sums over the 4 waves (rows < count)
    if (rt < count) {
      constexpr int WS = TR * LDR / 4;  // one wave's rows, in 16-byte vectors
      tvec ov, ok;
#pragma unroll
      for (int h4 = 0; h4 < EPT / 4; ++h4) {
        const f32x4* rv0 = (const f32x4*)&RedV[0][rt * LDR + rq * EPT + 4 * h4];
        const f32x4* rk0 = (const f32x4*)&RedK[0][rt * LDR + rq * EPT + 4 * h4];
        const f32x4 v = (rv0[0] + rv0[WS]) + (rv0[2 * WS] + rv0[3 * WS]);
        const f32x4 k = (rk0[0] + rk0[WS]) + (rk0[2 * WS] + rk0[3 * WS]);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          ov[4 * h4 + i] = cvt<T>(to_f32(cdv[4 * h4 + i]) + v[i]);
          ok[4 * h4 + i] = cvt<T>(to_f32(cdk[4 * h4 + i]) + k[i]);
        }
      }
      const size_t o = (size_t)(start + rt) * D + rq * EPT;
      *(tvec*)(dVh + o) = ov;
      *(tvec*)(dKh + o) = ok;
    }
    __syncthreads();
  }

  // dW partial of (head, segment): added to what the reverse walk left there
  float* dwp = a.dW_part + (head * a.P + p) * (size_t)M * D;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int et = 0; et < ET; ++et)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const size_t i = (size_t)(w * FW + 16 * mt + 4 * g + r) * D + 16 * et + c;
        dwp[i] += dWacc[mt][et][r];
      }
}

template <class G>
hipError_t launch_carry(const CarryArgs& a, hipStream_t s) {
  if (a.P < 2) return hipSuccess;
  hipLaunchKernelGGL(carry_kernel<G>, dim3(a.P - 1, a.H, a.B), dim3(256), 0, s, a);
  return hipGetLastError();
}

#define SLIM_INST_CARRY(T, D, FW, TR, KIND) \
  template hipError_t launch_carry<Cfg<T, D, FW, TR, KIND>>(const CarryArgs&, hipStream_t);
SLIM_FOR_EACH_CONFIG(SLIM_INST_CARRY)

}  // namespace slim
