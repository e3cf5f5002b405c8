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
// After the exponentials, Q~ and K~ live only in LDS (bf16 for bf16
// problems) and every later product reads its operand fragments from there;
// this keeps the per-wave register set to the state, the cotangent, the dW
// accumulators and the W fragments.  Cross-feature sums (N, D, dV, dq, dk) go
// through a cross-wave reduction in LDS that reuses each wave's transpose
// buffer.  dW partials of every workgroup are summed by dw_reduce in a fixed
// order, so results are deterministic.
#include "slim_common.hpp"
#include "slim_kernels.hpp"

namespace slim {

template <class G>
struct BwdLds {
  typedef typename G::T T;
  static constexpr int D = G::D, FW = G::FW, TR = G::TR, ZR = G::ZR, LDQ = G::LDQ, LDR = G::LDR;
  static constexpr int LDZK = TR + 8;  // [feature][row] buffers (K~, dK~.K~)
  static constexpr int LDZF = FW + 8;  // [row or e][feature] buffers (Q~, S, G, dQ~.Q~)
  static constexpr int LDZT = TR + 8;  // [row][row] buffers (A^T, dA^T)
  // shared tiles
  static constexpr size_t TILE = al16((size_t)TR * LDQ * sizeof(T));
  static constexpr size_t oQ = 0, oK = oQ + TILE, oV = oK + TILE, odY = oV + TILE, odN = odY + TILE;
  static constexpr size_t oF = odN + TILE;  // floats: qn kn qmx[4] dDs rsum[4] dzs[4]
  static constexpr size_t NF = 2 * TR + 4 * TR + TR + 4 * TR + 4 * FW;
  static constexpr size_t odDb = oF + al16(NF * sizeof(float));
  static constexpr size_t oW = odDb + al16((TR + 8) * sizeof(T));
  // per-wave regions
  static constexpr size_t ZK = al16((size_t)ZR * LDZK * sizeof(T));
  static constexpr size_t ZQ = al16((size_t)TR * LDZF * sizeof(T));
  static constexpr size_t X1 = (size_t)TR * LDZT * sizeof(T), X2 = (size_t)TR * LDZF * sizeof(T),
                          X3 = (size_t)ZR * LDZK * sizeof(T);
  static constexpr size_t ZX = al16(X1 > X2 ? (X1 > X3 ? X1 : X3) : (X2 > X3 ? X2 : X3));
  static constexpr size_t ZDA = al16((size_t)TR * LDZT * sizeof(T));
  static constexpr size_t R1 = (size_t)TR * LDR * sizeof(float), R2 = (size_t)D * LDZF * sizeof(T);
  static constexpr size_t ZRS = al16(R1 > R2 ? R1 : R2);
  static constexpr size_t oZk = 0, oZq = oZk + ZK, oZx = oZq + ZQ, oZdA = oZx + ZX, oZrs = oZdA + ZDA;
  static constexpr size_t WAVE = oZrs + ZRS;
  static constexpr size_t TOTAL = oW + 4 * WAVE;
};

// DROP: value dropout on (its masks are generated only in that instantiation)
template <class G, bool DROP>
__global__ __launch_bounds__(256, 1) void bwd_walk_kernel(BwdArgs a) {
  typedef typename G::T T;
  typedef typename FragT<T>::type F;
  typedef BwdLds<G> Lay;
  constexpr int D = G::D, FW = G::FW, M = G::M, TR = G::TR, MT = G::MT, MB = G::MB, ET = G::ET, EB = G::EB,
                RT = G::RT, RB = G::RB, LDQ = G::LDQ, LDR = G::LDR, ZR = G::ZR;
  constexpr int LDZK = Lay::LDZK, LDZF = Lay::LDZF, LDZT = Lay::LDZT;
  constexpr bool ODD = (MT & 1) != 0;  // last 32-deep feature block holds 16 features

  // one arena, so that the compiler sees every alias between phases
  __shared__ __attribute__((aligned(16))) char arena[Lay::TOTAL];
  T* Qs = (T*)(arena + Lay::oQ);
  T* Ks = (T*)(arena + Lay::oK);
  T* Vs = (T*)(arena + Lay::oV);
  T* dYs = (T*)(arena + Lay::odY);
  T* dNs = (T*)(arena + Lay::odN);
  float* fl = (float*)(arena + Lay::oF);
  float* qn = fl;
  float* kn = qn + TR;
  float* qmx = kn + TR;        // [4][TR]
  float* dDs = qmx + 4 * TR;   // [TR]
  float* rsum = dDs + TR;      // [4][TR]
  float* dzs = rsum + 4 * TR;  // [4][FW]
  T* dDb = (T*)(arena + Lay::odDb);

  const int w = wave_id(), g = lane_g(), c = lane_c();
  char* wz = arena + Lay::oW + (size_t)w * Lay::WAVE;
  T* Zk = (T*)(wz + Lay::oZk);    // K~ as [m][s], whole tile
  T* Zq = (T*)(wz + Lay::oZq);    // Q~ as [t][m], whole tile
  T* ZA = (T*)(wz + Lay::oZx);    // A^T as [t][s]; then dQ~.Q~ as [t][m]; then dK~.K~ as [m][s]
  T* ZP = ZA;
  T* ZPk = ZA;
  T* ZdA = (T*)(wz + Lay::oZdA);  // dA^T as [t][s]
  T* ZS = (T*)(wz + Lay::oZrs);   // S as [e][m]; G as [e][m]
  float* Redw = (float*)(wz + Lay::oZrs);  // this wave's partial sums [row][e]
  auto red = [&](int ww) -> float* { return (float*)(arena + Lay::oW + (size_t)ww * Lay::WAVE + Lay::oZrs); };

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

  // W fragments come from the fragment-ordered copy (L2-resident), loaded
  // where they are used instead of being held for the whole walk
  typedef WFragLayout<G> WL;
  const F* Wfr = reinterpret_cast<const F*>(a.Wfrag);
  const int lane = lane_id();

  const size_t SZ = (size_t)M * (D + 1);
  const size_t sidx = (head * a.P + p) * SZ;
  const float* bend = a.bounds + (head * a.bound_stride + (size_t)(p + 1) * a.bound_step) * SZ;
  float r0 = 1.f;
  if (G::KIND == kFavor && a.init_shift != nullptr) r0 = fast_exp2((a.init_shift[head] - a.kshift[head]) * kLog2e);

  // the cotangent starts at dstate_out in the last segment, else at zero
  // (earlier segments get the cotangent of later ones added by carry_kernel)
  const float* g0 = (p == a.P - 1 && a.dstate_out != nullptr) ? a.dstate_out + head * SZ : nullptr;
  f32x4 S[MT][ET + 1], Gs[MT][ET + 1], dWacc[MT][ET];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const size_t row = (size_t)(w * FW + 16 * mt + 4 * g + r) * (D + 1);
#pragma unroll
      for (int et = 0; et < ET; ++et) {
        S[mt][et][r] = bend[row + 16 * et + c];
        Gs[mt][et][r] = g0 ? g0[row + 16 * et + c] : 0.f;
      }
      S[mt][ET][r] = bend[row + D];
      Gs[mt][ET][r] = g0 ? g0[row + D] : 0.f;
    }
#pragma unroll
    for (int et = 0; et < ET; ++et) dWacc[mt][et] = zero4();
  }

  // this wave's buffers start at zero: pad rows of Zk must read as zero
  for (size_t i = lane_id() * 16; i < Lay::WAVE; i += 64 * 16) *reinterpret_cast<uint4*>(wz + i) = uint4{0, 0, 0, 0};

  const TileMap tm(a.L, a.C, TR);
  const int n_tiles = tm.count_tiles();
  const int j0 = (int)((int64_t)p * n_tiles / a.P), j1 = (int)((int64_t)(p + 1) * n_tiles / a.P);
  // exact states at the starts of the sub-segments inside this segment: the
  // walk resets to them instead of downdating, so downdates never run past
  // one sub-segment (the last reset is the segment's own start)
  const int P2 = a.bound_stride - 1;
  int qreset = (p + 1) * a.bound_step - 1;
  int jreset = (int)((int64_t)qreset * n_tiles / P2);
  const float half_log2M = 0.5f * __log2f((float)M);
  const float koff = (G::KIND == kFavor) ? a.kshift[head] * kLog2e + half_log2M : 0.f;
  constexpr int TPR = 256 / TR, EPT = D / TPR;

  RowStage<T, D, TR, 256> sq, sk, sv, sdy;
  const Drop drop{a.drop_seed, a.drop_t, a.C, head};
  if (j1 > j0) {
    int st0, cn0;
    tm.tile(j1 - 1, st0, cn0);
    sq.fetch(Qh + (size_t)st0 * D, cn0, threadIdx.x);
    sk.fetch(Kh + (size_t)st0 * D, cn0, threadIdx.x);
    sv.fetch(Vh + (size_t)st0 * D, cn0, threadIdx.x);
    sdy.fetch(dYh + (size_t)st0 * D, cn0, threadIdx.x);
  }

  // [V|1] operand over rows [32 rb, 32 rb + 32) for value tile et (et == ET: ones)
  auto v_frag = [&](int rb, int et, int count) -> F {
    if (et < ET) return frag_tr(Vs, LDQ, 32 * rb, 16 * et);
    F f;
#pragma unroll
    for (int s = 0; s < 8; ++s) f[s] = cvt<T>((32 * rb + kp(g, s) < count) ? 1.f : 0.f);
    return f;
  };
  auto half_m = [&](int kb) -> bool { return ODD && kb == MB - 1; };

  for (int j = j1 - 1; j >= j0; --j) {
    int start, count;
    tm.tile(j, start, count);
    // W of this wave's features for the logits, with the low parts of a bf16 split
    F Wf[MT][EB], Wl[MT][EB];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int kb = 0; kb < EB; ++kb) {
        Wf[mt][kb] = Wfr[WL::a(w, mt, kb) * 64 + lane];
        if constexpr (kSplitW<T>) Wl[mt][kb] = Wfr[WL::alo(w, mt, kb) * 64 + lane];
      }
    sq.template store<LDQ>(Qs, G::KIND == kFavor ? qn : nullptr, threadIdx.x);
    sk.template store<LDQ>(Ks, G::KIND == kFavor ? kn : nullptr, threadIdx.x);
    // (value dropout: dropped elements of the value rows zeroed when staged)
    if (DROP) sv.drop(drop, start, threadIdx.x);
    sv.template store<LDQ>(Vs, nullptr, threadIdx.x);
    sdy.template store<LDQ>(dYs, nullptr, threadIdx.x);
    if (j > j0) {  // next tile's loads overlap this tile's compute
      int sn, cnn;
      tm.tile(j - 1, sn, cnn);
      sq.fetch(Qh + (size_t)sn * D, cnn, threadIdx.x);
      sk.fetch(Kh + (size_t)sn * D, cnn, threadIdx.x);
      sv.fetch(Vh + (size_t)sn * D, cnn, threadIdx.x);
      sdy.fetch(dYh + (size_t)sn * D, cnn, threadIdx.x);
    }
    __syncthreads();

    // ---- features: logits, shifts, exponentials; Q~ -> Zq[t][m], K~ -> Zk[m][s]
    // (the logits stay live for the square map's chain rule; for the other
    // maps nothing reads them after this phase)
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
          if constexpr (kSplitW<T>) {
#pragma unroll
            for (int kb = 0; kb < EB; ++kb) acc = mma(acc, Wl[mt][kb], frag_rm(Qs, LDQ, 16 * tt, 32 * kb));
          }
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
          if constexpr (kSplitW<T>) {
#pragma unroll
            for (int kb = 0; kb < EB; ++kb) acc = mma(acc, frag_rm(Ks, LDQ, 16 * st, 32 * kb), Wl[mt][kb]);
          }
          Lk[st][mt] = acc;
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
          if (g == 0) qmx[w * TR + 16 * tt + c] = v;
        }
      }
#pragma unroll
      for (int st = 0; st < RT; ++st)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          f32x4 kv = Lk[st][mt];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const bool ok = 16 * st + 4 * g + r < count;
            kv[r] = !ok ? 0.f : (G::KIND == kFavor) ? fast_exp2(kv[r] * kLog2e - koff) : plain_feature<G::KIND>(kv[r], a.relu_eps);
          }
          store_tile_T<T>(Zk, LDZK, kv, 16 * st, 16 * mt);
        }
      __syncthreads();
#pragma unroll
      for (int tt = 0; tt < RT; ++tt) {
        const int t = 16 * tt + c;
        float qs = 0.f;
        if (G::KIND == kFavor)
          qs = fmaxf(fmaxf(qmx[t], qmx[TR + t]), fmaxf(qmx[2 * TR + t], qmx[3 * TR + t])) * kLog2e;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          f32x4 qv = Lq[mt][tt];
#pragma unroll
          for (int r = 0; r < 4; ++r)
            qv[r] = (t >= count) ? 0.f : (G::KIND == kFavor) ? fast_exp2(qv[r] * kLog2e - qs) : plain_feature<G::KIND>(qv[r], a.relu_eps);
          store_tile_T<T>(Zq, LDZF, qv, 16 * mt, 16 * tt);
        }
      }
    }
    __syncthreads();

    // ---- b1: state before the tile
    if (j == jreset) {
      const float* bq = a.bounds + (head * a.bound_stride + (size_t)qreset) * SZ;
      --qreset;
      jreset = (int)((int64_t)qreset * n_tiles / P2);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const size_t row = (size_t)(w * FW + 16 * mt + 4 * g + r) * (D + 1);
#pragma unroll
          for (int et = 0; et < ET; ++et) S[mt][et][r] = bq[row + 16 * et + c];
          S[mt][ET][r] = bq[row + D];
        }
    } else {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int et = 0; et <= ET; ++et) {
          const F vf = v_frag(rb, et, count);
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            F kf = frag_rm(Zk, LDZK, 16 * mt, 32 * rb);  // K~ contracting over rows
#pragma unroll
            for (int s = 0; s < 8; ++s) kf[s] = -kf[s];
            S[mt][et] = mma(S[mt][et], kf, vf);
          }
        }
    }

    // ---- b2: scores A^T[s][t] (this wave's features), causal, -> ZA[t][s]
#pragma unroll
    for (int tt = 0; tt < RT; ++tt)
#pragma unroll
      for (int st = 0; st < RT; ++st) {
        f32x4 acc = zero4();
        if (st <= tt) {
#pragma unroll
          for (int kb = 0; kb < MB; ++kb)
            acc = mma(acc, frag_tr(Zk, LDZK, 32 * kb, 16 * st), frag_rm_h(Zq, LDZF, 16 * tt, 32 * kb, half_m(kb)));
          if (st == tt) {
#pragma unroll
            for (int r = 0; r < 4; ++r)
              if (4 * g + r > c) acc[r] = 0.f;
          }
        }
        store_tile_T<T>(ZA, LDZT, acc, 16 * st, 16 * tt);
      }
    // N^T[e][t] = [V|1]^T A^T + [S|z]^T Q~^T, this wave's features; reduction rows [t][e]
#pragma unroll
    for (int tt = 0; tt < RT; ++tt)
#pragma unroll
      for (int et = 0; et <= ET; ++et) {
        f32x4 acc = zero4();
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
          if (2 * rb <= tt) acc = mma(acc, v_frag(rb, et, count), frag_rm(ZA, LDZT, 16 * tt, 32 * rb));
#pragma unroll
        for (int kb = 0; kb < MB; ++kb)
          acc = mma(acc, pair_or_half<T>(S[2 * kb][et], S[half_m(kb) ? 2 * kb : 2 * kb + 1][et], !half_m(kb)),
                    frag_rm_h(Zq, LDZF, 16 * tt, 32 * kb, half_m(kb)));
        if (et < ET) {
          store_tile_T<float>(Redw, LDR, acc, 16 * et, 16 * tt);
        } else if (g == 0) {
          Redw[(16 * tt + c) * LDR + D] = acc[0];
        }
      }
    __syncthreads();

    // ---- b3: dN, dD per row (threads: TPR per row)
    {
      const int t = threadIdx.x / TPR, q = threadIdx.x % TPR;
      const bool ok = t < count;
      float dy[EPT];
      float dot = 0.f;
      const float den = red(0)[t * LDR + D] + red(1)[t * LDR + D] + red(2)[t * LDR + D] + red(3)[t * LDR + D];
      const float inv = ok ? 1.f / den : 0.f;
      // (value dropout: Y = s N / D with the output scale s; 1 without dropout)
      const float invs = inv * a.drop_scale;
#pragma unroll
      for (int i = 0; i < EPT; ++i) {
        const int e = q * EPT + i;
        dy[i] = to_f32(dYs[t * LDQ + e]);
        const float n = red(0)[t * LDR + e] + red(1)[t * LDR + e] + red(2)[t * LDR + e] + red(3)[t * LDR + e];
        dot += dy[i] * (n * invs);
      }
      dot = sum_lane_group<TPR>(dot);
#pragma unroll
      for (int i = 0; i < EPT; ++i) dNs[t * LDQ + q * EPT + i] = cvt<T>(dy[i] * invs);
      if (q == 0) {
        const float dd = ok ? -dot * inv : 0.f;
        dDs[t] = dd;
        dDb[t] = cvt<T>(dd);
      }
    }
    __syncthreads();

    // ---- b4: dA^T[s][t] = sum_e V[s][e] dN[t][e] + dD[t], causal, -> ZdA[t][s]
#pragma unroll
    for (int tt = 0; tt < RT; ++tt) {
      const float ddt = dDs[16 * tt + c];
#pragma unroll
      for (int st = 0; st < RT; ++st) {
        f32x4 acc = zero4();
        if (st <= tt) {
          acc = f32x4{ddt, ddt, ddt, ddt};
#pragma unroll
          for (int kb = 0; kb < EB; ++kb)
            acc = mma(acc, frag_rm(Vs, LDQ, 16 * st, 32 * kb), frag_rm(dNs, LDQ, 16 * tt, 32 * kb));
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int sr = 16 * st + 4 * g + r;
            if ((st == tt && 4 * g + r > c) || sr >= count) acc[r] = 0.f;
          }
        }
        store_tile_T<T>(ZdA, LDZT, acc, 16 * st, 16 * tt);
      }
    }

    // ---- b7: dV^T[e][s] = sum_m dS[m][e] K~[s][m] + sum_t dN[t][e] A^T[s][t]; reduction rows [s][e]
#pragma unroll
    for (int st = 0; st < RT; ++st)
#pragma unroll
      for (int et = 0; et < ET; ++et) {
        f32x4 acc = zero4();
#pragma unroll
        for (int kb = 0; kb < MB; ++kb)
          acc = mma(acc, pair_or_half<T>(Gs[2 * kb][et], Gs[half_m(kb) ? 2 * kb : 2 * kb + 1][et], !half_m(kb)),
                    frag_tr(Zk, LDZK, 32 * kb, 16 * st));
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
          acc = mma(acc, frag_tr(dNs, LDQ, 32 * rb, 16 * et), frag_tr(ZA, LDZT, 32 * rb, 16 * st));
        store_tile_T<float>(Redw, LDR, acc, 16 * et, 16 * st);
      }
    __syncthreads();
    {
      const int t = threadIdx.x / TPR, q = threadIdx.x % TPR;
      if (t < count) {
        const unsigned keep = DROP ? drop_keep_bits<EPT>(drop, start + t, q * EPT) : ~0u;
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
          const int e = q * EPT + i;
          const float v = red(0)[t * LDR + e] + red(1)[t * LDR + e] + red(2)[t * LDR + e] + red(3)[t * LDR + e];
          dVh[(size_t)(start + t) * D + e] = cvt<T>((keep >> i) & 1u ? v : 0.f);
        }
      }
    }
    __syncthreads();

    // ---- b5: dQ~^T[m][t] = sum_e S[m][e] dN[t][e] + z[m] dD[t] + sum_s K~[s][m] dA^T[s][t]
    //          P = dQ~ . Q~ (FAVOR+) or dQ~ masked (ReLU) -> ZP[t][m]
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int et = 0; et < ET; ++et) store_tile_T<T>(ZS, LDZF, S[mt][et], 16 * mt, 16 * et);
    __syncthreads();
    {
      float rs[RT];
#pragma unroll
      for (int tt = 0; tt < RT; ++tt) rs[tt] = 0.f;
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
            acc = mma(acc, frag_rm(Zk, LDZK, 16 * mt, 32 * rb), frag_rm(ZdA, LDZT, 16 * tt, 32 * rb));
          const f32x4 qv = load_tile_T(Zq, LDZF, 16 * mt, 16 * tt);
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            acc[r] = vjp_factor<G::KIND>(acc[r], qv[r], Lq[mt][tt][r], a.relu_eps);
            rs[tt] += acc[r];
          }
          store_tile_T<T>(ZP, LDZF, acc, 16 * mt, 16 * tt);
        }
      if (G::KIND == kFavor) {
#pragma unroll
        for (int tt = 0; tt < RT; ++tt) {
          const float v = wave_sum_over_g(rs[tt]);
          if (g == 0) rsum[w * TR + 16 * tt + c] = v;
        }
      }
    }
    __syncthreads();  // ZS reads done before the reduction rows are rewritten; ZP visible
    // dq^T[e][t] = sum_m W[m][e] P[m][t]; reduction rows [t][e]
#pragma unroll
    for (int tt = 0; tt < RT; ++tt)
#pragma unroll
      for (int et = 0; et < ET; ++et) {
        f32x4 acc = zero4();
#pragma unroll
        for (int kb = 0; kb < MB; ++kb)
          acc = mma(acc, Wfr[WL::b(w, kb, et) * 64 + lane], frag_rm_h(ZP, LDZF, 16 * tt, 32 * kb, half_m(kb)));
        store_tile_T<float>(Redw, LDR, acc, 16 * et, 16 * tt);
      }
    // dW[m][e] += sum_t P[m][t] Q[t][e]
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const F pf = frag_tr(ZP, LDZF, 32 * rb, 16 * mt);
#pragma unroll
        for (int et = 0; et < ET; ++et) dWacc[mt][et] = mma(dWacc[mt][et], pf, frag_tr(Qs, LDQ, 32 * rb, 16 * et));
      }
    __syncthreads();
    {
      const int t = threadIdx.x / TPR, q = threadIdx.x % TPR;
      if (t < count) {
        const float rsv = (G::KIND == kFavor) ? rsum[t] + rsum[TR + t] + rsum[2 * TR + t] + rsum[3 * TR + t] : 0.f;
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
          const int e = q * EPT + i;
          float v = red(0)[t * LDR + e] + red(1)[t * LDR + e] + red(2)[t * LDR + e] + red(3)[t * LDR + e];
          if (G::KIND == kFavor) v -= to_f32(Qs[t * LDQ + e]) * rsv;
          dQh[(size_t)(start + t) * D + e] = cvt<T>(v);
        }
      }
    }
    __syncthreads();

    // ---- b6: dK~[s][m] = sum_e V[s][e] G[m][e] + dz[m] + sum_t dA^T[s][t] Q~[t][m]
    //          Pk = dK~ . K~ (FAVOR+) or masked (ReLU) -> ZPk[m][s]
    T* ZG = ZS;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
      for (int et = 0; et < ET; ++et) store_tile_T<T>(ZG, LDZF, Gs[mt][et], 16 * mt, 16 * et);
      if (c == 0) {
#pragma unroll
        for (int r = 0; r < 4; ++r) dzs[w * FW + 16 * mt + 4 * g + r] = Gs[mt][ET][r];
      }
    }
    __syncthreads();
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
          f32x4 acc;
          const float dz = dzs[w * FW + 16 * mt + c];
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[r] = (16 * st + 4 * g + r < count) ? dz : 0.f;
#pragma unroll
          for (int kb = 0; kb < EB; ++kb)
            acc = mma(acc, frag_rm(Vs, LDQ, 16 * st, 32 * kb), frag_tr(ZG, LDZF, 32 * kb, 16 * mt));
#pragma unroll
          for (int rb = 0; rb < RB; ++rb)
            acc = mma(acc, frag_tr(ZdA, LDZT, 32 * rb, 16 * st), frag_tr(Zq, LDZF, 32 * rb, 16 * mt));
          const f32x4 kv = load_tile_T(Zk, LDZK, 16 * st, 16 * mt);
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            acc[r] = vjp_factor<G::KIND>(acc[r], kv[r], Lk[st][mt][r], a.relu_eps);
            rk[st][r] += acc[r];
          }
          store_tile_T<T>(ZPk, LDZK, acc, 16 * st, 16 * mt);
        }
      if (G::KIND == kFavor) {
#pragma unroll
        for (int st = 0; st < RT; ++st)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float v = wave_sum_over_c(rk[st][r]);
            if (c == 0) rsum[w * TR + 16 * st + 4 * g + r] = v;
          }
      }
    }
    __syncthreads();  // ZG reads done before the reduction rows are rewritten; ZPk visible
    // dW[m][e] += sum_s Pk[s][m] K[s][e]
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const F pf = frag_rm(ZPk, LDZK, 16 * mt, 32 * rb);
#pragma unroll
        for (int et = 0; et < ET; ++et) dWacc[mt][et] = mma(dWacc[mt][et], pf, frag_tr(Ks, LDQ, 32 * rb, 16 * et));
      }
    // dk^T[e][s] = sum_m W[m][e] Pk[s][m]; reduction rows [s][e]
#pragma unroll
    for (int st = 0; st < RT; ++st)
#pragma unroll
      for (int et = 0; et < ET; ++et) {
        f32x4 acc = zero4();
#pragma unroll
        for (int kb = 0; kb < MB; ++kb)
          acc = mma(acc, Wfr[WL::b(w, kb, et) * 64 + lane], frag_tr(ZPk, LDZK, 32 * kb, 16 * st));
        store_tile_T<float>(Redw, LDR, acc, 16 * et, 16 * st);
      }
    __syncthreads();
    {
      const int t = threadIdx.x / TPR, q = threadIdx.x % TPR;
      if (t < count) {
        const float rsv = (G::KIND == kFavor) ? rsum[t] + rsum[TR + t] + rsum[2 * TR + t] + rsum[3 * TR + t] : 0.f;
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
          const int e = q * EPT + i;
          float v = red(0)[t * LDR + e] + red(1)[t * LDR + e] + red(2)[t * LDR + e] + red(3)[t * LDR + e];
          if (G::KIND == kFavor) v -= to_f32(Ks[t * LDQ + e]) * rsv;
          dKh[(size_t)(start + t) * D + e] = cvt<T>(v);
        }
      }
    }

    // ---- b8: G[m][e] += sum_t Q~[t][m] [dN|dD][t][e]
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const F qf = frag_tr(Zq, LDZF, 32 * rb, 16 * mt);
#pragma unroll
        for (int et = 0; et <= ET; ++et) {
          F bfr;
          if (et < ET) {
            bfr = frag_tr(dNs, LDQ, 32 * rb, 16 * et);
          } else {
#pragma unroll
            for (int s = 0; s < 8; ++s) bfr[s] = dDb[32 * rb + kp(g, s)];
          }
          Gs[mt][et] = mma(Gs[mt][et], qf, bfr);
        }
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
  // cotangent the walk ends with (several segments), or the state cotangent
  // before the sequence (one segment)
  float* gout = a.g_final != nullptr ? a.g_final + sidx
                                     : ((p == 0 && a.dstate_in != nullptr) ? a.dstate_in + head * SZ : nullptr);
  if (a.g_final != nullptr) r0 = 1.f;
  if (gout != nullptr) {
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

// dW[m][e] = sum over workgroups of the partials, in a fixed order: a block
// covers 64 entries; its 4 thread groups sum interleaved quarters of the
// partials, then the 4 group sums are added in group order
// dW = sum of the n_parts partials [n_parts][n] in a fixed order: block b
// takes 64 groups of 4 consecutive entries (16-byte loads); its 16 waves sum
// every 16th partial each, and the 16 wave sums are added in wave order.
__global__ __launch_bounds__(1024) void dw_reduce_kernel(const float* part, int nparts, int n, float* dW) {
  __shared__ f32x4 acc[16][64];
  const int e = threadIdx.x & 63, q = threadIdx.x >> 6;
  const int i = (blockIdx.x * 64 + e) * 4;  // n is a multiple of 4
  f32x4 s = zero4();
  if (i < n) {
    // (four partials' loads issued together, added in the same order)
    int k = q;
    for (; k + 48 < nparts; k += 64) {
      f32x4 x[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) x[j] = *(const f32x4*)&part[(size_t)(k + 16 * j) * n + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) s += x[j];
    }
    for (; k < nparts; k += 16) s += *(const f32x4*)&part[(size_t)k * n + i];
  }
  acc[q][e] = s;
  __syncthreads();
  if (q == 0 && i < n) {
    f32x4 t = acc[0][e];
#pragma unroll
    for (int j = 1; j < 16; ++j) t += acc[j][e];
#pragma unroll
    for (int j = 0; j < 4; ++j) dW[i + j] = t[j];  // dW is only 4-byte aligned
  }
}

template <class G>
hipError_t launch_bwd_walk(const BwdArgs& a, hipStream_t s) {
  if (a.drop_t != 0) hipLaunchKernelGGL((bwd_walk_kernel<G, true>), dim3(a.P, a.H, a.B), dim3(256), 0, s, a);
  else hipLaunchKernelGGL((bwd_walk_kernel<G, false>), dim3(a.P, a.H, a.B), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_dw_reduce(const float* part, int n_parts, int n, float* dW, hipStream_t s) {
  hipLaunchKernelGGL(dw_reduce_kernel, dim3((n / 4 + 63) / 64), dim3(1024), 0, s, part, n_parts, n, dW);
  return hipGetLastError();
}

#define SLIM_INST_BWD(T, D, FW, TR, KIND) \
  template hipError_t launch_bwd_walk<Cfg<T, D, FW, TR, KIND>>(const BwdArgs&, hipStream_t);
SLIM_FOR_EACH_CONFIG(SLIM_INST_BWD)

}  // namespace slim
