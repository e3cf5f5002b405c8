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
// CS workgroups per (segment p < P - 1, batch, head), each taking a part of
// the segment's rows in 32-row tiles (no causal coupling between rows here).
// Per tile, wave w first maps its own M/4 features (K~ and Pk into LDS, its
// rows of dW in registers); then it owns a quarter of the tile's dV and dk
// outputs and contracts them over all M features straight from LDS, so no
// partial sums cross waves.  G_end(p) sits in LDS, W in registers.
#include "slim_common.hpp"
#include "slim_kernels.hpp"

namespace slim {

// DROP: value dropout on (its masks are generated only in that instantiation)
template <class G, bool DROP>
__global__ __launch_bounds__(256, 2) void carry_kernel(CarryArgs a) {
  typedef typename G::T T;
  typedef typename FragT<T>::type F;
  typedef WFragLayout<G> WL;
  constexpr int D = G::D, FW = G::FW, M = G::M, TR = G::TR, MT = G::MT, ET = G::ET, EB = G::EB, RT = G::RT,
                LDQ = G::LDQ;
  constexpr int NT = 256;
  constexpr int KB = M / 32;       // 32-deep blocks over all features
  constexpr int LDK = M + 8;       // pitch of the [row][feature] tiles
  constexpr int LDG = D + 8;       // pitch of G_end [feature][value column]
  static_assert((LDG - D) * sizeof(T) >= sizeof(float) && (D * sizeof(T)) % sizeof(float) == 0, "ones column in the padding");
  constexpr int NO = ET * RT / 4;  // output tiles (column tile, row half) per wave
  static_assert(RT == 2 && G::RB == 1, "32-row tiles");
  static_assert(NO >= 1 && ET * RT == 4 * NO, "output tiles shared evenly by the 4 waves");

  __shared__ __attribute__((aligned(16))) T Ks[TR * LDQ];
  __shared__ __attribute__((aligned(16))) T Vs[TR * LDQ];
  __shared__ __attribute__((aligned(16))) T Kt[TR * LDK];  // K~ [s][m]
  __shared__ __attribute__((aligned(16))) T Pk[TR * LDK];  // Pk [s][m]
  __shared__ __attribute__((aligned(16))) T Gs[M * LDG];   // G_end [m][e]; e = D: a float in the padding
  __shared__ float rsum[4][TR];                            // per-wave parts of rowsum(Pk[s])
  __shared__ float kn[TR];

  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = lane_id();
  const int p = blockIdx.x / a.CS, part = blockIdx.x % a.CS, hd = blockIdx.y, b = blockIdx.z;
  const size_t head = (size_t)b * a.H + hd;
  const size_t hoff = head * (size_t)a.L * D;
  const T* Kh = (const T*)a.K + hoff;
  const T* Vh = (const T*)a.V + hoff;
  T* dKh = (T*)a.dK + hoff;
  T* dVh = (T*)a.dV + hoff;
  const size_t SZ = (size_t)M * (D + 1);
  const float* Ge = a.gend + (head * a.P + p) * SZ;  // G_end(p), rows m, columns e (column D: ones)

  // G_end into LDS: columns e < D in the element type, the ones column
  // (e = D) as a float in the row's padding
  {
    constexpr int PER = M * D / NT, U = PER < 16 ? PER : 16;  // loads in flight per thread
    static_assert(PER % U == 0, "whole batches");
    const int tid = fresh_tid();
#pragma unroll
    for (int u0 = 0; u0 < PER; u0 += U) {
      float v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = tid + (u0 + u) * NT, m = i / D, e = i - (i / D) * D;
        v[u] = Ge[(size_t)m * (D + 1) + e];
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = tid + (u0 + u) * NT, m = i / D, e = i - (i / D) * D;
        Gs[m * LDG + e] = cvt<T>(v[u]);
      }
    }
    for (int m = tid; m < M; m += NT) *(float*)&Gs[m * LDG + D] = Ge[(size_t)m * (D + 1) + D];
  }

  // output tiles of this wave: column tile eo, row halves so(i)
  const int eo = (w * NO) / RT;
  auto so = [&](int i) { return (w * NO + i) % RT; };

  // W operand fragments (one table shared by every head)
  const __amdgpu_buffer_rsrc_t wrs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(a.Wfrag), (short)0, (int)(WL::TOTAL * 64 * sizeof(F)), 0x00020000);
  auto wfrag = [&](int idx) -> F {
    typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
    u32x4 v[sizeof(F) / 16];
#pragma unroll
    for (int i = 0; i < (int)(sizeof(F) / 16); ++i)
      v[i] = __builtin_amdgcn_raw_buffer_load_b128(wrs, lane * (int)sizeof(F) + 16 * i, idx * 64 * (int)sizeof(F), 0);
    return __builtin_bit_cast(F, v);
  };
  F Wl[MT][EB];  // low parts of Wf (bf16 split of the float32 W)
  F Wf[MT][EB];  // slot s = W[w FW + 16 mt + c][32 kb + kp]: K~ of this wave's features
  F Wc[KB];      // slot s = W[32 kb + kp][16 eo + c]: dk of this wave's column tile
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int kb = 0; kb < EB; ++kb) {
      Wf[mt][kb] = wfrag(WL::a(w, mt, kb));
      if constexpr (kSplitW<T>) Wl[mt][kb] = wfrag(WL::alo(w, mt, kb));
    }
#pragma unroll
  for (int kb = 0; kb < KB; ++kb) Wc[kb] = wfrag(WL::c(kb, eo));

  f32x4 dWacc[MT][ET];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int et = 0; et < ET; ++et) dWacc[mt][et] = zero4();

  // rows of this part of segment p
  const TileMap tm(a.L, a.C, TR);
  const int n_tiles = tm.count_tiles();
  const int s0 = (int)((int64_t)p * n_tiles / a.P), s1 = (int)((int64_t)(p + 1) * n_tiles / a.P);
  const int j0 = s0 + (s1 - s0) * part / a.CS, j1 = s0 + (s1 - s0) * (part + 1) / a.CS;
  int row0 = 0, row1 = 0;
  if (j1 > j0) {
    int s_, c_;
    tm.tile(j0, row0, c_);
    tm.tile(j1 - 1, s_, c_);
    row1 = s_ + c_;
  }
  const float half_log2M = 0.5f * __log2f((float)M);
  const float koff = (G::KIND == kFavor) ? a.kshift[head] * kLog2e + half_log2M : 0.f;

  // this part's rows through range resources: the ragged end of the last
  // block reads as zero and its stores are dropped
  const size_t part_bytes = (size_t)(row1 - row0) * D * sizeof(T);
  const __amdgpu_buffer_rsrc_t rK = range_rsrc(Kh + (size_t)row0 * D, part_bytes);
  const __amdgpu_buffer_rsrc_t rV = range_rsrc(Vh + (size_t)row0 * D, part_bytes);
  const __amdgpu_buffer_rsrc_t rdK = range_rsrc(dKh + (size_t)row0 * D, part_bytes);
  const __amdgpu_buffer_rsrc_t rdV = range_rsrc(dVh + (size_t)row0 * D, part_bytes);

  RowStage<T, D, TR, NT> sk, sv;
  // dV and dK entries of the next block in the output layout: lane (g, c) of
  // output tile i holds row 16 so(i) + c, columns 16 eo + 4 g + [0, 4)
  typedef T t4 __attribute__((ext_vector_type(4)));
  typedef BufIO<sizeof(t4)> IO;
  t4 pdv[NO], pdk[NO];
  auto out_off = [&](const Lane& L, int r, int i) {  // r: block start relative to row0
    return ((r + 16 * so(i) + L.c) * D + 16 * eo + 4 * L.g) * (int)sizeof(T);
  };
  auto fetch_block = [&](int r) {
    sk.fetch(rK, r, fresh_tid());
    sv.fetch(rV, r, fresh_tid());
    const Lane L = fresh_lane();
#pragma unroll
    for (int i = 0; i < NO; ++i) {
      pdv[i] = IO::template load<t4>(rdV, out_off(L, r, i));
      pdk[i] = IO::template load<t4>(rdK, out_off(L, r, i));
    }
  };
  // value dropout: dropped value elements zeroed when staged, and their dV
  // contributions dropped
  const Drop drop{a.drop_seed, a.drop_t, a.C, head};
  if (row1 > row0) fetch_block(0);
  for (int start = row0; start < row1; start += TR) {
    const int count = min(TR, row1 - start);
    const int rel = start - row0;
    sk.template store<LDQ>(Ks, G::KIND == kFavor ? kn : nullptr, fresh_tid());
    if (DROP) sv.drop(drop, start, fresh_tid());
    sv.template store<LDQ>(Vs, nullptr, fresh_tid());
    t4 cdv[NO], cdk[NO];
#pragma unroll
    for (int i = 0; i < NO; ++i) {
      cdv[i] = pdv[i];
      cdk[i] = pdk[i];
    }
    fetch_block(rel + TR);  // past the part's end: zeros, no traffic
    __syncthreads();

    // this wave's features: K~ and Pk for every row of the tile
    {
      const Lane L = fresh_lane();
#pragma unroll
      for (int st = 0; st < RT; ++st) {
        const bool col_ok = 16 * st + L.c < count;
        f32x4 kt[MT], kl[MT];  // features and (square map) logits
        // exponent offset of the column's key row, the row term -|k|^2/2
        // included; rows past the block: infinite (features exactly zero)
        const float kc = (G::KIND == kFavor) ? (col_ok ? koff + 0.5f * kLog2e * kn[16 * st + L.c] : INFINITY) : 0.f;
        F kfr[EB];
#pragma unroll
        for (int kb = 0; kb < EB; ++kb) kfr[kb] = frag_rm(L, Ks, LDQ, 16 * st, 32 * kb);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          f32x4 acc = zero4();
#pragma unroll
          for (int kb = 0; kb < EB; ++kb) acc = mma(acc, Wf[mt][kb], kfr[kb]);
          if constexpr (kSplitW<T>) {
#pragma unroll
            for (int kb = 0; kb < EB; ++kb) acc = mma(acc, Wl[mt][kb], kfr[kb]);
          }
          kl[mt] = acc;
#pragma unroll
          for (int r = 0; r < 4; ++r)
            acc[r] = (G::KIND == kFavor) ? fast_exp2(acc[r] * kLog2e - kc)
                                         : (col_ok ? plain_feature<G::KIND>(acc[r], a.relu_eps) : 0.f);
          kt[mt] = acc;
          store_tile_T<T>(L, Kt, LDK, acc, w * FW + 16 * mt, 16 * st);
        }
        // dK~^T[m][s] = sum_e G[m][e] V[s][e] + z-cotangent[m]; Pk^T = dK~^T . K~^T (FAVOR+),
        // masked (ReLU) or times 2 l (square)
        // (columns past the block have K~ = 0, hence Pk = 0)
        float sum = 0.f;
        F vfr[EB];
#pragma unroll
        for (int kb = 0; kb < EB; ++kb) vfr[kb] = frag_rm(L, Vs, LDQ, 16 * st, 32 * kb);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          f32x4 acc;
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[r] = *(const float*)&Gs[(w * FW + 16 * mt + 4 * L.g + r) * LDG + D];
#pragma unroll
          for (int kb = 0; kb < EB; ++kb) acc = mma(acc, frag_rm(L, Gs, LDG, w * FW + 16 * mt, 32 * kb), vfr[kb]);
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            acc[r] = vjp_factor<G::KIND>(acc[r], kt[mt][r], kl[mt][r], a.relu_eps);
            sum += acc[r];
          }
          store_tile_T<T>(L, Pk, LDK, acc, w * FW + 16 * mt, 16 * st);
        }
        if (G::KIND == kFavor) {
          sum = wave_sum_over_g(sum);
          if (L.g == 0) rsum[w][16 * st + L.c] = sum;
        }
      }
    }
    __syncthreads();

    // this wave's output tiles, contracted over all M features
    {
      const Lane L = fresh_lane();
#pragma unroll
      for (int i = 0; i < NO; ++i) {
        const int st = so(i);
        // dV^T[e][s] = sum_m G[m][e] K~[s][m]
        f32x4 acc = zero4();
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) acc = mma(acc, frag_tr(L, Gs, LDG, 32 * kb, 16 * eo), frag_rm(L, Kt, LDK, 16 * st, 32 * kb));
        {
          const unsigned keep = DROP ? drop_keep_bits<4>(drop, start + 16 * st + L.c, 16 * eo + 4 * L.g) : ~0u;
          t4 o;
#pragma unroll
          for (int r = 0; r < 4; ++r) o[r] = cvt<T>(to_f32(cdv[i][r]) + ((keep >> r) & 1u ? acc[r] : 0.f));
          IO::store(o, rdV, out_off(L, rel, i));
        }
        // dk^T[e][s] = sum_m W[m][e] Pk[s][m] - k[s][e] rowsum(Pk[s])
        if (G::KIND == kFavor) {
          const int sr = 16 * st + L.c;
          const float rs = (rsum[0][sr] + rsum[1][sr]) + (rsum[2][sr] + rsum[3][sr]);
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[r] = -to_f32(Ks[sr * LDQ + 16 * eo + 4 * L.g + r]) * rs;
        } else {
          acc = zero4();
        }
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) acc = mma(acc, Wc[kb], frag_rm(L, Pk, LDK, 16 * st, 32 * kb));
        {
          t4 o;
#pragma unroll
          for (int r = 0; r < 4; ++r) o[r] = cvt<T>(to_f32(cdk[i][r]) + acc[r]);
          IO::store(o, rdK, out_off(L, rel, i));
        }
      }
      // dW[m][e] += sum_s Pk[s][m] K[s][e] (this wave's rows m)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const F pf = frag_tr(L, Pk, LDK, 0, w * FW + 16 * mt);
#pragma unroll
        for (int et = 0; et < ET; ++et) dWacc[mt][et] = mma(dWacc[mt][et], pf, frag_tr(L, Ks, LDQ, 0, 16 * et));
      }
    }
    __syncthreads();
  }

  // dW partial: part 0 adds to what the reverse walk left for (head,
  // segment); part q > 0 writes its own slot after the walk's B H P slots
  const size_t n_walk = (size_t)a.B * a.H * a.P;
  const size_t slot = part == 0 ? head * a.P + p : n_walk + ((size_t)(part - 1) * a.B * a.H + head) * (a.P - 1) + p;
  float* dwp = a.dW_part + slot * (size_t)M * D;
  const Lane L = fresh_lane();
  float* dwl = dwp + (size_t)(w * FW + 4 * L.g) * D + L.c;  // + (16 mt + r) D + 16 et
  if (part == 0) {
    // all loads first, then the stores
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int et = 0; et < ET; ++et)
#pragma unroll
        for (int r = 0; r < 4; ++r) dWacc[mt][et][r] += dwl[(16 * mt + r) * D + 16 * et];
  }
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int et = 0; et < ET; ++et)
#pragma unroll
      for (int r = 0; r < 4; ++r) dwl[(16 * mt + r) * D + 16 * et] = dWacc[mt][et][r];
}

template <class G>
hipError_t launch_carry(const CarryArgs& a, hipStream_t s) {
  if (a.P < 2) return hipSuccess;
  const dim3 grid((a.P - 1) * a.CS, a.H, a.B);
  if (a.drop_t != 0) hipLaunchKernelGGL((carry_kernel<G, true>), grid, dim3(256), 0, s, a);
  else hipLaunchKernelGGL((carry_kernel<G, false>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

#define SLIM_INST_CARRY(T, D, FW, TR, KIND) \
  template hipError_t launch_carry<Cfg<T, D, FW, TR, KIND>>(const CarryArgs&, hipStream_t);
SLIM_FOR_EACH_CONFIG(SLIM_INST_CARRY)

}  // namespace slim
