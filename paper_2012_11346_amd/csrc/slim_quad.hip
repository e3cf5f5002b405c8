// The slice evaluated as a whole: Algorithm 1 with the masked quadratic form
// of eq. 2 inside each slice (Sec. 3.2).  Slices are processed one after
// another, as in the paper; inside a slice every 32-row query tile t is
// independent given the state B^(n-1) before the slice:
//
//   N_t = Q~_t [S|z] + sum_{u <= t in the slice} tril_u=t(Q~_t K~_u^T) [V_u|1],
//   Y_t = N_t / D_t,
//
// so the work per row grows with the slice length C (C / 2 key tiles on
// average), where the tile walks of the other kernels carry the state from
// tile to tile and do the same work for every C.  Four waves per workgroup,
// wave w owning features [w FW, (w + 1) FW); each wave sums its features'
// share of N over the key tiles and the shares meet in LDS once per query
// tile.  Key features are recomputed for every (query, key) tile pair: no
// buffer of size C is kept.
#include "slim_common.hpp"
#include "slim_kernels.hpp"

namespace slim {

template <class G>
struct QuadLds {
  typedef typename G::T T;
  static constexpr int D = G::D, FW = G::FW, TR = G::TR;
  static constexpr int LDQ = D + 8;        // row tiles
  static constexpr int LDZ = TR + 8;       // K~ as [feature][row], per wave
  static constexpr int LDR = D + 4;        // reduction rows (floats)
  static constexpr size_t TILE = al16((size_t)TR * LDQ * sizeof(T));
  static constexpr size_t oQ = 0, oK = TILE, oV = 2 * TILE;
  static constexpr size_t oF = 3 * TILE;   // floats: kn[TR], qmx[4][TR]
  static constexpr size_t oZ = oF + al16(5 * TR * sizeof(float));
  static constexpr size_t ZW = al16((size_t)FW * LDZ * sizeof(T));
  static constexpr size_t oR = oZ + 4 * ZW;
  static constexpr size_t RW = al16((size_t)TR * LDR * sizeof(float));
  static constexpr size_t TOTAL = oR + 4 * RW;
};

// W fragments of wave w's feature tile mt for the logits: the bf16 values and
// their low parts, from the fragment table
template <class G>
struct QuadW {
  typedef typename FragT<typename G::T>::type F;
  __amdgpu_buffer_rsrc_t rs;
  int lane_off;
  __device__ QuadW(const void* table) {
    rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(table), (short)0,
                                           (int)(WFragLayout<G>::TOTAL * 64 * sizeof(F)), 0x00020000);
    lane_off = lane_id() * (int)sizeof(F);
  }
  __device__ __forceinline__ F load(int idx) const {
    typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
    u32x4 v[sizeof(F) / 16];
#pragma unroll
    for (int i = 0; i < (int)(sizeof(F) / 16); ++i)
      v[i] = __builtin_amdgcn_raw_buffer_load_b128(rs, lane_off + 16 * i, idx * 64 * (int)sizeof(F), 0);
    return __builtin_bit_cast(F, v);
  }
  __device__ __forceinline__ void get(int w, int mt, F (&hi)[G::EB], F (&lo)[G::EB]) const {
#pragma unroll
    for (int kb = 0; kb < G::EB; ++kb) {
      hi[kb] = load(WFragLayout<G>::a(w, mt, kb));
      lo[kb] = load(WFragLayout<G>::alo(w, mt, kb));
    }
  }
};

// Forward of one slice: grid (nwg, H, B); workgroup x takes the slice's
// query tiles x, x + nwg, ...
template <class G, bool DROP>
__global__ __launch_bounds__(256, 2) void quad_fwd_kernel(QuadArgs a) {
  typedef typename G::T T;
  typedef typename FragT<T>::type F;
  typedef QuadLds<G> Lay;
  constexpr int D = G::D, FW = G::FW, M = G::M, TR = G::TR, MT = G::MT, MB = G::MB, ET = G::ET, RT = G::RT;
  constexpr int LDQ = Lay::LDQ, LDZ = Lay::LDZ, LDR = Lay::LDR;
  constexpr int TPR = 256 / TR, EPT = D / TPR;
  static_assert(RT == 2 && G::RB == 1 && MT % 2 == 0, "32-row tiles, whole 32-deep feature blocks");

  __shared__ __attribute__((aligned(16))) char arena[Lay::TOTAL];
  T* Qs = (T*)(arena + Lay::oQ);
  T* Ks = (T*)(arena + Lay::oK);
  T* Vs = (T*)(arena + Lay::oV);
  float* kn = (float*)(arena + Lay::oF);
  float* qmx = kn + TR;  // [4][TR]
  const int w = wave_id();
  T* Zk = (T*)(arena + Lay::oZ + w * Lay::ZW);  // K~ as [m][s]
  auto red = [&](int ww) -> float* { return (float*)(arena + Lay::oR + ww * Lay::RW); };

  const int hd = blockIdx.y, b = blockIdx.z;
  const size_t head = (size_t)b * a.H + hd;
  const size_t hoff = head * (size_t)a.L * D;
  const T* Qh = (const T*)a.Q + hoff;
  const T* Kh = (const T*)a.K + hoff;
  const T* Vh = (const T*)a.V + hoff;
  T* Yh = (T*)a.Y + hoff;
  const QuadW<G> wt(a.Wfrag);
  const Drop drop{a.drop_seed, a.drop_t, a.C, head};
  const float half_log2M = 0.5f * __log2f((float)M);
  const float koff = (G::KIND == kFavor) ? a.kshift[head] * kLog2e + half_log2M : 0.f;

  // this wave's share of the state before the slice: S[mt][et] rows m,
  // columns e; S[mt][ET] the ones column (z) replicated over 16 columns
  f32x4 S[MT][ET + 1];
  {
    const Lane L = this_lane();
    const float* sp = a.S + head * (size_t)M * (D + 1);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const size_t row = (size_t)(w * FW + 16 * mt + 4 * L.g + r) * (D + 1);
#pragma unroll
        for (int et = 0; et < ET; ++et) S[mt][et][r] = sp[row + 16 * et + L.c];
        S[mt][ET][r] = sp[row + D];
      }
  }
  // the state as operands contracting over this wave's features, columns e
  F sf[MB][ET + 1];
#pragma unroll
  for (int kb = 0; kb < MB; ++kb)
#pragma unroll
    for (int et = 0; et <= ET; ++et) sf[kb][et] = tile_pair_frag<T>(S[2 * kb][et], S[2 * kb + 1][et]);

  const int nt = (a.rows + TR - 1) / TR;
  for (int t = blockIdx.x; t < nt; t += gridDim.x) {
    const int q0 = a.row0 + t * TR, qcount = min(TR, a.rows - t * TR);
    __syncthreads();  // the previous tile's readers of Qs and the reduction rows are done
    load_rows<T, D, TR, LDQ, 256>(Qs, Qh + (size_t)q0 * D, qcount, nullptr);
    __syncthreads();
    Lane L = fresh_lane();
    // query logits Lq[mt][tt]: rows m, columns t (the -|q|^2/2 term cancels
    // against the row shift)
    f32x4 Lq[MT][RT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      F hi[G::EB], lo[G::EB];
      wt.get(w, mt, hi, lo);
#pragma unroll
      for (int tt = 0; tt < RT; ++tt) {
        f32x4 acc = zero4();
#pragma unroll
        for (int kb = 0; kb < G::EB; ++kb) {
          const F qf = frag_rm(L, Qs, LDQ, 16 * tt, 32 * kb);
          acc = mma(acc, hi[kb], qf);
          acc = mma(acc, lo[kb], qf);
        }
        Lq[mt][tt] = acc;
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
        if (L.g == 0) qmx[w * TR + 16 * tt + L.c] = v;
      }
      __syncthreads();
#pragma unroll
      for (int tt = 0; tt < RT; ++tt) {
        const int tr = 16 * tt + L.c;
        const float qs = fmaxf(fmaxf(qmx[tr], qmx[TR + tr]), fmaxf(qmx[2 * TR + tr], qmx[3 * TR + tr])) * kLog2e;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int r = 0; r < 4; ++r) Lq[mt][tt][r] = fast_exp2(Lq[mt][tt][r] * kLog2e - qs);
      }
    } else {
#pragma unroll
      for (int tt = 0; tt < RT; ++tt)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int r = 0; r < 4; ++r) Lq[mt][tt][r] = plain_feature<G::KIND>(Lq[mt][tt][r], a.relu_eps);
    }
    // Q~ contracting over this wave's features, columns t
    F qf[MB][RT];
#pragma unroll
    for (int kb = 0; kb < MB; ++kb)
#pragma unroll
      for (int tt = 0; tt < RT; ++tt) qf[kb][tt] = tile_pair_frag<T>(Lq[2 * kb][tt], Lq[2 * kb + 1][tt]);

    // this wave's share of N^T[e][t]: the state before the slice first
    f32x4 nacc[ET + 1][RT];
#pragma unroll
    for (int et = 0; et <= ET; ++et)
#pragma unroll
      for (int tt = 0; tt < RT; ++tt) {
        f32x4 acc = zero4();
#pragma unroll
        for (int kb = 0; kb < MB; ++kb) acc = mma(acc, sf[kb][et], qf[kb][tt]);
        nacc[et][tt] = acc;
      }

    // then every key tile of the slice up to the diagonal
    for (int u = 0; u <= t; ++u) {
      const int k0 = a.row0 + u * TR, kcount = min(TR, a.rows - u * TR);
      __syncthreads();  // readers of the previous key tile are done
      load_rows<T, D, TR, LDQ, 256>(Ks, Kh + (size_t)k0 * D, kcount, G::KIND == kFavor ? kn : nullptr);
      if constexpr (DROP) {
        // value rows with the dropped elements zeroed (16-byte chunks)
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
      __syncthreads();
      L = fresh_lane();
      // key features of this wave's features -> Zk[m][s] (rows past the
      // tile: zero)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        F hi[G::EB], lo[G::EB];
        wt.get(w, mt, hi, lo);
#pragma unroll
        for (int st = 0; st < RT; ++st) {
          f32x4 acc = zero4();
#pragma unroll
          for (int kb = 0; kb < G::EB; ++kb) {
            const F kf = frag_rm(L, Ks, LDQ, 16 * st, 32 * kb);
            acc = mma(acc, kf, hi[kb]);
            acc = mma(acc, kf, lo[kb]);
          }
          // acc: rows s = 16 st + 4 g + r, columns m = 16 mt + c
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int s = 16 * st + 4 * L.g + r;
            if (G::KIND == kFavor) {
              const float kc = s < kcount ? koff + 0.5f * kLog2e * kn[s] : INFINITY;
              acc[r] = fast_exp2(acc[r] * kLog2e - kc);
            } else {
              acc[r] = s < kcount ? plain_feature<G::KIND>(acc[r], a.relu_eps) : 0.f;
            }
          }
          store_tile_T<T>(L, Zk, LDZ, acc, 16 * st, 16 * mt);
        }
      }
      // scores A^T[s][t] over this wave's features (causal on the diagonal
      // tile), then N^T += [V|1]^T A^T
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

    // the waves' shares of N meet in LDS; Y = s N / D
    L = fresh_lane();
#pragma unroll
    for (int tt = 0; tt < RT; ++tt) {
#pragma unroll
      for (int et = 0; et < ET; ++et) store_tile_T<float>(L, red(w), LDR, nacc[et][tt], 16 * et, 16 * tt);
      if (L.g == 0) red(w)[(16 * tt + L.c) * LDR + D] = nacc[ET][tt][0];
    }
    __syncthreads();
    {
      const int tid = fresh_tid();
      const int tr = tid / TPR, q = tid % TPR;
      if (tr < qcount) {
        const float den = (red(0)[tr * LDR + D] + red(1)[tr * LDR + D]) + (red(2)[tr * LDR + D] + red(3)[tr * LDR + D]);
        const float inv = a.drop_scale / den;
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
          const int e = q * EPT + i;
          const float n = (red(0)[tr * LDR + e] + red(1)[tr * LDR + e]) + (red(2)[tr * LDR + e] + red(3)[tr * LDR + e]);
          Yh[(size_t)(q0 + tr) * D + e] = cvt<T>(n * inv);
        }
      }
    }
  }
}

// out = f * in + sign * sum_p part[p], one thread per state entry
__global__ __launch_bounds__(256) void state_combine_kernel(const float* in, size_t in_stride, const float* in_shift,
                                                            const float* shift, const float* part, int P2, float sign,
                                                            float* out, int SZ) {
  const int head = blockIdx.y;
  const int el = blockIdx.x * 256 + threadIdx.x;
  if (el >= SZ) return;
  float v = 0.f;
  if (in != nullptr) {
    const float f = (in_shift != nullptr && shift != nullptr) ? fast_exp2((in_shift[head] - shift[head]) * kLog2e) : 1.f;
    v = f * in[(size_t)head * in_stride + el];
  }
  float s = 0.f;
  for (int p = 0; p < P2; ++p) s += part[((size_t)head * P2 + p) * SZ + el];
  out[(size_t)head * SZ + el] = v + sign * s;
}

hipError_t launch_state_combine(const float* in, size_t in_stride, const float* in_shift, const float* shift,
                                const float* part, int P2, float sign, float* out, int BH, int SZ, hipStream_t s) {
  hipLaunchKernelGGL(state_combine_kernel, dim3((SZ + 255) / 256, BH), dim3(256), 0, s, in, in_stride, in_shift, shift,
                     part, P2, sign, out, SZ);
  return hipGetLastError();
}

template <class G>
hipError_t launch_quad_fwd(const QuadArgs& a, int nwg, hipStream_t s) {
  const dim3 grid(nwg, a.H, a.B);
  if (a.drop_t != 0) hipLaunchKernelGGL((quad_fwd_kernel<G, true>), grid, dim3(256), 0, s, a);
  else hipLaunchKernelGGL((quad_fwd_kernel<G, false>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

#define SLIM_INST_QUAD(T, D, FW, TR, KIND) \
  template hipError_t launch_quad_fwd<Cfg<T, D, FW, TR, KIND>>(const QuadArgs&, int, hipStream_t);
SLIM_FOR_EACH_QUAD_CONFIG(SLIM_INST_QUAD)

}  // namespace slim
