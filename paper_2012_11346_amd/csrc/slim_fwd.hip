// Forward sweep (Algorithm 1, one layer) and the stand-alone feature map.
//
// fwd_walk: one workgroup per (batch, head, segment) walks its tiles in
// order.  Per tile of C_t <= TR rows (never straddling a slice), with the
// state B = (S, z) of everything before the tile held in registers:
//   a1  logits of Q and K against W on the matrix cores, with -|x|^2/2 folded
//       into the accumulator start; FAVOR+ features are exp2 of the shifted
//       logits (one shift per query row, one running shift per head for keys;
//       when the key shift grows the state is rescaled, so that all keys seen
//       so far share one shift).  ReLU: max(., 0) + eps.
//   a2  scores A^T = tril(K~ Q~^T) restricted to the tile (eq. 2, first line)
//   a3+a4  N^T = [V|1]^T A^T + [S|z]^T Q~^T, per wave over its features
//   a5  cross-wave sum of N, then Y = N / D
//   a6  [S|z] += K~^T [V|1]                       (eqs. 14-16, carried state)
// For slices longer than TR rows the tiles of a slice are chained through
// the same running state, which is the block-iterative evaluation of the
// in-slice prefix sum (Appendix B) with block TR.
#include "slim_common.hpp"
#include "slim_kernels.hpp"

namespace slim {

// W fragments of wave w's features for the logits: Wf the bf16 values of W,
// Wl their low parts (bf16 problems; unused for fp32)
template <class G>
__device__ __forceinline__ void load_w_frags(typename FragT<typename G::T>::type (&Wf)[G::MT][G::EB],
                                             typename FragT<typename G::T>::type (&Wl)[G::MT][G::EB],
                                             const float* W, int w) {
  const int g = lane_g(), c = lane_c();
#pragma unroll
  for (int mt = 0; mt < G::MT; ++mt)
#pragma unroll
    for (int kb = 0; kb < G::EB; ++kb)
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const float x = W[(size_t)(w * G::FW + 16 * mt + c) * G::D + 32 * kb + kp(g, s)];
        Wf[mt][kb][s] = cvt<typename G::T>(x);
        Wl[mt][kb][s] = w_lo<typename G::T>(x);
      }
}

// operand fragment of [V|1] over rows [k0, k0 + 32) for value tile et (et ==
// ET is the all-ones column block, zero on rows >= count)
template <class G>
__device__ __forceinline__ typename FragT<typename G::T>::type v_frag(const Lane& L, const typename G::T* Vs, int k0,
                                                                        int et, int count) {
  typedef typename G::T T;
  if (et < G::ET) return frag_tr(L, Vs, G::LDQ, k0, 16 * et);
  if constexpr (sizeof(T) == 2) return ones_rows_frag(L, k0, count);
  typename FragT<T>::type f;
  const int rem = count - k0 - 4 * L.g;  // rows k0 + kp(g, s) < count
#pragma unroll
  for (int s = 0; s < 8; ++s) f[s] = cvt<T>(((s & 3) + 16 * (s >> 2) < rem) ? 1.f : 0.f);
  return f;
}

// Query logits w_m . q_t, transposed: Lq[mt][tt] holds rows m (features of
// this wave), columns t.  (The FAVOR+ term -|q_t|^2/2 cancels against the
// query row shift, so it is never formed.)
template <class G>
__device__ __forceinline__ void query_logits(const Lane& L, f32x4 (&Lq)[G::MT][G::RT],
                                             const typename FragT<typename G::T>::type (&Wf)[G::MT][G::EB],
                                             const typename FragT<typename G::T>::type (&Wl)[G::MT][G::EB],
                                             const typename G::T* Qs) {
#pragma unroll
  for (int tt = 0; tt < G::RT; ++tt) {
    typename FragT<typename G::T>::type qf[G::EB];
#pragma unroll
    for (int kb = 0; kb < G::EB; ++kb) qf[kb] = frag_rm(L, Qs, G::LDQ, 16 * tt, 32 * kb);
#pragma unroll
    for (int mt = 0; mt < G::MT; ++mt) {
      f32x4 acc = zero4();
#pragma unroll
      for (int kb = 0; kb < G::EB; ++kb) {
        if constexpr (kSplitW<typename G::T>) acc = mma(acc, Wl[mt][kb], qf[kb]);
        acc = mma(acc, Wf[mt][kb], qf[kb]);
      }
      Lq[mt][tt] = acc;
    }
  }
}

// Key logits w_m . k_s: Lk[st][mt] holds rows s, columns m (features of this
// wave).  The FAVOR+ row term -|k_s|^2/2 enters with the exponent.
template <class G>
__device__ __forceinline__ void key_logits(const Lane& L, f32x4 (&Lk)[G::RT][G::MT],
                                           const typename FragT<typename G::T>::type (&Wf)[G::MT][G::EB],
                                           const typename FragT<typename G::T>::type (&Wl)[G::MT][G::EB],
                                           const typename G::T* Ks) {
#pragma unroll
  for (int st = 0; st < G::RT; ++st) {
    typename FragT<typename G::T>::type kf[G::EB];
#pragma unroll
    for (int kb = 0; kb < G::EB; ++kb) kf[kb] = frag_rm(L, Ks, G::LDQ, 16 * st, 32 * kb);
#pragma unroll
    for (int mt = 0; mt < G::MT; ++mt) {
      f32x4 acc = zero4();
#pragma unroll
      for (int kb = 0; kb < G::EB; ++kb) {
        if constexpr (kSplitW<typename G::T>) acc = mma(acc, kf[kb], Wl[mt][kb]);
        acc = mma(acc, kf[kb], Wf[mt][kb]);
      }
      Lk[st][mt] = acc;
    }
  }
}

// MODE kWalkOutputs: Y and the final state; kWalkSums: only the keys, the
// state each segment adds.
// (two workgroups per compute unit; DROP: value dropout on, its masks are
// generated only in that instantiation)
template <class G, int MODE, bool DROP>
__global__ __launch_bounds__(256, 2) void fwd_walk_kernel(FwdArgs a) {
  typedef typename G::T T;
  typedef typename FragT<T>::type F;
  constexpr int D = G::D, FW = G::FW, M = G::M, TR = G::TR, MT = G::MT, MB = G::MB, ET = G::ET, EB = G::EB,
                RT = G::RT, RB = G::RB, LDQ = G::LDQ, LDZ = G::LDZ, ZR = G::ZR, LDR = G::LDR, LDF = G::LDF;
  constexpr bool QSIDE = MODE != kWalkSums;
  // rows of the tile: keys and values double-buffered (tile j reads buffer
  // (j - j0) & 1), queries single-buffered (read only before the first barrier)
  constexpr int TQ = TR * LDQ;
  __shared__ __attribute__((aligned(16))) T Qbuf[QSIDE ? TQ : 8];
  __shared__ __attribute__((aligned(16))) T Kbuf[2 * TQ];
  __shared__ __attribute__((aligned(16))) T Vbuf[2 * TQ];
  __shared__ __attribute__((aligned(16))) T Zk[4][QSIDE ? ZR * LDZ : 8];
  __shared__ __attribute__((aligned(16))) float Red[4][QSIDE ? TR * LDR : 4];
  __shared__ __attribute__((aligned(16))) float knb[2][TR];  // key row norms, read as 16-byte vectors
  // row maxima of the query logits per wave, double-buffered by tile: the
  // output phase of a tile reads them (for logD) while a faster wave may
  // already write the next tile's
  __shared__ float qmx[2][4][TR], kmx[4];

  const int w = wave_id(), g = lane_g(), c = lane_c();
  const int p = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const size_t head = (size_t)b * a.H + h;
  const T* Qh = (const T*)a.Q + head * (size_t)a.L * D;
  const T* Kh = (const T*)a.K + head * (size_t)a.L * D;
  const T* Vh = (const T*)a.V + head * (size_t)a.L * D;

  // W of this wave's features for the logits: the bf16 values in registers;
  // the low parts (bf16 problems) in registers too, or, with 64 features per
  // wave and queries (where registers are short), read from the fragment
  // table a.Wfrag at every tile, behind the products of the high parts
  constexpr bool LO_TABLE = kSplitW<T> && MT == 4 && QSIDE;
  constexpr int MR = LO_TABLE ? 1 : MT, ER = LO_TABLE ? 1 : EB;
  F Wf[MR][ER], Wl[MR][ER];
  if constexpr (!LO_TABLE) load_w_frags<G>(Wf, Wl, a.W, w);
  // (table form: both parts of the fragments of half of the features at a
  // time, fetched at the start of every tile)
  typedef WFragLayout<G> WL;
  const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(a.Wfrag), (short)0, LO_TABLE ? (int)(WL::TOTAL * 64 * sizeof(F)) : 0, 0x00020000);

  // running state of this wave's features: S[mt][et] rows m, columns e;
  // S[mt][ET] holds z replicated over its 16 columns
  f32x4 S[MT][ET + 1];
  float cur = -INFINITY;  // key shift the state is relative to (FAVOR+)
  const bool fixed = a.fixed_shift != nullptr;
  if (G::KIND == kFavor && fixed) cur = a.fixed_shift[head];
  const size_t sidx = (head * a.P + p) * (size_t)M * (D + 1);
  const size_t sstate = head * a.seg_stride + (size_t)p * a.seg_step;
  const float* sin = a.seg_state ? a.seg_state + sstate * (size_t)M * (D + 1) : nullptr;
  if (sin != nullptr) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const size_t row = (size_t)(w * FW + 16 * mt + 4 * g + r) * (D + 1);
#pragma unroll
        for (int et = 0; et < ET; ++et) S[mt][et][r] = sin[row + 16 * et + c];
        S[mt][ET][r] = sin[row + D];
      }
    if (G::KIND == kFavor && !fixed) cur = a.seg_shift[sstate];
  } else {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int et = 0; et <= ET; ++et) S[mt][et] = zero4();
  }

  // pad rows of the transposed key buffer stay zero
  if constexpr (QSIDE)
    for (int i = FW * LDZ + lane_id(); i < ZR * LDZ; i += 64) Zk[w][i] = cvt<T>(0.f);

  const TileMap tm(a.L, a.C, TR);
  const int n_tiles = tm.count_tiles();
  const int j0 = (int)((int64_t)p * n_tiles / a.P), j1 = (int)((int64_t)(p + 1) * n_tiles / a.P);
  const float half_log2M = 0.5f * __log2f((float)M);
  constexpr int TPR = 256 / TR, EPT = D / TPR;

  // Rows two tiles ahead are fetched into registers; at the start of tile j
  // the rows of tile j + 1 go into the other buffer (its readers, tile j - 1,
  // finished before tile j - 1's last barrier) and become visible at tile j's
  // barriers.
  RowStage<T, D, TR, 256> sq, sk, sv;
  // range-checked loads without branches (an empty range past the last
  // tile), so that waits for them count exactly and never include the
  // output stores issued after them
  auto fetch = [&](int jj) {
    int s0, n0;
    tm.tile(min(jj, j1 - 1), s0, n0);
    const size_t nb = jj < j1 ? (size_t)n0 * D * sizeof(T) : 0;
    const int tid = fresh_tid();
    if constexpr (QSIDE) sq.fetch(range_rsrc(Qh + (size_t)s0 * D, nb), 0, tid);
    sk.fetch(range_rsrc(Kh + (size_t)s0 * D, nb), 0, tid);
    sv.fetch(range_rsrc(Vh + (size_t)s0 * D, nb), 0, tid);
  };
  auto store_q = [&](int bf) {
    if constexpr (QSIDE) sq.template store<LDQ>(Qbuf, nullptr, fresh_tid());
  };
  const Drop drop{a.drop_seed, a.drop_t, a.C, head};
  // value rows of tile jj, dropped elements zeroed (value dropout)
  auto store_kv = [&](int bf, int jj) {
    const int tid = fresh_tid();
    if (DROP) {
      int s0, n0;
      tm.tile(jj, s0, n0);
      sv.drop(drop, s0, tid);
    }
    sk.template store<LDQ>(Kbuf + bf * TQ, G::KIND == kFavor ? knb[bf] : nullptr, tid);
    sv.template store<LDQ>(Vbuf + bf * TQ, nullptr, tid);
  };
  if (j1 > j0) {
    fetch(j0);
    store_q(0);
    store_kv(0, j0);
    fetch(j0 + 1);
  }
  __syncthreads();

  // Y of a tile: EPT consecutive entries of one row per thread, stored as
  // PB-byte pieces at the end of the tile
  typedef T tvec __attribute__((ext_vector_type(EPT)));
  constexpr int PB = sizeof(tvec) >= 16 ? 16 : (int)sizeof(tvec);  // bytes per store (8 or 16)
  constexpr int NV = (int)(sizeof(tvec) / PB);
  static_assert(sizeof(tvec) % PB == 0 && (PB == 8 || PB == 16), "8- or 16-byte pieces");
  typedef unsigned pvec __attribute__((ext_vector_type(PB / 4)));
  pvec y_hold[NV] = {};
  __amdgpu_buffer_rsrc_t y_rs = range_rsrc(a.Y, 0);  // empty until the first tile's Y
  int y_off = 0;
  auto flush_y = [&]() {
    if constexpr (QSIDE) {
#pragma unroll
      for (int v = 0; v < NV; ++v) BufIO<PB>::store(y_hold[v], y_rs, y_off + PB * v);
    }
  };

  for (int j = j0; j < j1; ++j) {
    int start, count;
    tm.tile(j, start, count);
    const int bf = (j - j0) & 1;
    Lane L = fresh_lane();
    int g = L.g, c = L.c;
    if (j + 1 < j1) store_kv(bf ^ 1, j + 1);
    const T* Qs = Qbuf;
    const T* Ks = Kbuf + bf * TQ;
    const T* Vs = Vbuf + bf * TQ;
    const float* kn = knb[bf];

    f32x4 Lq[QSIDE ? MT : 1][RT], Lk[RT][MT];
    if constexpr (LO_TABLE) {
      // per half of the feature tiles: both parts of W from the table, then
      // the high-part and low-part products (row operands re-read from LDS)
      typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
      const int wlane = (fresh_tid() & 63) * (int)sizeof(F);
#pragma unroll
      for (int m2 = 0; m2 < MT; m2 += 2) {
        F Wh[2][EB], Wt[2][EB];
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int kb = 0; kb < EB; ++kb) {
            Wh[i][kb] = __builtin_bit_cast(
                F, __builtin_amdgcn_raw_buffer_load_b128(wrs, wlane, WL::a(w, m2 + i, kb) * 64 * (int)sizeof(F), 0));
            Wt[i][kb] = __builtin_bit_cast(
                F, __builtin_amdgcn_raw_buffer_load_b128(wrs, wlane, WL::alo(w, m2 + i, kb) * 64 * (int)sizeof(F), 0));
          }
#pragma unroll
        for (int tt = 0; tt < RT; ++tt) {
          F qf[EB], kf[EB];
#pragma unroll
          for (int kb = 0; kb < EB; ++kb) {
            qf[kb] = frag_rm(L, Qs, LDQ, 16 * tt, 32 * kb);
            kf[kb] = frag_rm(L, Ks, LDQ, 16 * tt, 32 * kb);
          }
#pragma unroll
          for (int i = 0; i < 2; ++i) {
            f32x4 q = zero4(), k = zero4();
#pragma unroll
            for (int kb = 0; kb < EB; ++kb) {
              q = mma(q, Wh[i][kb], qf[kb]);
              k = mma(k, kf[kb], Wh[i][kb]);
            }
#pragma unroll
            for (int kb = 0; kb < EB; ++kb) {
              q = mma(q, Wt[i][kb], qf[kb]);
              k = mma(k, kf[kb], Wt[i][kb]);
            }
            Lq[m2 + i][tt] = q;
            Lk[tt][m2 + i] = k;
          }
        }
      }
    } else {
      if constexpr (QSIDE) query_logits<G>(L, Lq, Wf, Wl, Qs);
      key_logits<G>(L, Lk, Wf, Wl, Ks);
    }

    if (G::KIND == kFavor) {
      if constexpr (QSIDE) {
#pragma unroll
        for (int tt = 0; tt < RT; ++tt) {
          float v = -INFINITY;
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int r = 0; r < 4; ++r) v = fmaxf(v, Lq[mt][tt][r]);
          v = wave_max_over_g(v);
          if (g == 0) qmx[bf][w][16 * tt + c] = v;
        }
      }
      if (!fixed) {
        float v = -INFINITY;
#pragma unroll
        for (int st = 0; st < RT; ++st)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            float u = -INFINITY;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) u = fmaxf(u, Lk[st][mt][r]);
            if (16 * st + 4 * g + r < count) v = fmaxf(v, u - 0.5f * kn[16 * st + 4 * g + r]);
          }
        v = wave_max(v);
        if ((fresh_tid() & 63) == 0) kmx[w] = v;
      }
    }
    // row maxima of all waves (and, with queries, the previous tile's
    // reduction reads are finished before N overwrites them)
    if (QSIDE || (G::KIND == kFavor && !fixed)) {
      __syncthreads();
      L = fresh_lane();
      g = L.g;
      c = L.c;
    }
    // queries of the next tile: every wave has read this tile's
    if (j + 1 < j1) store_q(bf ^ 1);
    fetch(j + 2);

    if (G::KIND == kFavor) {
      if (!fixed) {
        const float km = fmaxf(fmaxf(kmx[0], kmx[1]), fmaxf(kmx[2], kmx[3]));
        if (km > cur) {
          const float sc = fast_exp2((cur - km) * kLog2e);
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int et = 0; et <= ET; ++et) S[mt][et] *= sc;
          cur = km;
        }
      }
      // exponent offsets of the key rows (row term included); rows past the
      // tile: infinite, so their features are exactly zero
      const float koff = cur * kLog2e + half_log2M;
#pragma unroll
      for (int st = 0; st < RT; ++st) {
        const f32x4 knv = *(const f32x4*)&kn[16 * st + 4 * g];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float kc = 16 * st + 4 * g + r < count ? koff + 0.5f * kLog2e * knv[r] : INFINITY;
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) Lk[st][mt][r] = fast_exp2(Lk[st][mt][r] * kLog2e - kc);
        }
      }
      if constexpr (QSIDE) {
#pragma unroll
        for (int tt = 0; tt < RT; ++tt) {
          const int t = 16 * tt + c;
          const float qs = fmaxf(fmaxf(qmx[bf][0][t], qmx[bf][1][t]), fmaxf(qmx[bf][2][t], qmx[bf][3][t])) * kLog2e;
          // (rows past the tile get finite features; their outputs are not stored)
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int r = 0; r < 4; ++r) Lq[mt][tt][r] = fast_exp2(Lq[mt][tt][r] * kLog2e - qs);
        }
      }
    } else {
#pragma unroll
      for (int st = 0; st < RT; ++st)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            Lk[st][mt][r] = (16 * st + 4 * g + r < count) ? plain_feature<G::KIND>(Lk[st][mt][r], a.relu_eps) : 0.f;
      if constexpr (QSIDE) {
#pragma unroll
        for (int tt = 0; tt < RT; ++tt)
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int r = 0; r < 4; ++r) Lq[mt][tt][r] = plain_feature<G::KIND>(Lq[mt][tt][r], a.relu_eps);
      }
    }

    // K~ contracting over the tile's rows, rounded once for the state update
    // and (with queries) for the transposed copy the scores read
    F kt[RB][MT];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) kt[rb][mt] = tile_pair_frag<T>(Lk[2 * rb][mt], Lk[2 * rb + 1][mt]);

    F vf[RB][ET + 1];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int et = 0; et <= ET; ++et) vf[rb][et] = v_frag<G>(L, Vs, 32 * rb, et, count);

    if constexpr (QSIDE) {
      // keys transposed into this wave's buffer: Zk[m][s]
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          store_half_T(L, Zk[w], LDZ, frag_lo(kt[rb][mt]), 32 * rb, 16 * mt);
          store_half_T(L, Zk[w], LDZ, frag_hi(kt[rb][mt]), 32 * rb + 16, 16 * mt);
        }

      F qf[MB][RT];
#pragma unroll
      for (int kb = 0; kb < MB; ++kb)
#pragma unroll
        for (int tt = 0; tt < RT; ++tt)
          qf[kb][tt] = (2 * kb + 1 < MT) ? tile_pair_frag<T>(Lq[2 * kb][tt], Lq[2 * kb + 1][tt])
                                         : tile_half_frag<T>(Lq[2 * kb][tt]);

      // scores A^T[s][t] = sum_m K~[s][m] Q~[t][m], causal
      f32x4 At[RT][RT];
#pragma unroll
      for (int tt = 0; tt < RT; ++tt)
#pragma unroll
        for (int st = 0; st < RT; ++st) {
          At[st][tt] = zero4();
          if (st > tt) continue;
#pragma unroll
          for (int kb = 0; kb < MB; ++kb)
            At[st][tt] = mma(At[st][tt], frag_tr(L, Zk[w], LDZ, 32 * kb, 16 * st), qf[kb][tt]);
          if (st == tt) {
#pragma unroll
            for (int r = 0; r < 4; ++r)
              if (4 * g + r > c) At[st][tt][r] = 0.f;
          }
        }

      F sf[MB][ET + 1];
#pragma unroll
      for (int kb = 0; kb < MB; ++kb)
#pragma unroll
        for (int et = 0; et <= ET; ++et)
          sf[kb][et] = (2 * kb + 1 < MT) ? tile_pair_frag<T>(S[2 * kb][et], S[2 * kb + 1][et])
                                         : tile_half_frag<T>(S[2 * kb][et]);

      // N^T[e][t] over this wave's features, into the reduction buffer as [t][e]
#pragma unroll
      for (int tt = 0; tt < RT; ++tt)
#pragma unroll
        for (int et = 0; et <= ET; ++et) {
          f32x4 acc = zero4();
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) {
            if (2 * rb > tt) continue;
            const F af = (2 * rb + 1 <= tt) ? tile_pair_frag<T>(At[2 * rb][tt], At[2 * rb + 1][tt])
                                            : tile_half_frag<T>(At[2 * rb][tt]);
            acc = mma(acc, vf[rb][et], af);
          }
#pragma unroll
          for (int kb = 0; kb < MB; ++kb) acc = mma(acc, sf[kb][et], qf[kb][tt]);
          if (et < ET) {
            store_tile_T<float>(L, Red[w], LDR, acc, 16 * et, 16 * tt);
          } else if (g == 0) {
            Red[w][(16 * tt + c) * LDR + D] = acc[0];
          }
        }
    }

    // state update [S|z] += K~^T [V|1]
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int et = 0; et <= ET; ++et)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
          S[mt][et] = mma(S[mt][et], kt[rb][mt], vf[rb][et]);

    __syncthreads();
    if constexpr (QSIDE) {
      // Y = N / D over all features (vector reads of the reduction rows)
      static_assert(EPT % 4 == 0, "");
      // (rows past the tile are computed and dropped by the range-checked
      // stores: no branch, so later waits count exactly)
      const int tid = fresh_tid();
      const int t = tid / TPR, q = tid % TPR;
      // (value dropout: the output scale 1 / (1 - p) folded in)
      const float den = (Red[0][t * LDR + D] + Red[1][t * LDR + D]) + (Red[2][t * LDR + D] + Red[3][t * LDR + D]);
      const float inv = a.drop_scale / den;
      tvec o;
#pragma unroll
      for (int h4 = 0; h4 < EPT / 4; ++h4) {
        const int idx = t * LDR + q * EPT + 4 * h4;
        const f32x4 n = (*(const f32x4*)&Red[0][idx] + *(const f32x4*)&Red[1][idx]) +
                        (*(const f32x4*)&Red[2][idx] + *(const f32x4*)&Red[3][idx]);
        if constexpr (sizeof(T) == 2) {
          const bf16x2 lo = pk_bf16(n[0] * inv, n[1] * inv), hi = pk_bf16(n[2] * inv, n[3] * inv);
          o[4 * h4] = lo[0];
          o[4 * h4 + 1] = lo[1];
          o[4 * h4 + 2] = hi[0];
          o[4 * h4 + 3] = hi[1];
        } else {
#pragma unroll
          for (int i = 0; i < 4; ++i) o[4 * h4 + i] = cvt<T>(n[i] * inv);
        }
      }
      y_rs = range_rsrc((T*)a.Y + head * (size_t)a.L * D + (size_t)start * D, (size_t)count * D * sizeof(T));
      y_off = (t * D + q * EPT) * (int)sizeof(T);
      const pvec* ov = (const pvec*)&o;
#pragma unroll
      for (int v = 0; v < NV; ++v) y_hold[v] = ov[v];
      flush_y();
      // logD: log2 of the row's denominator D in the units of the true
      // features phi (the row shift and the key shift added back), so that
      // phi(q)_m / D = exp2(w_m.q log2(e) - logD) for FAVOR+ and
      // phi(q)_m exp2(-logD) otherwise; one thread per row, rows past the
      // tile dropped by the range check
      {
        const float qs = (G::KIND == kFavor)
                             ? fmaxf(fmaxf(qmx[bf][0][t], qmx[bf][1][t]), fmaxf(qmx[bf][2][t], qmx[bf][3][t])) * kLog2e
                             : 0.f;
        const float l2 = (G::KIND == kFavor) ? qs + __log2f(den) + cur * kLog2e : __log2f(den);
        const __amdgpu_buffer_rsrc_t lrs =
            range_rsrc(a.logD != nullptr ? a.logD + head * (size_t)a.L + start : nullptr,
                       a.logD != nullptr ? (size_t)count * sizeof(float) : 0);
        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(l2), lrs, q == 0 ? t * 4 : INT_MAX - 3, 0, 0);
      }
    }
  }

  // outputs of the segment
  float* sout = nullptr;
  if (MODE == kWalkOutputs) {
    if (p == a.P - 1 && a.state_out != nullptr) sout = a.state_out + head * (size_t)M * (D + 1);
  } else {
    sout = a.seg_out + sidx;
  }
  if (sout != nullptr) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const size_t row = (size_t)(w * FW + 16 * mt + 4 * g + r) * (D + 1);
#pragma unroll
        for (int et = 0; et < ET; ++et) sout[row + 16 * et + c] = S[mt][et][r];
        if (c == 0) sout[row + D] = S[mt][ET][r];
      }
  }
  if (G::KIND == kFavor && threadIdx.x == 0) {
    if (MODE == kWalkSums && a.seg_shift_out != nullptr) a.seg_shift_out[head * a.P + p] = cur;
    if (MODE == kWalkOutputs && p == a.P - 1 && a.kshift_out != nullptr) a.kshift_out[head] = cur;
  }
}

// ---------------------------------------------------------------------------
// Stand-alone feature map.

// per-head key shift: max over rows and features of w_m . k - |k|^2 / 2
template <class G>
__global__ __launch_bounds__(256, 1) void key_shift_kernel(FeatArgs a) {
  typedef typename G::T T;
  typedef typename FragT<T>::type F;
  constexpr int D = G::D, TR = G::TR, MT = G::MT, EB = G::EB, RT = G::RT, LDQ = G::LDQ;
  __shared__ __attribute__((aligned(16))) T Ks[TR * LDQ];
  __shared__ float kn[TR], kmx[4];
  const int w = wave_id(), g = lane_g();
  const size_t head = (size_t)blockIdx.z * a.H + blockIdx.y;
  const T* Kh = (const T*)a.X + head * (size_t)a.L * D;
  F Wf[MT][EB], Wl[MT][EB];
  load_w_frags<G>(Wf, Wl, a.W, w);
  float best = -INFINITY;
  for (int start = 0; start < a.L; start += TR) {
    const int count = min(TR, a.L - start);
    load_rows<T, D, TR, LDQ, 256>(Ks, Kh + (size_t)start * D, count, kn);
    __syncthreads();
    f32x4 Lk[RT][MT];
    key_logits<G>(this_lane(), Lk, Wf, Wl, Ks);
#pragma unroll
    for (int st = 0; st < RT; ++st)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int s = 16 * st + 4 * g + r;
          if (s < count) best = fmaxf(best, Lk[st][mt][r] - 0.5f * kn[s]);
        }
    __syncthreads();
  }
  best = wave_max(best);
  if (lane_id() == 0) kmx[w] = best;
  __syncthreads();
  if (threadIdx.x == 0) a.shift[head] = fmaxf(fmaxf(kmx[0], kmx[1]), fmaxf(kmx[2], kmx[3]));
}

// phi_hat for one tile of TR rows per workgroup
template <class G>
__global__ __launch_bounds__(256, 1) void featmap_kernel(FeatArgs a) {
  typedef typename G::T T;
  typedef typename FragT<T>::type F;
  constexpr int D = G::D, FW = G::FW, M = G::M, TR = G::TR, MT = G::MT, EB = G::EB, RT = G::RT, LDQ = G::LDQ;
  __shared__ __attribute__((aligned(16))) T Xs[TR * LDQ];
  __shared__ float xn[TR], qmx[4][TR];
  const int w = wave_id(), g = lane_g(), c = lane_c();
  const size_t head = (size_t)blockIdx.z * a.H + blockIdx.y;
  const int start = blockIdx.x * TR;
  const int count = min(TR, a.L - start);
  const T* Xh = (const T*)a.X + head * (size_t)a.L * D;
  float* Ph = a.phi + head * (size_t)a.L * M;
  F Wf[MT][EB], Wl[MT][EB];
  load_w_frags<G>(Wf, Wl, a.W, w);
  load_rows<T, D, TR, LDQ, 256>(Xs, Xh + (size_t)start * D, count, G::KIND == kFavor ? xn : nullptr);
  __syncthreads();
  const float half_log2M = 0.5f * __log2f((float)M);
  if (a.role == 0) {
    f32x4 Lq[MT][RT];
    query_logits<G>(this_lane(), Lq, Wf, Wl, Xs);
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
    for (int tt = 0; tt < RT; ++tt) {
      const int t = 16 * tt + c;
      if (t >= count) continue;
      float qs = 0.f;
      if (G::KIND == kFavor) {
        qs = fmaxf(fmaxf(qmx[0][t], qmx[1][t]), fmaxf(qmx[2][t], qmx[3][t]));
        if (w == 0 && g == 0 && a.shift != nullptr) a.shift[head * a.L + start + t] = qs - 0.5f * xn[t];
      }
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = w * FW + 16 * mt + 4 * g + r;
          const float x = Lq[mt][tt][r];
          Ph[(size_t)(start + t) * M + m] =
              (G::KIND == kFavor) ? fast_exp2((x - qs) * kLog2e - half_log2M) : plain_feature<G::KIND>(x, a.relu_eps);
        }
    }
  } else {
    f32x4 Lk[RT][MT];
    key_logits<G>(this_lane(), Lk, Wf, Wl, Xs);
    const float ks = (G::KIND == kFavor) ? a.shift[head] : 0.f;
#pragma unroll
    for (int st = 0; st < RT; ++st)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int s = 16 * st + 4 * g + r;
          if (s >= count) continue;
          const int m = w * FW + 16 * mt + c;
          const float x = Lk[st][mt][r] - (G::KIND == kFavor ? 0.5f * xn[s] : 0.f);
          Ph[(size_t)(start + s) * M + m] =
              (G::KIND == kFavor) ? fast_exp2((x - ks) * kLog2e - half_log2M) : plain_feature<G::KIND>(x, a.relu_eps);
        }
  }
}

// ---------------------------------------------------------------------------
// Fragment-ordered copy of W: one block per fragment, one thread per lane.
template <class G>
__global__ __launch_bounds__(64) void wfrag_kernel(WfragArgs a) {
  typedef typename G::T T;
  typedef typename FragT<T>::type F;
  typedef WFragLayout<G> WL;
  const int f = blockIdx.x, lane = threadIdx.x;
  const int g = lane >> 4, c = lane & 15;
  const int w = f / WL::PER_WAVE;
  int i = f - w * WL::PER_WAVE;
  F v;
  if (f >= 4 * WL::PER_WAVE + WL::NC) {
    // block A': low parts of block A
    i = f - 4 * WL::PER_WAVE - WL::NC;
    const int wl = i / WL::NA;
    i -= wl * WL::NA;
    const int mt = i / G::EB, kb = i - (i / G::EB) * G::EB;
#pragma unroll
    for (int s = 0; s < 8; ++s) v[s] = w_lo<T>(a.W[(size_t)(wl * G::FW + 16 * mt + c) * G::D + 32 * kb + kp(g, s)]);
  } else if (w >= 4) {
    i = f - 4 * WL::PER_WAVE;
    const int kb = i / G::ET, et = i - (i / G::ET) * G::ET;
#pragma unroll
    for (int s = 0; s < 8; ++s) v[s] = cvt<T>(a.W[(size_t)(32 * kb + kp(g, s)) * G::D + 16 * et + c]);
  } else if (i < WL::NA) {
    const int mt = i / G::EB, kb = i - (i / G::EB) * G::EB;
#pragma unroll
    for (int s = 0; s < 8; ++s) v[s] = cvt<T>(a.W[(size_t)(w * G::FW + 16 * mt + c) * G::D + 32 * kb + kp(g, s)]);
  } else {
    i -= WL::NA;
    const int kb = i / G::ET, et = i - (i / G::ET) * G::ET;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const int m = 32 * kb + kp(g, s);
      v[s] = cvt<T>(m < G::FW ? a.W[(size_t)(w * G::FW + m) * G::D + 16 * et + c] : 0.f);
    }
  }
  reinterpret_cast<F*>(a.out)[(size_t)f * 64 + lane] = v;
}

// ---------------------------------------------------------------------------
// launchers

template <class G>
size_t wfrag_bytes() {
  return (size_t)WFragLayout<G>::TOTAL * 64 * sizeof(typename FragT<typename G::T>::type);
}

template <class G>
hipError_t launch_wfrag(const WfragArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(wfrag_kernel<G>, dim3(WFragLayout<G>::TOTAL), dim3(64), 0, s, a);
  return hipGetLastError();
}

template <class G>
hipError_t launch_fwd_walk(const FwdArgs& a, int mode, hipStream_t s) {
  const dim3 grid(a.P, a.H, a.B);
  const bool drop = a.drop_t != 0;
  if (mode == kWalkOutputs) {
    if (drop) hipLaunchKernelGGL((fwd_walk_kernel<G, kWalkOutputs, true>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((fwd_walk_kernel<G, kWalkOutputs, false>), grid, dim3(256), 0, s, a);
  } else if (mode == kWalkSums) {
    if (drop) hipLaunchKernelGGL((fwd_walk_kernel<G, kWalkSums, true>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((fwd_walk_kernel<G, kWalkSums, false>), grid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

template <class G>
hipError_t launch_featmap(const FeatArgs& a, hipStream_t s) {
  if (a.role == 1 && G::KIND == kFavor) {
    hipLaunchKernelGGL(key_shift_kernel<G>, dim3(1, a.H, a.B), dim3(256), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(featmap_kernel<G>, dim3((a.L + G::TR - 1) / G::TR, a.H, a.B), dim3(256), 0, s, a);
  return hipGetLastError();
}

#define SLIM_INST_FWD(T, D, FW, TR, KIND)                                                     \
  template size_t wfrag_bytes<Cfg<T, D, FW, TR, KIND>>();                                     \
  template hipError_t launch_wfrag<Cfg<T, D, FW, TR, KIND>>(const WfragArgs&, hipStream_t);  \
  template hipError_t launch_fwd_walk<Cfg<T, D, FW, TR, KIND>>(const FwdArgs&, int, hipStream_t); \
  template hipError_t launch_featmap<Cfg<T, D, FW, TR, KIND>>(const FeatArgs&, hipStream_t);
SLIM_FOR_EACH_CONFIG(SLIM_INST_FWD)

}  // namespace slim
