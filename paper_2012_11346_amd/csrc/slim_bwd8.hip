// Backward sweep (Algorithm 1, one layer) with 8 waves per workgroup.
//
// Same computation as bwd_walk_kernel (reverse walk over the tiles of one
// segment: downdate of the state B by eq. 17, recomputation of the tile,
// gradients, update of the state cotangent G by eq. 18), with the work of a
// feature slice shared by a pair of waves so that each wave holds half of
// the running state:
//
//   wave w = 4 h + f   feature slice f (features [f FW, (f + 1) FW)), half h
//   value columns      wave h owns the columns [16 EH h, 16 EH (h + 1)) of
//                      S = sum K~^T V, of G and of its dW rows; half 0 also
//                      owns the ones column (z = sum K~ and its cotangent)
//   tile rows          products whose output rows are tile rows and whose
//                      contraction runs over all value columns (dQ~, dK~) are
//                      split by 16-row halves of the tile: half h takes rows
//                      [16 h, 16 h + 16)
//
// The features (logits) of a slice are split between the two waves of its
// pair by feature tiles.  Both waves of a pair compute the in-tile scores A^T
// of their slice.  Cross-slice sums (N, dV, and dq, dk with d = 32) go
// through per-wave reduction rows in LDS; with d = 64 the two waves of a pair
// exchange partial dq and dk tiles over halves of the features.  The
// per-wave register set (state half, cotangent half, dW half) is about half
// of the 4-wave kernel's, which removes its register spills at M = 256 and
// puts two waves on every SIMD.
//
// Phases of one tile (| = workgroup barrier):
//   features (Q and K logits of half of the slice's features) | Q~ -> LDS,
//   downdate, scores, N partials | dN, dD | dA^T, dV partials | dV sums,
//   S -> LDS | dQ~ (this wave's 16 rows), P = dQ~ . Q~ | dq partials, dW | dq
//   sums, G -> LDS | dK~ (16 rows), Pk, G update | dk partials, dW | dk sums,
//   next tile's rows -> LDS |
#include "slim_common.hpp"
#include "slim_kernels.hpp"

namespace slim {

template <class G>
struct Bwd8Lds {
  typedef typename G::T T;
  static constexpr int D = G::D, FW = G::FW, TR = G::TR, ZR = G::ZR;
  static constexpr int EH = G::ET / 2;          // value tiles per wave
  // bf16 tiles are swizzled (SwzLane): rows padded by 16 elements
  static constexpr int LDQ = D + 16;            // Q, K, V, dY / dN rows (kSwzRows)
  static constexpr int LDZK = TR + 16;          // [feature][row] buffers (K~, Pk)
  static constexpr int LDZF = FW + 16;          // [row or value column][feature] buffers (Q~, P, S, G)
  static constexpr int LDZT = TR + 16;          // [row][row] buffers (A^T, dA^T)
  static_assert(LDZT == LDZK, "A^T, dA^T share the lane offsets of K~");
  static constexpr int LDRH = 16 * EH + 4;      // reduction row pitch (floats)
  // floats between the reduction rows of the two value halves (d = 32: the
  // offset keeps the halves of a row in different banks for 8-byte reads)
  static constexpr int REDH = TR * LDRH + (D == 32 ? 16 : 0);
  // shared: Q, K, V, dY (dN overwrites dY), floats, dD as T
  static constexpr size_t TILE = al16((size_t)TR * LDQ * sizeof(T));
  static constexpr size_t oQ = 0, oK = TILE, oV = 2 * TILE, odY = 3 * TILE, oF = 4 * TILE;
  // floats: kn[TR] qmx[TR][8] dDs[TR] zs[4][FW] dzs[4][FW]
  static constexpr size_t NF = TR + 8 * TR + TR + 8 * FW;
  static constexpr size_t odDb = oF + al16(NF * sizeof(float));
  static constexpr size_t oP = odDb + al16((TR + 8) * sizeof(T));
  // per pair: one block holding all of the pair's buffers, so that a lane
  // reaches every buffer of its pair from one address register per access
  // pattern plus immediate offsets
  static constexpr size_t ZK = al16((size_t)ZR * LDZK * sizeof(T));
  static constexpr size_t ZQ = al16((size_t)TR * LDZF * sizeof(T));
  static constexpr size_t ZDA = al16((size_t)TR * LDZT * sizeof(T));
  static constexpr size_t max3(size_t a, size_t b, size_t c) { return a > b ? (a > c ? a : c) : (b > c ? b : c); }
  static constexpr size_t RED = 2 * (size_t)REDH * sizeof(float);  // reduction rows of both waves
  static constexpr size_t REDZ = RED + (size_t)TR * sizeof(float);  // then the ones column of N
  static constexpr size_t ZSG = (size_t)D * LDZF * sizeof(T);
  // Y: N / dV reduction rows (+ the ones column of N), then P (as [t][m]), then G (as [e][m]),
  // then dk reduction rows
  static constexpr size_t ZY = al16(max3(REDZ, (size_t)TR * LDZF * sizeof(T), ZSG));
  // X: A^T, then S (as [e][m]), then dq reduction rows, then Pk (as [m][s])
  static constexpr size_t ZX = al16(max3((size_t)TR * LDZT * sizeof(T), ZSG,
                                         RED > (size_t)ZR * LDZK * sizeof(T) ? RED : (size_t)ZR * LDZK * sizeof(T)));
  static constexpr size_t pY = 0, pX = ZY, pZk = pX + ZX, pZq = pZk + ZK, pZdA = pZq + ZQ, PAIR = pZdA + ZDA;
  static constexpr size_t TOTAL = oP + 4 * PAIR;
  static_assert(TOTAL <= 160 * 1024, "LDS budget of one workgroup");
};

// DROP: value dropout on (its masks are generated only in that instantiation)
// HY: the forward's output Y is given; dD = -rowdot(dY, Y) / D then needs
// only the ones column of N (the denominators), not its value columns.
// HL (with HY): the forward's logD too; then D comes from it, N is not
// recomputed at all, and the row cotangents are formed in the scores phase
// (one barrier fewer per tile).
template <class G, bool DROP, bool HY, bool HL>
__global__ __launch_bounds__(512, 1) void bwd_walk8_kernel(BwdArgs a) {
  typedef typename G::T T;
  typedef typename FragT<T>::type F;
  typedef Bwd8Lds<G> Lay;
  typedef WFragLayout<G> WL;
  constexpr int D = G::D, FW = G::FW, M = G::M, TR = G::TR, MT = G::MT, MB = G::MB, ET = G::ET, EB = G::EB,
                RT = G::RT;
  constexpr int EH = Lay::EH, LDQ = Lay::LDQ, LDZK = Lay::LDZK, LDZF = Lay::LDZF, LDRH = Lay::LDRH,
                REDH = Lay::REDH;
  typedef SwzLane<LDQ, kSwzRows> OR;   // row tiles
  typedef SwzLane<LDZK, kSwzInter> OK;  // K~, Pk, A^T, dA^T
  typedef SwzLane<LDZF, kSwzInter> OF;  // Q~, P, S, G
  constexpr bool ODD = (MT & 1) != 0;  // last 32-deep feature block holds 16 features
  constexpr bool FULL = (ET == 4);      // d = 64: dq and dk tiles over half of the features
  constexpr int MH = MT / 2;            // feature tiles of a wave in the logits
  constexpr int NT = 512, TPR = NT / TR, EPT = D / TPR;
  static_assert(RT == 2 && G::RB == 1, "the two waves of a pair take one 16-row half of the tile each");
  static_assert(ET % 2 == 0 && EPT >= 1, "");
  // (an odd tile count would leave pad rows in buffers that alias float rows)
  static_assert(!ODD, "features per wave must be a multiple of 32");
  static_assert(MT % 2 == 0, "the pair splits the slice's feature tiles");

  __shared__ __attribute__((aligned(16))) char arena[Lay::TOTAL];
  T* Qs = (T*)(arena + Lay::oQ);
  T* Ks = (T*)(arena + Lay::oK);
  T* Vs = (T*)(arena + Lay::oV);
  T* dYs = (T*)(arena + Lay::odY);
  T* dNs = dYs;  // dN = dY / D overwrites dY row by row
  float* fl = (float*)(arena + Lay::oF);
  float* kn = fl;
  float* qmx = kn + TR;        // [TR][8]: row maxima of the query logits per (slice, feature half)
  float* dDs = qmx + 8 * TR;   // [TR]
  float* zs = dDs + TR;        // [4][FW]
  float* dzs = zs + 4 * FW;    // [4][FW]
  T* dDb = (T*)(arena + Lay::odDb);

  // wave-uniform indices live in scalar registers
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), f = w & 3, h = w >> 2;
  const int g = lane_g(), c = lane_c(), lane = lane_id();
  // per-lane offsets of the swizzled tiles; refreshed through an opaque copy
  // at every phase so that addresses derived from them are formed per phase
  OR oR(this_lane());
  OK oK(this_lane());
  OF oF(this_lane());
  auto fresh_offsets = [&]() {
    asm volatile("" : "+v"(oR.a), "+v"(oR.b), "+v"(oK.a), "+v"(oK.b), "+v"(oF.a), "+v"(oF.b));
  };
  // Only wave h = 0 of a pair carries the ones column (z = sum K~ and its
  // cotangent): its products and its writes are skipped by wave h = 1.
  const bool zown = (h == 0);
  char* pz = arena + Lay::oP + f * Lay::PAIR;
  T* Zk = (T*)(pz + Lay::pZk);     // K~ as [m][s]
  T* Zq = (T*)(pz + Lay::pZq);     // Q~ as [t][m]
  // dA^T as [t][s]: one copy for the workgroup (in pair 0's block); its
  // upper-right quarter (s in [16, 32), t in [0, 16)) is never written and
  // stays zero from the initial fill
  T* ZdA = (T*)(arena + Lay::oP + Lay::pZdA);
  T* ZA = (T*)(pz + Lay::pX);      // A^T as [t][s]
  T* ZS = ZA;                                       // S as [e][m]
  T* ZPk = ZA;                                      // Pk as [m][s]
  float* RedX = (float*)(pz + Lay::pX) + h * REDH;  // dq partial rows [t][e']
  T* ZP = (T*)(pz + Lay::pY);      // P as [t][m]
  T* ZG = ZP;                                       // G as [e][m]
  float* RedY = (float*)(pz + Lay::pY) + h * REDH;  // N, dV, dk partial rows [t][e']
  float* RedYz = (float*)(pz + Lay::pY) + 2 * REDH;  // ones column of N [t]
  // row of the reduction threads: the TPR = 16 threads of a row are 16
  // consecutive lanes, and lanes 16 apart take rows 8 apart (their 16-byte
  // reads of the reduction rows then fall into different banks)
  static_assert(TPR == 16 && TR == 32, "reduction thread mapping");
  auto red_row = [](int tid) -> int { return (tid >> 6) + 8 * ((tid >> 4) & 3); };
  // sums over the 4 slices of the EPT consecutive reduction entries
  // [t][col .. col + EPT) of value half hh (vector reads: one row of 16
  // threads covers all banks)
  typedef float fvec __attribute__((ext_vector_type(EPT)));
  static_assert((16 * EH) % EPT == 0 && (LDRH * 4) % 16 == 0, "");
  auto sum_x = [&](int hh, int idx) -> fvec {
    const char* r = arena + Lay::oP + Lay::pX + (hh * REDH + idx) * 4;
    const fvec a0 = *(const fvec*)r, a1 = *(const fvec*)(r + Lay::PAIR);
    const fvec a2 = *(const fvec*)(r + 2 * Lay::PAIR), a3 = *(const fvec*)(r + 3 * Lay::PAIR);
    return (a0 + a1) + (a2 + a3);
  };
  auto sum_y = [&](int hh, int idx) -> fvec {
    const char* r = arena + Lay::oP + Lay::pY + (hh * REDH + idx) * 4;
    const fvec a0 = *(const fvec*)r, a1 = *(const fvec*)(r + Lay::PAIR);
    const fvec a2 = *(const fvec*)(r + 2 * Lay::PAIR), a3 = *(const fvec*)(r + 3 * Lay::PAIR);
    return (a0 + a1) + (a2 + a3);
  };
  auto sum_y1 = [&](int t) -> float {
    const float* r = (const float*)(arena + Lay::oP + Lay::pY) + 2 * REDH + t;
    constexpr int S4 = Lay::PAIR / sizeof(float);
    return (r[0] + r[S4]) + (r[2 * S4] + r[3 * S4]);
  };

  const int p = blockIdx.x, hd = blockIdx.y, b = blockIdx.z;
  const size_t head = (size_t)b * a.H + hd;
  const size_t hoff = head * (size_t)a.L * D;
  const T* Qh = (const T*)a.Q + hoff;
  const T* Kh = (const T*)a.K + hoff;
  const T* Vh = (const T*)a.V + hoff;
  const T* dYh = (const T*)a.dY + hoff;
  const T* Yh = HY ? (const T*)a.Y + hoff : nullptr;
  const float* lDh = HL ? a.logD + head * (size_t)a.L : nullptr;
  // 1 / D of the walk's units from logD: the row shift and the key shift
  // (FAVOR+) taken out again
  const float kshl = (HL && G::KIND == kFavor) ? a.kshift[head] * kLog2e : 0.f;
  T* dQh = (T*)a.dQ + hoff;
  T* dKh = (T*)a.dK + hoff;
  T* dVh = (T*)a.dV + hoff;
  // W fragments through a buffer resource: scalar base and fragment offset,
  // one lane offset register for every fragment
  const __amdgpu_buffer_rsrc_t wrs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(a.Wfrag), (short)0, (int)(WL::TOTAL * 64 * sizeof(F)), 0x00020000);
  const int wlane = lane * (int)sizeof(F);
  auto wfrag = [&](int idx) -> F {
    typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
    u32x4 v[sizeof(F) / 16];
#pragma unroll
    for (int i = 0; i < (int)(sizeof(F) / 16); ++i)
      v[i] = __builtin_amdgcn_raw_buffer_load_b128(wrs, wlane + 16 * i, idx * 64 * (int)sizeof(F), 0);
    return __builtin_bit_cast(F, v);
  };
  // d = 64: the partial dq / dk tile of row tile rt computed by the partner
  // wave, as the result fragment of each lane (X of the pair for dq, Y for dk)
  auto part_x = [&](int rt) -> f32x4* { return (f32x4*)(pz + Lay::pX + rt * 1024 + wlane); };
  auto part_y = [&](int rt) -> f32x4* { return (f32x4*)(pz + Lay::pY + rt * 1024 + wlane); };
  const int e0 = 16 * EH * h;  // first value column of this wave

  const size_t SZ = (size_t)M * (D + 1);
  const size_t sidx = (head * a.P + p) * SZ;
  const float* bend = a.bounds + (head * a.bound_stride + (size_t)(p + 1) * a.bound_step) * SZ;

  // the cotangent starts at the cotangent after the segment when the caller
  // has it (g_init); else at dstate_out in the last segment and at zero in
  // the others (they get the cotangent of later ones added by the carry pass)
  const float* g0 = a.g_init != nullptr ? a.g_init + (head * a.P + p) * SZ
                    : ((p == a.P - 1 && a.dstate_out != nullptr) ? a.dstate_out + head * SZ : nullptr);
  // running state after the current tile (this wave's columns), its cotangent, dW rows
  f32x4 S[MT][EH], Sz[MT], Gs[MT][EH], Gz[MT], dWacc[MT][EH];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const size_t row = (size_t)(f * FW + 16 * mt + 4 * g + r) * (D + 1);
#pragma unroll
      for (int et = 0; et < EH; ++et) {
        S[mt][et][r] = bend[row + e0 + 16 * et + c];
        Gs[mt][et][r] = g0 ? g0[row + e0 + 16 * et + c] : 0.f;
      }
      Sz[mt][r] = bend[row + D];
      Gz[mt][r] = g0 ? g0[row + D] : 0.f;
    }
#pragma unroll
    for (int et = 0; et < EH; ++et) dWacc[mt][et] = zero4();
  }

  // every buffer starts at zero: pad rows of the [feature][row] buffers must read as zero
  for (size_t i = (size_t)threadIdx.x * 16; i < Lay::TOTAL; i += (size_t)NT * 16)
    *reinterpret_cast<uint4*>(arena + i) = uint4{0, 0, 0, 0};

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

  // row staging: threads 0..255 carry Q and K, threads 256..511 carry V and dY
  // (wave-uniform: the range resources of the prefetch live in scalar registers)
  const int sh = __builtin_amdgcn_readfirstlane(threadIdx.x >> 8), stid = threadIdx.x & 255;
  const T* srcA = sh ? Vh : Qh;
  const T* srcB = sh ? dYh : Kh;
  T* dstA = sh ? Vs : Qs;
  T* dstB = sh ? dYs : Ks;
  // (the query norm cancels against the query row shift: only key norms are kept)
  float* nrmA = nullptr;
  float* nrmB = (G::KIND == kFavor && !sh) ? kn : nullptr;
  RowStage<T, D, TR, 256> stA, stB;
  // value dropout: the dropped elements of the value rows are zeroed when
  // staged (threads 256..511 stage V), and those of dV before it is stored
  const Drop drop{a.drop_seed, a.drop_t, a.C, head};
  const bool dropv = DROP && sh;
  __syncthreads();  // zero fill done
  if (j1 > j0) {
    int s0, n0;
    tm.tile(j1 - 1, s0, n0);
    stA.fetch(srcA + (size_t)s0 * D, n0, stid);
    stB.fetch(srcB + (size_t)s0 * D, n0, stid);
    if (dropv) stA.drop(drop, s0, stid);
    stA.template store_swz<LDQ>(dstA, nrmA, stid);
    stB.template store_swz<LDQ>(dstB, nrmB, stid);
  }
  __syncthreads();

  // V operand over the tile's 32 rows, value columns [col, col + 16)
  auto v_frag = [&](int col) -> F { return sfrag_tr(oR, Vs, 0, col); };
  // the ones column of [V|1] over the tile's rows (zero past the tile)
  auto ones_frag = [&](const Lane& L, int count) -> F { return ones_rows_frag(L, 0, count); };
  // operand contracting over this slice's features m in [32 kb, 32 kb + 32),
  // columns = own value tile el of X (el == EH: the ones column Xz)
  auto feat_frag = [&](const f32x4 (&X)[MT][EH], const f32x4 (&Xz)[MT], int el, int kb) -> F {
    return tile_pair_frag<T>(el < EH ? X[2 * kb][el] : Xz[2 * kb], el < EH ? X[2 * kb + 1][el] : Xz[2 * kb + 1]);
  };

  // Output rows are written with range-checked stores (rows past the tile
  // are dropped, no branches) and after the waits for this wave's W
  // fragments in program order: on gfx9 a wait for a load also waits for
  // every earlier store.  dV is held from its reduction to the dq store; dk
  // of a tile is stored in the next tile after its logits.
  typedef unsigned u32e __attribute__((ext_vector_type(EPT / 2)));
  static_assert(EPT == 2 || EPT == 4, "8- or 4-byte row pieces");
  auto cvt_row = [&](const fvec& v) -> u32e {
    u32e o;
#pragma unroll
    for (int i = 0; i < EPT / 2; ++i) o[i] = __builtin_bit_cast(unsigned, pk_bf16(v[2 * i], v[2 * i + 1]));
    return o;
  };
  auto store_piece = [&](const u32e& v, __amdgpu_buffer_rsrc_t rs, int off) {
    if constexpr (EPT == 4) __builtin_amdgcn_raw_buffer_store_b64(v, rs, off, 0, 0);
    else __builtin_amdgcn_raw_buffer_store_b32(v[0], rs, off, 0, 0);
  };
  u32e dk_hold = {};
  f32x4 dk_part;
  // W fragments of the logits, fetched one tile ahead (at the end of the
  // previous tile) so that the features phase starts with them resident
  F Wf[MH][EB];
  auto fetch_wf = [&]() {
#pragma unroll
    for (int i = 0; i < MH; ++i)
#pragma unroll
      for (int kb = 0; kb < EB; ++kb) Wf[i][kb] = wfrag(WL::a(f, MH * h + i, kb));
  };
  fetch_wf();
  __amdgpu_buffer_rsrc_t dk_rs = range_rsrc(dKh, 0);
  int dk_off = 0;
  for (int j = j1 - 1; j >= j0; --j) {
    Lane L = fresh_lane();
    int g = L.g, c = L.c;
    fresh_offsets();
    int start, count;
    tm.tile(j, start, count);
    u32e dv_hold;
    // W fragments of the dq and dk products: with d = 64 (FULL) a wave
    // computes the output tiles of value columns [16 f, 16 f + 16) over both
    // row tiles, contracting over the features of slices 2 h and 2 h + 1 (it
    // reads their P and Pk from LDS); the pair adds its two halves through
    // LDS, and wave h keeps the rows [16 h, 16 h + 16).  With d = 32 each wave
    // contracts over its own slice and the slices are summed in LDS.
    F Wb[FULL ? 1 : MB][FULL ? 1 : EH];
    F Wc[FULL ? 2 * MB : 1];
    f32x4 dq_part;

    // ---- features: Q and K logits of this wave's feature tiles over all tile
    //      rows (the pair splits the slice's features: wave h takes the tiles
    //      [MH h, MH (h + 1)), so each wave reads half of the slice's W);
    //      K~ -> Zk[m][s], row maxima of the query logits -> qmx[t][2 f + h]
    f32x4 Lq[MH][RT];  // rows m = 16 (MH h + i) + 4 g + r, columns t = 16 tt + c
    {
      // low parts of the logits' W fragments (bf16 split of the float32 W),
      // fetched here and used after every high-part product of the phase
      F Wl[MH][EB];
#pragma unroll
      for (int i = 0; i < MH; ++i)
#pragma unroll
        for (int kb = 0; kb < EB; ++kb) Wl[i][kb] = wfrag(WL::alo(f, MH * h + i, kb));
      // raw logits w.q: the query row shift max_m(w.q - |q|^2/2) absorbs the norm term
      F qfr[RT][EB];
#pragma unroll
      for (int tt = 0; tt < RT; ++tt)
#pragma unroll
        for (int kb = 0; kb < EB; ++kb) qfr[tt][kb] = sfrag_rm(oR, Qs, 16 * tt, 32 * kb);
#pragma unroll
      for (int i = 0; i < MH; ++i)
#pragma unroll
        for (int tt = 0; tt < RT; ++tt) {
          f32x4 acc = zero4();
#pragma unroll
          for (int kb = 0; kb < EB; ++kb) acc = mma(acc, Wf[i][kb], qfr[tt][kb]);
          Lq[i][tt] = acc;
        }
      // the low-part products of the queries
#pragma unroll
      for (int i = 0; i < MH; ++i)
#pragma unroll
        for (int tt = 0; tt < RT; ++tt)
#pragma unroll
          for (int kb = 0; kb < EB; ++kb) Lq[i][tt] = mma(Lq[i][tt], Wl[i][kb], qfr[tt][kb]);
      // key rows: exp2(log2e (w.k - |k|^2/2 - shift) - log2(M)/2), the row term folded into the exponent
      // (rows past the tile: an infinite offset gives exactly zero features)
      float kc[RT][4];
      if (G::KIND == kFavor) {
#pragma unroll
        for (int st = 0; st < RT; ++st) {
          const f32x4 knv = *(const f32x4*)&kn[16 * st + 4 * g];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float v = koff + 0.5f * kLog2e * knv[r];
            kc[st][r] = 16 * st + 4 * g + r < count ? v : INFINITY;
          }
        }
      }
      F kfr[RT][EB];  // the tile's key rows as operands
#pragma unroll
      for (int st = 0; st < RT; ++st)
#pragma unroll
        for (int kb = 0; kb < EB; ++kb) kfr[st][kb] = sfrag_rm(oR, Ks, 16 * st, 32 * kb);
      f32x4 Lk[MH][RT];
#pragma unroll
      for (int i = 0; i < MH; ++i)
#pragma unroll
        for (int st = 0; st < RT; ++st) {
          f32x4 kv = zero4();
#pragma unroll
          for (int kb = 0; kb < EB; ++kb) kv = mma(kv, kfr[st][kb], Wf[i][kb]);
          Lk[i][st] = kv;
        }
      // the low-part products of the keys
#pragma unroll
      for (int i = 0; i < MH; ++i)
#pragma unroll
        for (int st = 0; st < RT; ++st)
#pragma unroll
          for (int kb = 0; kb < EB; ++kb) Lk[i][st] = mma(Lk[i][st], kfr[st][kb], Wl[i][kb]);
#pragma unroll
      for (int i = 0; i < MH; ++i)
#pragma unroll
        for (int st = 0; st < RT; ++st) {
          f32x4 kv = Lk[i][st];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            if (G::KIND == kFavor) {
              kv[r] = fast_exp2(kv[r] * kLog2e - kc[st][r]);
            } else {
              const bool ok = 16 * st + 4 * g + r < count;
              kv[r] = ok ? fmaxf(kv[r], 0.f) + a.relu_eps : 0.f;
            }
          }
          sstore_tile_T(oK, Zk, kv, 16 * st, 16 * (MH * h + i));
        }
      if (G::KIND == kFavor) {
#pragma unroll
        for (int tt = 0; tt < RT; ++tt) {
          float v = -INFINITY;
#pragma unroll
          for (int i = 0; i < MH; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) v = fmaxf(v, Lq[i][tt][r]);
          v = wave_max_over_g(v);
          if (g == 0) qmx[(16 * tt + c) * 8 + 2 * f + h] = v;
        }
      }
    }
    __syncthreads();
    L = fresh_lane();
    g = L.g;
    c = L.c;
    fresh_offsets();

    // dk of the previous tile (an empty range before the first)
    store_piece(dk_hold, dk_rs, dk_off);

    // Y (given): the EPT entries of its row that this thread takes in the
    // dN, dD phase, loaded here so that the load is complete by then (rows
    // past the tile read row 0 of the tile and are not used)
    u32e yv = {};
    float lv = 0.f;
    if constexpr (HY) {
      const int tid = fresh_tid();
      const int t = red_row(tid), tc = t < count ? t : 0;
      yv = *(const u32e*)(Yh + (size_t)(start + tc) * D + (tid % TPR) * EPT);
      if constexpr (HL) lv = lDh[start + tc];
    }

    // ---- Q~ of this wave's feature tiles -> Zq[t][m].  Rows past the tile
    //      (zero in LDS) get finite features and need no mask: their dN, dD
    //      are zero, so they add nothing to G, dA, P or dW.
    // (the operands of the downdate are read first, ahead of their use)
    F kfd[MT], vfd[EH];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) kfd[mt] = sfrag_rm(oK, Zk, 16 * mt, 0);  // K~ contracting over rows
#pragma unroll
    for (int el = 0; el < EH; ++el) vfd[el] = v_frag(e0 + 16 * el);
    {
      float qs[RT] = {};
      if (G::KIND == kFavor) {
#pragma unroll
        for (int tt = 0; tt < RT; ++tt) {
          const f32x4 m0 = *(const f32x4*)&qmx[(16 * tt + c) * 8], m1 = *(const f32x4*)&qmx[(16 * tt + c) * 8 + 4];
          qs[tt] = fmaxf(fmaxf(fmaxf(m0[0], m0[1]), fmaxf(m0[2], m0[3])),
                         fmaxf(fmaxf(m1[0], m1[1]), fmaxf(m1[2], m1[3]))) * kLog2e;
        }
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < MH; ++i)
#pragma unroll
        for (int tt = 0; tt < RT; ++tt) {
          f32x4 x = Lq[i][tt];
#pragma unroll
          for (int r = 0; r < 4; ++r)
            x[r] = (G::KIND == kFavor) ? fast_exp2(x[r] * kLog2e - qs[tt]) : fmaxf(x[r], 0.f) + a.relu_eps;
          sstore_tile_T(oF, Zq, x, 16 * (MH * h + i), 16 * tt);
        }
    }

    // ---- state before the tile: downdate (eq. 17), or the exact segment start
    if (j == jreset) {
      const float* bs = a.bounds + (head * a.bound_stride + (size_t)qreset) * SZ + (size_t)(f * FW) * (D + 1) + e0;
      --qreset;
      jreset = (int)((int64_t)qreset * n_tiles / P2);
      int lo = 4 * g * (D + 1) + c;
      asm volatile("" : "+v"(lo));  // lane offsets are formed here, not kept live through the walk
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float* row = bs + lo + (16 * mt + r) * (D + 1);
#pragma unroll
          for (int et = 0; et < EH; ++et) S[mt][et][r] = row[16 * et];
          Sz[mt][r] = row[D - e0 - c];
        }
      // complete these loads here: otherwise the first use of S after the
      // branches would wait for every outstanding load on the common path
      // too, including the next tile's rows (gfx9 encoding: vmcnt(0) only)
      __builtin_amdgcn_s_waitcnt(0x0F70);
    } else {
      // S -= K~^T [V|1]: the [V|1] operands negated once (sign bits of the
      // packed pairs), not every K~ operand
      typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
      auto neg = [](const F& x) { return __builtin_bit_cast(F, __builtin_bit_cast(u32x4, x) ^ 0x80008000u); };
      const F nones = neg(ones_frag(L, count));
      F nv[EH];
#pragma unroll
      for (int el = 0; el < EH; ++el) nv[el] = neg(vfd[el]);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int el = 0; el < EH; ++el) S[mt][el] = mma(S[mt][el], kfd[mt], nv[el]);
      if (zown) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) Sz[mt] = mma(Sz[mt], kfd[mt], nones);
      }
    }

    __syncthreads();  // both halves of Q~ in Zq
    L = fresh_lane();
    g = L.g;
    c = L.c;
    fresh_offsets();
    F qf[MB][RT];  // Q~ contracting over this slice's features, columns t
#pragma unroll
    for (int kb = 0; kb < MB; ++kb)
#pragma unroll
      for (int tt = 0; tt < RT; ++tt) qf[kb][tt] = sfrag_rm(oF, Zq, 16 * tt, 32 * kb);
    F kT[MB][RT];  // K~ contracting over this slice's features, columns s
#pragma unroll
    for (int kb = 0; kb < MB; ++kb)
#pragma unroll
      for (int st = 0; st < RT; ++st) kT[kb][st] = sfrag_tr(oK, Zk, 32 * kb, 16 * st);
    F vT[EH];  // V contracting over the tile's rows, own value columns (for N)
#pragma unroll
    for (int el = 0; el < EH; ++el) vT[el] = HY ? F{} : v_frag(e0 + 16 * el);
    // (every operand of the phase is read before its first product)
    __builtin_amdgcn_sched_barrier(0);

    // ---- scores A^T[s][t] over this slice's features, causal -> ZA[t][s] (for dV)
    f32x4 At[RT][RT];
#pragma unroll
    for (int tt = 0; tt < RT; ++tt)
#pragma unroll
      for (int st = 0; st < RT; ++st) {
        f32x4 acc = zero4();
        if (st <= tt) {
#pragma unroll
          for (int kb = 0; kb < MB; ++kb) acc = mma(acc, kT[kb][st], qf[kb][tt]);
        }
        if (st == tt) {
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (4 * g + r > c) acc[r] = 0.f;
        }
        At[st][tt] = acc;
      }
    F af[RT];  // A^T contracting over rows s, columns t (rounded once, also -> ZA)
#pragma unroll
    for (int tt = 0; tt < RT; ++tt) {
      af[tt] = tile_pair_frag<T>(At[0][tt], At[1][tt]);
      if (zown) {  // (both waves of the pair hold the same scores)
        sstore_half_T(oK, ZA, frag_lo(af[tt]), 0, 16 * tt);
        sstore_half_T(oK, ZA, frag_hi(af[tt]), 16, 16 * tt);
      }
    }
    // ---- dN = dY / D, dD = -(dY . N) / D^2 per row (TPR threads per row)
    auto row_cotangents = [&]() {
      const int tid = fresh_tid();
      const int t = red_row(tid), q = tid % TPR;
      const bool ok = t < count;
      float inv;
      if constexpr (HL) {
        // D from logD, in the walk's units: 2^(row shift + key shift - logD)
        float qsh = 0.f;
        if (G::KIND == kFavor) {
          const f32x4 m0 = *(const f32x4*)&qmx[t * 8], m1 = *(const f32x4*)&qmx[t * 8 + 4];
          qsh = fmaxf(fmaxf(fmaxf(m0[0], m0[1]), fmaxf(m0[2], m0[3])), fmaxf(fmaxf(m1[0], m1[1]), fmaxf(m1[2], m1[3]))) *
                    kLog2e + kshl;
        }
        inv = ok ? fast_exp2(qsh - lv) : 0.f;
      } else {
        const float den = sum_y1(t);
        inv = ok ? 1.f / den : 0.f;
      }
      // (value dropout: Y = s N / D with the output scale s; 1 without dropout)
      const float invs = inv * a.drop_scale;
      const int e = q * EPT, hh = e / (16 * EH), col = e - hh * 16 * EH;
      float dy[EPT];
      float dot = 0.f;
      if constexpr (HY) {
        // Y = s N / D as the forward wrote it
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
          dy[i] = to_f32(dYs[swz_off<LDQ, kSwzRows>(t, e) + i]);
          const unsigned u = yv[i / 2];
          dot += dy[i] * __uint_as_float((i & 1) ? (u & 0xFFFF0000u) : (u << 16));
        }
      } else {
        const fvec n = sum_y(hh, t * LDRH + col);
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
          dy[i] = to_f32(dYs[swz_off<LDQ, kSwzRows>(t, e) + i]);
          dot += dy[i] * (n[i] * invs);
        }
      }
      dot = sum_lane_group<TPR>(dot);
      u32e dn;
#pragma unroll
      for (int i = 0; i < EPT / 2; ++i) dn[i] = __builtin_bit_cast(unsigned, pk_bf16(dy[2 * i] * invs, dy[2 * i + 1] * invs));
      *(u32e*)&dNs[swz_off<LDQ, kSwzRows>(t, e)] = dn;
      if (q == 0) {
        const float dd = ok ? -dot * inv : 0.f;
        dDs[t] = dd;
        dDb[t] = cvt<T>(dd);
      }
    };
    if constexpr (HL) {
      // (nothing of N is needed; dY is not read before this point of the tile)
      row_cotangents();
    } else {
      // N^T[e][t] = [V|1]^T A^T + [S|z]^T Q~^T over this slice, own columns -> RedY[t][e']
      // (with Y given only the ones column, D)
#pragma unroll
      for (int tt = 0; tt < RT; ++tt) {
#pragma unroll
        for (int el = HY ? EH : 0; el <= EH; ++el) {
          if (el == EH && !zown) break;
          f32x4 acc = mma(zero4(), el < EH ? vT[el < EH ? el : 0] : ones_frag(L, count), af[tt]);
#pragma unroll
          for (int kb = 0; kb < MB; ++kb) acc = mma(acc, feat_frag(S, Sz, el, kb), qf[kb][tt]);
          if (el < EH) {
            store_tile_T<float>(L, RedY, LDRH, acc, 16 * el, 16 * tt);
          } else if (g == 0) {
            RedYz[16 * tt + c] = acc[0];
          }
        }
      }
      __syncthreads();
      L = fresh_lane();
      g = L.g;
      c = L.c;
      fresh_offsets();
      row_cotangents();
    }
    __syncthreads();
    L = fresh_lane();
    g = L.g;
    c = L.c;
    fresh_offsets();

    // ---- dA^T[s][t] = sum_e V[s][e] dN[t][e] + dD[t], causal -> ZdA[t][s], once per
    //      workgroup: wave 0 takes the tile (s, t) in ([0,16), [0,16)), wave 1
    //      ([0,16), [16,32)), wave 2 ([16,32), [16,32)).  A row s past the tile has
    //      V[s] = 0 and is reached only from rows t >= s, whose dD is zero.
    if (w < 3) {
      const int st = w >> 1, tt = (w + 1) >> 1;
      const float ddt = dDs[16 * tt + c];
      F vr[EB], dr[EB];
#pragma unroll
      for (int kb = 0; kb < EB; ++kb) {
        vr[kb] = sfrag_rm(oR, Vs, 16 * st, 32 * kb);
        dr[kb] = sfrag_rm(oR, dNs, 16 * tt, 32 * kb);
      }
      __builtin_amdgcn_sched_barrier(0);
      f32x4 acc = f32x4{ddt, ddt, ddt, ddt};
#pragma unroll
      for (int kb = 0; kb < EB; ++kb) acc = mma(acc, vr[kb], dr[kb]);
      if (st == tt) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (4 * g + r > c) acc[r] = 0.f;
      }
      sstore_tile_T(oK, ZdA, acc, 16 * st, 16 * tt);
    }
    // dV^T[e][s] = sum_m G[m][e] K~[s][m] + sum_t dN[t][e] A^T[s][t], own columns -> RedY[s][e']
    // (per row tile, its operands are read before its products)
    {
      F dnT[EH];
#pragma unroll
      for (int el = 0; el < EH; ++el) dnT[el] = sfrag_tr(oR, dNs, 0, 16 * (h * EH + el));
#pragma unroll
      for (int st = 0; st < RT; ++st) {
        const F aT = sfrag_tr(oK, ZA, 0, 16 * st);
        F kT[MB];
#pragma unroll
        for (int kb = 0; kb < MB; ++kb) kT[kb] = sfrag_tr(oK, Zk, 32 * kb, 16 * st);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int el = 0; el < EH; ++el) {
          f32x4 acc = mma(zero4(), dnT[el], aT);
#pragma unroll
          for (int kb = 0; kb < MB; ++kb) acc = mma(acc, feat_frag(Gs, Gz, el, kb), kT[kb]);
          store_tile_T<float>(L, RedY, LDRH, acc, 16 * el, 16 * st);
        }
      }
    }
    __syncthreads();
    L = fresh_lane();
    g = L.g;
    c = L.c;
    fresh_offsets();

    // ---- dV = sum over slices (held); S (own columns) -> ZS[e][m], z -> zs
    {
      const int tid = fresh_tid();
      const int t = red_row(tid), q = tid % TPR;
      const int e = q * EPT, hh = e / (16 * EH), col = e - hh * 16 * EH;
      fvec dvs = sum_y(hh, t * LDRH + col);
      if (DROP) {
        const unsigned keep = drop_keep_bits<EPT>(drop, start + t, e);
#pragma unroll
        for (int i = 0; i < EPT; ++i) dvs[i] = (keep >> i) & 1u ? dvs[i] : 0.f;
      }
      dv_hold = cvt_row(dvs);
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
      for (int el = 0; el < EH; ++el) sstore_tile_T(oF, ZS, S[mt][el], 16 * mt, e0 + 16 * el);
      if (zown && c == 0) {
#pragma unroll
        for (int r = 0; r < 4; ++r) zs[f * FW + 16 * mt + 4 * g + r] = Sz[mt][r];
      }
    }
    __syncthreads();
    L = fresh_lane();
    g = L.g;
    c = L.c;
    fresh_offsets();

    // ---- dQ~^T[m][t] = sum_e S[m][e] dN[t][e] + z[m] dD[t] + sum_s K~[s][m] dA^T[s][t]
    //      for this wave's rows t in [16 h, 16 h + 16); P = dQ~ . Q~ (FAVOR+) or
    //      dQ~ masked (ReLU) -> ZP[t][m]
    // (the W fragments of the dq and dk products are fetched here, a phase
    // ahead of their first use)
    if constexpr (FULL) {
#pragma unroll
      for (int i = 0; i < 2 * MB; ++i) Wc[i] = wfrag(WL::c(2 * h * MB + i, f));
    } else {
#pragma unroll
      for (int kb = 0; kb < MB; ++kb)
#pragma unroll
        for (int el = 0; el < EH; ++el) Wb[kb][el] = wfrag(WL::b(f, kb, h * EH + el));
    }
    // rows of the next tile, stored into LDS at the end of this one; issued
    // after the W fragments so that waiting for those does not wait for
    // these, and half a tile ahead of the logits' W fragments (fetched at the
    // end of the tile), so that those do not queue behind them.  Range-checked
    // loads without branches (an empty range after the last tile) keep the
    // count of outstanding loads exact.
    {
      const int st2 = fresh_tid() & 255;
      int sn, cn;
      tm.tile(j > j0 ? j - 1 : j, sn, cn);
      const size_t nb = j > j0 ? (size_t)cn * D * sizeof(T) : 0;
      stA.fetch(range_rsrc(srcA + (size_t)sn * D, nb), 0, st2);
      stB.fetch(range_rsrc(srcB + (size_t)sn * D, nb), 0, st2);
    }
    {
      // the operands shared by every feature tile, then per feature tile
      // all of its operands before its products (the fence keeps the
      // compiler from putting a wait before each product)
      const float ddt = dDs[16 * h + c];
      F dnf[EB];
#pragma unroll
      for (int kb = 0; kb < EB; ++kb) dnf[kb] = sfrag_rm(oR, dNs, 16 * h, 32 * kb);
      const F daf = sfrag_rm(oK, ZdA, 16 * h, 0);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const f32x4 zv = *(const f32x4*)&zs[f * FW + 16 * mt + 4 * g];
        F zsf[EB];
#pragma unroll
        for (int kb = 0; kb < EB; ++kb) zsf[kb] = sfrag_tr(oF, ZS, 32 * kb, 16 * mt);
        const F zkf = sfrag_rm(oK, Zk, 16 * mt, 0);
        const f32x4 qv = sload_tile_T(oF, Zq, 16 * mt, 16 * h);
        __builtin_amdgcn_sched_barrier(0);
        f32x4 acc = zv * ddt;
#pragma unroll
        for (int kb = 0; kb < EB; ++kb) acc = mma(acc, zsf[kb], dnf[kb]);
        acc = mma(acc, zkf, daf);
#pragma unroll
        for (int r = 0; r < 4; ++r)
          acc[r] = (G::KIND == kFavor) ? acc[r] * qv[r] : (qv[r] > a.relu_eps ? acc[r] : 0.f);
        sstore_tile_T(oF, ZP, acc, 16 * mt, 16 * h);
      }
    }
    __syncthreads();
    L = fresh_lane();
    g = L.g;
    c = L.c;
    fresh_offsets();

    // ---- dq^T[e][t] = sum_m W[m][e] P[t][m] (FULL: columns [16 f, 16 f + 16)
    //      over the features of slices 2 h, 2 h + 1, the partner's row tile ->
    //      LDS, the own one held; else own columns over this slice -> RedX[t][e']);
    //      dW[m][e] += sum_t P[t][m] Q[t][e].  The FAVOR+ chain rule also has
    //      -q[t] sum_m P[t][m], which is zero: Y is homogeneous of degree 0 in
    //      each query feature vector, so sum_m Q~[t][m] dQ~[t][m] = 0.
    if constexpr (FULL) {
      // P of one slice at a time (both row tiles), read before its products
      f32x4 acc[RT] = {};
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const T* Ps = (const T*)(arena + Lay::oP + (2 * h + i) * Lay::PAIR + Lay::pY);
        F pa[RT][MB];
#pragma unroll
        for (int tt = 0; tt < RT; ++tt)
#pragma unroll
          for (int kb = 0; kb < MB; ++kb) pa[tt][kb] = sfrag_rm(oF, Ps, 16 * tt, 32 * kb);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int tt = 0; tt < RT; ++tt)
#pragma unroll
          for (int kb = 0; kb < MB; ++kb) acc[tt] = mma(acc[tt], Wc[i * MB + kb], pa[tt][kb]);
      }
      *part_x(1 - h) = h ? acc[0] : acc[1];
      dq_part = h ? acc[1] : acc[0];
      F pT[MT], qT[EH];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) pT[mt] = sfrag_tr(oF, ZP, 0, 16 * mt);
#pragma unroll
      for (int el = 0; el < EH; ++el) qT[el] = sfrag_tr(oR, Qs, 0, e0 + 16 * el);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int el = 0; el < EH; ++el) dWacc[mt][el] = mma(dWacc[mt][el], pT[mt], qT[el]);
    } else {
      // every operand of the phase is read before its first product
      F pr[RT][MB], pT[MT], qT[EH];
#pragma unroll
      for (int tt = 0; tt < RT; ++tt)
#pragma unroll
        for (int kb = 0; kb < MB; ++kb) pr[tt][kb] = sfrag_rm(oF, ZP, 16 * tt, 32 * kb);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) pT[mt] = sfrag_tr(oF, ZP, 0, 16 * mt);
#pragma unroll
      for (int el = 0; el < EH; ++el) qT[el] = sfrag_tr(oR, Qs, 0, e0 + 16 * el);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int tt = 0; tt < RT; ++tt) {
#pragma unroll
        for (int el = 0; el < EH; ++el) {
          f32x4 acc = zero4();
#pragma unroll
          for (int kb = 0; kb < MB; ++kb) acc = mma(acc, Wb[kb][el], pr[tt][kb]);
          store_tile_T<float>(L, RedX, LDRH, acc, 16 * el, 16 * tt);
        }
      }
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int el = 0; el < EH; ++el) dWacc[mt][el] = mma(dWacc[mt][el], pT[mt], qT[el]);
    }
    __syncthreads();
    L = fresh_lane();
    g = L.g;
    c = L.c;
    fresh_offsets();

    // ---- dq = sum over slices; G (own columns) -> ZG[e][m], dz -> dzs
    {
      const int tid = fresh_tid();
      const int t = red_row(tid), q = tid % TPR;
      const int e = q * EPT, hh = e / (16 * EH), col = e - hh * 16 * EH;
      const int off = (t * D + e) * (int)sizeof(T);
      const size_t nb = (size_t)count * D * sizeof(T);
      if constexpr (FULL) {
        // lane (g, c) of the wave's tile: row 16 h + c, columns 16 f + 4 g + [0, 4)
        const Lane Lq = fresh_lane();
        const u32e dq = __builtin_bit_cast(u32e, pk_bf16x4(dq_part + *part_x(h)));
        store_piece(dq, range_rsrc(dQh + (size_t)start * D, nb), ((16 * h + Lq.c) * D + 16 * f + 4 * Lq.g) * (int)sizeof(T));
      } else {
        store_piece(cvt_row(sum_x(hh, t * LDRH + col)), range_rsrc(dQh + (size_t)start * D, nb), off);
      }
      store_piece(dv_hold, range_rsrc(dVh + (size_t)start * D, nb), off);
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
      for (int el = 0; el < EH; ++el) sstore_tile_T(oF, ZG, Gs[mt][el], 16 * mt, e0 + 16 * el);
      if (zown && c == 0) {
#pragma unroll
        for (int r = 0; r < 4; ++r) dzs[f * FW + 16 * mt + 4 * g + r] = Gz[mt][r];
      }
    }
    __syncthreads();
    L = fresh_lane();
    g = L.g;
    c = L.c;
    fresh_offsets();

    // ---- dK~[s][m] = sum_e V[s][e] G[m][e] + dz[m] + sum_t dA^T[s][t] Q~[t][m] for this
    //      wave's rows s in [16 h, 16 h + 16); Pk = dK~ . K~ (FAVOR+) or masked (ReLU)
    //      -> ZPk[m][s] (rows past the tile have K~ = 0, hence Pk = 0)
    //      and G[m][e] += sum_t Q~[t][m] [dN|dD][t][e] (eq. 18), own columns.
    //      (FULL: the W fragments of the dk product are fetched again here, a
    //      phase ahead, so that they are not held through the phases between)
    //      The operands shared by every feature tile are read first, then per
    //      feature tile all of its operands before its products (the fence
    //      keeps the compiler from putting a wait before each product); the
    //      Q~ operand serves both products.
    if constexpr (FULL) {
#pragma unroll
      for (int i = 0; i < 2 * MB; ++i) Wc[i] = wfrag(WL::c(2 * h * MB + i, f));
    }
    {
      F vfr[EB], dnT[EH];
#pragma unroll
      for (int kb = 0; kb < EB; ++kb) vfr[kb] = sfrag_rm(oR, Vs, 16 * h, 32 * kb);
      const F daT = sfrag_tr(oK, ZdA, 0, 16 * h);
#pragma unroll
      for (int el = 0; el < EH; ++el) dnT[el] = sfrag_tr(oR, dNs, 0, e0 + 16 * el);
      F dd;
#pragma unroll
      for (int s = 0; s < 8; ++s) dd[s] = dDb[kp(g, s)];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const float dz = dzs[f * FW + 16 * mt + c];
        F gfr[EB];
#pragma unroll
        for (int kb = 0; kb < EB; ++kb) gfr[kb] = sfrag_tr(oF, ZG, 32 * kb, 16 * mt);
        const F qf = sfrag_tr(oF, Zq, 0, 16 * mt);
        const f32x4 kv = sload_tile_T(oK, Zk, 16 * h, 16 * mt);
        __builtin_amdgcn_sched_barrier(0);
        f32x4 acc = {dz, dz, dz, dz};
#pragma unroll
        for (int kb = 0; kb < EB; ++kb) acc = mma(acc, vfr[kb], gfr[kb]);
        acc = mma(acc, daT, qf);
#pragma unroll
        for (int el = 0; el < EH; ++el) Gs[mt][el] = mma(Gs[mt][el], qf, dnT[el]);
        if (zown) Gz[mt] = mma(Gz[mt], qf, dd);
#pragma unroll
        for (int r = 0; r < 4; ++r)
          acc[r] = (G::KIND == kFavor) ? acc[r] * kv[r] : (kv[r] > a.relu_eps ? acc[r] : 0.f);
        sstore_tile_T(oK, ZPk, acc, 16 * h, 16 * mt);
      }
    }
    __syncthreads();
    L = fresh_lane();
    g = L.g;
    c = L.c;
    fresh_offsets();

    // ---- dW[m][e] += sum_s Pk[s][m] K[s][e]; dk^T[e][s] = sum_m W[m][e] Pk[s][m] - k[s][e] rowsum_f(Pk)[s]
    //      own columns -> RedY[s][e'], with rowsum_f(Pk)[s] (over this slice's features) from
    //      a product with an all-ones operand
    {
      // the key operands first, then per feature tile its Pk operand
      F kT[EH];
#pragma unroll
      for (int el = 0; el < EH; ++el) kT[el] = sfrag_tr(oR, Ks, 0, e0 + 16 * el);
      F pf[MT];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) pf[mt] = sfrag_rm(oK, ZPk, 16 * mt, 0);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int el = 0; el < EH; ++el) dWacc[mt][el] = mma(dWacc[mt][el], pf[mt], kT[el]);
    }
    if constexpr (FULL) {
      // dk^T[e][s] = sum_m W[m][e] Pk[s][m] - k[s][e] rowsum(Pk)[s] for columns
      // [16 f, 16 f + 16) over the features of slices 2 h, 2 h + 1 (both terms
      // are sums over features, so the halves add up; the rowsum from products
      // with an all-ones operand); the partner's row tile -> LDS, the own one
      // held and completed in the next phase
      bf16x4 ke[RT];
#pragma unroll
      for (int st = 0; st < RT; ++st)
        ke[st] = G::KIND == kFavor ? *(const bf16x4*)&Ks[oR.a + 16 * st * LDQ + 16 * f] : bf16x4{};
      F ones;
#pragma unroll
      for (int s2 = 0; s2 < 8; ++s2) ones[s2] = cvt<T>(1.f);
      f32x4 acc[RT] = {}, rs[RT] = {};
      // Pk of one slice at a time (both row tiles), read before its products
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const T* Pks = (const T*)(arena + Lay::oP + (2 * h + i) * Lay::PAIR + Lay::pX);
        F pa[RT][MB];
#pragma unroll
        for (int st = 0; st < RT; ++st)
#pragma unroll
          for (int kb = 0; kb < MB; ++kb) pa[st][kb] = sfrag_tr(oK, Pks, 32 * kb, 16 * st);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int st = 0; st < RT; ++st)
#pragma unroll
          for (int kb = 0; kb < MB; ++kb) {
            acc[st] = mma(acc[st], Wc[i * MB + kb], pa[st][kb]);
            if (G::KIND == kFavor) rs[st] = mma(rs[st], ones, pa[st][kb]);
          }
      }
      if (G::KIND == kFavor) {
#pragma unroll
        for (int st = 0; st < RT; ++st) {
          const float rsv = rs[st][0];  // every row of the product holds the sums of the columns s
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[st][r] += (float)ke[st][r] * (-rsv);
        }
      }
      *part_y(1 - h) = h ? acc[0] : acc[1];
      dk_part = h ? acc[1] : acc[0];
      dk_rs = range_rsrc(dKh + (size_t)start * D, (size_t)count * D * sizeof(T));
      dk_off = ((16 * h + c) * D + 16 * f + 4 * g) * (int)sizeof(T);
    } else {
    // every operand of the dk products first: Pk over this slice and the key entries
    F pkk[RT][MB];
    bf16x4 kent[RT][EH];
#pragma unroll
    for (int st = 0; st < RT; ++st) {
#pragma unroll
      for (int kb = 0; kb < MB; ++kb) pkk[st][kb] = sfrag_tr(oK, ZPk, 32 * kb, 16 * st);
#pragma unroll
      for (int el = 0; el < EH; ++el)
        kent[st][el] = G::KIND == kFavor ? *(const bf16x4*)&Ks[oR.a + 16 * st * LDQ + 16 * (h * EH + el)] : bf16x4{};
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int st = 0; st < RT; ++st) {
      const F (&pk)[MB] = pkk[st];
      float rsv = 0.f;
      if (G::KIND == kFavor) {
        F ones;
#pragma unroll
        for (int s2 = 0; s2 < 8; ++s2) ones[s2] = cvt<T>(1.f);
        f32x4 rs = zero4();
#pragma unroll
        for (int kb = 0; kb < MB; ++kb) rs = mma(rs, ones, pk[kb]);
        rsv = rs[0];  // every row of the product holds the sums of the columns s
      }
#pragma unroll
      for (int el = 0; el < EH; ++el) {
        f32x4 acc;
        if (G::KIND == kFavor) {
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[r] = (float)kent[st][el][r] * (-rsv);
        } else {
          acc = zero4();
        }
#pragma unroll
        for (int kb = 0; kb < MB; ++kb)
          acc = mma(acc, Wb[kb][el], pk[kb]);
        store_tile_T<float>(L, RedY, LDRH, acc, 16 * el, 16 * st);
      }
    }
    }
    __syncthreads();
    L = fresh_lane();
    g = L.g;
    c = L.c;
    fresh_offsets();

    // ---- dk = sum over slices or feature halves (held); rows of the next
    //      tile -> LDS (their readers are done)
    if constexpr (FULL) {
      dk_hold = __builtin_bit_cast(u32e, pk_bf16x4(dk_part + *part_y(h)));
    } else {
      const int tid = fresh_tid();
      const int t = red_row(tid), q = tid % TPR;
      const int e = q * EPT, hh = e / (16 * EH), col = e - hh * 16 * EH;
      dk_hold = cvt_row(sum_y(hh, t * LDRH + col));
      dk_rs = range_rsrc(dKh + (size_t)start * D, (size_t)count * D * sizeof(T));
      dk_off = (t * D + e) * (int)sizeof(T);
    }
    if (j > j0) {
      const int st2 = fresh_tid() & 255;
      if (dropv) {
        int sn, cn;
        tm.tile(j - 1, sn, cn);
        stA.drop(drop, sn, st2);
      }
      stA.template store_swz<LDQ>(dstA, nrmA, st2);
      stB.template store_swz<LDQ>(dstB, nrmB, st2);
    }
    fetch_wf();
    __syncthreads();
    L = fresh_lane();
    g = L.g;
    c = L.c;
    fresh_offsets();
  }

  store_piece(dk_hold, dk_rs, dk_off);

  // per-workgroup dW partial: this wave's rows and columns
  float* dwp = a.dW_part + (head * a.P + p) * (size_t)M * D;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int el = 0; el < EH; ++el)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        dwp[(size_t)(f * FW + 16 * mt + 4 * g + r) * D + e0 + 16 * el + c] = dWacc[mt][el][r];
  // cotangent the walk ends with (several segments), or the state cotangent
  // before the sequence (one segment)
  float* gout = a.g_final != nullptr ? a.g_final + sidx
                                     : ((p == 0 && a.dstate_in != nullptr) ? a.dstate_in + head * SZ : nullptr);
  // (the caller's initial state has its own key shift: its cotangent scales by exp(init_shift - kshift))
  float r0 = 1.f;
  if (G::KIND == kFavor && a.init_shift != nullptr && a.g_final == nullptr)
    r0 = fast_exp2((a.init_shift[head] - a.kshift[head]) * kLog2e);
  if (gout != nullptr) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const size_t row = (size_t)(f * FW + 16 * mt + 4 * g + r) * (D + 1);
#pragma unroll
        for (int el = 0; el < EH; ++el) gout[row + e0 + 16 * el + c] = r0 * Gs[mt][el][r];
        if (zown && c == 0) gout[row + D] = r0 * Gz[mt][r];
      }
  }
}

template <class G>
hipError_t launch_bwd_walk8(const BwdArgs& a, hipStream_t s) {
  const dim3 grid(a.P, a.H, a.B);
  const bool hy = a.Y != nullptr, hl = hy && a.logD != nullptr;
  if (a.drop_t != 0) {
    if (hl) hipLaunchKernelGGL((bwd_walk8_kernel<G, true, true, true>), grid, dim3(512), 0, s, a);
    else if (hy) hipLaunchKernelGGL((bwd_walk8_kernel<G, true, true, false>), grid, dim3(512), 0, s, a);
    else hipLaunchKernelGGL((bwd_walk8_kernel<G, true, false, false>), grid, dim3(512), 0, s, a);
  } else {
    if (hl) hipLaunchKernelGGL((bwd_walk8_kernel<G, false, true, true>), grid, dim3(512), 0, s, a);
    else if (hy) hipLaunchKernelGGL((bwd_walk8_kernel<G, false, true, false>), grid, dim3(512), 0, s, a);
    else hipLaunchKernelGGL((bwd_walk8_kernel<G, false, false, false>), grid, dim3(512), 0, s, a);
  }
  return hipGetLastError();
}

#define SLIM_INST_BWD8(T, D, FW, TR, KIND) \
  template hipError_t launch_bwd_walk8<Cfg<T, D, FW, TR, KIND>>(const BwdArgs&, hipStream_t);
SLIM_FOR_EACH_BF16_CONFIG(SLIM_INST_BWD8)

}  // namespace slim
