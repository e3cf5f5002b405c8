// Carried state cotangent of the segmented reverse walk, 8-wave form for
// bf16 problems with M = 128 or 256 features (the arithmetic of carry_kernel:
// rows of segment p < P - 1 receive the contribution of G_end(p), the
// cotangent after the segment, eq. 18 summed over the later segments):
//   dV[s]  += K~[s] G_end(p)
//   Pk[s]   = ([V[s] | 1] G_end(p)^T) . K~[s]          (FAVOR+; ReLU: masked where w.k <= 0)
//   dk[s]  += Pk[s] W - k[s] rowsum(Pk[s])              (FAVOR+; ReLU: Pk[s] W)
//   dW     += sum_s Pk[s]^T k[s]
//
// Schedule.  The rows of every head's segments 0 .. P-2 are cut into chunks
// of 32 rows that never straddle a segment boundary; the chunks of all heads,
// in order, are dealt to the workgroups in contiguous runs of equal length
// (one workgroup per compute unit), so every workgroup gets the same work.
// Each workgroup keeps its own dW partial over everything it visits (dW is
// shared by all heads).
//
// Per chunk, wave w first maps its M/8 features for all rows of the chunk:
// key logits and features, dK~ from G_end, Pk, the wave's part of
// rowsum(Pk), K~ and Pk into LDS ([row][feature]) and its rows of dW.  After
// the chunk's one barrier it computes its share of the chunk's dV and dk
// tiles, contracting over all M features from LDS.  G_end of the current
// segment lives in registers in the two operand layouts it is used in and is
// reloaded when a run crosses a segment boundary.  Row tiles are
// triple-buffered and the K~/Pk tiles double-buffered, so the one barrier per
// chunk orders every LDS hazard: a buffer written during chunk i was last
// read during chunk i - 2 (row tiles: i - 2, their readers finish before
// barrier i - 1).
#include "slim_common.hpp"
#include "slim_kernels.hpp"

namespace slim {

namespace {

constexpr int kCarryRows = 32;  // rows per chunk

// rows [a0, a1) of segment p of a head (segments cut at the walk's 32-row tiles)
__host__ __device__ inline void carry_seg_rows(const TileMap& tm, int n_tiles, int P, int p, int& a0, int& a1) {
  const int j0 = (int)((int64_t)p * n_tiles / P), j1 = (int)((int64_t)(p + 1) * n_tiles / P);
  int c_;
  tm.tile(j0, a0, c_);
  a1 = a0;
  if (j1 > j0) {
    int s_;
    tm.tile(j1 - 1, s_, c_);
    a1 = s_ + c_;
  }
}

// position of one chunk in the (head, segment, chunk) order, with its rows'
// byte range in a [B,H,L,D] bf16 tensor; wave-uniform
struct ChunkPos {
  int head, p, k, nk, a0, a1;
  int cnt;       // rows of the chunk
  int nbytes;    // bytes of its rows; 0 for a chunk past the workgroup's run
  int64_t boff;  // byte offset of its first row
  __device__ void finish(int L, int row_bytes, bool valid) {
    const int r0 = a0 + k * kCarryRows;
    cnt = min(kCarryRows, a1 - r0);
    nbytes = valid ? cnt * row_bytes : 0;
    boff = ((int64_t)head * L + r0) * row_bytes;
    // the fields in scalar registers (values computed with vector
    // instructions, such as 64-bit divisions, would otherwise turn every
    // buffer access based on them into a loop over lanes)
    head = __builtin_amdgcn_readfirstlane(head);
    p = __builtin_amdgcn_readfirstlane(p);
    k = __builtin_amdgcn_readfirstlane(k);
    nk = __builtin_amdgcn_readfirstlane(nk);
    a0 = __builtin_amdgcn_readfirstlane(a0);
    a1 = __builtin_amdgcn_readfirstlane(a1);
    cnt = __builtin_amdgcn_readfirstlane(cnt);
    nbytes = __builtin_amdgcn_readfirstlane(nbytes);
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)boff);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(boff >> 32));
    boff = (int64_t)(((uint64_t)hi << 32) | lo);
  }
  // range resource over the chunk's rows of tensor X (loads past them read
  // zero, stores past them are dropped)
  __device__ __amdgpu_buffer_rsrc_t rsrc(const void* X) const {
    return range_rsrc((const char*)X + boff, (size_t)nbytes);
  }
};

}  // namespace

int carry8_chunks_per_head(int L, int C, int P) {
  const TileMap tm(L, C, 32);
  const int n_tiles = tm.count_tiles();
  int n = 0;
  for (int p = 0; p < P - 1; ++p) {
    int a0, a1;
    carry_seg_rows(tm, n_tiles, P, p, a0, a1);
    n += (a1 - a0 + kCarryRows - 1) / kCarryRows;
  }
  return n;
}

// DROP: value dropout on (its masks are generated only in that instantiation)
template <class G, bool DROP>
__global__ __launch_bounds__(512, 1) void carry8_kernel(CarryArgs a) {
  typedef bf16 T;
  typedef bf16x8 F;
  typedef WFragLayout<G> WL;
  constexpr int D = G::D, M = G::M, EB = G::EB, ET = G::ET;
  constexpr int CR = kCarryRows;
  constexpr int RT = CR / 16;         // 16-row tiles per chunk
  constexpr int MW = M / 8;           // features per wave
  constexpr int MT = MW / 16;         // 16-feature tiles per wave
  constexpr int KB = M / 32;          // 32-deep blocks over all features
  constexpr int NJ = 2 * ET * RT / 8; // output jobs per wave (tile x {dV, dk})
  constexpr int LDQ = D + 16;         // row tiles, swizzled (kSwzRows)
  constexpr int LDK = M + 16;         // [row][feature] tiles, swizzled (kSwzInter)
  constexpr int TQ = CR * LDQ, TK = CR * LDK;
  constexpr int SZ = M * (D + 1);
  constexpr int RB = D * (int)sizeof(T);  // bytes per row
  constexpr int CPR = RB / 16;            // 16-byte chunks per row
  constexpr int NSW = CR * CPR / 64;      // waves staging the rows of one tensor, a chunk per lane
  typedef SwzLane<LDQ, kSwzRows> OR;
  typedef SwzLane<LDK, kSwzInter> OK;
  static_assert(G::M == 128 || G::M == 256, "M/8 features per wave in 16-feature tiles");
  static_assert(MT == 1 || MT == 2, "one 32-deep feature block per wave");
  static_assert(NJ == 1 || NJ == 2, "dV and dk tiles shared evenly by the 8 waves");
  static_assert(2 * MT == G::MT, "a wave's features are half of a 4-wave slice");
  static_assert(NSW >= 1 && 2 * NSW <= 8 && (CR * CPR) % 64 == 0, "K and V rows staged by whole waves");

  __shared__ __attribute__((aligned(16))) T Kb[3 * TQ];
  __shared__ __attribute__((aligned(16))) T Vb[3 * TQ];
  __shared__ __attribute__((aligned(16))) float knb[3][CR];
  __shared__ __attribute__((aligned(16))) T Ktb[2 * TK];    // K~ [s][m]
  __shared__ __attribute__((aligned(16))) T Pkb[2 * TK];    // Pk [s][m]
  __shared__ __attribute__((aligned(16))) float rsb[2][CR * 8];  // [s][wave]: the waves' parts of rowsum(Pk[s])

  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = lane_id();
  const Lane L = this_lane();
  const OR oR(L);
  const OK oK(L);
  const int BH = a.B * a.H;
  const TileMap tm(a.L, a.C, 32);
  const int n_tiles = tm.count_tiles();

  // this workgroup's run of chunks [i0, i0 + n_run)
  const int64_t total = (int64_t)BH * a.nch_head;
  const int i0 = __builtin_amdgcn_readfirstlane((int)((int64_t)blockIdx.x * total / a.NWG));
  const int n_run = __builtin_amdgcn_readfirstlane((int)((int64_t)(blockIdx.x + 1) * total / a.NWG) - i0);

  auto seek = [&](int idx, bool valid) {
    ChunkPos c;
    c.head = idx / a.nch_head;
    int rem = idx - c.head * a.nch_head;
    c.p = 0;
    for (;;) {
      carry_seg_rows(tm, n_tiles, a.P, c.p, c.a0, c.a1);
      c.nk = (c.a1 - c.a0 + CR - 1) / CR;
      if (rem < c.nk || c.p == a.P - 2) break;
      rem -= c.nk;
      ++c.p;
    }
    c.k = rem;
    c.finish(a.L, RB, valid);
    return c;
  };
  auto advance = [&](ChunkPos& c, bool valid) {
    if (++c.k >= c.nk) {
      c.k = 0;
      for (int guard = 0; guard < a.P; ++guard) {
        if (++c.p == a.P - 1) {
          c.p = 0;
          ++c.head;
        }
        carry_seg_rows(tm, n_tiles, a.P, c.p, c.a0, c.a1);
        c.nk = (c.a1 - c.a0 + CR - 1) / CR;
        if (c.nk > 0) break;
      }
    }
    c.finish(a.L, RB, valid);
  };

  // W operand fragments (one table shared by every head)
  const __amdgpu_buffer_rsrc_t wrs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(a.Wfrag), (short)0, (int)(WL::TOTAL * 64 * sizeof(F)), 0x00020000);
  auto wfrag = [&](int idx) -> F {
    return __builtin_bit_cast(F, __builtin_amdgcn_raw_buffer_load_b128(wrs, lane * (int)sizeof(F), idx * 64 * (int)sizeof(F), 0));
  };

  // output jobs of this wave: job j = w NJ + jj is tile o = j / 2 (value
  // columns 16 eo, rows 16 so of the chunk), dV when j is even, dk when odd
  auto job_is_dk = [&](int jj) { return ((w * NJ + jj) & 1) != 0; };
  const int eo = ((w * NJ) >> 1) % ET, so = ((w * NJ) >> 1) / ET;  // the same tile for both jobs when NJ = 2
  auto job_tensor = [&](int jj) { return job_is_dk(jj) ? a.dK : a.dV; };
  // lane (g, c) of an output tile: row 16 so + c, columns 16 eo + 4 g + [0, 4)
  const int out_off = ((16 * so + L.c) * D + 16 * eo + 4 * L.g) * (int)sizeof(T);

  // row staging: waves [0, NSW) carry K, waves [NSW, 2 NSW) V, one 16-byte
  // chunk per lane; the other waves load nothing (an offset past any range)
  const bool stage_k = w < NSW, stage_v = w >= NSW && w < 2 * NSW;
  const int sch = (w % NSW) * 64 + lane, srow = sch / CPR, scc = sch % CPR;
  const int s_goff = stage_k || stage_v ? (srow * D + scc * 8) * (int)sizeof(T) : INT_MAX - 15;
  const int s_loff = srow * LDQ + 8 * (scc ^ ((srow >> 3) & 1));  // kSwzRows: chunk cc of row r at cc ^ sw(r) / 2
  uint4 stage;
  auto fetch_rows = [&](const ChunkPos& c) { stage = BufIO<16>::load<uint4>(c.rsrc(stage_k ? a.K : a.V), s_goff); };
  // value dropout: dropped value elements zeroed when staged (the chunk's
  // head and first row give their positions), their dV contributions dropped
  auto drop_of = [&](const ChunkPos& c) { return Drop{a.drop_seed, a.drop_t, a.C, (uint64_t)c.head}; };
  auto put_rows = [&](int buf, const ChunkPos& c) {
    if (DROP && stage_v) drop_chunk<T>(stage, drop_of(c), c.a0 + c.k * CR + srow, scc * 8);
    if (stage_k) {
      *(uint4*)(Kb + buf * TQ + s_loff) = stage;
      if (G::KIND == kFavor) {
        const bf16x8 e = __builtin_bit_cast(bf16x8, stage);
        float n2 = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) n2 += (float)e[i] * (float)e[i];
        n2 = sum_lane_group<CPR>(n2);
        if (scc == 0) knb[buf][srow] = n2;
      }
    } else if (stage_v) {
      *(uint4*)(Vb + buf * TQ + s_loff) = stage;
    }
  };

  F Wf[MT][EB];  // slot s = W[w MW + 16 mt + c][32 kb + kp(g, s)]: logits of this wave's features
  F Wc[KB];      // slot s = W[32 kb + kp(g, s)][16 eo + c]: dk of this wave's output tile
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int kb = 0; kb < EB; ++kb) Wf[mt][kb] = wfrag(WL::a(w >> 1, (w & 1) * MT + mt, kb));
#pragma unroll
  for (int kb = 0; kb < KB; ++kb) Wc[kb] = wfrag(WL::c(kb, eo));
  F ones;
#pragma unroll
  for (int i = 0; i < 8; ++i) ones[i] = (T)1.f;

  // G_end(p) of the current segment in the two operand layouts
  F GA[MT][EB];    // slot s = G[w MW + 16 mt + c][32 kb + kp(g, s)]: dK~ of this wave's features
  float gz[MT][4]; // G[w MW + 16 mt + 4 g + r][D]: the ones column
  F GB[KB];        // slot s = G[32 kb + kp(g, s)][16 eo + c]: dV of this wave's output tile
  float koff = 0.f;  // FAVOR+: the head's key shift in log2 units, plus log2(M)/2
  const float half_log2M = 0.5f * __log2f((float)M);
  auto load_g = [&](const ChunkPos& c) {
    const float* Ge = a.gend + ((size_t)c.head * a.P + c.p) * SZ;
    if (G::KIND == kFavor) koff = a.kshift[c.head] * kLog2e + half_log2M;
    // lane coordinates rebuilt here, so that no address of these rare loads
    // stays live across the loop
    const Lane Lg = fresh_lane();
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const float* gr = Ge + (w * MW + 16 * mt + Lg.c) * (D + 1);
#pragma unroll
      for (int kb = 0; kb < EB; ++kb)
#pragma unroll
        for (int s = 0; s < 8; ++s) GA[mt][kb][s] = (T)gr[32 * kb + kp(Lg.g, s)];
#pragma unroll
      for (int r = 0; r < 4; ++r) gz[mt][r] = Ge[(w * MW + 16 * mt + 4 * Lg.g + r) * (D + 1) + D];
    }
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int s = 0; s < 8; ++s) GB[kb][s] = (T)Ge[(32 * kb + kp(Lg.g, s)) * (D + 1) + 16 * eo + Lg.c];
  };

  f32x4 dWacc[MT][ET];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int et = 0; et < ET; ++et) dWacc[mt][et] = zero4();

  typedef T t4 __attribute__((ext_vector_type(4)));
  typedef BufIO<sizeof(t4)> IO;

  if (n_run > 0) {
    ChunkPos cur = seek(i0, true), c1 = cur, c2;
    advance(c1, n_run > 1);
    c2 = c1;
    advance(c2, n_run > 2);
    t4 pd[NJ];  // prior dV / dK entries of the current chunk's output tiles
    fetch_rows(cur);
    put_rows(0, cur);
    fetch_rows(c1);
#pragma unroll
    for (int jj = 0; jj < NJ; ++jj) pd[jj] = IO::template load<t4>(cur.rsrc(job_tensor(jj)), out_off);
    load_g(cur);
    int g_head = cur.head, g_p = cur.p;
    // vmcnt(0): G_end is complete before the loop, as after every reload, so
    // the loop never waits on it (nor on the output stores issued after it)
    __builtin_amdgcn_s_waitcnt(0x0F70);
    __syncthreads();

    int b0 = 0, b1 = 1, z = 0;  // row buffer of this chunk and of the next; K~/Pk buffer
    // low parts of the logits' W fragments (bf16 split of the float32 W),
    // read from the table for every chunk at the end of the one before,
    // ahead of that chunk's output stores and of the next chunk's loads, so
    // that waiting for them waits for nothing else
    F Wl[MT][EB];
    auto fetch_wl = [&]() {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int kb = 0; kb < EB; ++kb) Wl[mt][kb] = wfrag(WL::alo(w >> 1, (w & 1) * MT + mt, kb));
    };
    fetch_wl();
    for (int it = 0; it < n_run; ++it) {
      // rows of chunk it + 1 into their buffer, rows of chunk it + 2 into
      // registers
      put_rows(b1, c1);
      fetch_rows(c2);
      if (cur.head != g_head || cur.p != g_p) {
        load_g(cur);
        g_head = cur.head;
        g_p = cur.p;
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this branch's loads complete inside it
      }
      const T* Ks = Kb + b0 * TQ;
      const T* Vs = Vb + b0 * TQ;
      const float* kn = knb[b0];
      T* Kt = Ktb + z * TK;
      T* Pk = Pkb + z * TK;
      float* rs = rsb[z];

      // ---- this wave's features for every row of the chunk
      {
        // every operand read of the phase first (the fence keeps them ahead)
        F kf[RT][EB], vf[RT][EB];
        float knv[RT];
#pragma unroll
        for (int st = 0; st < RT; ++st) {
#pragma unroll
          for (int kb = 0; kb < EB; ++kb) {
            kf[st][kb] = sfrag_rm(oR, Ks, 16 * st, 32 * kb);
            vf[st][kb] = sfrag_rm(oR, Vs, 16 * st, 32 * kb);
          }
          knv[st] = kn[16 * st + L.c];
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int st = 0; st < RT; ++st) {
          // exponent offset of the column's key row, -|k|^2/2 included; rows
          // past the chunk: infinite (features exactly zero)
          const bool col_ok = 16 * st + L.c < cur.cnt;
          const float kc = (G::KIND == kFavor) ? (col_ok ? koff + 0.5f * kLog2e * knv[st] : INFINITY) : 0.f;
          f32x4 kt[MT], pk[MT];
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            // K~^T[m][s] and dK~^T[m][s] = G[m][D] + sum_e G[m][e] V[s][e]
            f32x4 x = zero4();
#pragma unroll
            for (int kb = 0; kb < EB; ++kb) x = mma(x, Wf[mt][kb], kf[st][kb]);
            if constexpr (kSplitW<T>) {
#pragma unroll
              for (int kb = 0; kb < EB; ++kb) x = mma(x, Wl[mt][kb], kf[st][kb]);
            }
            f32x4 dk = f32x4{gz[mt][0], gz[mt][1], gz[mt][2], gz[mt][3]};
#pragma unroll
            for (int kb = 0; kb < EB; ++kb) dk = mma(dk, GA[mt][kb], vf[st][kb]);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              if (G::KIND == kFavor) {
                kt[mt][r] = fast_exp2(x[r] * kLog2e - kc);
                pk[mt][r] = dk[r] * kt[mt][r];
              } else {
                kt[mt][r] = col_ok ? fmaxf(x[r], 0.f) + a.relu_eps : 0.f;
                pk[mt][r] = kt[mt][r] > a.relu_eps ? dk[r] : 0.f;
              }
            }
          }
          // rounded once: the LDS copies and the operand of the rowsum
          const F kfr = MT == 2 ? tile_pair_frag<T>(kt[0], kt[MT - 1]) : tile_half_frag<T>(kt[0]);
          const F pfr = MT == 2 ? tile_pair_frag<T>(pk[0], pk[MT - 1]) : tile_half_frag<T>(pk[0]);
          sstore_half_T(oK, Kt, frag_lo(kfr), w * MW, 16 * st);
          sstore_half_T(oK, Pk, frag_lo(pfr), w * MW, 16 * st);
          if (MT == 2) {
            sstore_half_T(oK, Kt, frag_hi(kfr), w * MW + 16, 16 * st);
            sstore_half_T(oK, Pk, frag_hi(pfr), w * MW + 16, 16 * st);
          }
          if (G::KIND == kFavor) {
            // this wave's part of rowsum(Pk[s]): every row of the product holds it
            const f32x4 rsum = mma(zero4(), ones, pfr);
            if (L.g == 0) rs[(16 * st + L.c) * 8 + w] = rsum[0];
          }
        }
        // dW[m][e] += sum_s Pk[s][m] K[s][e]: the wave reads back its own
        // Pk columns (LDS operations of one wave complete in order)
        F kT[ET];
#pragma unroll
        for (int et = 0; et < ET; ++et) kT[et] = sfrag_tr(oR, Ks, 0, 16 * et);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const F pf = sfrag_tr(oK, Pk, 0, w * MW + 16 * mt);
#pragma unroll
          for (int et = 0; et < ET; ++et) dWacc[mt][et] = mma(dWacc[mt][et], pf, kT[et]);
        }
      }
      __syncthreads();

      // ---- this wave's dV / dk tiles over all M features
      //   dV^T[e][s] = sum_m G[m][e] K~[s][m]
      //   dk^T[e][s] = sum_m W[m][e] Pk[s][m] - k[s][e] rowsum(Pk[s])
      {
        // the rowsum term of the dk tile (FAVOR+): the waves' parts of
        // rowsum(Pk[s]) and the key row's entries
        const bool has_dk = NJ == 2 || job_is_dk(0);
        f32x4 r0 = zero4(), r1 = zero4();
        bf16x4 kv = {};
        if (G::KIND == kFavor && has_dk) {
          const f32x4* rp = (const f32x4*)&rs[(16 * so + L.c) * 8];
          r0 = rp[0];
          r1 = rp[1];
          kv = *(const bf16x4*)(Ks + oR.a + 16 * so * LDQ + 16 * eo);
        }
        __builtin_amdgcn_sched_barrier(0);
        auto rowsum_term = [&]() {
          f32x4 kterm = zero4();
          if (G::KIND == kFavor && has_dk) {
            const float rsv = ((r0[0] + r0[1]) + (r0[2] + r0[3])) + ((r1[0] + r1[1]) + (r1[2] + r1[3]));
#pragma unroll
            for (int r = 0; r < 4; ++r) kterm[r] = -(float)kv[r] * rsv;
          }
          return kterm;
        };
        f32x4 acc[NJ];
        if constexpr (NJ == 2) {
          // both products of the tile, interleaved; every operand read is
          // issued before the first product (the fence keeps the compiler
          // from trading that for registers)
          F kfa[KB], pfa[KB];
#pragma unroll
          for (int kb = 0; kb < KB; ++kb) {
            kfa[kb] = sfrag_rm(oK, Kt, 16 * so, 32 * kb);
            pfa[kb] = sfrag_rm(oK, Pk, 16 * so, 32 * kb);
          }
          __builtin_amdgcn_sched_barrier(0);
          const f32x4 kterm = rowsum_term();
          acc[0] = zero4();
          acc[1] = kterm;
#pragma unroll
          for (int kb = 0; kb < KB; ++kb) {
            acc[0] = mma(acc[0], GB[kb], kfa[kb]);
            acc[1] = mma(acc[1], Wc[kb], pfa[kb]);
          }
        } else {
          const bool is_dk = job_is_dk(0);
          const T* Z = is_dk ? Pk : Kt;
          acc[0] = rowsum_term();
#pragma unroll
          for (int kb = 0; kb < KB; ++kb) acc[0] = mma(acc[0], is_dk ? Wc[kb] : GB[kb], sfrag_rm(oK, Z, 16 * so, 32 * kb));
        }
        // plus the prior outputs of this chunk (loaded a chunk ago); then
        // the same registers receive those of the next chunk
        fetch_wl();
#pragma unroll
        for (int jj = 0; jj < NJ; ++jj) {
          if (DROP && !job_is_dk(jj)) {
            const unsigned keep = drop_keep_bits<4>(drop_of(cur), cur.a0 + cur.k * CR + 16 * so + L.c, 16 * eo + 4 * L.g);
#pragma unroll
            for (int r = 0; r < 4; ++r) acc[jj][r] = (keep >> r) & 1u ? acc[jj][r] : 0.f;
          }
          t4 o;
#pragma unroll
          for (int r = 0; r < 4; ++r) o[r] = (T)((float)pd[jj][r] + acc[jj][r]);
          IO::store(o, cur.rsrc(job_tensor(jj)), out_off);
          pd[jj] = IO::template load<t4>(c1.rsrc(job_tensor(jj)), out_off);
        }
      }
      cur = c1;
      c1 = c2;
      advance(c2, it + 3 < n_run);
      b0 = b1;
      b1 = b1 == 2 ? 0 : b1 + 1;
      z ^= 1;
    }
  }

  // this workgroup's dW partial: slot B H P + blockIdx.x (after the walk's)
  const size_t slot = (size_t)BH * a.P + blockIdx.x;
  float* dwl = a.dW_part + slot * (size_t)M * D + (size_t)(w * MW + 4 * L.g) * D + L.c;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int et = 0; et < ET; ++et)
#pragma unroll
      for (int r = 0; r < 4; ++r) dwl[(16 * mt + r) * D + 16 * et] = dWacc[mt][et][r];
}

template <class G>
hipError_t launch_carry8(const CarryArgs& a, hipStream_t s) {
  if (a.P < 2 || a.NWG < 1) return hipSuccess;
  if (a.drop_t != 0) hipLaunchKernelGGL((carry8_kernel<G, true>), dim3(a.NWG), dim3(512), 0, s, a);
  else hipLaunchKernelGGL((carry8_kernel<G, false>), dim3(a.NWG), dim3(512), 0, s, a);
  return hipGetLastError();
}

#define SLIM_INST_CARRY8(T, D, FW, TR, KIND) \
  template hipError_t launch_carry8<Cfg<T, D, FW, TR, KIND>>(const CarryArgs&, hipStream_t);
SLIM_FOR_EACH_BF16_CONFIG(SLIM_INST_CARRY8)

}  // namespace slim
