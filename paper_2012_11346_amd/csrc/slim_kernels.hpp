// Kernel argument blocks and launcher declarations shared by the host API
// (slim_api.cpp) and the kernel translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace slim {

// Sets the calling thread's slim_last_error() text (cleared for SLIM_OK)
// and returns `status`.
int report(int status, const char* msg);

// Walk modes of the forward kernel
enum WalkMode {
  kWalkOutputs = 0,  // Y and the final state (forward sweep)
  kWalkSums = 1,     // keys only: the state each segment adds (segment sums)
};

struct FwdArgs {
  const void* Q;
  const void* K;
  const void* V;
  const float* W;
  const void* Wfrag;        // fragment-ordered W (WFragLayout)
  void* Y;                  // kWalkOutputs
  float* logD;              // kWalkOutputs: [B,H,L] row normalisers (slim_fwd's logD), or nullptr
  float* state_out;         // kWalkOutputs: [B,H,M,D+1] or nullptr (written by the last segment)
  float* kshift_out;        // kWalkOutputs: [B,H] or nullptr
  const float* seg_state;   // [B,H,seg_stride,M,D+1] state each segment starts from, or nullptr (zero)
  int seg_stride;           // states per head in seg_state
  int seg_step;             // segment p starts from state p * seg_step of its head
  const float* seg_shift;   // [B,H,seg_stride] key shift of seg_state (FAVOR+), same indexing
  const float* fixed_shift; // [B,H] key shift used throughout (no online rescaling), or nullptr
  float* seg_out;           // kWalkSums: [B,H,P,M,D+1]
  float* seg_shift_out;     // kWalkSums: [B,H,P]
  int B, H, L, C, P;
  float relu_eps;
  // value dropout (Drop): seed, keep threshold t (0: none), output scale 1 / (1 - p)
  uint64_t drop_seed;
  uint32_t drop_t;
  float drop_scale;
};

struct ScanArgs {
  const float* seg;        // [B,H,P,M,D+1] per-segment sums
  const float* seg_shift;  // [B,H,P] their key shifts (forward), or nullptr (common shift)
  const float* init;       // [B,H,M,D+1] state before the first segment, or nullptr (zero)
  const float* init_shift; // [B,H] key shift of init (forward) / of init relative to `shift` (backward)
  const float* shift;      // [B,H] common key shift (backward), or nullptr
  float* out;              // forward: [B,H,P,...] segment starts; backward: [B,H,P+1,...] boundaries
  float* out_shift;        // forward: [B,H,P]
  float* total;            // reverse scan: [B,H,M,D+1] scaled total, or nullptr
  int BH, P, SZ, favor;
  int step;                // reverse scan: out holds every step-th entry (P / step per head); 0 or 1: all
};

struct WfragArgs {
  const float* W;
  void* out;  // fragment-ordered W (WFragLayout), element type of the problem
};

struct FeatArgs {
  const void* X;
  const float* W;
  float* phi;
  float* shift;
  int B, H, L, role;
  float relu_eps;
};

struct BwdArgs {
  const void* Q;
  const void* K;
  const void* V;
  const void* dY;
  const void* Y;            // [B,H,L,d] the forward's output, or nullptr (recomputed); 8-wave walk only
  const float* logD;        // [B,H,L] the forward's row normalisers (with Y), or nullptr; 8-wave walk only
  const float* W;
  const void* Wfrag;        // fragment-ordered W (WFragLayout)
  const float* kshift;      // [B,H] key shift of every state below (FAVOR+)
  const float* bounds;      // [B,H,bound_stride,M,D+1] exact states at (sub-)segment boundaries
  int bound_stride, bound_step;  // segment p spans boundaries p * bound_step .. (p + 1) * bound_step
  const float* dstate_out;  // [B,H,M,D+1] cotangent of the final state (segment P-1 starts from it), or nullptr
  float* g_final;           // [B,H,P,M,D+1] cotangent each segment's walk ends with (P > 1), or nullptr
  const float* g_init;      // [B,H,P,M,D+1] cotangent after each segment, which its walk starts from
                            // (8-wave walk; then g_final, dstate_in and the carry are not used), or nullptr
  const float* init_shift;  // [B,H] key shift of the caller's initial state (scales dstate_in), or nullptr
  float* dstate_in;         // [B,H,M,D+1] state cotangent before the sequence (P == 1 only), or nullptr
  void* dQ;
  void* dK;
  void* dV;
  float* dW_part;           // [B,H,P,M,D] per-workgroup partial dW
  float* dW;                // [M,D] sum of the partials
  int B, H, L, C, P;
  float relu_eps;
  // value dropout (Drop): seed, keep threshold t (0: none), output scale 1 / (1 - p)
  uint64_t drop_seed;
  uint32_t drop_t;
  float drop_scale;
};

// Carried cotangent: adds the contribution of G_end(p) (the cotangent after
// segment p, from all later segments) to dK, dV and dW of segment p's rows.
struct CarryArgs {
  const void* K;
  const void* V;
  const void* Wfrag;
  const float* kshift;  // [B,H] (FAVOR+)
  const float* gend;    // [B,H,P,M,D+1] G_end(p)
  void* dK;             // in/out
  void* dV;             // in/out
  float* dW_part;       // [B,H,P,M,D] in/out, then (CS-1) x [B,H,P-1,M,D] written
  int B, H, L, C, P;
  int CS;  // workgroups (row parts) per segment (carry_kernel)
  int nch_head;  // 32-row chunks per head over segments 0 .. P-2 (carry8_kernel)
  int NWG;       // workgroups (carry8_kernel); dW_part slot B H P + i is workgroup i's
  float relu_eps;
  // value dropout (Drop): seed, keep threshold t (0: none), output scale 1 / (1 - p)
  uint64_t drop_seed;
  uint32_t drop_t;
  float drop_scale;
};

// Key sums of contiguous parts of each head (ksum_kernel): per part, the
// state it adds relative to a fixed key shift, or the largest key exponent.
enum KsumMode { kSumStates = 0, kSumMax = 1, kSumQuery = 2 };
struct KsumArgs {
  const void* K;       // keys (kSumQuery: the queries)
  const void* V;       // values (kSumQuery: dY)
  const void* Y;       // kSumQuery: the forward's Y
  const float* logD;   // kSumQuery: [B,H,L] the forward's row normalisers
  const float* W;
  const void* Wfrag;   // fragment-ordered W (WFragLayout)
  const float* shift;  // kSumStates, kSumQuery, FAVOR+: [B,H] key shift of the sums
  // kSumStates, FAVOR+, instead of `shift`: the key maxima of n_part_max
  // parts per head ([B,H,n_part_max], from kSumMax) and init_shift ([B,H] or
  // nullptr); the shift is their largest, written to shift_out by part 0
  const float* part_max;
  const float* init_shift;
  float* shift_out;
  int n_part_max;
  float* out;          // kSumStates, kSumQuery: [B,H,P2,M,D+1]; kSumMax: [B,H,P2]
  int B, H, L, C, P2;
  int tile_begin, tile_end;  // the parts cover tiles [tile_begin, tile_end) of each head (0, 0: all)
  int align;                 // > 0: parts start at multiples of `align` tiles from tile_begin (slices)
  float relu_eps;
  // value dropout (Drop): seed, keep threshold t (0: none), output scale 1 / (1 - p)
  uint64_t drop_seed;
  uint32_t drop_t;
  float drop_scale;
};

// In-slice masked quadratic form (the slice evaluated as a whole, Sec. 3.2
// with eq. 2 inside the slice): slices are processed one after another,
// the query (or key) tiles of a slice in parallel.
struct QuadArgs {
  const void* Q;
  const void* K;
  const void* V;
  const void* dY;
  const void* Wfrag;      // fragment-ordered W (WFragLayout), with the low parts
  const float* kshift;    // [B,H] key shift (FAVOR+)
  const float* S;         // [B,H,M,D+1] state before the slice (relative to kshift)
  const void* Sfrag;      // its fragment tables (StateFragLayout), backward query pass
  const float* Gc;        // [B,H,M,D+1] state cotangent after the slice (backward key pass)
  const void* Gfrag;      // its fragment tables
  void* Y;                // forward: out [B,H,L,D]
  float* DN;              // backward: [B,H,C,D+4] per row of the slice: dN[0,D), dD, the query row shift
  void* dQ;
  void* dK;
  void* dV;
  float* dW_part;         // [B,H,gridDim.x][M,D] partial dW per workgroup, accumulated (+=)
  float* out;             // cotangent sums: [B,H,gridDim.x][M,D+1] per part
  int B, H, L, C;
  int row0, rows;         // the slice: rows [row0, row0 + rows)
  float relu_eps;
  uint64_t drop_seed;
  uint32_t drop_t;
  float drop_scale;
};

// Sum of per-part states: out = f * in + sign * sum_p part[p] per head, with
// f = exp(in_shift - shift) when both shifts are given (FAVOR+), else 1;
// in may be nullptr (zero); head h of `in` starts at in + h * in_stride,
// of `out` at out + h * SZ, its parts at part + (h * P2 + p) * SZ.
hipError_t launch_state_combine(const float* in, size_t in_stride, const float* in_shift, const float* shift,
                                const float* part, int P2, float sign, float* out, int BH, int SZ, hipStream_t s);
template <class G>
hipError_t launch_quad_fwd(const QuadArgs& a, int nwg, hipStream_t s);
// backward of one slice: the query pass (dN, dD, dQ, dW), the key pass
// (dK, dV, dW), the sum of Q~^T [dN|dD] over the slice in nwg parts
template <class G>
hipError_t launch_quad_dq(const QuadArgs& a, int nwg, hipStream_t s);
template <class G>
hipError_t launch_quad_dk(const QuadArgs& a, int nwg, hipStream_t s);
template <class G>
hipError_t launch_quad_gsum(const QuadArgs& a, int nwg, hipStream_t s);
// fragment tables of n states [BH][M][D+1] (n = 1 or 2: X0 -> F0, X1 -> F1)
template <class G>
hipError_t launch_state_frag(const float* X0, void* F0, const float* X1, void* F1, int BH, hipStream_t s);
template <class G>
size_t state_frag_bytes();

template <class G>
hipError_t launch_fwd_walk(const FwdArgs& a, int mode, hipStream_t s);
template <class G>
hipError_t launch_ksum(const KsumArgs& a, int mode, hipStream_t s);
// kshift[h] = max(init_shift[h] (if given), max_p part_max[h][p])
hipError_t launch_kshift_reduce(const float* part_max, int P2, const float* init_shift, float* kshift, int BH,
                                hipStream_t s);
// exclusive scan of segment states (forward: with key-shift rescaling)
hipError_t launch_scan_fwd(const ScanArgs& a, hipStream_t s);
// inclusive boundaries of segment states under one common shift (backward)
hipError_t launch_scan_bwd(const ScanArgs& a, hipStream_t s);
// reverse scan of state cotangents: out[p] = init + sum_{q > p} seg[q]; with
// `total` also total = r0 (init + sum_q seg[q]), r0 = exp(init_shift - shift)
// (FAVOR+, when init_shift is given) else 1
hipError_t launch_scan_rev(const ScanArgs& a, hipStream_t s);
template <class G>
hipError_t launch_featmap(const FeatArgs& a, hipStream_t s);
template <class G>
hipError_t launch_wfrag(const WfragArgs& a, hipStream_t s);
template <class G>
size_t wfrag_bytes();
template <class G>
hipError_t launch_bwd_walk(const BwdArgs& a, hipStream_t s);
// the same walk with 8 waves per workgroup (two per feature slice); bf16
// problems with 32 or 64 features per slice
template <class G>
hipError_t launch_bwd_walk8(const BwdArgs& a, hipStream_t s);
template <class G>
hipError_t launch_carry(const CarryArgs& a, hipStream_t s);
// the same pass with 8 waves and a balanced run of 32-row chunks per
// workgroup; bf16 problems with 32 or 64 features per 4-wave slice
template <class G>
hipError_t launch_carry8(const CarryArgs& a, hipStream_t s);
int carry8_chunks_per_head(int L, int C, int P);
// dW = sum of the n_parts partials [n_parts][n], in a fixed order
hipError_t launch_dw_reduce(const float* part, int n_parts, int n, float* dW, hipStream_t s);

// every compiled (element type, head dim, features per wave, tile rows, kind);
// fp32 problems serve exactness checks and are compiled for d * M <= 4096;
// the square map is compiled for M = 64 (16 features per wave)
#define SLIM_FOR_EACH_CONFIG(X)                                                           \
  X(bf16, 64, 64, 32, kFavor) X(bf16, 64, 32, 32, kFavor) X(bf16, 64, 16, 32, kFavor) \
  X(bf16, 32, 64, 32, kFavor) X(bf16, 32, 32, 32, kFavor) X(bf16, 32, 16, 32, kFavor) \
  X(bf16, 64, 64, 32, kRelu) X(bf16, 64, 32, 32, kRelu) X(bf16, 64, 16, 32, kRelu)    \
  X(bf16, 32, 64, 32, kRelu) X(bf16, 32, 32, 32, kRelu) X(bf16, 32, 16, 32, kRelu)    \
  X(float, 64, 16, 32, kFavor) X(float, 32, 32, 32, kFavor) X(float, 32, 16, 32, kFavor) \
  X(float, 64, 16, 32, kRelu) X(float, 32, 32, 32, kRelu) X(float, 32, 16, 32, kRelu)    \
  X(bf16, 64, 16, 32, kSquare) X(bf16, 32, 16, 32, kSquare)                               \
  X(float, 64, 16, 32, kSquare) X(float, 32, 16, 32, kSquare)

// Explicit prefix-sum within-slice mode (slim_ps.hip): the states of every
// row of a slice written out, then used; streaming kernels for any
// configuration.  Launch selector `which`:
enum PsKernel {
  kPsKmax = 0,   // part[head][wg]: largest key exponent of the rows a workgroup visits
  kPsTerms = 1,  // U[head][i] = g(k)^T [v | 1] for the slice's rows
  kPsScan0 = 2,  // prefix sums of U from S_in (or zero); S_out = the last
  kPsScan1 = 3,  // S_out = S_in - sum U (eq. 17), then prefix sums from it
  kPsScan2 = 4,  // S_out = S_in (exact), then prefix sums from it
  kPsOut = 5,    // Y of the slice's rows from U
  kPsGq = 6,     // dq, dW (queries), query terms g(q) [dN | dD] -> Gh
  kPsRscan = 7,  // reverse prefix sums of Gh from G_in (or zero); G_out = the first
  kPsGk = 8,     // dk, dv, dW (keys) from Gh
  kPsSum = 9     // part[head][r][m][e]: what the rows of slices [r NS / P2, (r + 1) NS / P2) add
};
struct PsArgs {
  const void* Q;
  const void* K;
  const void* V;
  const void* dY;
  const float* W;       // [M, d]
  const float* kshift;  // [B H] FAVOR+ key shift
  void* Y;
  void* dQ;
  void* dK;
  void* dV;
  float* U;             // [B H][C][d + 1][M] the slice's states (or its rows' terms)
  float* Gh;            // [B H][C][d + 1][M] query terms, then the states' cotangents
  const float* S_in;    // state of head h at S_in + h in_stride ([m][d + 1])
  size_t in_stride;
  float* S_out;         // [B H][M][d + 1]
  const float* G_in;    // [B H][M][d + 1] cotangent after the slice, or nullptr (zero)
  float* G_out;         // [B H][M][d + 1] cotangent before the slice
  float* part;          // kPsKmax: [B H][workgroups]; kPsSum: [B H][P2][M][d + 1]
  float* dW_part;       // [B H][nslot][M][d], added to (workgroup w of head h: slot h nslot + w)
  int nslot;
  int B, H, L, d, M, C;  // C: rows of U and Gh per head (the longest slice)
  int row0, rows;        // the slice
  int kind;              // Kind
  float relu_eps;
  int bf16;              // element type of Q, K, V, dY, Y, dQ, dK, dV: bf16 (1) or float (0)
};
// grid (nwg, B H); extra: kPsSum's slice count
hipError_t launch_ps(int which, const PsArgs& a, int nwg, int extra, hipStream_t s);

// configurations of the whole-slice quadratic form (bf16, 32 or 64 features
// per wave)
#define SLIM_FOR_EACH_QUAD_CONFIG(X)                                                  \
  X(bf16, 64, 64, 32, kFavor) X(bf16, 64, 32, 32, kFavor) X(bf16, 32, 64, 32, kFavor) \
  X(bf16, 32, 32, 32, kFavor) X(bf16, 64, 64, 32, kRelu) X(bf16, 64, 32, 32, kRelu)  \
  X(bf16, 32, 64, 32, kRelu) X(bf16, 32, 32, 32, kRelu)

// configurations served by the 8-wave backward walk
#define SLIM_FOR_EACH_BF16_CONFIG(X)                                                  \
  X(bf16, 64, 64, 32, kFavor) X(bf16, 64, 32, 32, kFavor) X(bf16, 32, 64, 32, kFavor) \
  X(bf16, 32, 32, 32, kFavor) X(bf16, 64, 64, 32, kRelu) X(bf16, 64, 32, 32, kRelu)  \
  X(bf16, 32, 64, 32, kRelu) X(bf16, 32, 32, 32, kRelu)

}  // namespace slim
