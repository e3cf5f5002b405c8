// Host side of the C ABI declared in include/slim.h: argument validation,
// workspace layout, segment planning and kernel dispatch.
#include <hip/hip_runtime.h>

#include <climits>
#include <cstdint>
#include <initializer_list>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <mutex>
#include <string>

#include "../../include/slim.h"
#include "slim_common.hpp"
#include "slim_kernels.hpp"

namespace {

thread_local std::string g_last_error;

// events set by slim_time_walk, per phase; consumed by the next call
struct WalkTimer {
  hipEvent_t before = nullptr, after = nullptr;
};
thread_local WalkTimer g_timer[2];

// launch `run` between the phase's timing events, if any were set
template <class F>
hipError_t timed_launch(int phase, hipStream_t s, F run) {
  WalkTimer t = g_timer[phase];
  g_timer[phase] = WalkTimer();
  hipError_t e = hipSuccess;
  if (t.before != nullptr && (e = hipEventRecord(t.before, s)) != hipSuccess) return e;
  e = run();
  if (e != hipSuccess) return e;
  if (t.after != nullptr) e = hipEventRecord(t.after, s);
  return e;
}

int fail(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return status;
}

int ok() {
  g_last_error.clear();
  return SLIM_OK;
}

}  // namespace

// error reporting shared with the other entry points of the library
int slim::report(int status, const char* msg) {
  if (status == SLIM_OK) g_last_error.clear();
  else g_last_error = msg;
  return status;
}

namespace {

int hip_fail(hipError_t e, const char* what) {
  return fail(SLIM_EHIP, "%s: %s", what, hipGetErrorString(e));
}

constexpr int kTileRows = 32;

int check_problem(const slim_problem* p) {
  if (p == nullptr) return fail(SLIM_EINVAL, "problem is NULL");
  if (p->B < 1 || p->H < 1 || p->L < 1) return fail(SLIM_EINVAL, "B, H, L must be >= 1");
  if (p->C < 1) return fail(SLIM_EINVAL, "slice length C must be >= 1 (got %d)", (int)p->C);
  if (p->dtype != SLIM_F32 && p->dtype != SLIM_BF16) return fail(SLIM_EINVAL, "unknown dtype %d", (int)p->dtype);
  if (p->kind != SLIM_FAVOR_PLUS && p->kind != SLIM_RELU && p->kind != SLIM_SQUARE)
    return fail(SLIM_EINVAL, "unknown kind %d", (int)p->kind);
  if (p->d != 32 && p->d != 64) return fail(SLIM_EUNSUPPORTED, "head dim d=%d not supported (32 or 64)", (int)p->d);
  if (p->M != 64 && p->M != 128 && p->M != 256)
    return fail(SLIM_EUNSUPPORTED, "feature count M=%d not supported (64, 128 or 256)", (int)p->M);
  if (p->L > (int64_t)INT_MAX / 2) return fail(SLIM_EUNSUPPORTED, "L=%lld too long", (long long)p->L);
  // one head's rows are addressed with 32-bit byte offsets (range-checked buffer accesses)
  if (p->L * p->d * (p->dtype == SLIM_F32 ? 4 : 2) > ((int64_t)1 << 30))
    return fail(SLIM_EUNSUPPORTED, "L=%lld too long: one head's rows must fit in 1 GiB", (long long)p->L);
  if (p->B * p->H > 65535) return fail(SLIM_EUNSUPPORTED, "B*H=%lld too large", (long long)(p->B * p->H));
  if (p->B > 65535 || p->H > 65535) return fail(SLIM_EUNSUPPORTED, "B or H above 65535");
  if (p->kind == SLIM_RELU && !(p->relu_eps > 0.f)) return fail(SLIM_EINVAL, "relu_eps must be > 0");
  if (p->kind == SLIM_SQUARE && p->M != 64)
    return fail(SLIM_EUNSUPPORTED, "the square map is built for M=64 (got M=%d)", (int)p->M);
  if (!(p->dropout >= 0.f && p->dropout < 1.f)) return fail(SLIM_EINVAL, "dropout must be in [0, 1)");
  if (p->within != SLIM_WITHIN_ITER && p->within != SLIM_WITHIN_QUADRATIC && p->within != SLIM_WITHIN_PS)
    return fail(SLIM_EINVAL, "unknown within-slice mode %d", (int)p->within);
  if (p->dtype == SLIM_F32 && (int64_t)p->d * p->M > 4096 && p->within != SLIM_WITHIN_PS)
    return fail(SLIM_EUNSUPPORTED, "fp32 problems need d*M <= 4096 (got d=%d, M=%d) outside the PS mode", (int)p->d,
                (int)p->M);
  if (p->within == SLIM_WITHIN_PS && p->dropout != 0.f)
    return fail(SLIM_EUNSUPPORTED, "the PS within-slice mode has no dropout");
  if (p->reserved != 0) return fail(SLIM_EINVAL, "reserved field must be 0");
  if (p->within == SLIM_WITHIN_QUADRATIC &&
      (p->dtype != SLIM_BF16 || (p->M != 128 && p->M != 256) || p->kind == SLIM_SQUARE))
    return fail(SLIM_EUNSUPPORTED, "the quadratic within-slice mode is built for bf16, M=128 or 256, FAVOR+ or ReLU");
  return SLIM_OK;
}

bool quad(const slim_problem* p) { return p->within == SLIM_WITHIN_QUADRATIC; }
bool ps(const slim_problem* p) { return p->within == SLIM_WITHIN_PS; }

// value dropout parameters of the kernels: keep threshold t = round(p 65536)
// on 16-bit fields (0: nothing dropped) and the output scale 1 / (1 - p)
struct DropPlan {
  uint64_t seed;
  uint32_t t;
  float scale;
};
DropPlan drop_plan(const slim_problem* p) {
  const double q = p->dropout;
  return DropPlan{p->seed, (uint32_t)std::lround(q * 65536.0), (float)(1.0 / (1.0 - q))};
}
template <class A>
void set_drop(A& a, const DropPlan& d) {
  a.drop_seed = d.seed;
  a.drop_t = d.t;
  a.drop_scale = d.scale;
}

bool misaligned(const void* ptr, size_t a) { return ptr != nullptr && ((uintptr_t)ptr & (a - 1)) != 0; }

int check_alignment(std::initializer_list<const void*> rows, std::initializer_list<const void*> words) {
  for (const void* q : rows)
    if (misaligned(q, 16)) return fail(SLIM_EINVAL, "row tensors and the workspace must be 16-byte aligned");
  for (const void* q : words)
    if (misaligned(q, 4)) return fail(SLIM_EINVAL, "float tensors must be 4-byte aligned");
  return SLIM_OK;
}

int clamp_C(const slim_problem* p) { return (int)(p->C > p->L ? p->L : p->C); }

// Workgroups per device the segment plans aim for: the reverse walk runs one
// workgroup per compute unit (256 CUs), the forward-family walks two.
constexpr int kTargetWorkgroups = 256;
constexpr int kTargetWorkgroupsForward = 512;
// Segments shorter than this many tiles are not worth their start-up cost.
constexpr int kMinTilesPerSegment = 4;

int count_tiles(const slim_problem* p) {
  return slim::TileMap((int)p->L, clamp_C(p), kTileRows).count_tiles();
}

// Segments per head.  The walk inside a segment is sequential; segments run
// in parallel and are stitched together by exact scans of their states.  The
// count depends on B*H and the device size, not on L once L is long enough,
// so workspace stays flat in L.  It is rounded down, so that the workgroups
// are all resident on the device at once.  SLIM_SEGMENTS (debugging) forces a count.
int plan_segments_for(const slim_problem* p, int target) {
  const int n_tiles = count_tiles(p);
  const char* env = getenv("SLIM_SEGMENTS");
  if (env != nullptr && atoi(env) > 0) return std::max(1, std::min(atoi(env), n_tiles));
  const int64_t heads = p->B * p->H;
  int P = (int)std::min<int64_t>(target / heads, 1 << 20);
  P = std::min(P, std::max(1, n_tiles / kMinTilesPerSegment));
  return std::max(1, P);
}
bool has_ksum(const slim_problem* p);
size_t state_elems(const slim_problem* p) { return (size_t)p->M * (size_t)(p->d + 1); }
// segments of the backward (and of slim_num_segments)
int plan_segments(const slim_problem* p) { return plan_segments_for(p, kTargetWorkgroups); }

// Boundary states of the parts (one state of M (d + 1) floats per part and
// head) are the exact restarts of the reverse walk's downdates (eq. 17): a
// part's downdates start from the exact state at its end, so rounding never
// accumulates over more than one part.  Parts are made as short as this
// budget over all heads allows (one tile each for short sequences, where no
// downdate runs at all); beyond it their number per head stays fixed, so
// memory stays flat in L.
constexpr size_t kBoundaryBudgetBytes = (size_t)32 << 20;

// Parts per backward segment: the key sums are associative and the pass fits
// two workgroups per compute unit, so each segment's sum is split in two
// when that leaves enough tiles per part; and into more parts, down to one
// tile each, while the boundary states fit kBoundaryBudgetBytes.  Parts
// hold at least one tile.  SLIM_SUM_SPLIT (debugging) forces a count.
int plan_sum_split(const slim_problem* p, int P) {
  const char* env = getenv("SLIM_SUM_SPLIT");
  const int n_tiles = count_tiles(p);
  const int most = std::max(1, n_tiles / P);  // parts of at least one tile
  if (env != nullptr && atoi(env) >= 1) return std::min(atoi(env), most);
  int s2;
  if (has_ksum(p)) {
    s2 = 2 * P <= std::max(1, n_tiles / kMinTilesPerSegment) ? 2 : 1;
  } else {
    const int64_t wgs = p->B * p->H * (int64_t)P;
    s2 = (n_tiles >= 4 * P && 2 * wgs <= kTargetWorkgroupsForward) ? 2 : 1;
  }
  const size_t per_part = (size_t)p->B * p->H * state_elems(p) * sizeof(float);
  const int64_t budget_parts = (int64_t)(kBoundaryBudgetBytes / per_part);  // per head, over all segments
  return std::max(s2, (int)std::min<int64_t>(most, budget_parts / P));
}

// Segments of the forward.  Problems on the key-sum kernel walk one segment
// per part of the backward (two workgroups per compute unit), so that the
// boundary states serve both passes; the others aim for twice the
// backward's workgroups on their own.
int plan_fwd_segments(const slim_problem* p) {
  if (has_ksum(p)) {
    const int P = plan_segments(p);
    return P * plan_sum_split(p, P);
  }
  return plan_segments_for(p, kTargetWorkgroupsForward);
}

// Row parts per segment of the carry pass (several segments): enough
// workgroups to give two per compute unit, at least one tile per part.
// SLIM_CARRY_SPLIT (debugging) forces a count from 1 to 4.
int plan_carry_split(const slim_problem* p, int P) {
  if (P < 2) return 1;
  const int per_seg = count_tiles(p) / P;
  const int64_t wgs = p->B * p->H * (int64_t)(P - 1);
  const char* env = getenv("SLIM_CARRY_SPLIT");
  int cs = (env != nullptr && atoi(env) >= 1 && atoi(env) <= 4) ? atoi(env)
                                                                : (int)std::max<int64_t>(1, std::min<int64_t>(4, kTargetWorkgroupsForward / wgs));
  return std::max(1, std::min(cs, per_seg));
}

// Parts of the backward's segment boundaries: P segments, each split in S2.
int bwd_parts(const slim_problem* p) {
  const int P = plan_segments(p);
  return P * plan_sum_split(p, P);
}
// The forward hands its boundary states to the backward (slim_context_bytes)
// when it computes them with one key shift per head (the key-sum kernel):
// then its segments are the backward's parts.
bool context_used(const slim_problem* p) { return !quad(p) && !ps(p) && has_ksum(p) && plan_fwd_segments(p) > 1; }

// Parts of the forward's boundaries on the one-shift path
int fwd_parts(const slim_problem* p) { return plan_fwd_segments(p); }

size_t align256(size_t n) { return (n + 255) & ~(size_t)255; }

size_t wfrag_bytes_of(const slim_problem* p);

// forward workspace: W in fragment order (bf16 problems), segment sums and
// shifts, segment starts and shifts
struct FwdLayout {
  size_t wfrag, seg_sum, seg_shift, starts, start_shift, total;
};
FwdLayout fwd_layout(const slim_problem* p, int P) {
  FwdLayout l{0, 0, 0, 0, 0, 0};
  size_t off = 0;
  if (p->dtype == SLIM_BF16) {
    l.wfrag = off;
    off += align256(wfrag_bytes_of(p));
  }
  if (P <= 1) {
    l.total = off;
    return l;
  }
  const size_t n = (size_t)p->B * p->H * (has_ksum(p) ? P : P * plan_sum_split(p, P));
  l.seg_sum = off;
  off += align256(n * state_elems(p) * sizeof(float));
  l.seg_shift = off;
  off += align256(n * sizeof(float));
  l.starts = off;  // segment starts, or the P2 + 1 boundaries of each head (fixed key shift)
  off += align256((n + (size_t)p->B * p->H) * state_elems(p) * sizeof(float));
  l.start_shift = off;
  off += align256(n * sizeof(float));
  l.total = off;
  return l;
}

// backward workspace: W in fragment order, segment sums, segment
// boundaries, the cotangent each segment's walk ends with and the cotangent
// after each segment (several segments), dW partials
struct BwdLayout {
  size_t wfrag, seg_sum, bounds, gc, gend, dw_part, total;
};
size_t wfrag_bytes_of(const slim_problem* p);
bool has_carry8(const slim_problem* p);
// Workgroups of the 8-wave carry pass: one per compute unit, or one per
// chunk when there are fewer chunks.  SLIM_CARRY_WORKGROUPS (debugging)
// forces a smaller count, so that each workgroup's run crosses segments and
// heads.
int carry8_workgroups(const slim_problem* p, int P) {
  if (P < 2) return 0;
  const int64_t chunks = p->B * p->H * (int64_t)slim::carry8_chunks_per_head((int)p->L, clamp_C(p), P);
  int64_t n = std::min<int64_t>(kTargetWorkgroups, chunks);
  const char* env = getenv("SLIM_CARRY_WORKGROUPS");
  if (env != nullptr && atoi(env) >= 1) n = std::min<int64_t>(n, atoi(env));
  return (int)n;
}
// dW partials: one per (head, segment) from the walk, then the carry's
size_t dw_slots(const slim_problem* p, int P) {
  const size_t heads = (size_t)p->B * p->H;
  if (has_carry8(p)) return heads * P + carry8_workgroups(p, P);
  return heads * P + (P > 1 ? heads * (P - 1) * (plan_carry_split(p, P) - 1) : 0);
}
BwdLayout bwd_layout(const slim_problem* p, int P) {
  BwdLayout l{0, 0, 0, 0, 0, 0, 0};
  const size_t heads = (size_t)p->B * p->H;
  const size_t se = state_elems(p) * sizeof(float);
  size_t off = 0;
  l.wfrag = off;
  off += align256(wfrag_bytes_of(p));
  const int P2 = P * plan_sum_split(p, P);
  l.seg_sum = off;
  off += align256(heads * P2 * se);
  l.bounds = off;
  off += align256(heads * (P2 + 1) * se);
  if (P > 1) {
    l.gc = off;
    off += align256(heads * P * se);
    l.gend = off;
    off += align256(heads * P * se);
  }
  l.dw_part = off;  // the walk's B H P partials, then the carry's extra row parts
  off += align256(dw_slots(p, P) * (size_t)p->M * p->d * sizeof(float));
  l.total = off;
  return l;
}

// ---- the quadratic within-slice mode: slices one after another, the 32-row
// tiles of a slice in parallel
int quad_slices(const slim_problem* p) { return (int)((p->L + clamp_C(p) - 1) / clamp_C(p)); }
int quad_tiles(const slim_problem* p) { return (clamp_C(p) + kTileRows - 1) / kTileRows; }
// workgroups per head of the per-slice passes: one per query (key) tile, up
// to about eight per compute unit over all heads.  SLIM_QUAD_WORKGROUPS
// (debugging) forces fewer, so that workgroups take several tiles.
int quad_workgroups(const slim_problem* p) {
  int64_t n = std::min<int64_t>(quad_tiles(p), 2048 / (p->B * p->H));
  const char* env = getenv("SLIM_QUAD_WORKGROUPS");
  if (env != nullptr && atoi(env) > 0) n = std::min<int64_t>(n, atoi(env));
  return (int)std::max<int64_t>(1, n);
}
// parts of the per-slice key sums, and of the key maxima over the whole head
int quad_sum_parts(const slim_problem* p) {
  return (int)std::max<int64_t>(1, std::min<int64_t>((quad_tiles(p) + 3) / 4, kTargetWorkgroupsForward / (p->B * p->H)));
}
int quad_max_parts(const slim_problem* p) {
  return (int)std::max<int64_t>(1, std::min<int64_t>(std::max(1, count_tiles(p) / 4), kTargetWorkgroupsForward / (p->B * p->H)));
}
// states at exact restarts of the backward's downdates: the slices are cut
// into this many runs, and each run's downdates start from an exact state
int quad_runs(const slim_problem* p) {
  const char* env = getenv("SLIM_QUAD_RUNS");
  if (env != nullptr && atoi(env) > 0) return std::min(atoi(env), quad_slices(p));
  return std::min(quad_slices(p), 16);
}

struct QuadFwdLayout {
  size_t wfrag, kmax, sa, sb, parts, total;
};
QuadFwdLayout quad_fwd_layout(const slim_problem* p) {
  QuadFwdLayout l{0, 0, 0, 0, 0, 0};
  const size_t heads = (size_t)p->B * p->H, se = state_elems(p) * sizeof(float);
  size_t off = 0;
  l.wfrag = off;
  off += align256(wfrag_bytes_of(p));
  l.kmax = off;
  off += align256(heads * quad_max_parts(p) * sizeof(float));
  l.sa = off;
  off += align256(heads * se);
  l.sb = off;
  off += align256(heads * se);
  l.parts = off;
  off += align256(heads * quad_sum_parts(p) * se);
  l.total = off;
  return l;
}

// workgroups per head of the backward passes (each holds a dW partial)
int quad_bwd_workgroups(const slim_problem* p) {
  return std::min(quad_workgroups(p), (int)std::max<int64_t>(1, 1024 / (p->B * p->H)));
}
size_t state_frag_bytes_of(const slim_problem* p);
// backward workspace: W in fragment order; the run sums and the exact
// states at the run boundaries; states and cotangents (two each, used in
// turn); per-slice parts; fragment tables of the state and the cotangent;
// the query pass's rows [dN|dD|shift]; the dW partials
struct QuadBwdLayout {
  size_t wfrag, seg, bounds, s[2], g[2], parts, sfrag, gfrag, dn, dw_part, total;
};
QuadBwdLayout quad_bwd_layout(const slim_problem* p) {
  QuadBwdLayout l;
  std::memset(&l, 0, sizeof(l));
  const size_t heads = (size_t)p->B * p->H, se = state_elems(p) * sizeof(float);
  const int R = quad_runs(p);
  size_t off = 0;
  auto take = [&](size_t& at, size_t n) {
    at = off;
    off += align256(n);
  };
  take(l.wfrag, wfrag_bytes_of(p));
  take(l.seg, heads * R * se);
  take(l.bounds, heads * (R + 1) * se);
  take(l.s[0], heads * se);
  take(l.s[1], heads * se);
  take(l.g[0], heads * se);
  take(l.g[1], heads * se);
  take(l.parts, heads * std::max(quad_sum_parts(p), 1) * se);
  take(l.sfrag, heads * state_frag_bytes_of(p));
  take(l.gfrag, heads * state_frag_bytes_of(p));
  take(l.dn, heads * (size_t)clamp_C(p) * (p->d + 4) * sizeof(float));
  take(l.dw_part, heads * quad_bwd_workgroups(p) * (size_t)p->M * p->d * sizeof(float));
  l.total = off;
  return l;
}

typedef hipError_t (*fwd_fn)(const slim::FwdArgs&, int, hipStream_t);
typedef hipError_t (*feat_fn)(const slim::FeatArgs&, hipStream_t);
typedef hipError_t (*bwd_fn)(const slim::BwdArgs&, hipStream_t);
typedef hipError_t (*wfrag_fn)(const slim::WfragArgs&, hipStream_t);
typedef size_t (*size_fn)();
typedef hipError_t (*carry_fn)(const slim::CarryArgs&, hipStream_t);
typedef hipError_t (*ksum_fn)(const slim::KsumArgs&, int, hipStream_t);
typedef hipError_t (*quad_fn)(const slim::QuadArgs&, int, hipStream_t);
typedef hipError_t (*sfrag_fn)(const float*, void*, const float*, void*, int, hipStream_t);

struct Dispatch {
  fwd_fn fwd;
  feat_fn feat;
  bwd_fn bwd4;  // backward walk, 4 waves per workgroup
  bwd_fn bwd8;  // backward walk, 8 waves per workgroup (nullptr where not built)
  wfrag_fn wfrag;
  size_fn wfrag_bytes;
  carry_fn carry;
  carry_fn carry8;  // 8-wave carry pass (nullptr where not built)
  ksum_fn ksum;  // key sums of row ranges (nullptr where not built: the key-only walk serves)
  quad_fn quad_fwd;  // quadratic within-slice mode (nullptr where not built)
  quad_fn quad_dq, quad_dk, quad_gsum;
  sfrag_fn state_frag;
  size_fn state_frag_bytes;
};

template <class T, int D, int FW, int KIND>
Dispatch make_dispatch() {
  typedef slim::Cfg<T, D, FW, kTileRows, KIND> G;
  return Dispatch{&slim::launch_fwd_walk<G>, &slim::launch_featmap<G>, &slim::launch_bwd_walk<G>, nullptr,
                  &slim::launch_wfrag<G>,    &slim::wfrag_bytes<G>,     &slim::launch_carry<G>,    nullptr,
                  nullptr,                   nullptr,                   nullptr,
                  nullptr,                   nullptr,                   nullptr,
                  nullptr};
}
template <int D, int FW, int KIND>
Dispatch make_dispatch8() {
  Dispatch d = make_dispatch<slim::bf16, D, FW, KIND>();
  d.bwd8 = &slim::launch_bwd_walk8<slim::Cfg<slim::bf16, D, FW, kTileRows, KIND>>;
  d.ksum = &slim::launch_ksum<slim::Cfg<slim::bf16, D, FW, kTileRows, KIND>>;
  d.carry8 = &slim::launch_carry8<slim::Cfg<slim::bf16, D, FW, kTileRows, KIND>>;
  typedef slim::Cfg<slim::bf16, D, FW, kTileRows, KIND> G;
  d.quad_fwd = &slim::launch_quad_fwd<G>;
  d.quad_dq = &slim::launch_quad_dq<G>;
  d.quad_dk = &slim::launch_quad_dk<G>;
  d.quad_gsum = &slim::launch_quad_gsum<G>;
  d.state_frag = &slim::launch_state_frag<G>;
  d.state_frag_bytes = &slim::state_frag_bytes<G>;
  return d;
}

// Backward walk kernel: the 8-wave form where it is built (bf16, 32 or 64
// features per slice), else the 4-wave form.  SLIM_BWD_WAVES=4 (debugging)
// forces the 4-wave form.
bwd_fn pick_bwd(const Dispatch& d) {
  const char* env = getenv("SLIM_BWD_WAVES");
  if (d.bwd8 != nullptr && !(env != nullptr && atoi(env) == 4)) return d.bwd8;
  return d.bwd4;
}

template <int KIND>
Dispatch pick_bf16(int d, int M) {
  if (d == 64) {
    if (M == 256) return make_dispatch8<64, 64, KIND>();
    if (M == 128) return make_dispatch8<64, 32, KIND>();
    return make_dispatch<slim::bf16, 64, 16, KIND>();
  }
  if (M == 256) return make_dispatch8<32, 64, KIND>();
  if (M == 128) return make_dispatch8<32, 32, KIND>();
  return make_dispatch<slim::bf16, 32, 16, KIND>();
}

template <int KIND>
Dispatch pick_f32(int d, int M) {
  if (d == 64) return make_dispatch<float, 64, 16, KIND>();
  if (M == 128) return make_dispatch<float, 32, 32, KIND>();
  return make_dispatch<float, 32, 16, KIND>();
}

// the square map (M = 64): the 4-wave kernels with 16 features per wave
Dispatch pick_square(int dtype, int d) {
  if (dtype == SLIM_BF16)
    return d == 64 ? make_dispatch<slim::bf16, 64, 16, slim::kSquare>() : make_dispatch<slim::bf16, 32, 16, slim::kSquare>();
  return d == 64 ? make_dispatch<float, 64, 16, slim::kSquare>() : make_dispatch<float, 32, 16, slim::kSquare>();
}

// callers have checked check_problem(p)
Dispatch dispatch(const slim_problem* p) {
  if (p->kind == SLIM_SQUARE) return pick_square(p->dtype, p->d);
  if (p->dtype == SLIM_BF16) return p->kind == SLIM_FAVOR_PLUS ? pick_bf16<slim::kFavor>(p->d, p->M)
                                                               : pick_bf16<slim::kRelu>(p->d, p->M);
  return p->kind == SLIM_FAVOR_PLUS ? pick_f32<slim::kFavor>(p->d, p->M) : pick_f32<slim::kRelu>(p->d, p->M);
}

size_t wfrag_bytes_of(const slim_problem* p) { return dispatch(p).wfrag_bytes(); }
size_t state_frag_bytes_of(const slim_problem* p) {
  const Dispatch d = dispatch(p);
  return d.state_frag_bytes != nullptr ? d.state_frag_bytes() : 0;
}
bool has_ksum(const slim_problem* p) { return dispatch(p).ksum != nullptr; }
bool has_carry8(const slim_problem* p) { return dispatch(p).carry8 != nullptr; }
size_t context_bytes(const slim_problem* p) {
  if (!context_used(p)) return 0;
  return (size_t)p->B * p->H * (bwd_parts(p) + 1) * state_elems(p) * sizeof(float);
}

// ---- the explicit prefix-sum within-slice mode: slices one after another;
// the row kernels run ps_workgroups per head (rows dealt round-robin), the
// backward restarts from exact states at ps_parts part boundaries (whole
// slices) and downdates inside a part (eq. 17)
int ps_slices(const slim_problem* p) { return (int)((p->L + clamp_C(p) - 1) / clamp_C(p)); }
int ps_workgroups(const slim_problem* p) {
  const int64_t BH = p->B * p->H;
  return (int)std::max<int64_t>(1, std::min<int64_t>(64, (1024 + BH - 1) / BH));
}
int ps_parts(const slim_problem* p) { return std::min(ps_slices(p), 64); }
struct PsLayout {
  size_t kmax, U, Gh, s[2], g[2], parts, bounds, dw, total;
};
PsLayout ps_layout(const slim_problem* p, int phase) {
  PsLayout l;
  std::memset(&l, 0, sizeof(l));
  size_t off = 0;
  auto take = [&](size_t& at, size_t bytes) {
    at = off;
    off += align256(bytes);
  };
  const size_t BH = (size_t)p->B * p->H, SZ = state_elems(p), NW = ps_workgroups(p);
  const size_t rows = (size_t)clamp_C(p) * BH * SZ * sizeof(float);  // one slice's states
  take(l.U, rows);
  take(l.s[0], BH * SZ * sizeof(float));
  take(l.s[1], BH * SZ * sizeof(float));
  if (phase == SLIM_PHASE_FWD) {
    take(l.kmax, BH * NW * sizeof(float));
  } else {
    const size_t P2 = ps_parts(p);
    take(l.Gh, rows);
    take(l.g[0], BH * SZ * sizeof(float));
    take(l.g[1], BH * SZ * sizeof(float));
    take(l.parts, BH * P2 * SZ * sizeof(float));
    take(l.bounds, BH * (P2 + 1) * SZ * sizeof(float));
    take(l.dw, 2 * BH * NW * (size_t)p->M * p->d * sizeof(float));
  }
  l.total = off;
  return l;
}

size_t fwd_ws_bytes(const slim_problem* p) {
  if (ps(p)) return ps_layout(p, SLIM_PHASE_FWD).total;
  if (quad(p)) return quad_fwd_layout(p).total;
  return fwd_layout(p, plan_fwd_segments(p)).total;
}
size_t bwd_ws_bytes(const slim_problem* p) {
  if (ps(p)) return ps_layout(p, SLIM_PHASE_BWD).total;
  if (quad(p)) return quad_bwd_layout(p).total;
  return bwd_layout(p, plan_segments(p)).total;
}

}  // namespace

extern "C" {

const char* slim_status_string(int status) {
  switch (status) {
    case SLIM_OK:
      return "ok";
    case SLIM_EINVAL:
      return "invalid argument";
    case SLIM_EUNSUPPORTED:
      return "unsupported problem";
    case SLIM_EWORKSPACE:
      return "workspace missing or too small";
    case SLIM_EHIP:
      return "HIP runtime error";
    default:
      return "unknown status";
  }
}

const char* slim_last_error(void) { return g_last_error.c_str(); }

int slim_time_walk(int phase, void* before, void* after) {
  if (phase != SLIM_PHASE_FWD && phase != SLIM_PHASE_BWD) return fail(SLIM_EINVAL, "unknown phase %d", phase);
  if ((before == nullptr) != (after == nullptr)) return fail(SLIM_EINVAL, "set both events or neither");
  g_timer[phase].before = (hipEvent_t)before;
  g_timer[phase].after = (hipEvent_t)after;
  return ok();
}

int slim_num_segments(const slim_problem* p) {
  if (check_problem(p) != SLIM_OK) return 0;
  return plan_segments(p);
}

size_t slim_context_bytes(const slim_problem* p) {
  if (check_problem(p) != SLIM_OK) return 0;
  return context_bytes(p);
}

size_t slim_workspace_bytes(const slim_problem* p, int phase) {
  if (check_problem(p) != SLIM_OK) return 0;
  if (phase == SLIM_PHASE_FWD) return fwd_ws_bytes(p);
  if (phase == SLIM_PHASE_BWD) return bwd_ws_bytes(p);
  fail(SLIM_EINVAL, "unknown phase %d", phase);
  return 0;
}

int slim_featmap(const slim_problem* p, const void* X, const float* W, int role, float* phi, float* shift,
                 void* stream) {
  int st = check_problem(p);
  if (st != SLIM_OK) return st;
  if (X == nullptr || W == nullptr || phi == nullptr) return fail(SLIM_EINVAL, "X, W and phi must be non-NULL");
  if (role != SLIM_QUERY && role != SLIM_KEY) return fail(SLIM_EINVAL, "unknown role %d", role);
  if (p->kind == SLIM_FAVOR_PLUS && shift == nullptr) return fail(SLIM_EINVAL, "FAVOR+ needs a shift buffer");
  st = check_alignment({X}, {W, phi, shift});
  if (st != SLIM_OK) return st;
  slim::FeatArgs a;
  a.X = X;
  a.W = W;
  a.phi = phi;
  a.shift = shift;
  a.B = (int)p->B;
  a.H = (int)p->H;
  a.L = (int)p->L;
  a.role = role;
  a.relu_eps = p->relu_eps;
  hipError_t e = dispatch(p).feat(a, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "feature-map launch");
  return ok();
}

}  // extern "C"

namespace {

// Forward in the quadratic within-slice mode (arguments checked by fwd_impl):
//   (0) one key shift per head: the largest key exponent of every part and
//       of the initial state;
//   (1) the state before the first slice: the initial state, rescaled to
//       that shift;
//   (2) per slice: the outputs of its query tiles from the state before it
//       and its keys up to each row; what its keys add, in parts; the state
//       after it = the state before + the parts.
int quad_fwd_impl(const slim_problem* p, const Dispatch& dp, const void* Q, const void* K, const void* V,
                  const float* W, const float* state_in, const float* kshift_in, void* Y, float* state_out,
                  float* kshift_out, char* w, hipStream_t s) {
  const QuadFwdLayout lay = quad_fwd_layout(p);
  const bool favor = p->kind == SLIM_FAVOR_PLUS;
  const int BH = (int)(p->B * p->H), SZ = (int)state_elems(p);
  const int C = clamp_C(p), NS = quad_slices(p), tps = quad_tiles(p);
  hipError_t e;
  slim::WfragArgs wf;
  wf.W = W;
  wf.out = w + lay.wfrag;
  e = dp.wfrag(wf, s);
  if (e != hipSuccess) return hip_fail(e, "W-fragment launch");
  slim::KsumArgs ks;
  std::memset(&ks, 0, sizeof(ks));
  set_drop(ks, drop_plan(p));
  ks.K = K;
  ks.V = V;
  ks.W = W;
  ks.Wfrag = wf.out;
  ks.B = (int)p->B;
  ks.H = (int)p->H;
  ks.L = (int)p->L;
  ks.C = C;
  ks.relu_eps = p->relu_eps;
  if (favor) {
    ks.out = (float*)(w + lay.kmax);
    ks.P2 = quad_max_parts(p);
    e = dp.ksum(ks, slim::kSumMax, s);
    if (e != hipSuccess) return hip_fail(e, "key-maximum launch");
    e = slim::launch_kshift_reduce(ks.out, ks.P2, state_in != nullptr ? kshift_in : nullptr, kshift_out, BH, s);
    if (e != hipSuccess) return hip_fail(e, "key-shift launch");
    ks.shift = kshift_out;
  }
  float* Sa = (float*)(w + lay.sa);
  float* Sb = (float*)(w + lay.sb);
  float* parts = (float*)(w + lay.parts);
  e = slim::launch_state_combine(state_in, SZ, favor ? kshift_in : nullptr, favor ? kshift_out : nullptr, nullptr, 0,
                                 1.f, Sa, BH, SZ, s);
  if (e != hipSuccess) return hip_fail(e, "state launch");
  slim::QuadArgs qa;
  std::memset(&qa, 0, sizeof(qa));
  set_drop(qa, drop_plan(p));
  qa.Q = Q;
  qa.K = K;
  qa.V = V;
  qa.Wfrag = wf.out;
  qa.kshift = favor ? kshift_out : nullptr;
  qa.Y = Y;
  qa.B = (int)p->B;
  qa.H = (int)p->H;
  qa.L = (int)p->L;
  qa.C = C;
  qa.relu_eps = p->relu_eps;
  ks.out = parts;
  ks.P2 = quad_sum_parts(p);
  e = timed_launch(SLIM_PHASE_FWD, s, [&]() -> hipError_t {
    for (int n = 0; n < NS; ++n) {
      qa.row0 = n * C;
      qa.rows = (int)std::min<int64_t>(C, p->L - (int64_t)n * C);
      qa.S = Sa;
      hipError_t er = dp.quad_fwd(qa, quad_workgroups(p), s);
      if (er != hipSuccess) return er;
      if (n == NS - 1 && state_out == nullptr) break;
      ks.tile_begin = n * tps;
      ks.tile_end = n * tps + (qa.rows + kTileRows - 1) / kTileRows;
      er = dp.ksum(ks, slim::kSumStates, s);
      if (er != hipSuccess) return er;
      er = slim::launch_state_combine(Sa, SZ, nullptr, nullptr, parts, ks.P2, 1.f, n == NS - 1 ? state_out : Sb, BH, SZ,
                                      s);
      if (er != hipSuccess) return er;
      std::swap(Sa, Sb);
    }
    return hipSuccess;
  });
  if (e != hipSuccess) return hip_fail(e, "quadratic-mode forward launches");
  return ok();
}

// Backward in the quadratic within-slice mode (arguments checked by slim_bwd):
//   (1) exact states at the boundaries of R runs of whole slices (slice-
//       aligned key sums, then their prefix from the initial state);
//   (2) the slices in reverse, each with the state before it (the exact
//       state at a run's first slice, else the state after it downdated by
//       what the slice's keys add, eq. 17) and the cotangent after it: the
//       query pass, the key pass, then the cotangent before it (eq. 18);
//   (3) dstate_in, and dW from the workgroups' partials in a fixed order.
int quad_bwd_impl(const slim_problem* p, const Dispatch& dp, const void* Q, const void* K, const void* V,
                  const float* W, const float* state_in, const float* kshift_in, const float* kshift, const void* dY,
                  const float* dstate_out, void* dQ, void* dK, void* dV, float* dW, float* dstate_in, char* w,
                  hipStream_t s) {
  const QuadBwdLayout lay = quad_bwd_layout(p);
  const bool favor = p->kind == SLIM_FAVOR_PLUS;
  const int BH = (int)(p->B * p->H), SZ = (int)state_elems(p);
  const int C = clamp_C(p), NS = quad_slices(p), tps = quad_tiles(p), R = quad_runs(p);
  const int P2 = quad_sum_parts(p), NW = quad_bwd_workgroups(p);
  hipError_t e;
  slim::WfragArgs wf;
  wf.W = W;
  wf.out = w + lay.wfrag;
  e = dp.wfrag(wf, s);
  if (e != hipSuccess) return hip_fail(e, "W-fragment launch");
  slim::KsumArgs ks;
  std::memset(&ks, 0, sizeof(ks));
  set_drop(ks, drop_plan(p));
  ks.K = K;
  ks.V = V;
  ks.W = W;
  ks.Wfrag = wf.out;
  ks.shift = favor ? kshift : nullptr;
  ks.B = (int)p->B;
  ks.H = (int)p->H;
  ks.L = (int)p->L;
  ks.C = C;
  ks.relu_eps = p->relu_eps;
  // (1)
  ks.out = (float*)(w + lay.seg);
  ks.P2 = R;
  ks.align = tps;
  e = dp.ksum(ks, slim::kSumStates, s);
  if (e != hipSuccess) return hip_fail(e, "run-sum launch");
  const float* bounds = (const float*)(w + lay.bounds);
  const size_t bstride = (size_t)(R + 1) * SZ;  // between heads of one boundary
  {
    slim::ScanArgs sc;
    std::memset(&sc, 0, sizeof(sc));
    sc.seg = ks.out;
    sc.init = state_in;
    sc.init_shift = favor ? kshift_in : nullptr;
    sc.shift = favor ? kshift : nullptr;
    sc.out = (float*)(w + lay.bounds);
    sc.BH = BH;
    sc.P = R;
    sc.SZ = SZ;
    sc.favor = favor ? 1 : 0;
    e = slim::launch_scan_bwd(sc, s);
    if (e != hipSuccess) return hip_fail(e, "boundary-scan launch");
  }
  ks.align = 0;
  ks.out = (float*)(w + lay.parts);
  ks.P2 = P2;
  float* dw_part = (float*)(w + lay.dw_part);
  e = slim::launch_state_combine(nullptr, 0, nullptr, nullptr, nullptr, 0, 1.f, dw_part, BH * NW, (int)(p->M * p->d), s);
  if (e != hipSuccess) return hip_fail(e, "dW-partial launch");
  float* parts = (float*)(w + lay.parts);
  float* sbuf[2] = {(float*)(w + lay.s[0]), (float*)(w + lay.s[1])};
  float* gbuf[2] = {(float*)(w + lay.g[0]), (float*)(w + lay.g[1])};
  const float* Gafter = dstate_out;
  int gb = 0;
  if (Gafter == nullptr) {
    e = slim::launch_state_combine(nullptr, 0, nullptr, nullptr, nullptr, 0, 1.f, gbuf[1], BH, SZ, s);
    if (e != hipSuccess) return hip_fail(e, "cotangent launch");
    Gafter = gbuf[1];
  }
  slim::QuadArgs qa;
  std::memset(&qa, 0, sizeof(qa));
  set_drop(qa, drop_plan(p));
  qa.Q = Q;
  qa.K = K;
  qa.V = V;
  qa.dY = dY;
  qa.Wfrag = wf.out;
  qa.kshift = favor ? kshift : nullptr;
  qa.Sfrag = w + lay.sfrag;
  qa.Gfrag = w + lay.gfrag;
  qa.DN = (float*)(w + lay.dn);
  qa.dQ = dQ;
  qa.dK = dK;
  qa.dV = dV;
  qa.dW_part = dw_part;
  qa.out = parts;
  qa.B = (int)p->B;
  qa.H = (int)p->H;
  qa.L = (int)p->L;
  qa.C = C;
  qa.relu_eps = p->relu_eps;
  auto first_of_run = [&](int r) { return (int)((int64_t)r * NS / R); };
  // (2)
  e = timed_launch(SLIM_PHASE_BWD, s, [&]() -> hipError_t {
    hipError_t er;
    int r = R - 1, sb = 0;
    const float* Safter = nullptr;  // the state after slice n, unless n ends its run
    for (int n = NS - 1; n >= 0; --n) {
      while (first_of_run(r) > n) --r;
      const int rows = (int)std::min<int64_t>(C, p->L - (int64_t)n * C);
      const bool run_end = (n == first_of_run(r + 1) - 1);
      float* Sb = sbuf[sb];
      sb ^= 1;
      if (n == first_of_run(r)) {
        er = slim::launch_state_combine(bounds + (size_t)r * SZ, bstride, nullptr, nullptr, nullptr, 0, 1.f, Sb, BH, SZ,
                                        s);
      } else {
        ks.tile_begin = n * tps;
        ks.tile_end = n * tps + (rows + kTileRows - 1) / kTileRows;
        er = dp.ksum(ks, slim::kSumStates, s);
        if (er != hipSuccess) return er;
        if (run_end) er = slim::launch_state_combine(bounds + (size_t)(r + 1) * SZ, bstride, nullptr, nullptr, parts, P2,
                                                     -1.f, Sb, BH, SZ, s);
        else er = slim::launch_state_combine(Safter, SZ, nullptr, nullptr, parts, P2, -1.f, Sb, BH, SZ, s);
      }
      if (er != hipSuccess) return er;
      Safter = Sb;
      er = dp.state_frag(Sb, w + lay.sfrag, Gafter, w + lay.gfrag, BH, s);
      if (er != hipSuccess) return er;
      qa.S = Sb;
      qa.Gc = Gafter;
      qa.row0 = n * C;
      qa.rows = rows;
      er = dp.quad_dq(qa, NW, s);
      if (er != hipSuccess) return er;
      er = dp.quad_dk(qa, NW, s);
      if (er != hipSuccess) return er;
      if (n > 0 || dstate_in != nullptr) {
        er = dp.quad_gsum(qa, P2, s);
        if (er != hipSuccess) return er;
        er = slim::launch_state_combine(Gafter, SZ, nullptr, nullptr, parts, P2, 1.f, gbuf[gb], BH, SZ, s);
        if (er != hipSuccess) return er;
        Gafter = gbuf[gb];
        gb ^= 1;
      }
    }
    return hipSuccess;
  });
  if (e != hipSuccess) return hip_fail(e, "quadratic-mode backward launches");
  // (3) the cotangent of state_in, relative to kshift_in (FAVOR+ with an initial state)
  if (dstate_in != nullptr) {
    e = slim::launch_state_combine(Gafter, SZ, favor ? kshift_in : nullptr, favor ? kshift : nullptr, nullptr, 0, 1.f,
                                   dstate_in, BH, SZ, s);
    if (e != hipSuccess) return hip_fail(e, "dstate_in launch");
  }
  e = slim::launch_dw_reduce(dw_part, BH * NW, (int)(p->M * p->d), dW, s);
  if (e != hipSuccess) return hip_fail(e, "dW-reduction launch");
  return ok();
}

// Arguments common to the PS kernels
slim::PsArgs ps_args(const slim_problem* p, const void* Q, const void* K, const void* V, const float* W) {
  slim::PsArgs a;
  std::memset(&a, 0, sizeof(a));
  a.Q = Q;
  a.K = K;
  a.V = V;
  a.W = W;
  a.B = (int)p->B;
  a.H = (int)p->H;
  a.L = (int)p->L;
  a.d = (int)p->d;
  a.M = (int)p->M;
  a.C = clamp_C(p);
  a.kind = p->kind == SLIM_FAVOR_PLUS ? slim::kFavor : p->kind == SLIM_RELU ? slim::kRelu : slim::kSquare;
  a.relu_eps = p->relu_eps;
  a.bf16 = p->dtype == SLIM_BF16 ? 1 : 0;
  a.nslot = ps_workgroups(p);
  return a;
}

// Forward in the explicit prefix-sum mode (arguments checked by fwd_impl):
//   (0) FAVOR+: one key shift per head, the largest key exponent over all
//       rows and the initial state's;
//   (1) the state before the first slice: the initial state at that shift;
//   (2) per slice: each row's term g(k)^T [v | 1]; their prefix sums from the
//       state before the slice, written out for every row (the last is the
//       state after the slice); the outputs from them.
int ps_fwd_impl(const slim_problem* p, const void* Q, const void* K, const void* V, const float* W,
                const float* state_in, const float* kshift_in, void* Y, float* state_out, float* kshift_out, char* w,
                hipStream_t s) {
  const PsLayout lay = ps_layout(p, SLIM_PHASE_FWD);
  const bool favor = p->kind == SLIM_FAVOR_PLUS;
  const int BH = (int)(p->B * p->H), SZ = (int)state_elems(p), C = clamp_C(p), NS = ps_slices(p);
  const int NW = ps_workgroups(p);
  slim::PsArgs a = ps_args(p, Q, K, V, W);
  a.U = (float*)(w + lay.U);
  a.Y = Y;
  hipError_t e;
  if (favor) {
    a.part = (float*)(w + lay.kmax);
    e = slim::launch_ps(slim::kPsKmax, a, NW, 0, s);
    if (e != hipSuccess) return hip_fail(e, "key-maximum launch");
    e = slim::launch_kshift_reduce(a.part, NW, state_in != nullptr ? kshift_in : nullptr, kshift_out, BH, s);
    if (e != hipSuccess) return hip_fail(e, "key-shift launch");
    a.kshift = kshift_out;
  }
  float* S[2] = {(float*)(w + lay.s[0]), (float*)(w + lay.s[1])};
  e = slim::launch_state_combine(state_in, SZ, favor ? kshift_in : nullptr, favor ? kshift_out : nullptr, nullptr, 0,
                                 1.f, S[0], BH, SZ, s);
  if (e != hipSuccess) return hip_fail(e, "state launch");
  e = timed_launch(SLIM_PHASE_FWD, s, [&]() -> hipError_t {
    int cur = 0;
    for (int n = 0; n < NS; ++n) {
      a.row0 = n * C;
      a.rows = (int)std::min<int64_t>(C, p->L - (int64_t)n * C);
      const int nwg = std::min(NW, a.rows);
      hipError_t er = slim::launch_ps(slim::kPsTerms, a, nwg, 0, s);
      if (er != hipSuccess) return er;
      a.S_in = S[cur];
      a.in_stride = (size_t)SZ;
      a.S_out = (n == NS - 1 && state_out != nullptr) ? state_out : S[cur ^ 1];
      er = slim::launch_ps(slim::kPsScan0, a, 0, 0, s);
      if (er != hipSuccess) return er;
      er = slim::launch_ps(slim::kPsOut, a, nwg, 0, s);
      if (er != hipSuccess) return er;
      cur ^= 1;
    }
    return hipSuccess;
  });
  if (e != hipSuccess) return hip_fail(e, "PS-mode forward launches");
  return ok();
}

// Backward in the explicit prefix-sum mode (arguments checked by slim_bwd):
//   (1) exact states at the boundaries of P2 parts of whole slices (what
//       each part's rows add, then their prefix from the initial state);
//   (2) the slices in reverse: each row's term again, the state before the
//       slice (the exact one at a part's first slice, else the state after
//       it minus the slice's terms, eq. 17) and the prefix sums from it; the
//       queries' gradient and their terms g(q) [dN | dD]; the reverse prefix
//       sums of those from the cotangent after the slice (the last is the
//       cotangent before it, eq. 18); the keys' and values' gradient;
//   (3) dstate_in, and dW from the workgroups' partials in a fixed order.
int ps_bwd_impl(const slim_problem* p, const void* Q, const void* K, const void* V, const float* W,
                const float* state_in, const float* kshift_in, const float* kshift, const void* dY,
                const float* dstate_out, void* dQ, void* dK, void* dV, float* dW, float* dstate_in, char* w,
                hipStream_t s) {
  const PsLayout lay = ps_layout(p, SLIM_PHASE_BWD);
  const bool favor = p->kind == SLIM_FAVOR_PLUS;
  const int BH = (int)(p->B * p->H), SZ = (int)state_elems(p), C = clamp_C(p), NS = ps_slices(p);
  const int NW = ps_workgroups(p), P2 = ps_parts(p);
  const size_t MD = (size_t)p->M * p->d;
  slim::PsArgs a = ps_args(p, Q, K, V, W);
  a.kshift = favor ? kshift : nullptr;
  a.U = (float*)(w + lay.U);
  a.Gh = (float*)(w + lay.Gh);
  a.dY = dY;
  a.dQ = dQ;
  a.dK = dK;
  a.dV = dV;
  hipError_t e;
  // (1)
  a.part = (float*)(w + lay.parts);
  e = slim::launch_ps(slim::kPsSum, a, P2, NS, s);
  if (e != hipSuccess) return hip_fail(e, "part-sum launch");
  const float* bounds = (const float*)(w + lay.bounds);
  {
    slim::ScanArgs sc;
    std::memset(&sc, 0, sizeof(sc));
    sc.seg = a.part;
    sc.init = state_in;
    sc.init_shift = favor ? kshift_in : nullptr;
    sc.shift = favor ? kshift : nullptr;
    sc.out = (float*)(w + lay.bounds);
    sc.BH = BH;
    sc.P = P2;
    sc.SZ = SZ;
    sc.favor = favor ? 1 : 0;
    e = slim::launch_scan_bwd(sc, s);
    if (e != hipSuccess) return hip_fail(e, "boundary-scan launch");
  }
  float* dw_part = (float*)(w + lay.dw);
  e = slim::launch_state_combine(nullptr, 0, nullptr, nullptr, nullptr, 0, 1.f, dw_part, 2 * BH * NW, (int)MD, s);
  if (e != hipSuccess) return hip_fail(e, "dW-partial launch");
  float* sb[2] = {(float*)(w + lay.s[0]), (float*)(w + lay.s[1])};
  float* gb[2] = {(float*)(w + lay.g[0]), (float*)(w + lay.g[1])};
  const size_t bstride = (size_t)(P2 + 1) * SZ;  // between heads of one boundary
  auto first_of_part = [&](int r) { return (int)((int64_t)r * NS / P2); };
  const float* Gafter = dstate_out;  // nullptr: zero
  // (2)
  e = timed_launch(SLIM_PHASE_BWD, s, [&]() -> hipError_t {
    hipError_t er;
    int r = P2 - 1, cs = 0, cg = 0;
    const float* Safter = nullptr;
    for (int n = NS - 1; n >= 0; --n) {
      while (first_of_part(r) > n) --r;
      a.row0 = n * C;
      a.rows = (int)std::min<int64_t>(C, p->L - (int64_t)n * C);
      const int nwg = std::min(NW, a.rows);
      er = slim::launch_ps(slim::kPsTerms, a, nwg, 0, s);
      if (er != hipSuccess) return er;
      int mode;
      if (n == first_of_part(r)) {
        mode = slim::kPsScan2;
        a.S_in = bounds + (size_t)r * SZ;
        a.in_stride = bstride;
      } else if (n == first_of_part(r + 1) - 1) {
        mode = slim::kPsScan1;
        a.S_in = bounds + (size_t)(r + 1) * SZ;
        a.in_stride = bstride;
      } else {
        mode = slim::kPsScan1;
        a.S_in = Safter;
        a.in_stride = (size_t)SZ;
      }
      a.S_out = sb[cs];
      er = slim::launch_ps(mode, a, 0, 0, s);
      if (er != hipSuccess) return er;
      Safter = sb[cs];
      cs ^= 1;
      a.dW_part = dw_part;
      er = slim::launch_ps(slim::kPsGq, a, nwg, 0, s);
      if (er != hipSuccess) return er;
      a.G_in = Gafter;
      a.G_out = gb[cg];
      er = slim::launch_ps(slim::kPsRscan, a, 0, 0, s);
      if (er != hipSuccess) return er;
      Gafter = gb[cg];
      cg ^= 1;
      a.dW_part = dw_part + (size_t)BH * NW * MD;
      er = slim::launch_ps(slim::kPsGk, a, nwg, 0, s);
      if (er != hipSuccess) return er;
    }
    return hipSuccess;
  });
  if (e != hipSuccess) return hip_fail(e, "PS-mode backward launches");
  // (3) the cotangent of state_in, relative to kshift_in (FAVOR+ with an initial state)
  if (dstate_in != nullptr) {
    e = slim::launch_state_combine(Gafter, SZ, favor ? kshift_in : nullptr, favor ? kshift : nullptr, nullptr, 0, 1.f,
                                   dstate_in, BH, SZ, s);
    if (e != hipSuccess) return hip_fail(e, "dstate_in launch");
  }
  e = slim::launch_dw_reduce(dw_part, 2 * BH * NW, (int)MD, dW, s);
  if (e != hipSuccess) return hip_fail(e, "dW-reduction launch");
  return ok();
}

// The forward of slim_fwd on a given workspace (the caller's, or the
// library's static scratch for slim_fwd_noalloc).
int fwd_impl(const slim_problem* p, const void* Q, const void* K, const void* V, const float* W,
             const float* state_in, const float* kshift_in, void* Y, float* logD, float* state_out, float* kshift_out,
             float* ctx, void* ws, size_t ws_bytes, void* stream) {
  int st = check_problem(p);
  if (st != SLIM_OK) return st;
  if (Q == nullptr || K == nullptr || V == nullptr || W == nullptr || Y == nullptr)
    return fail(SLIM_EINVAL, "Q, K, V, W and Y must be non-NULL");
  if (p->kind == SLIM_FAVOR_PLUS) {
    if (kshift_out == nullptr) return fail(SLIM_EINVAL, "FAVOR+ needs kshift_out");
    if (state_in != nullptr && kshift_in == nullptr) return fail(SLIM_EINVAL, "state_in needs kshift_in (FAVOR+)");
  }
  st = check_alignment({Q, K, V, Y, ws}, {W, state_in, kshift_in, state_out, kshift_out, ctx, logD});
  if (st != SLIM_OK) return st;
  if (logD != nullptr && (ps(p) || quad(p)))
    return fail(SLIM_EUNSUPPORTED, "logD is written by the tile-walk mode (within = SLIM_WITHIN_ITER) only");
  if (!context_used(p)) ctx = nullptr;
  const size_t need = fwd_ws_bytes(p);
  if (need > 0 && (ws == nullptr || ws_bytes < need))
    return fail(SLIM_EWORKSPACE, "forward workspace needs %zu bytes, got %zu", need, ws == nullptr ? 0 : ws_bytes);
  if (ps(p))
    return ps_fwd_impl(p, Q, K, V, W, state_in, kshift_in, Y, state_out, kshift_out, (char*)ws, (hipStream_t)stream);
  const Dispatch dp = dispatch(p);
  if (quad(p))
    return quad_fwd_impl(p, dp, Q, K, V, W, state_in, kshift_in, Y, state_out, kshift_out, (char*)ws,
                         (hipStream_t)stream);
  const int P = plan_fwd_segments(p);
  const FwdLayout lay = fwd_layout(p, P);
  const bool favor = p->kind == SLIM_FAVOR_PLUS;
  hipStream_t s = (hipStream_t)stream;
  char* w = (char*)ws;
  slim::FwdArgs a;
  std::memset(&a, 0, sizeof(a));
  set_drop(a, drop_plan(p));
  a.Q = Q;
  a.K = K;
  a.V = V;
  a.W = W;
  a.B = (int)p->B;
  a.H = (int)p->H;
  a.L = (int)p->L;
  a.C = clamp_C(p);
  a.P = P;
  a.relu_eps = p->relu_eps;
  hipError_t e = hipSuccess;
  if (p->dtype == SLIM_BF16) {
    // W in fragment order, with the low parts of its bf16 split (logits)
    slim::WfragArgs wf;
    wf.W = W;
    wf.out = w + lay.wfrag;
    e = dp.wfrag(wf, s);
    if (e != hipSuccess) return hip_fail(e, "W-fragment launch");
    a.Wfrag = wf.out;
  }
  if (P > 1 && dp.ksum != nullptr) {
    // One key shift for the whole head: (0) the largest key exponent of every
    // part and of the initial state; (1) what each part adds relative to it;
    // (2) the exact state at every part boundary; (3) the walk, each segment
    // starting from its boundary, with no rescaling.
    const int P2 = fwd_parts(p), S2 = P2 / P;
    const int BH = (int)(p->B * p->H);
    slim::KsumArgs ks;
    std::memset(&ks, 0, sizeof(ks));
    set_drop(ks, drop_plan(p));
    ks.K = K;
    ks.V = V;
    ks.W = W;
    ks.Wfrag = a.Wfrag;
    ks.B = (int)p->B;
    ks.H = (int)p->H;
    ks.L = (int)p->L;
    ks.C = clamp_C(p);
    ks.P2 = P2;
    ks.relu_eps = p->relu_eps;
    if (favor) {
      ks.out = (float*)(w + lay.seg_shift);
      e = dp.ksum(ks, slim::kSumMax, s);
      if (e != hipSuccess) return hip_fail(e, "key-maximum launch");
      // (the sums take the head's shift as the largest part maximum
      // themselves and write it to kshift_out)
      ks.part_max = ks.out;
      ks.n_part_max = P2;
      ks.init_shift = state_in != nullptr ? kshift_in : nullptr;
      ks.shift_out = kshift_out;
    }
    ks.out = (float*)(w + lay.seg_sum);
    e = dp.ksum(ks, slim::kSumStates, s);
    if (e != hipSuccess) return hip_fail(e, "key-sum launch");
    slim::ScanArgs sc;
    std::memset(&sc, 0, sizeof(sc));
    sc.seg = ks.out;
    sc.init = state_in;
    sc.init_shift = favor ? kshift_in : nullptr;
    sc.shift = favor ? kshift_out : nullptr;
    sc.out = ctx != nullptr ? ctx : (float*)(w + lay.starts);
    sc.BH = BH;
    sc.P = P2;
    sc.SZ = (int)state_elems(p);
    sc.favor = favor ? 1 : 0;
    e = slim::launch_scan_bwd(sc, s);
    if (e != hipSuccess) return hip_fail(e, "boundary-scan launch");
    a.seg_state = sc.out;
    a.seg_stride = P2 + 1;
    a.seg_step = S2;
    a.fixed_shift = favor ? kshift_out : nullptr;
    a.Y = Y;
    a.state_out = state_out;
    a.logD = logD;
    e = timed_launch(SLIM_PHASE_FWD, s, [&] { return dp.fwd(a, slim::kWalkOutputs, s); });
    if (e != hipSuccess) return hip_fail(e, "forward launch");
    return ok();
  }
  if (P > 1) {
    // (1) what each sub-segment adds, with its own running key shift
    const int S2 = plan_sum_split(p, P), P2 = P * S2;
    slim::FwdArgs k = a;
    k.P = P2;
    k.seg_out = (float*)(w + lay.seg_sum);
    k.seg_shift_out = (float*)(w + lay.seg_shift);
    e = dp.fwd(k, slim::kWalkSums, s);
    if (e != hipSuccess) return hip_fail(e, "segment-sum launch");
    // (2) the exact state each segment starts from
    slim::ScanArgs sc;
    std::memset(&sc, 0, sizeof(sc));
    sc.seg = k.seg_out;
    sc.seg_shift = favor ? k.seg_shift_out : nullptr;
    sc.init = state_in;
    sc.init_shift = favor ? kshift_in : nullptr;
    sc.out = (float*)(w + lay.starts);
    sc.out_shift = (float*)(w + lay.start_shift);
    sc.BH = (int)(p->B * p->H);
    sc.P = P2;
    sc.SZ = (int)state_elems(p);
    sc.favor = favor ? 1 : 0;
    e = slim::launch_scan_fwd(sc, s);
    if (e != hipSuccess) return hip_fail(e, "segment-scan launch");
    a.seg_state = sc.out;
    a.seg_shift = sc.out_shift;
    a.seg_stride = P2;
    a.seg_step = S2;
  } else {
    a.seg_state = state_in;
    a.seg_shift = kshift_in;
    a.seg_stride = 1;
    a.seg_step = 1;
  }
  // (3) the walk proper
  a.Y = Y;
  a.logD = logD;
  a.state_out = state_out;
  a.kshift_out = favor ? kshift_out : nullptr;
  e = timed_launch(SLIM_PHASE_FWD, s, [&] { return dp.fwd(a, slim::kWalkOutputs, s); });
  if (e != hipSuccess) return hip_fail(e, "forward launch");
  return ok();
}

// Static device scratch of slim_fwd_noalloc: one copy per device, held until
// the process ends.  In host code `scratch` names a host-side stand-in, not
// the device array: its device address comes from hipGetSymbolAddress (per
// device, kept in g_scratch), and only that address is passed to kernels.
constexpr size_t kNoallocScratchBytes = SLIM_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

// device address of the current device's scratch, looked up once per device
int scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(SLIM_EUNSUPPORTED, "device index %d beyond %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch[dev] == nullptr) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (ptr == nullptr) return fail(SLIM_EHIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch[dev] = ptr;
  }
  *out = g_scratch[dev];
  return SLIM_OK;
}

}  // namespace

extern "C" {

int slim_fwd(const slim_problem* p, const void* Q, const void* K, const void* V, const float* W,
             const float* state_in, const float* kshift_in, void* Y, float* logD, float* state_out, float* kshift_out,
             float* ctx, void* ws, size_t ws_bytes, void* stream) {
  return fwd_impl(p, Q, K, V, W, state_in, kshift_in, Y, logD, state_out, kshift_out, ctx, ws, ws_bytes, stream);
}

size_t slim_noalloc_scratch_bytes(void) { return kNoallocScratchBytes; }

int slim_fwd_noalloc(const slim_problem* p, const void* Q, const void* K, const void* V, const float* W,
                     const float* state_in, const float* kshift_in, void* Y, float* logD, float* state_out,
                     float* kshift_out, float* ctx, void* stream) {
  int st = check_problem(p);
  if (st != SLIM_OK) return st;
  const size_t need = fwd_ws_bytes(p);
  if (need > kNoallocScratchBytes)
    return fail(SLIM_EUNSUPPORTED, "slim_fwd_noalloc: the forward needs %zu bytes of scratch, the static scratch holds %zu",
                need, kNoallocScratchBytes);
  void* ws = nullptr;
  if (need > 0) {
    st = scratch_address(&ws);
    if (st != SLIM_OK) return st;
  }
  return fwd_impl(p, Q, K, V, W, state_in, kshift_in, Y, logD, state_out, kshift_out, ctx, ws, kNoallocScratchBytes,
                  stream);
}

int slim_bwd(const slim_problem* p, const void* Q, const void* K, const void* V, const float* W,
             const float* state_in, const float* kshift_in, const float* kshift, const void* dY, const void* Y,
             const float* logD, const float* dstate_out, void* dQ, void* dK, void* dV, float* dW, float* dstate_in,
             const float* ctx, void* ws, size_t ws_bytes, void* stream) {
  int st = check_problem(p);
  if (st != SLIM_OK) return st;
  if (Q == nullptr || K == nullptr || V == nullptr || W == nullptr || dY == nullptr || dQ == nullptr ||
      dK == nullptr || dV == nullptr || dW == nullptr)
    return fail(SLIM_EINVAL, "Q, K, V, W, dY, dQ, dK, dV and dW must be non-NULL");
  const bool favor = p->kind == SLIM_FAVOR_PLUS;
  if (favor) {
    if (kshift == nullptr) return fail(SLIM_EINVAL, "FAVOR+ needs kshift (kshift_out of slim_fwd)");
    if (state_in != nullptr && kshift_in == nullptr) return fail(SLIM_EINVAL, "state_in needs kshift_in (FAVOR+)");
  }
  if (logD != nullptr && Y == nullptr) return fail(SLIM_EINVAL, "logD is used together with Y");
  st = check_alignment({Q, K, V, dY, Y, dQ, dK, dV, ws},
                       {W, state_in, kshift_in, kshift, dstate_out, dW, dstate_in, ctx, logD});
  if (st != SLIM_OK) return st;
  if (!context_used(p)) ctx = nullptr;
  const size_t need = bwd_ws_bytes(p);
  if (ws == nullptr || ws_bytes < need)
    return fail(SLIM_EWORKSPACE, "backward workspace needs %zu bytes, got %zu", need, ws == nullptr ? 0 : ws_bytes);
  if (ps(p))
    return ps_bwd_impl(p, Q, K, V, W, state_in, kshift_in, kshift, dY, dstate_out, dQ, dK, dV, dW, dstate_in, (char*)ws,
                       (hipStream_t)stream);
  const Dispatch dp = dispatch(p);
  if (quad(p))
    return quad_bwd_impl(p, dp, Q, K, V, W, state_in, kshift_in, kshift, dY, dstate_out, dQ, dK, dV, dW, dstate_in,
                         (char*)ws, (hipStream_t)stream);
  const int P = plan_segments(p);
  const BwdLayout lay = bwd_layout(p, P);
  hipStream_t s = (hipStream_t)stream;
  char* w = (char*)ws;
  const int BH = (int)(p->B * p->H);
  const int SZ = (int)state_elems(p);
  hipError_t e;

  slim::FwdArgs f;
  std::memset(&f, 0, sizeof(f));
  set_drop(f, drop_plan(p));
  f.Q = Q;
  f.K = K;
  f.V = V;
  f.W = W;
  f.fixed_shift = favor ? kshift : nullptr;
  f.B = (int)p->B;
  f.H = (int)p->H;
  f.L = (int)p->L;
  f.C = clamp_C(p);
  f.P = P;
  f.relu_eps = p->relu_eps;

  // (1) segment sums with the shift the reverse walk uses, so that every
  //     downdate subtracts exactly the rounded features that were added;
  //     (2) exact states at the segment boundaries.  Both come from the
  //     forward's context when the caller passes it.
  const int S2 = plan_sum_split(p, P), P2 = P * S2;
  // W in fragment order (with the low parts of its bf16 split), for every
  // kernel below
  slim::WfragArgs wf;
  wf.W = W;
  wf.out = w + lay.wfrag;
  e = dp.wfrag(wf, s);
  if (e != hipSuccess) return hip_fail(e, "W-fragment launch");
  const float* bounds = ctx;
  if (bounds == nullptr) {
  if (dp.ksum != nullptr) {
    slim::KsumArgs ks;
    std::memset(&ks, 0, sizeof(ks));
    set_drop(ks, drop_plan(p));
    ks.K = K;
    ks.V = V;
    ks.W = W;
    ks.Wfrag = wf.out;
    ks.shift = favor ? kshift : nullptr;
    ks.out = (float*)(w + lay.seg_sum);
    ks.B = (int)p->B;
    ks.H = (int)p->H;
    ks.L = (int)p->L;
    ks.C = clamp_C(p);
    ks.P2 = P2;
    ks.relu_eps = p->relu_eps;
    e = dp.ksum(ks, slim::kSumStates, s);
  } else {
    slim::FwdArgs k = f;
    k.P = P2;
    k.seg_out = (float*)(w + lay.seg_sum);
    e = dp.fwd(k, slim::kWalkSums, s);
  }
  if (e != hipSuccess) return hip_fail(e, "segment-sum launch");
  // (2) exact states at the segment boundaries
  slim::ScanArgs sc;
  std::memset(&sc, 0, sizeof(sc));
  sc.seg = (float*)(w + lay.seg_sum);
  sc.init = state_in;
  sc.init_shift = favor ? kshift_in : nullptr;
  sc.shift = favor ? kshift : nullptr;
  sc.out = (float*)(w + lay.bounds);
  sc.BH = BH;
  sc.P = P2;
  sc.SZ = SZ;
  sc.favor = favor ? 1 : 0;
  e = slim::launch_scan_bwd(sc, s);
  if (e != hipSuccess) return hip_fail(e, "boundary-scan launch");
  bounds = sc.out;
  }
  // (3) the reverse walk of every segment; each starts from a zero
  //     cotangent except the last (dstate_out)
  slim::BwdArgs a;
  std::memset(&a, 0, sizeof(a));
  set_drop(a, drop_plan(p));
  a.Q = Q;
  a.K = K;
  a.V = V;
  a.dY = dY;
  a.Y = Y;  // read by the 8-wave walk (the other walks recompute N)
  a.logD = logD;
  a.W = W;
  a.Wfrag = wf.out;
  a.kshift = favor ? kshift : nullptr;
  a.bounds = bounds;
  a.bound_stride = P2 + 1;
  a.bound_step = S2;
  a.dstate_out = dstate_out;
  a.g_final = P > 1 ? (float*)(w + lay.gc) : nullptr;
  a.init_shift = favor ? kshift_in : nullptr;
  a.dstate_in = P > 1 ? nullptr : dstate_in;
  a.dQ = dQ;
  a.dK = dK;
  a.dV = dV;
  a.dW_part = (float*)(w + lay.dw_part);
  a.dW = dW;
  a.B = (int)p->B;
  a.H = (int)p->H;
  a.L = (int)p->L;
  a.C = clamp_C(p);
  a.P = P;
  a.relu_eps = p->relu_eps;
  const bwd_fn walk = pick_bwd(dp);
  // With the forward's Y and logD the cotangent after every segment is known
  // before the walks (eq. 18 summed over the later rows, the row cotangents
  // from Y and D): a query-sum pass and a reverse scan give it, each walk
  // starts from it, and no carry pass follows.
  const bool direct = P > 1 && logD != nullptr && dp.ksum != nullptr && walk == dp.bwd8;
  if (direct) {
    slim::KsumArgs qs;
    std::memset(&qs, 0, sizeof(qs));
    qs.K = Q;
    qs.V = dY;
    qs.Y = Y;
    qs.logD = logD;
    qs.W = W;
    qs.Wfrag = wf.out;
    qs.shift = favor ? kshift : nullptr;
    qs.out = (float*)(w + lay.seg_sum);
    qs.B = (int)p->B;
    qs.H = (int)p->H;
    qs.L = (int)p->L;
    qs.C = clamp_C(p);
    qs.P2 = P2;
    qs.relu_eps = p->relu_eps;
    qs.drop_scale = drop_plan(p).scale;
    e = dp.ksum(qs, slim::kSumQuery, s);
    if (e != hipSuccess) return hip_fail(e, "query-sum launch");
    slim::ScanArgs rv;
    std::memset(&rv, 0, sizeof(rv));
    rv.seg = qs.out;
    rv.init = dstate_out;
    rv.out = (float*)(w + lay.gend);
    rv.total = dstate_in;
    rv.init_shift = favor ? kshift_in : nullptr;
    rv.shift = favor ? kshift : nullptr;
    rv.BH = BH;
    rv.P = P2;
    rv.SZ = SZ;
    rv.favor = favor ? 1 : 0;
    rv.step = S2;
    e = slim::launch_scan_rev(rv, s);
    if (e != hipSuccess) return hip_fail(e, "cotangent-scan launch");
    a.g_init = rv.out;
    a.g_final = nullptr;
    a.dstate_in = nullptr;
  }
  e = timed_launch(SLIM_PHASE_BWD, s, [&] { return walk(a, s); });
  if (e != hipSuccess) return hip_fail(e, "backward launch");
  if (P > 1 && !direct) {
    // (4) cotangent after each segment (reverse scan of what the walks ended
    //     with; eq. 18 summed over the later segments) and before the
    //     sequence; then its contribution to the rows of each earlier segment
    slim::ScanArgs rv;
    std::memset(&rv, 0, sizeof(rv));
    rv.seg = a.g_final;
    rv.out = (float*)(w + lay.gend);
    rv.total = dstate_in;
    rv.init_shift = favor ? kshift_in : nullptr;
    rv.shift = favor ? kshift : nullptr;
    rv.BH = BH;
    rv.P = P;
    rv.SZ = SZ;
    rv.favor = favor ? 1 : 0;
    e = slim::launch_scan_rev(rv, s);
    if (e != hipSuccess) return hip_fail(e, "cotangent-scan launch");
    slim::CarryArgs ca;
    std::memset(&ca, 0, sizeof(ca));
    set_drop(ca, drop_plan(p));
    ca.K = K;
    ca.V = V;
    ca.Wfrag = a.Wfrag;
    ca.kshift = favor ? kshift : nullptr;
    ca.gend = rv.out;
    ca.dK = dK;
    ca.dV = dV;
    ca.dW_part = a.dW_part;
    ca.B = a.B;
    ca.H = a.H;
    ca.L = a.L;
    ca.C = a.C;
    ca.P = P;
    ca.CS = plan_carry_split(p, P);
    ca.relu_eps = p->relu_eps;
    if (dp.carry8 != nullptr) {
      ca.nch_head = slim::carry8_chunks_per_head(a.L, a.C, P);
      ca.NWG = carry8_workgroups(p, P);
      e = dp.carry8(ca, s);
    } else {
      e = dp.carry(ca, s);
    }
    if (e != hipSuccess) return hip_fail(e, "carry launch");
  }
  // (5) dW: the workgroups' partials summed in a fixed order (the walks'
  //     only, without the carry pass)
  const int slots = direct ? BH * P : (int)dw_slots(p, P);
  e = slim::launch_dw_reduce(a.dW_part, slots, (int)(p->M * p->d), dW, s);
  if (e != hipSuccess) return hip_fail(e, "dW-reduction launch");
  return ok();
}

}  // extern "C"
