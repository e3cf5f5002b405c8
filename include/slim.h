/*
 * slim.h - C ABI of the slice-wise causal linear attention library (gfx950).
 *
 * The library computes exact causal linear attention with a positive random
 * feature map g (Sec. 2.1, eq. 2) for a batch of heads,
 *
 *     Y_l = sum_{l' <= l} (g(Q_l) . g(K_l')) V_l' / sum_{l' <= l} g(Q_l) . g(K_l'),
 *
 * slice by slice in the manner of Algorithm 1 (Sec. 3.2-3.3): the forward
 * pass carries the running state B = (sum_l g(K_l) V_l^T, sum_l g(K_l)) from
 * slice to slice (eqs. 14-16); the backward pass walks the slices in reverse,
 * downdating B by each slice's contribution (eq. 17), recomputing the slice
 * and carrying the state cotangent G (eq. 18).  Extra device memory is
 * state-sized: it does not grow with the sequence length L.
 *
 * Feature maps (W in R^{M x d}, one row w_m per feature):
 *   SLIM_FAVOR_PLUS  g(x)_m = exp(w_m . x - |x|^2 / 2) / sqrt(M)
 *   SLIM_RELU        g(x)_m = max(w_m . x, 0) + relu_eps
 *   SLIM_SQUARE      g(x)_m = (w_m . x)^2; with W = I (M = d) this is the
 *                    element-wise square of the paper's experiments (Sec. 4)
 * The FAVOR+ map is evaluated with max-stabilisers that cancel exactly:
 * one shift per query row and one shift per (batch, head) shared by all keys;
 * the state is stored relative to the key shift (true state =
 * stored state * exp(kshift)).  The ReLU and square maps use no shifts.
 * Range: features are formed in float32, so a key whose exponent
 * w_m . k - |k|^2 / 2 lies more than about 87 below the head's key shift for
 * every m contributes exactly zero; a row l whose keys l' <= l all do so has
 * a zero denominator and a non-finite Y_l (and gradients).  Inputs scaled
 * like attention projections (entries of order d^-1/4) are far from it.
 *
 * Conventions for every entry point:
 *   - Tensors are dense, contiguous, row-major, in device memory:
 *       Q, K, V, Y, dY, dQ, dK, dV : [B, H, L, d], element type `dtype`
 *       W, dW                      : [M, d] float32, W shared by all heads
 *       state tensors              : [B, H, M, d + 1] float32; column j < d of
 *                                    row m holds sum_l g(K_l)_m V_l[j], column
 *                                    d holds sum_l g(K_l)_m
 *       kshift tensors             : [B, H] float32 (FAVOR+ only)
 *     Q, K, V, Y, dY, dQ, dK, dV and the workspace must be 16-byte aligned
 *     (rows are moved as 16-byte vectors); other tensors 4-byte aligned.
 *   - The caller owns every buffer.  The library never allocates or frees
 *     device memory; scratch space is the caller's workspace `ws`, whose size
 *     slim_workspace_bytes() gives.  The workspace holds nothing between calls.
 *   - Calls are asynchronous on `stream` (a hipStream_t passed as void*; NULL is
 *     the default stream).  No call synchronises the device.
 *   - Arguments are validated on the host before anything is launched; on a
 *     validation error nothing is launched and the output buffers are untouched.
 *     The return value is a slim_status; slim_last_error() describes the last
 *     failure of the calling thread.
 *   - The library keeps no state between calls and may be called from several
 *     threads; calls that share a workspace or outputs must not overlap.
 */
#ifndef SLIM_H_
#define SLIM_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SLIM_OK = 0,
  SLIM_EINVAL = -1,       /* null pointer, size < 1, unknown enum value */
  SLIM_EUNSUPPORTED = -2, /* well-formed problem outside the kernels' coverage */
  SLIM_EWORKSPACE = -3,   /* workspace null or smaller than slim_workspace_bytes() */
  SLIM_EHIP = -4          /* a HIP runtime call or a kernel launch failed */
} slim_status;

typedef enum { SLIM_FAVOR_PLUS = 0, SLIM_RELU = 1, SLIM_SQUARE = 2 } slim_kind;
typedef enum { SLIM_F32 = 0, SLIM_BF16 = 1 } slim_dtype;
typedef enum { SLIM_QUERY = 0, SLIM_KEY = 1 } slim_role;
typedef enum { SLIM_PHASE_FWD = 0, SLIM_PHASE_BWD = 1 } slim_phase;
/* How the prefix sums inside a slice are evaluated (Sec. 3.2, Appendix B):
 *   SLIM_WITHIN_ITER       block-iteratively, the state carried from one
 *                          32-row tile to the next (the tiles of a slice never
 *                          leave the chip; the work per row does not depend
 *                          on C)
 *   SLIM_WITHIN_QUADRATIC  the slice as one masked quadratic form (eq. 2
 *                          inside the slice), slices one after another and the
 *                          32-row tiles of a slice in parallel: the work per
 *                          row grows with C (bf16 problems with M of 128 or
 *                          256, FAVOR+ or ReLU)
 *   SLIM_WITHIN_PS         the explicit prefix sum the paper benchmarks as
 *                          "PS": the state after every row of a slice is
 *                          written out (C M (d + 1) floats per head, twice in
 *                          the backward, in the workspace), then used; slices
 *                          one after another.  Memory grows with C.  Any
 *                          dtype, map and shape (float32 with d M up to 16384
 *                          included); no dropout (SLIM_EUNSUPPORTED) */
typedef enum { SLIM_WITHIN_ITER = 0, SLIM_WITHIN_QUADRATIC = 1, SLIM_WITHIN_PS = 2 } slim_within;

/* Problem description shared by all entry points.
 *   B, H, L  batch, heads, sequence length (each >= 1; B H <= 65535 and one
 *            head's rows, L d elements, within 1 GiB, else SLIM_EUNSUPPORTED)
 *   d        head dimension: 32 or 64
 *   M        number of features: 64, 128 or 256 (SLIM_SQUARE: 64); with
 *            SLIM_F32, d M <= 4096 except in SLIM_WITHIN_PS
 *   C        slice length (Sec. 3.2): >= 1; values above L act as L.  The
 *            sequence is cut into N = ceil(L / C) slices, the last one ragged.
 *   dtype    slim_dtype of Q, K, V, Y, dY, dQ, dK, dV.  With SLIM_BF16 every
 *            product runs on bf16 matrix cores with float32 accumulation: W
 *            enters the logits w_m . x as the pair hi = bf16(w), lo =
 *            bf16(w - hi) (one product each, about 16 significant bits of
 *            W) and the chain rule (dq, dk) as hi; with SLIM_F32 products
 *            are float32.  SLIM_WITHIN_PS computes everything in float32
 *            from the float32 W for either dtype.
 *   kind     slim_kind
 *   relu_eps additive constant of the ReLU map (the usual value is 1e-3)
 *   dropout  probability p in [0, 1) of value dropout (0: none), and
 *   seed     its seed.  With dropout (Sec. 5: each slice n has its own
 *            seed, reused by the forward and the backward pass through it)
 *            value element (b, h, l, e) enters the attention multiplied by
 *            m in {0, 1}, and the output is scaled by s = 1 / (1 - p):
 *                Y_l = s sum_{l' <= l} a_ll' (m_l' * V_l') / sum_{l' <= l} a_ll'.
 *            m = 1 when 16-bit field e % 16 (word (e % 16) / 4, bits
 *            16 ((e % 16) % 4) and up) of Philox4x64-10 (Salmon et al.,
 *            SC 2011) with counter (r, e / 16, b H + h, 0) and key
 *            (seed, n) is >= round(p 65536), where n = l / C is the slice
 *            of row l and r = l - n C its row in the slice.  Rows are
 *            counted from the start of the call.  state_out then holds
 *            sum_l g(K_l) (m_l * V_l)^T (unscaled) in columns 0 .. d-1; dV
 *            is the cotangent of V itself (masked).
 *   within   slim_within: how the slice is evaluated (results agree up to
 *            rounding).
 * Work split: each head's sequence is cut into segments walked in parallel
 * (slim_num_segments) and each segment into parts whose exact boundary
 * states restart the backward's downdates; the counts are planned for a
 * device of 256 compute units (MI355X) and depend on B H, never on L once L
 * is long enough.  Parts are one tile (32 rows) each while their boundary
 * states fit 32 MiB over all heads.  A downdate subtracts in float32 what
 * the part's keys added; where a part's early keys have features orders of
 * magnitude below its later ones, the early states it recovers lose that
 * much relative precision (eq. 17 itself; the exact restarts bound it to
 * one part). */
typedef struct {
  int64_t B, H, L;
  int32_t d, M, C;
  int32_t dtype;
  int32_t kind;
  float relu_eps;
  float dropout;
  uint64_t seed;
  int32_t within; /* slim_within */
  int32_t reserved; /* must be 0 */
} slim_problem;

/* Bytes of device workspace slim_fwd (phase SLIM_PHASE_FWD) or slim_bwd
 * (SLIM_PHASE_BWD) need for problem *p.  Independent of L beyond the point
 * where the sequence is split into its maximum number of segments.  Returns 0
 * for an invalid problem (slim_last_error() says why).  Memory-only query:
 * makes no HIP call. */
size_t slim_workspace_bytes(const slim_problem* p, int phase);

/* Bytes of the optional context slim_fwd can hand to slim_bwd for problem
 * *p, or 0 when the problem uses none (then ctx is ignored and may be NULL).
 * The context holds the exact states at the segment boundaries of every
 * head ([B, H, P2 + 1, M, d + 1] float32: the state B^(n) of eqs. 14-16 at
 * each of the P2 + 1 boundaries of the head's parts, relative to kshift_out).
 * Its size depends on B H and the device, not on L: like the state itself it
 * is flat in the sequence length.  This is the state hand-off from the
 * forward to the backward pass beyond B^(N) (state_out) and the key shift
 * (kshift_out); the quadratic within-slice mode uses none.  Memory-only
 * query: makes no HIP call. */
size_t slim_context_bytes(const slim_problem* p);

/* Feature map of Sec. 2.1 (the map g of eq. 2) on its own, for inspection.
 *   X      [B, H, L, d] queries (role SLIM_QUERY) or keys (role SLIM_KEY), dtype
 *   W      [M, d] float32
 *   phi    out [B, H, L, M] float32: the stabilised map phi_hat
 *   shift  out, FAVOR+ only (NULL allowed for ReLU): queries [B, H, L], keys
 *          [B, H].  g(x) = phi_hat * exp(shift).  The query shift of row l is
 *          max_m(w_m . x_l) - |x_l|^2 / 2; the key shift of a head is the same
 *          maximum taken over all its rows.
 * The products use the same precision as slim_fwd (bf16 matrix cores for
 * SLIM_BF16). */
int slim_featmap(const slim_problem* p, const void* X, const float* W, int role, float* phi,
                 float* shift, void* stream);

/* Forward sweep of Algorithm 1 (one layer): Y for every row, and the state
 * B^(N) after the last slice.
 *   state_in   optional [B, H, M, d + 1]: the state B^(0) the sequence starts
 *              from (a previous call's state_out); NULL means zero
 *   kshift_in  [B, H], required with state_in for FAVOR+: the key shift
 *              state_in is relative to
 *   Y          out [B, H, L, d]
 *   logD       optional out [B, H, L] float32 (NULL: not written): for each row
 *              t the row normaliser log2(D_t) of eq. 4, Y_t = N_t / D_t, in
 *              the units of the true feature map g (its key shifts added
 *              back), so that g(q_t)_m / D_t = exp2(w_m . q_t log2(e) - logD_t)
 *              for FAVOR+ and g(q_t)_m exp2(-logD_t) for ReLU and the square
 *              map.  An output like Y (4 bytes per row): slim_bwd given Y and
 *              logD finds the state cotangent of every segment before its
 *              reverse walk.  Written by the tile-walk mode only: the
 *              quadratic and prefix-sum modes return SLIM_EUNSUPPORTED for a
 *              non-NULL logD
 *   state_out  out [B, H, M, d + 1], may be NULL: B^(N) relative to kshift_out
 *   kshift_out out [B, H] (FAVOR+: required; ReLU: ignored, may be NULL)
 *   ctx        optional out of slim_context_bytes(p) bytes (NULL: none): the
 *              segment boundary states, for the slim_bwd call on the same
 *              inputs
 *   ws         workspace of at least slim_workspace_bytes(p, SLIM_PHASE_FWD) */
int slim_fwd(const slim_problem* p, const void* Q, const void* K, const void* V, const float* W,
             const float* state_in, const float* kshift_in, void* Y, float* logD, float* state_out,
             float* kshift_out, float* ctx, void* ws, size_t ws_bytes, void* stream);

/* Bytes of the static device scratch slim_fwd_noalloc uses (a compile-time
 * constant, SLIM_NOALLOC_SCRATCH_BYTES). */
#define SLIM_NOALLOC_SCRATCH_BYTES ((size_t)72 << 20)
size_t slim_noalloc_scratch_bytes(void);

/* slim_fwd without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, serving loops, harnesses that
 * forbid hipMalloc).  Same arguments, results and errors as slim_fwd, except
 * that the scratch space is a static device array of
 * SLIM_NOALLOC_SCRATCH_BYTES inside the library: each device the library
 * runs on holds one copy, from the first call on that device until the
 * process ends.  The call allocates nothing (no hipMalloc, hipFree or
 * allocating library routine); the caller still passes every input and
 * output.  Problems whose forward needs more scratch than that
 * (slim_workspace_bytes(p, SLIM_PHASE_FWD) > SLIM_NOALLOC_SCRATCH_BYTES) are
 * rejected with SLIM_EUNSUPPORTED before anything is launched.  The scratch
 * of the current device (hipGetDevice) is used, so `stream` must belong to
 * it.  All calls on one device share its scratch: calls that may overlap on
 * one device (other host threads, or streams not ordered with each other)
 * race and must be serialised by the caller. */
int slim_fwd_noalloc(const slim_problem* p, const void* Q, const void* K, const void* V, const float* W,
                     const float* state_in, const float* kshift_in, void* Y, float* logD, float* state_out,
                     float* kshift_out, float* ctx, void* stream);

/* Backward sweep of Algorithm 1 (one layer) for the loss
 * sum(dY * Y) + <dstate_out, state_out>.
 *   Q, K, V, W, state_in, kshift_in  as given to slim_fwd
 *   kshift     [B, H]: kshift_out of slim_fwd (FAVOR+; ignored for ReLU)
 *   dY         [B, H, L, d] cotangent of Y
 *   Y          optional [B, H, L, d]: the Y slim_fwd wrote for these inputs
 *              (and the same seed), or NULL.  Given, the row cotangents of
 *              the recomputed slice (dN = dY / D, dD = -rowdot(dY, Y) / D,
 *              from eq. 2) take the rowdot from it, so the walk recomputes
 *              only the denominators D, not the numerators N.  Used by the
 *              bf16 tile walk with d = 32 or 64 and M / 4 in {32, 64}; the
 *              other configurations and within-slice modes recompute N and
 *              ignore it.  Y is rounded to the dtype, so the results differ
 *              from those without it within that rounding.
 *   logD       optional [B, H, L]: the logD slim_fwd wrote with Y (requires
 *              Y; SLIM_EINVAL otherwise), or NULL.  Given to the bf16 tile
 *              walk on a sequence split into several segments, the state
 *              cotangent after every segment (eq. 18 summed over the later
 *              rows) is summed from Q, dY, Y and logD before the walks, each
 *              walk starts from it, and the pass that otherwise adds the later
 *              segments' cotangent to every earlier row is skipped.  Ignored
 *              elsewhere.
 *   dstate_out optional [B, H, M, d + 1]: cotangent G^(N) of state_out (in the
 *              same kshift scaling as state_out); NULL means zero
 *   dQ, dK, dV out [B, H, L, d]
 *   dW         out [M, d] float32, overwritten: summed over heads, rows and the
 *              query and key branches
 *   dstate_in  out, may be NULL: [B, H, M, d + 1] cotangent G^(0) of state_in
 *              (relative to kshift_in; relative to kshift when state_in is NULL)
 *   ctx        optional: the context slim_fwd wrote for these inputs (and the
 *              same state_in, kshift_in), or NULL
 *   ws         workspace of at least slim_workspace_bytes(p, SLIM_PHASE_BWD)
 * The reverse walk starts from B^(N) and downdates it tile by tile (eq. 17).
 * B^(N) and the states at the segment boundaries come from ctx, or, without
 * one, are rebuilt here from the keys and values with the key shift
 * `kshift`; either way each downdate subtracts exactly the rounded features
 * that were added.  Nothing of size O(L) is kept between slim_fwd and
 * slim_bwd.  The key shifts are constants of the computation
 * (stop-gradient); they cancel exactly in Y. */
int slim_bwd(const slim_problem* p, const void* Q, const void* K, const void* V, const float* W,
             const float* state_in, const float* kshift_in, const float* kshift, const void* dY, const void* Y,
             const float* logD, const float* dstate_out, void* dQ, void* dK, void* dV, float* dW, float* dstate_in,
             const float* ctx, void* ws, size_t ws_bytes, void* stream);

/* Kernel-timing instrumentation.  before and after are hipEvent_t handles
 * (passed as void*) created by the caller with timing enabled.  The next
 * slim_fwd (phase SLIM_PHASE_FWD) or slim_bwd (SLIM_PHASE_BWD) call made by
 * this host thread records `before` and `after` on its stream immediately
 * around the launch of its main walk kernel (the forward walk that writes Y,
 * the reverse walk of the backward), so the caller can read that kernel's
 * own duration; the other launches of the call fall outside the pair (in the
 * quadratic within-slice mode the pair brackets the launches of all
 * slices).  The setting is consumed by that one call.  NULL for both clears
 * it.
 * Returns SLIM_OK, or SLIM_EINVAL for an unknown phase or only one NULL. */
int slim_time_walk(int phase, void* before, void* after);

/* Static description of a status code. */
const char* slim_status_string(int status);

/* Description of the last failure of the calling thread ("" if none). */
const char* slim_last_error(void);

/* Number of segments the sequence of each head is split into for parallel
 * processing (1 means one workgroup walks the whole sequence), or 0 for an
 * invalid problem.  Memory-only query. */
int slim_num_segments(const slim_problem* p);

#ifdef __cplusplus
}
#endif

#endif /* SLIM_H_ */
