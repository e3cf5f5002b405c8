/*
 * slim_model.h - C ABI of the low-memory training step of an s-layer
 * Performer language model (gfx950): Algorithm 1 with Algorithm 2 (Sec.
 * 3.2-3.3) over the model of Sec. 2.2 (eqs. 5-10).
 *
 * The model, for a batch of token sequences p in {0, ..., vocab - 1}^L:
 *
 *     X0_l  = E[p_l] + PE(l)              token embedding plus sinusoids,
 *                                         PE(l, 2i) = sin(l / 10000^(2i/D)),
 *                                         PE(l, 2i+1) = cos(...), l from 0
 *     for r = 1..s:
 *       A   = [Att(X Wq_j, X Wk_j, X Wv_j)]_j   (eqs. 7-8; head j takes
 *                                                columns [64 j, 64 j + 64))
 *       H   = LN1(A) + X                         (eq. 5)
 *       X   = LN2(GeLU(H W1 + b1) W2 + b2) + H   (eqs. 6, 9)
 *     loss  = mean over the batch of (L - 1)^-1 sum_{l < L} CE(X Wout + bout, p_{l+1})   (eq. 10)
 *
 * Att is causal linear attention (eq. 2) with the element-wise square map
 * g(x) = (x_i^2) and M = d = 64 (Sec. 4), evaluated by slim_fwd / slim_bwd
 * (include/slim.h, kind SLIM_SQUARE with W = I, float32).  LN is layer
 * normalisation with eps = ln_eps; GeLU is x Phi(x) (exact).
 *
 * slim_model_step computes the loss and its gradient by Algorithm 1: the
 * forward walks the slices of C rows in order and, inside a slice, the
 * layers in order, carrying only the attention states B_r of every layer;
 * the backward walks the slices in reverse, recovers B_r before each slice
 * by subtracting what the slice added (eq. 17), recomputes the slice through
 * all layers, back-propagates through it and carries the state cotangents
 * G_r (eq. 18).  Device memory beyond parameters, gradients and tokens is
 * the workspace: the activations of one slice plus the states, so it grows
 * with C and not with L.
 *
 * Everything is float32.  Matrix products run on the float32 matrix cores
 * in the library's own kernels (long reductions split over workgroups and
 * summed in a fixed order); every call is asynchronous on `stream`; the
 * library allocates nothing; results are deterministic (fixed summation
 * orders, no atomics).
 */
#ifndef SLIM_MODEL_H_
#define SLIM_MODEL_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Model and step description.
 *   B, L    batch of sequences and their length (L >= 2)
 *   D       d_model: a multiple of 64 (k = D / 64 heads of dimension 64), <= 4096
 *   s       layers (>= 1)
 *   vocab   alphabet size (2 .. 65536)
 *   F       d_ff (the paper uses 4 D): a multiple of 4
 *   C       slice length (>= 1; values above L act as L; B * min(C, L) <= 65535 * 64)
 *   ln_eps  layer-normalisation epsilon (the usual value is 1e-5) */
typedef struct {
  int64_t B, L;
  int32_t D, s, vocab, F, C;
  float ln_eps;
} slim_model;

/* Number of parameter tensors: 11 s + 3, in this order:
 *   emb [vocab, D];
 *   per layer r: Wq [D, D], Wk [D, D], Wv [D, D], ln1_g [D], ln1_b [D],
 *                W1 [D, F], b1 [F], W2 [F, D], b2 [D], ln2_g [D], ln2_b [D];
 *   Wout [D, vocab], bout [vocab].
 * All float32, row-major, contiguous, in device memory. */
int slim_model_num_params(const slim_model* m);

/* Bytes of device workspace slim_model_step needs (0 for an invalid
 * description).  Memory-only query. */
size_t slim_model_workspace_bytes(const slim_model* m);

/* One forward + backward pass of Algorithm 1.
 *   tokens  [B, L] int32, device; every entry in [0, vocab)
 *   params  host array of slim_model_num_params(m) device pointers (above)
 *   grads   host array of the same count of device pointers, same shapes:
 *           overwritten with the gradient of the loss
 *   loss    device pointer to one float: overwritten with the loss
 *   ws      workspace of at least slim_model_workspace_bytes(m) bytes,
 *           256-byte aligned
 * Returns a slim_status (include/slim.h); on a validation error nothing is
 * launched. */
int slim_model_step(const slim_model* m, const int32_t* tokens, const float* const* params, float* const* grads,
                    float* loss, void* ws, size_t ws_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SLIM_MODEL_H_ */
