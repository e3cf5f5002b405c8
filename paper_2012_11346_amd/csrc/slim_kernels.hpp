// Kernel argument blocks and launcher declarations shared by the host API
// (slim_api.cpp) and the kernel translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace slim {

struct FwdArgs {
  const void* Q;
  const void* K;
  const void* V;
  const float* W;
  void* Y;                 // nullptr: segment-sum mode (no outputs, only seg_sum_out)
  float* state_out;        // [B,H,M,D+1] or nullptr
  float* kshift_out;       // [B,H] or nullptr
  const float* seg_state;  // [B,H,P,M,D+1] state each segment starts from, or nullptr (zero)
  const float* seg_shift;  // [B,H,P] key shift of seg_state
  float* seg_sum_out;      // segment-sum mode: [B,H,P,M,D+1] state after the segment
  float* seg_shift_out;    // segment-sum mode: [B,H,P]
  int B, H, L, C, P;
  float relu_eps;
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
  const float* W;
  const float* kshift;      // [B,H] (FAVOR+)
  const float* seg_start;   // [B,H,P,M,D+1] exact state at each segment start (nullptr: zero)
  const float* start_shift; // [B,H,P] key shift seg_start is relative to (nullptr: kshift)
  const float* seg_end;     // [B,H,P,M,D+1] state at each segment end
  const float* seg_gend;    // [B,H,P,M,D+1] state cotangent at each segment end (nullptr: zero)
  float* seg_gstart;        // [B,H,P,M,D+1] state cotangent at each segment start (out), or nullptr
  void* dQ;
  void* dK;
  void* dV;
  float* dW_part;           // [B,H,P,M,D] per-workgroup partial dW
  float* dW;                // [M,D] sum of the partials
  float* gsum_out;          // G-contribution mode: [B,H,P,M,D+1] sum over the segment of Q~^T [dN|dD]
  int B, H, L, C, P;
  float relu_eps;
};

template <class G>
hipError_t launch_fwd_walk(const FwdArgs& a, hipStream_t s);
template <class G>
hipError_t launch_featmap(const FeatArgs& a, hipStream_t s);
template <class G>
hipError_t launch_bwd_walk(const BwdArgs& a, hipStream_t s);

// every compiled (element type, head dim, features per wave, tile rows, kind);
// fp32 problems serve exactness checks and are compiled for d * M <= 4096
#define SLIM_FOR_EACH_CONFIG(X)                                                           \
  X(bf16, 64, 64, 32, kFavor) X(bf16, 64, 32, 32, kFavor) X(bf16, 64, 16, 32, kFavor) \
  X(bf16, 32, 64, 32, kFavor) X(bf16, 32, 32, 32, kFavor) X(bf16, 32, 16, 32, kFavor) \
  X(bf16, 64, 64, 32, kRelu) X(bf16, 64, 32, 32, kRelu) X(bf16, 64, 16, 32, kRelu)    \
  X(bf16, 32, 64, 32, kRelu) X(bf16, 32, 32, 32, kRelu) X(bf16, 32, 16, 32, kRelu)    \
  X(float, 64, 16, 32, kFavor) X(float, 32, 32, 32, kFavor) X(float, 32, 16, 32, kFavor) \
  X(float, 64, 16, 32, kRelu) X(float, 32, 32, 32, kRelu) X(float, 32, 16, 32, kRelu)

}  // namespace slim
