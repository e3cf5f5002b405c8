// Scans over segment states: the sequence of each head is split into P
// segments walked in parallel; these kernels turn per-segment sums into the
// exact state each segment starts from (forward and backward) and into the
// state cotangent each segment ends with (backward).  Grid: (state entries /
// 256, heads); one thread per state entry walks the segments in order.
#include "slim_common.hpp"
#include "slim_kernels.hpp"

namespace slim {

// out[p] = state before segment p, with key shift out_shift[p]:
//   s_0 = init (shift init_shift) or zero; s_{p+1} = s_p (+) seg_p, where (+)
//   brings both operands to the larger shift before adding.
__global__ __launch_bounds__(256) void scan_fwd_kernel(ScanArgs a) {
  const int head = blockIdx.y;
  const size_t SZ = a.SZ;
  const int el = blockIdx.x * 256 + threadIdx.x;
  if (el < a.SZ) {
    float v = a.init ? a.init[head * SZ + el] : 0.f;
    float vs = a.favor ? (a.init ? a.init_shift[head] : -INFINITY) : 0.f;
    for (int p = 0; p < a.P; ++p) {
      const size_t idx = ((size_t)head * a.P + p) * SZ + el;
      a.out[idx] = v;
      if (a.favor) {
        if (el == 0) a.out_shift[(size_t)head * a.P + p] = vs;
        const float ss = a.seg_shift[(size_t)head * a.P + p];
        const float m = fmaxf(vs, ss);
        v = v * fast_exp2((vs - m) * kLog2e) + a.seg[idx] * fast_exp2((ss - m) * kLog2e);
        vs = m;
      } else {
        v += a.seg[idx];
      }
    }
  }
}

// out[p] for p = 0..P: state at the boundary before segment p (p = P: after the
// last one), all relative to the common shift; init is relative to init_shift.
__global__ __launch_bounds__(256) void scan_bwd_kernel(ScanArgs a) {
  const int head = blockIdx.y;
  const size_t SZ = a.SZ;
  float r0 = 1.f;
  if (a.favor && a.init != nullptr) r0 = fast_exp2((a.init_shift[head] - a.shift[head]) * kLog2e);
  const int el = blockIdx.x * 256 + threadIdx.x;
  if (el < a.SZ) {
    float v = a.init ? r0 * a.init[head * SZ + el] : 0.f;
    const float* seg = a.seg + (size_t)head * a.P * SZ + el;
    float* out = a.out + (size_t)head * (a.P + 1) * SZ + el;
    // (eight segments' loads issued together; the sums stay in order)
    int p = 0;
    for (; p + 8 <= a.P; p += 8) {
      float x[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) x[i] = seg[(size_t)(p + i) * SZ];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        out[(size_t)(p + i) * SZ] = v;
        v += x[i];
      }
    }
    for (; p < a.P; ++p) {
      out[(size_t)p * SZ] = v;
      v += seg[(size_t)p * SZ];
    }
    out[(size_t)a.P * SZ] = v;
  }
}

// out[p] = init + sum_{q > p} seg[q]: the state cotangent after segment p;
// total = r0 (init + sum over all segments): the cotangent before segment 0.
// With step > 1 the P entries are parts of P / step segments and out holds
// the cotangent after each segment: out[i] = init + sum_{q >= (i + 1) step} seg[q].
__global__ __launch_bounds__(256) void scan_rev_kernel(ScanArgs a) {
  const int head = blockIdx.y;
  const size_t SZ = a.SZ;
  const int st = a.step > 1 ? a.step : 1, no = a.P / st;
  const int el = blockIdx.x * 256 + threadIdx.x;
  if (el < a.SZ) {
    float v = a.init ? a.init[head * SZ + el] : 0.f;
    const float* seg = a.seg + (size_t)head * a.P * SZ + el;
    auto step_to = [&](int p, float x) {
      if ((p + 1) % st == 0) a.out[((size_t)head * no + (p + 1) / st - 1) * SZ + el] = v;
      v += x;
    };
    // (eight segments' loads issued together; the sums stay in order)
    int p = a.P - 1;
    for (; p >= 7; p -= 8) {
      float x[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) x[i] = seg[(size_t)(p - i) * SZ];
#pragma unroll
      for (int i = 0; i < 8; ++i) step_to(p - i, x[i]);
    }
    for (; p >= 0; --p) step_to(p, seg[(size_t)p * SZ]);
    if (a.total != nullptr) {
      float r0 = 1.f;
      if (a.favor && a.init_shift != nullptr) r0 = fast_exp2((a.init_shift[head] - a.shift[head]) * kLog2e);
      a.total[head * SZ + el] = r0 * v;
    }
  }
}

static dim3 scan_grid(const ScanArgs& a) { return dim3((a.SZ + 255) / 256, a.BH); }

hipError_t launch_scan_fwd(const ScanArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(scan_fwd_kernel, scan_grid(a), dim3(256), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_scan_bwd(const ScanArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(scan_bwd_kernel, scan_grid(a), dim3(256), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_scan_rev(const ScanArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(scan_rev_kernel, scan_grid(a), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace slim
