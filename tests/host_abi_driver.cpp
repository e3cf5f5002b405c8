// Host-side exercise of the C ABI (include/slim.h, include/slim_model.h)
// for a build with AddressSanitizer and UndefinedBehaviorSanitizer on the
// host code: every sizing query over a grid of problem descriptions, valid
// and invalid, at the edges of the documented ranges, and every entry point
// with arguments that validation must reject before any device call.  No
// GPU is touched.  Exit status 0 when every status code is the expected one
// (a sanitizer finding aborts the program).
#include <climits>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "../include/slim.h"
#include "../include/slim_model.h"

static int failures = 0;
#define EXPECT(cond)                                                       \
  do {                                                                     \
    if (!(cond)) {                                                         \
      std::fprintf(stderr, "%s:%d: expected %s\n", __FILE__, __LINE__, #cond); \
      ++failures;                                                          \
    }                                                                      \
  } while (0)

static slim_problem problem(int64_t B, int64_t H, int64_t L, int d, int M, int C, int dtype, int kind, int within) {
  slim_problem p;
  std::memset(&p, 0, sizeof(p));
  p.B = B;
  p.H = H;
  p.L = L;
  p.d = d;
  p.M = M;
  p.C = C;
  p.dtype = dtype;
  p.kind = kind;
  p.relu_eps = 1e-3f;
  p.within = within;
  return p;
}

int main() {
  // a fake, aligned device address: validation must reject the calls below
  // before anything is dereferenced or launched
  alignas(256) static unsigned char block[4096];
  void* A = block;

  // ---- sizing over a grid of descriptions (int64 arithmetic at the edges)
  const int64_t Bs[] = {1, 3, 65535, 65536};
  const int64_t Ls[] = {1, 31, 32, 33, 4096, 262144, (int64_t)1 << 22, (int64_t)INT_MAX / 2, (int64_t)INT_MAX};
  const int Cs[] = {0, 1, 7, 32, 64, 1000, 32768, INT_MAX};
  const int ds[] = {16, 32, 64};
  const int Ms[] = {32, 64, 128, 256};
  size_t n_ok = 0, n_rejected = 0;
  for (int64_t B : Bs)
    for (int64_t L : Ls)
      for (int C : Cs)
        for (int d : ds)
          for (int M : Ms)
            for (int dtype = 0; dtype < 3; ++dtype)
              for (int kind = 0; kind < 4; ++kind)
                for (int within = 0; within < 4; ++within) {
                  const slim_problem p = problem(B, 1, L, d, M, C, dtype, kind, within);
                  const size_t f = slim_workspace_bytes(&p, SLIM_PHASE_FWD);
                  const size_t b = slim_workspace_bytes(&p, SLIM_PHASE_BWD);
                  (void)slim_context_bytes(&p);
                  (void)slim_num_segments(&p);
                  const bool valid = B <= 65535 && L >= 1 && C >= 1 && (d == 32 || d == 64) &&
                                     (M == 64 || M == 128 || M == 256) && dtype < 2 && kind < 3 && within < 3;
                  if (!valid) {
                    EXPECT(f == 0 && b == 0);
                    ++n_rejected;
                  } else if (f > 0 && b > 0) {
                    ++n_ok;
                  }
                }
  EXPECT(n_ok > 0 && n_rejected > 0);
  EXPECT(slim_workspace_bytes(nullptr, SLIM_PHASE_FWD) == 0);
  EXPECT(slim_noalloc_scratch_bytes() > 0);
  {
    slim_problem p = problem(1, 1, 64, 64, 256, 64, SLIM_BF16, SLIM_FAVOR_PLUS, SLIM_WITHIN_ITER);
    EXPECT(slim_workspace_bytes(&p, 7) == 0);
    p.reserved = 1;
    EXPECT(slim_workspace_bytes(&p, SLIM_PHASE_FWD) == 0);
    p.reserved = 0;
    p.dropout = 1.0f;
    EXPECT(slim_workspace_bytes(&p, SLIM_PHASE_FWD) == 0);
  }

  // ---- entry points rejected before any device call
  const slim_problem p = problem(2, 3, 1000, 64, 256, 64, SLIM_BF16, SLIM_FAVOR_PLUS, SLIM_WITHIN_ITER);
  float* F = (float*)block;
  EXPECT(slim_fwd(&p, nullptr, A, A, F, nullptr, nullptr, A, nullptr, F, F, nullptr, A, 1 << 20, nullptr) ==
         SLIM_EINVAL);
  EXPECT(slim_fwd(&p, A, A, A, F, nullptr, nullptr, A, nullptr, F, nullptr, nullptr, A, 1 << 20, nullptr) ==
         SLIM_EINVAL);
  EXPECT(slim_fwd(&p, A, A, A, F, nullptr, nullptr, A, nullptr, F, F, nullptr, A, 0, nullptr) == SLIM_EWORKSPACE);
  EXPECT(slim_fwd(&p, (char*)A + 2, A, A, F, nullptr, nullptr, A, nullptr, F, F, nullptr, A, 1 << 20, nullptr) ==
         SLIM_EINVAL);
  {
    // logD: misaligned; and in a mode that does not write it
    EXPECT(slim_fwd(&p, A, A, A, F, nullptr, nullptr, A, (float*)((char*)A + 2), F, F, nullptr, A, 1 << 20,
                    nullptr) == SLIM_EINVAL);
    slim_problem q = p;
    q.within = SLIM_WITHIN_QUADRATIC;
    EXPECT(slim_fwd(&q, A, A, A, F, nullptr, nullptr, A, F, F, F, nullptr, A, 1 << 30, nullptr) ==
           SLIM_EUNSUPPORTED);
  }
  EXPECT(slim_bwd(&p, A, A, A, F, nullptr, nullptr, F, A, nullptr, nullptr, nullptr, nullptr, A, A, F, nullptr,
                  nullptr, A, 1 << 20, nullptr) == SLIM_EINVAL);
  EXPECT(slim_bwd(&p, A, A, A, F, nullptr, nullptr, F, A, nullptr, nullptr, nullptr, A, A, A, F, nullptr, nullptr, A,
                  0, nullptr) == SLIM_EWORKSPACE);
  EXPECT(slim_bwd(&p, A, A, A, F, nullptr, nullptr, F, A, (char*)A + 2, nullptr, nullptr, A, A, A, F, nullptr,
                  nullptr, A, 1 << 20, nullptr) == SLIM_EINVAL);
  // logD without Y
  EXPECT(slim_bwd(&p, A, A, A, F, nullptr, nullptr, F, A, nullptr, F, nullptr, A, A, A, F, nullptr, nullptr, A,
                  1 << 20, nullptr) == SLIM_EINVAL);
  EXPECT(slim_featmap(&p, nullptr, F, SLIM_QUERY, F, F, nullptr) == SLIM_EINVAL);
  EXPECT(slim_featmap(&p, A, F, 5, F, F, nullptr) == SLIM_EINVAL);
  {
    const slim_problem bad = problem(1, 1, 0, 64, 256, 64, SLIM_BF16, SLIM_FAVOR_PLUS, SLIM_WITHIN_ITER);
    EXPECT(slim_fwd_noalloc(&bad, A, A, A, F, nullptr, nullptr, A, nullptr, F, F, nullptr, nullptr) == SLIM_EINVAL);
    const slim_problem big = problem(64, 64, 262144, 64, 256, 64, SLIM_BF16, SLIM_FAVOR_PLUS, SLIM_WITHIN_ITER);
    EXPECT(slim_fwd_noalloc(&big, A, A, A, F, nullptr, nullptr, A, nullptr, F, F, nullptr, nullptr) ==
           SLIM_EUNSUPPORTED);
  }
  EXPECT(slim_time_walk(9, nullptr, nullptr) == SLIM_EINVAL);
  EXPECT(slim_time_walk(SLIM_PHASE_FWD, A, nullptr) == SLIM_EINVAL);
  EXPECT(slim_time_walk(SLIM_PHASE_FWD, nullptr, nullptr) == SLIM_OK);
  for (int s = -6; s <= 1; ++s) EXPECT(slim_status_string(s) != nullptr);
  EXPECT(std::strlen(slim_last_error()) < 512);

  // ---- the model step
  slim_model m;
  std::memset(&m, 0, sizeof(m));
  m.B = 1;
  m.L = 16384;
  m.D = 1024;
  m.s = 3;
  m.vocab = 256;
  m.F = 4096;
  m.C = 512;
  m.ln_eps = 1e-5f;
  EXPECT(slim_model_num_params(&m) == 36);
  EXPECT(slim_model_workspace_bytes(&m) > 0);
  const int32_t Ds[] = {0, 64, 96, 4096, 4160};
  const int32_t Vs[] = {1, 2, 65536, 65537};
  const int64_t Ms_L[] = {1, 2, 1000, (int64_t)1 << 30, (int64_t)1 << 31};
  const int32_t Cm[] = {0, 1, 64, INT_MAX};
  for (int32_t D : Ds)
    for (int32_t V : Vs)
      for (int64_t L : Ms_L)
        for (int32_t C : Cm) {
          slim_model q = m;
          q.D = D;
          q.vocab = V;
          q.L = L;
          q.C = C;
          (void)slim_model_workspace_bytes(&q);
        }
  std::vector<void*> ptrs(36, A);
  EXPECT(slim_model_step(&m, nullptr, (const float* const*)ptrs.data(), (float* const*)ptrs.data(), F, A, 1 << 20,
                         nullptr) == SLIM_EINVAL);
  EXPECT(slim_model_step(&m, (const int32_t*)A, (const float* const*)ptrs.data(), (float* const*)ptrs.data(), F, A, 16,
                         nullptr) == SLIM_EWORKSPACE);
  EXPECT(slim_model_step(nullptr, (const int32_t*)A, nullptr, nullptr, F, A, 16, nullptr) == SLIM_EINVAL);

  std::printf("host ABI checks: %zu valid and %zu rejected descriptions sized; %d failures\n", n_ok, n_rejected,
              failures);
  return failures == 0 ? 0 : 1;
}
