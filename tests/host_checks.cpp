// Host-side checks of the library's argument validation, size arithmetic
// and workspace layout, built with AddressSanitizer and
// UndefinedBehaviorSanitizer on the host code only and run without a GPU.
// Every call below either fails validation (the status is checked) or, for
// the shapes marked "valid", passes validation and lays out its workspace,
// then reports the failed launch (no GPU in the process: the device code is
// compiled, and never runs).
// Exit status 0 when every status matched; sanitizer reports abort the run.
#include <climits>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <vector>

#include "specverify.h"

namespace {

int failures = 0;

void expect(const char* what, int line, spec_status got, spec_status want) {
  if (got != want) {
    std::printf("line %d (%s): status %d, expected %d\n", line, what, static_cast<int>(got), static_cast<int>(want));
    ++failures;
  }
}
void expect_not_ok(const char* what, int line, spec_status got) {
  if (got == SPEC_OK) {
    std::printf("line %d (%s): accepted\n", line, what);
    ++failures;
  }
}
#define EXPECT(call, want) expect(#call, __LINE__, (call), (want))
#define EXPECT_FAIL(call) expect_not_ok(#call, __LINE__, (call))

// Addresses that are never dereferenced on the host (device pointers in a
// real call): 256-byte aligned, and one that is not 16-byte aligned.
void* const P = reinterpret_cast<void*>(uintptr_t{1} << 20);
void* const Pmis = reinterpret_cast<void*>((uintptr_t{1} << 20) + 4);
const int32_t* const Ids = static_cast<const int32_t*>(P);
int32_t* const Out = static_cast<int32_t*>(P);
float* const F = static_cast<float*>(P);

spec_status verify(int B, int K, int V, spec_dtype dt, int64_t tsb, int64_t tsk, int64_t dsb, int64_t dsk,
                   void* ws, size_t wsb, const void* t = P, float Ts = 1.f, const int32_t* ids = Ids,
                   int32_t* acc = Out) {
  return spec_verify(t, tsb, tsk, P, dsb, dsk, dt, B, K, V, ids, nullptr, Ts, 1, 2, acc, Out, F, F, F, F, F, ws, wsb,
                     nullptr);
}

}  // namespace

int main() {
  const int maxV = SPEC_MAX_V;
  const int Ks[] = {-1, 0, 1, 3, 8, 9, INT_MAX};
  const int Bs[] = {INT_MIN, -1, 0, 1, 256, 65536, INT_MAX};
  const int Vs[] = {INT_MIN, -1, 0, 1, 8191, 8192, 151936, maxV, maxV + 1, INT_MAX};
  const spec_dtype dts[] = {SPEC_F32, SPEC_BF16, static_cast<spec_dtype>(7)};

  // size queries over every corner: never negative, never an overflowed
  // small value for a huge shape, 256-byte multiples, growing with B
  for (spec_dtype dt : dts)
    for (int K : Ks)
      for (int V : Vs) {
        size_t prev = 0;
        for (int B : Bs) {
          const size_t sizes[] = {spec_verify_workspace_size(B, K, V, dt), spec_tv_workspace_size(B, K, V, dt),
                                  spec_verify_gumbel_workspace_size(B, K, V, dt),
                                  spec_verify_target_only_workspace_size(B, K, V, dt),
                                  spec_diagnostics_workspace_size(B, K, V, dt), spec_kl_workspace_size(B, K, V, dt),
                                  spec_sample_workspace_size(B, V, dt), spec_sample_gumbel_workspace_size(B, V, dt)};
          for (size_t s : sizes)
            if (s % 256 != 0) {
              std::printf("size %zu for B=%d K=%d V=%d dt=%d is not a 256-byte multiple\n", s, B, K, V, dt);
              ++failures;
            }
          const size_t vs = sizes[0];
          if (vs != 0 && vs < prev) {
            std::printf("verify workspace shrinks with B at B=%d K=%d V=%d\n", B, K, V);
            ++failures;
          }
          if (vs) prev = vs;
        }
      }

  // spec_verify: one definite error per call
  const int B = 4, K = 3, V = 1000;
  const size_t need = spec_verify_workspace_size(B, K, V, SPEC_BF16);
  std::vector<unsigned char> none;
  EXPECT(verify(B, K, V, static_cast<spec_dtype>(7), 4000, 1000, 3000, 1000, P, need), SPEC_EUNSUPPORTED);
  EXPECT(verify(B, 9, V, SPEC_BF16, 10000, 1000, 9000, 1000, P, need), SPEC_EUNSUPPORTED);
  EXPECT(verify(0, K, V, SPEC_BF16, 4000, 1000, 3000, 1000, P, need), SPEC_EINVAL);
  EXPECT(verify(B, K, 0, SPEC_BF16, 4000, 1000, 3000, 1000, P, need), SPEC_EINVAL);
  EXPECT(verify(B, K, V, SPEC_BF16, -1, 1000, 3000, 1000, P, need), SPEC_EINVAL);
  EXPECT(verify(B, K, V, SPEC_BF16, 4000, 1000, 3000, -1000, P, need), SPEC_EINVAL);
  EXPECT(verify(B, K, V, SPEC_BF16, 4000, 1000, 3000, 1000, P, need, nullptr), SPEC_EINVAL);
  EXPECT(verify(B, K, V, SPEC_BF16, 4000, 1000, 3000, 1000, P, need, P, 0.f), SPEC_EINVAL);
  EXPECT(verify(B, K, V, SPEC_BF16, 4000, 1000, 3000, 1000, P, need, P, NAN), SPEC_EINVAL);
  EXPECT(verify(B, K, V, SPEC_BF16, 4000, 1000, 3000, 1000, P, need, P, INFINITY), SPEC_EINVAL);
  EXPECT(verify(B, K, V, SPEC_BF16, 4000, 1000, 3000, 1000, P, need, P, 1.f, nullptr), SPEC_EINVAL);
  EXPECT(verify(B, K, V, SPEC_BF16, 4000, 1000, 3000, 1000, P, need, P, 1.f, Ids, nullptr), SPEC_EINVAL);
  EXPECT(verify(B, K, V, SPEC_BF16, 4000, 1000, 3000, 1000, nullptr, need), SPEC_EWORKSPACE);
  EXPECT(verify(B, K, V, SPEC_BF16, 4000, 1000, 3000, 1000, P, need - 1), SPEC_EWORKSPACE);
  EXPECT(verify(B, K, V, SPEC_BF16, 4000, 1000, 3000, 1000, Pmis, need), SPEC_EINVAL);
  // strides whose products overflow 64 bits, and a vocabulary past the limit
  EXPECT_FAIL(verify(B, K, V, SPEC_BF16, INT64_MAX, INT64_MAX / 2, 3000, 1000, P, need));
  EXPECT_FAIL(verify(INT_MAX, K, V, SPEC_BF16, INT64_MAX / 4, 1000, 3000, 1000, P, SIZE_MAX));
  EXPECT_FAIL(verify(B, K, maxV + 1, SPEC_BF16, int64_t{1} << 33, int64_t{1} << 31, int64_t{1} << 33,
                     int64_t{1} << 31, P, SIZE_MAX));
  EXPECT_FAIL(verify(B, K, INT_MAX, SPEC_F32, INT64_MAX / 8, INT64_MAX / 64, 3000, 1000, P, SIZE_MAX));
  // launch controls
  spec_launch bad = {5, 0, 0}, neg = {SPEC_PATH_CHAIN, -1, 0}, shape = {SPEC_PATH_CHAIN, 0, 7};
  EXPECT(spec_verify_ex(P, 4000, 1000, P, 3000, 1000, SPEC_BF16, B, K, V, Ids, nullptr, 1.f, 1, 2, Out, Out, F, F, F,
                        F, F, P, need, nullptr, &bad),
         SPEC_EINVAL);
  EXPECT(spec_verify_ex(P, 4000, 1000, P, 3000, 1000, SPEC_BF16, B, K, V, Ids, nullptr, 1.f, 1, 2, Out, Out, F, F, F,
                        F, F, P, need, nullptr, &neg),
         SPEC_EINVAL);
  EXPECT(spec_verify_ex(P, 4000, 1000, P, 3000, 1000, SPEC_BF16, B, K, V, Ids, nullptr, 1.f, 1, 2, Out, Out, F, F, F,
                        F, F, P, need, nullptr, &shape),
         SPEC_EINVAL);
  // the entry point without a workspace: beyond its array, and argument errors
  EXPECT(spec_verify_noalloc(P, int64_t{262144} * 4, 262144, P, int64_t{262144} * 3, 262144, SPEC_BF16, 65536, 3,
                             262144, Ids, nullptr, 1.f, 1, 2, Out, Out, F, F, F, F, F, nullptr),
         SPEC_EWORKSPACE);
  EXPECT(spec_verify_noalloc(P, 4000, 1000, P, 3000, 1000, SPEC_BF16, B, K, V, Ids, nullptr, -1.f, 1, 2, Out, Out, F,
                             F, F, F, F, nullptr),
         SPEC_EINVAL);

  // the other entry points
  const size_t tvw = spec_tv_workspace_size(8, K, V, SPEC_BF16);
  EXPECT(spec_tv_loss_fwd_bwd(P, 3000, 1000, P, 3000, 1000, SPEC_BF16, 8, K, V, 1.f, static_cast<spec_tv_mode>(9),
                              1.f, F, F, F, P, tvw, nullptr),
         SPEC_EINVAL);
  EXPECT(spec_tv_loss_fwd_bwd(P, 3000, 1000, P, 3000, 1000, SPEC_BF16, 8, K, V, 0.f, SPEC_TV_E2E, 1.f, F, F, F, P,
                              tvw, nullptr),
         SPEC_EINVAL);
  EXPECT(spec_tv_loss_fwd_bwd(P, 3000, 1000, P, 3000, 1000, SPEC_BF16, 8, K, V, 1.f, SPEC_TV_E2E, 1.f, F, F, F, P,
                              tvw - 1, nullptr),
         SPEC_EWORKSPACE);
  EXPECT_FAIL(spec_tv_loss_fwd_bwd(P, INT64_MAX, INT64_MAX, P, 3000, 1000, SPEC_BF16, INT_MAX, K, V, 1.f,
                                   SPEC_TV_E2E, 1.f, F, F, F, P, SIZE_MAX, nullptr));
  const size_t klw = spec_kl_workspace_size(8, K, V, SPEC_F32);
  EXPECT(spec_kl_loss_fwd_bwd(P, 3000, 1000, P, 3000, 1000, SPEC_F32, 8, K, V, 1.f, static_cast<spec_kl_kind>(9),
                              1.f, F, F, F, P, klw, nullptr),
         SPEC_EINVAL);
  EXPECT(spec_kl_loss_fwd_bwd(P, 3000, 1000, P, 3000, 1000, SPEC_F32, 8, K, V, 1.f, SPEC_KL_FORWARD, 1.f, F, F, F, P,
                              klw - 1, nullptr),
         SPEC_EWORKSPACE);
  const size_t tow = spec_verify_target_only_workspace_size(B, K, V, SPEC_BF16);
  EXPECT(spec_verify_target_only(P, 4000, 1000, SPEC_BF16, B, K, V, nullptr, nullptr, 1.f, 1, 2, Out, Out, F, F, P,
                                 tow, nullptr),
         SPEC_EINVAL);
  EXPECT(spec_verify_target_only(P, 4000, 1000, SPEC_BF16, B, K, V, Ids, nullptr, 1.f, 1, 2, Out, Out, F, F, P,
                                 tow - 1, nullptr),
         SPEC_EWORKSPACE);
  const size_t sw = spec_sample_workspace_size(16, V, SPEC_BF16);
  EXPECT(spec_sample(P, 1000, SPEC_BF16, 16, V, nullptr, 1.f, 1, 2, nullptr, F, P, sw, nullptr), SPEC_EINVAL);
  EXPECT(spec_sample(P, -1, SPEC_BF16, 16, V, nullptr, 1.f, 1, 2, Out, F, P, sw, nullptr), SPEC_EINVAL);
  EXPECT_FAIL(spec_sample(P, INT64_MAX, SPEC_BF16, INT_MAX, V, nullptr, 1.f, 1, 2, Out, F, P, SIZE_MAX, nullptr));
  const size_t gw = spec_sample_gumbel_workspace_size(16, V, SPEC_BF16);
  EXPECT(spec_sample_gumbel(P, 1000, SPEC_BF16, 16, V, nullptr, 1.f, 1, 2, nullptr, P, gw, nullptr), SPEC_EINVAL);
  EXPECT(spec_sample_gumbel(P, 1000, SPEC_BF16, 16, V, nullptr, 1.f, 1, 2, Out, P, gw - 1, nullptr), SPEC_EWORKSPACE);
  const size_t vgw = spec_verify_gumbel_workspace_size(B, K, V, SPEC_BF16);
  EXPECT(spec_verify_gumbel(P, 4000, 1000, P, 3000, 1000, SPEC_BF16, B, K, V, nullptr, nullptr, 1.f, 1, 2, Out, Out, F,
                            F, F, F, F, P, vgw, nullptr),
         SPEC_EINVAL);
  const size_t dw = spec_diagnostics_workspace_size(B, K, V, SPEC_BF16);
  EXPECT(spec_diagnostics(P, 4000, 1000, P, 3000, 1000, SPEC_BF16, B, K, V, nullptr, 1.f, nullptr, Out, Out, P, dw,
                          nullptr),
         SPEC_EINVAL);
  EXPECT(spec_diagnostics(P, 4000, 1000, P, 3000, 1000, SPEC_BF16, B, K, V, nullptr, 1.f, F, Out, Out, P, dw - 1,
                          nullptr),
         SPEC_EWORKSPACE);

  // valid shapes: validation and the workspace layout run in full, then the
  // launch fails (no GPU in this process)
  for (int Kv : {1, 3, 8})
    for (int Vv : {1, 8191, 8193, 151936}) {
      const int Bv = 5;
      const int64_t tsk = (Vv + 7) / 8 * 8, tsb = tsk * (Kv + 1), dsb = tsk * Kv;
      const size_t w = spec_verify_workspace_size(Bv, Kv, Vv, SPEC_BF16);
      EXPECT_FAIL(verify(Bv, Kv, Vv, SPEC_BF16, tsb, tsk, dsb, tsk, P, w));
    }

  for (int s = -2; s < 12; ++s)
    if (spec_status_string(static_cast<spec_status>(s)) == nullptr) ++failures;
  if (spec_version() <= 0) ++failures;
  std::printf("%d failures\n", failures);
  return failures ? 1 : 0;
}
