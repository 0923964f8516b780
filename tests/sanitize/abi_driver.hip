// Host-only driver for the sanitizer test (tests/test_host_sanitizers.py).
// Built together with streamkl_api.hip, both with AddressSanitizer and
// UndefinedBehaviorSanitizer on the host side; the launchers of the other
// translation units are replaced by the counting stubs below, so no kernel of
// theirs exists here. Every call either fails validation, in which case the
// status is checked and no launcher may have been reached, or it reaches the
// stubs (or HIP, which fails without a GPU): what is checked there is that the
// host arithmetic on the way (extents, sizes, grids) stays defined.
#include <climits>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>

#include "kl_launch.hpp"
#include "streamkl.h"

namespace streamkl {
static int g_launches = 0;
static hipError_t stub() {
  ++g_launches;
  return hipSuccess;
}
hipError_t launch_fwd(int, int, bool, const FwdArgs&, int, float*) { return stub(); }
hipError_t launch_fwd_sigmoid(int, int, bool, const FwdArgs&) { return stub(); }
int fwd_rows_per_workgroup(int, int, int n_q, long long, bool, bool) { return n_q <= 32 ? 32 : n_q <= 128 ? 128 : 256; }
int fwd_merge_rows_per_workgroup() { return 4; }
hipError_t launch_bwd_dq_m1(int, int, bool, const BwdArgs&) { return stub(); }
hipError_t launch_bwd_dq_m2(int, int, bool, const BwdArgs&) { return stub(); }
hipError_t launch_bwd_dq_m3(int, int, bool, const BwdArgs&) { return stub(); }
hipError_t launch_bwd_dk_m1(int, int, bool, const BwdArgs&) { return stub(); }
hipError_t launch_bwd_dk_m2(int, int, bool, const BwdArgs&) { return stub(); }
hipError_t launch_bwd_dk_m3(int, int, bool, const BwdArgs&) { return stub(); }
hipError_t launch_bwd_dq_sig_m1(int, int, bool, const BwdArgs&) { return stub(); }
hipError_t launch_bwd_dq_sig_m2(int, int, bool, const BwdArgs&) { return stub(); }
hipError_t launch_bwd_dq_sig_m3(int, int, bool, const BwdArgs&) { return stub(); }
hipError_t launch_bwd_dk_sig_m1(int, int, bool, const BwdArgs&) { return stub(); }
hipError_t launch_bwd_dk_sig_m2(int, int, bool, const BwdArgs&) { return stub(); }
hipError_t launch_bwd_dk_sig_m3(int, int, bool, const BwdArgs&) { return stub(); }
bool bwd_fused_fits_m1(int, int) { return true; }
bool bwd_fused_fits_m2(int, int) { return true; }
bool bwd_fused_fits_m3(int da, int db) { return da + db <= 320; }
hipError_t launch_bwd_fused_m1(int, int, bool, const BwdArgs&) { return stub(); }
hipError_t launch_bwd_fused_m2(int, int, bool, const BwdArgs&) { return stub(); }
hipError_t launch_bwd_fused_m3(int, int, bool, const BwdArgs&) { return stub(); }
size_t bwd_rowstats_floats(int bh, int nq) { return (size_t)bh * ((nq + 31) / 32) * 129; }
hipError_t launch_bwd_rowstats(BwdArgs& a, float* stats) {
  a.pstats = stats;
  a.pfold = reinterpret_cast<const int*>(stats);
  return stub();
}
}  // namespace streamkl

static int g_failures = 0;
#define EXPECT(call, want)                                                                          \
  do {                                                                                              \
    const int before_ = streamkl::g_launches;                                                       \
    const int got_ = (call);                                                                        \
    if (got_ != (want) || streamkl::g_launches != before_) {                                        \
      std::fprintf(stderr, "FAIL line %d: status %d (want %d), launches %d\n", __LINE__, got_, (want), \
                   streamkl::g_launches - before_);                                                 \
      ++g_failures;                                                                                 \
    }                                                                                               \
  } while (0)

// fake device addresses: never dereferenced by the host code
static void* const P = reinterpret_cast<void*>(0x100000);
static void* const MIS2 = reinterpret_cast<void*>(0x100002);
static float* const F = reinterpret_cast<float*>(0x100000);

static int fwd(int B, int H, int nq, int nk, int d1, int d2, float s1 = 0.125f, float s2 = 0.125f, int causal = 0,
               int dir = 0, const void* q1 = P, float* kl = F) {
  return streamkl_fwd(q1, P, P, P, B, H, nq, nk, d1, d2, s1, s2, causal, dir, kl, F, F, nullptr);
}
static int bwd(int B, int H, int nq, int nk, int d1, int d2, float* dq2 = F, float* dk2 = F, const float* kl = F,
               int strategy = STREAMKL_BWD_SEPARATE, float* dq1 = nullptr, float* dk1 = nullptr) {
  return streamkl_bwd_ex(P, P, P, P, B, H, nq, nk, d1, d2, 0.125f, 0.125f, 0, 0, kl, F, F, nullptr, dq1, dk1, dq2,
                         dk2, strategy, nullptr);
}

int main() {
  const float inf = INFINITY, nan = NAN;
  // forward: argument checks (nothing launched)
  EXPECT(fwd(-1, 1, 64, 64, 64, 64), STREAMKL_ERR_INVALID_ARG);
  EXPECT(fwd(1, 1, -3, 64, 64, 64), STREAMKL_ERR_INVALID_ARG);
  EXPECT(fwd(1, 1, 64, INT_MIN, 64, 64), STREAMKL_ERR_INVALID_ARG);
  EXPECT(fwd(1, 1, 64, 64, 64, 64, 0.f), STREAMKL_ERR_INVALID_ARG);
  EXPECT(fwd(1, 1, 64, 64, 64, 64, inf), STREAMKL_ERR_INVALID_ARG);
  EXPECT(fwd(1, 1, 64, 64, 64, 64, 0.125f, nan), STREAMKL_ERR_INVALID_ARG);
  EXPECT(fwd(1, 1, 64, 64, 64, 64, 0.125f, 0.125f, 2), STREAMKL_ERR_INVALID_ARG);
  EXPECT(fwd(1, 1, 64, 64, 64, 64, 0.125f, 0.125f, 0, 7), STREAMKL_ERR_INVALID_ARG);
  EXPECT(fwd(1, 1, 64, 64, 64, 64, 0.125f, 0.125f, 0, 0, nullptr), STREAMKL_ERR_INVALID_ARG);
  EXPECT(fwd(1, 1, 64, 64, 64, 64, 0.125f, 0.125f, 0, 0, MIS2), STREAMKL_ERR_INVALID_ARG);
  EXPECT(fwd(1, 1, 64, 64, 64, 64, 0.125f, 0.125f, 0, 0, P, nullptr), STREAMKL_ERR_INVALID_ARG);
  for (int d : {0, 16, 48, 80, 257, 288, 512, INT_MAX, INT_MIN}) {
    EXPECT(fwd(1, 1, 64, 64, d, 64), STREAMKL_ERR_UNSUPPORTED);
    EXPECT(fwd(1, 1, 64, 64, 64, d), STREAMKL_ERR_UNSUPPORTED);
  }
  // extents whose products overflow 32 bits, or whose slabs leave 32-bit offsets
  EXPECT(fwd(70000, 70000, 64, 64, 64, 64), STREAMKL_ERR_UNSUPPORTED);
  EXPECT(fwd(INT_MAX, INT_MAX, INT_MAX, INT_MAX, 256, 256), STREAMKL_ERR_UNSUPPORTED);
  EXPECT(fwd(1, 1, 64, 4194304, 256, 64), STREAMKL_ERR_UNSUPPORTED);
  EXPECT(fwd(1, 1, INT_MAX, 64, 32, 32), STREAMKL_ERR_UNSUPPORTED);
  // zero extents are valid no-ops
  EXPECT(fwd(0, 5, 64, 64, 64, 64), STREAMKL_OK);
  EXPECT(fwd(1, 1, 0, 4194303, 256, 256, 0.125f, 0.125f, 0, 0, nullptr, nullptr), STREAMKL_OK);

  // backward
  EXPECT(bwd(1, 2, 64, 64, 64, 64, nullptr, nullptr), STREAMKL_ERR_INVALID_ARG);
  EXPECT(bwd(1, 2, 64, 64, 64, 64, reinterpret_cast<float*>(MIS2)), STREAMKL_ERR_INVALID_ARG);
  EXPECT(bwd(1, 2, 64, 64, 64, 64, F, F, nullptr), STREAMKL_ERR_INVALID_ARG);
  EXPECT(bwd(1, 2, 64, 64, 64, 64, F, F, F, 3), STREAMKL_ERR_INVALID_ARG);
  EXPECT(bwd(1, 2, 64, 64, 64, 100), STREAMKL_ERR_UNSUPPORTED);
  EXPECT(bwd(1, 1, 16, 65536, 256, 256, F, F, F, STREAMKL_BWD_FUSED, F, F), STREAMKL_ERR_UNSUPPORTED);
  EXPECT(bwd(INT_MAX, 2, 1, 1, 64, 64), STREAMKL_ERR_UNSUPPORTED);
  EXPECT(bwd(1, 1, 4194304, 64, 64, 256), STREAMKL_ERR_UNSUPPORTED);
  EXPECT(streamkl_bwd_act(P, P, P, P, 1, 1, 64, 64, 64, 64, 0.125f, 0.125f, 0, 0, 2, nullptr, nullptr, nullptr,
                          nullptr, nullptr, nullptr, F, F, nullptr),
         STREAMKL_ERR_INVALID_ARG);

  // split-K forward and its helpers
  EXPECT(streamkl_fwd_split(P, P, P, P, 1, 2, 16, 4096, 64, 64, 0.125f, 0.125f, 0, 0, 0, P, 1 << 20, F, F, F,
                            nullptr),
         STREAMKL_ERR_INVALID_ARG);
  EXPECT(streamkl_fwd_split(P, P, P, P, 1, 2, 16, 4096, 64, 64, 0.125f, 0.125f, 0, 0, 4, P, 10, F, F, F, nullptr),
         STREAMKL_ERR_INVALID_ARG);
  EXPECT(streamkl_fwd_split(P, P, P, P, 1024, 1024, 16384, 64, 64, 64, 0.125f, 0.125f, 0, 0, 2, P, SIZE_MAX, F,
                            F, F, nullptr),
         STREAMKL_ERR_UNSUPPORTED);
  EXPECT(streamkl_fwd_split_noalloc(P, P, P, P, 1, 1, 1 << 20, 64, 128, 128, 0.125f, 0.125f, 0, 0, 2, F, F, F,
                                    nullptr),
         STREAMKL_ERR_SCRATCH_LIMIT);
  EXPECT(streamkl_fwd_split_noalloc(P, P, P, P, 1, 1, 64, 64, 128, 128, 0.125f, 0.125f, 0, 0, INT_MAX, F, F, F,
                                    nullptr),
         STREAMKL_ERR_SCRATCH_LIMIT);
  volatile size_t sink = 0;
  for (int v : {0, 1, 2, 31, 32, 1000, INT_MAX, -1, INT_MIN}) {
    sink += streamkl_fwd_split_workspace_bytes(v, v, v, v);
    sink += streamkl_fwd_split_workspace_bytes(INT_MAX, INT_MAX, INT_MAX, v);
    sink += (size_t)streamkl_fwd_split_count(v, v, v, v, 128, 128);
    sink += (size_t)streamkl_fwd_split_count(1, 1, 1, v, 64, 64);
    sink += (size_t)streamkl_bwd_choose(v, v, v, v, 64, 64, 0, 0, 15);
    sink += (size_t)streamkl_bwd_choose(1, 1, v, INT_MAX, 96, 160, 1, 1, 5);
    sink += (size_t)streamkl_supported_head_dim(v);
  }
  for (int st = -2; st < 8; ++st) sink += std::strlen(streamkl_strerror(st));
  sink += std::strlen(streamkl_version());

  // valid calls that reach the launch stubs (or HIP): defined host arithmetic on the way
  const int launches0 = streamkl::g_launches;
  for (int d1 : {32, 96, 128, 256})
    for (int d2 : {32, 64, 224}) {
      (void)fwd(2, 3, 1000, 70000, d1, d2, 0.1f, 0.2f, 1, 1);
      (void)bwd(2, 3, 1000, 70000, d1, d2);
      (void)bwd(2, 3, 3, 70000, d1, d2, F, F, F, STREAMKL_BWD_AUTO, F, F);
      (void)bwd(1, 1, 4194303, 3, d1, d2 <= 64 ? d2 : 64);
      (void)streamkl_bwd_act(P, P, P, P, 1, 2, 77, 99, d1, d2, 0.1f, 0.1f, 1, 0, STREAMKL_ACT_SIGMOID, nullptr,
                             nullptr, nullptr, nullptr, F, F, F, F, nullptr);
      (void)streamkl_fwd_split(P, P, P, P, 4, 4, 16, 65536, d1, d2, 0.1f, 0.1f, 0, 0,
                               streamkl_fwd_split_count(4, 4, 16, 65536, d1, d2), P, SIZE_MAX, F, F, F, nullptr);
      (void)streamkl_fwd_split(P, P, P, P, 1, 1, 16, 4096, d1, d2, 0.1f, 0.1f, 1, 0, INT_MAX, P, SIZE_MAX, F, F, F,
                               nullptr);
    }
  if (streamkl::g_launches == launches0) {
    std::fprintf(stderr, "FAIL: no valid call reached a launcher\n");
    ++g_failures;
  }
  std::printf("abi driver: %d failures, %d launches, sink %zu\n", g_failures, streamkl::g_launches, (size_t)sink);
  return g_failures == 0 ? 0 : 1;
}
