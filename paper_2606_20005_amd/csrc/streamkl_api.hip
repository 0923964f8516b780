// C ABI of the attention-KL library: argument checking, resolution of the
// KL direction into (first slot, second slot) roles, and kernel dispatch.
// Every check happens before anything is enqueued, and no HIP call is made
// on an error path, so the checks are exercised on hosts without a GPU.
#include <atomic>
#include <cmath>
#include <cstdint>

#include "kl_launch.hpp"
#include "streamkl.h"

namespace {

using streamkl::BwdArgs;
using streamkl::FwdArgs;

constexpr float kLog2e = 1.4426950408889634f;
constexpr long long kMaxGrid = 0x7fffffffLL;

// Head dims: multiples of 32 up to 256. The kernels exist for multiples of
// 64; 32, 96, 160 and 224 run those of the next multiple of 64 with the real
// row length passed along (the extra columns read as zeros and gradients are
// written only for the real ones). The fused backward keeps to multiples of
// 64 (its end-of-tile wait counts every dQ atomic of the tile).
bool supported_dim(int d) { return d >= 32 && d <= 256 && d % 32 == 0; }
int kernel_dim(int d) { return (d + 63) / 64 * 64; }
bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }
bool scale_ok(float s) { return std::isfinite(s) && s > 0.f; }

// Checks shared by both passes. Returns STREAMKL_OK or an error code.
int check_common(const void* Q1, const void* K1, const void* Q2, const void* K2, int B, int H, int N_Q,
                 int N_K, int d1, int d2, float s1, float s2, int causal, int direction, bool* empty) {
  if (B < 0 || H < 0 || N_Q < 0 || N_K < 0) return STREAMKL_ERR_INVALID_ARG;
  if (causal != 0 && causal != 1) return STREAMKL_ERR_INVALID_ARG;
  if (direction != STREAMKL_KL_FWD && direction != STREAMKL_KL_REV) return STREAMKL_ERR_INVALID_ARG;
  if (!scale_ok(s1) || !scale_ok(s2)) return STREAMKL_ERR_INVALID_ARG;
  if (!supported_dim(d1) || !supported_dim(d2)) return STREAMKL_ERR_UNSUPPORTED;
  const long long bh = (long long)B * H;
  if (bh > kMaxGrid) return STREAMKL_ERR_UNSUPPORTED;
  // one workgroup per 128 rows of one head; element offsets are 64-bit in the kernels
  if (bh * ((N_Q + 127LL) / 128) > kMaxGrid || bh * ((N_K + 127LL) / 128) > kMaxGrid)
    return STREAMKL_ERR_UNSUPPORTED;
  // one (batch, head) slab of any tensor (bf16 inputs, fp32 gradients) is
  // addressed with 32-bit byte offsets
  const long long dmax = d1 > d2 ? d1 : d2;
  if ((long long)N_Q * dmax * 4 > 0xffffffffLL || (long long)N_K * dmax * 4 > 0xffffffffLL)
    return STREAMKL_ERR_UNSUPPORTED;
  *empty = bh == 0 || N_Q == 0;
  if (*empty) return STREAMKL_OK;
  if (!Q1 || !Q2) return STREAMKL_ERR_INVALID_ARG;
  if (N_K > 0 && (!K1 || !K2)) return STREAMKL_ERR_INVALID_ARG;
  if (!aligned(Q1, 16) || !aligned(Q2, 16) || (K1 && !aligned(K1, 16)) || (K2 && !aligned(K2, 16)))
    return STREAMKL_ERR_INVALID_ARG;
  return STREAMKL_OK;
}

int hip_status(hipError_t e) { return e == hipSuccess ? STREAMKL_OK : STREAMKL_ERR_HIP; }

// Zero fill by a kernel rather than hipMemsetAsync, so that the call stays
// safe to record into a HIP graph.
__global__ void zero_fill_kernel(float* __restrict__ p, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    p[i] = 0.f;
}

hipError_t zero_fill(float* p, size_t n, hipStream_t stream) {
  if (!p || n == 0) return hipSuccess;
  const size_t blocks = (n + 255) / 256;
  hipLaunchKernelGGL(zero_fill_kernel, dim3((unsigned)(blocks < 4096 ? blocks : 4096)), dim3(256), 0, stream, p, n);
  return hipGetLastError();
}

}  // namespace

// ---------------------------------------------------------------------------
// Static scratch of the allocation-free split-K forward
// (streamkl_fwd_split_noalloc): the five partial row statistics of every
// (chunk, row), in the layout the split-K kernels use for a caller's
// workspace. Every GPU the library runs on holds its own copy for the life of
// the process. In host code `scratch` only names the variable: its device
// address on a GPU comes from hipGetSymbolAddress with that GPU current, once
// per device, and only that address is ever handed to a kernel.
// ---------------------------------------------------------------------------
static __device__ __align__(256) float scratch[STREAMKL_NOALLOC_SCRATCH_BYTES / sizeof(float)];

namespace {

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_addr[kMaxDevices];

// Device address of the scratch array on the device of `stream`, which must
// be the current device. The first call on a device looks it up; concurrent
// first calls look up the same address, so the race is benign.
int scratch_address(hipStream_t stream, void** out) {
  int cur = -1;
  hipDevice_t sdev = -1;
  if (hipGetDevice(&cur) != hipSuccess || hipStreamGetDevice(stream, &sdev) != hipSuccess) return STREAMKL_ERR_HIP;
  if (sdev != cur) return STREAMKL_ERR_INVALID_ARG;
  if (cur < 0 || cur >= kMaxDevices) return STREAMKL_ERR_UNSUPPORTED;
  void* p = g_scratch_addr[cur].load(std::memory_order_acquire);
  if (!p) {
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return STREAMKL_ERR_HIP;
    g_scratch_addr[cur].store(p, std::memory_order_release);
  }
  *out = p;
  return STREAMKL_OK;
}

// use_scratch: the partials of a split-K call go to the static scratch array
// (workspace and workspace_bytes are ignored).
int fwd_common(const void* Q1, const void* K1, const void* Q2, const void* K2, int B, int H, int N_Q, int N_K, int d1,
               int d2, float s1, float s2, int causal, int direction, int splits, void* workspace,
               size_t workspace_bytes, bool use_scratch, float* kl, float* lse1, float* lse2, hipStream_t stream) {
  bool empty = false;
  const int st = check_common(Q1, K1, Q2, K2, B, H, N_Q, N_K, d1, d2, s1, s2, causal, direction, &empty);
  if (st != STREAMKL_OK) return st;
  if (splits < 1) return STREAMKL_ERR_INVALID_ARG;
  if (splits > 1) {
    const long long rows = (long long)B * H * N_Q;
    const int bq = streamkl::fwd_rows_per_workgroup(kernel_dim(d1), kernel_dim(d2), N_Q, (long long)B * H,
                                                    causal == 1, d1 % 64 != 0 || d2 % 64 != 0);
    const long long grid = (long long)B * H * ((N_Q + bq - 1) / bq) * splits;
    const long long merge_grid =
        (rows + streamkl::fwd_merge_rows_per_workgroup() - 1) / streamkl::fwd_merge_rows_per_workgroup();
    if (grid > kMaxGrid || merge_grid > kMaxGrid || rows * splits > (1LL << 40)) return STREAMKL_ERR_UNSUPPORTED;
    const size_t need = streamkl_fwd_split_workspace_bytes(B, H, N_Q, splits);
    if (use_scratch) {
      if (need > STREAMKL_NOALLOC_SCRATCH_BYTES) return STREAMKL_ERR_SCRATCH_LIMIT;
    } else if (!empty && (!workspace || !aligned(workspace, 4) || workspace_bytes < need)) {
      return STREAMKL_ERR_INVALID_ARG;
    }
  }
  if (empty) return STREAMKL_OK;
  if (!kl || !lse1 || !lse2) return STREAMKL_ERR_INVALID_ARG;
  if (!aligned(kl, 4) || !aligned(lse1, 4) || !aligned(lse2, 4)) return STREAMKL_ERR_INVALID_ARG;
  if (use_scratch && splits > 1) {
    const int sst = scratch_address(stream, &workspace);
    if (sst != STREAMKL_OK) return sst;
  }
  const bool rev = direction == STREAMKL_KL_REV;
  FwdArgs a;
  a.Qa = static_cast<const uint16_t*>(rev ? Q2 : Q1);
  a.Ka = static_cast<const uint16_t*>(rev ? K2 : K1);
  a.Qb = static_cast<const uint16_t*>(rev ? Q1 : Q2);
  a.Kb = static_cast<const uint16_t*>(rev ? K1 : K2);
  a.BH = B * H;
  a.NQ = N_Q;
  a.NK = N_K;
  a.dra = rev ? d2 : d1;
  a.drb = rev ? d1 : d2;
  a.ca = (rev ? s2 : s1) * kLog2e;
  a.cb = (rev ? s1 : s2) * kLog2e;
  a.kl = kl;
  a.lse_a = rev ? lse2 : lse1;
  a.lse_b = rev ? lse1 : lse2;
  a.stream = stream;
  return hip_status(streamkl::launch_fwd(kernel_dim(a.dra), kernel_dim(a.drb), causal == 1, a, splits,
                                         static_cast<float*>(workspace)));
}

}  // namespace

extern "C" int streamkl_fwd(const void* Q1, const void* K1, const void* Q2, const void* K2, int B, int H, int N_Q,
                            int N_K, int d1, int d2, float s1, float s2, int causal, int direction, float* kl,
                            float* lse1, float* lse2, hipStream_t stream) {
  return fwd_common(Q1, K1, Q2, K2, B, H, N_Q, N_K, d1, d2, s1, s2, causal, direction, 1, nullptr, 0, false, kl,
                    lse1, lse2, stream);
}

extern "C" int streamkl_fwd_act(const void* Q1, const void* K1, const void* Q2, const void* K2, int B, int H,
                                int N_Q, int N_K, int d1, int d2, float s1, float s2, int causal, int direction,
                                int activation, float* kl, float* stat1, float* stat2, hipStream_t stream) {
  if (activation == STREAMKL_ACT_SOFTMAX)
    return fwd_common(Q1, K1, Q2, K2, B, H, N_Q, N_K, d1, d2, s1, s2, causal, direction, 1, nullptr, 0, false, kl,
                      stat1, stat2, stream);
  if (activation != STREAMKL_ACT_SIGMOID) return STREAMKL_ERR_INVALID_ARG;
  bool empty = false;
  const int st = check_common(Q1, K1, Q2, K2, B, H, N_Q, N_K, d1, d2, s1, s2, causal, direction, &empty);
  if (st != STREAMKL_OK || empty) return st;
  if (!kl || !aligned(kl, 4) || (stat1 && !aligned(stat1, 4)) || (stat2 && !aligned(stat2, 4)))
    return STREAMKL_ERR_INVALID_ARG;
  const bool rev = direction == STREAMKL_KL_REV;
  FwdArgs a;
  a.Qa = static_cast<const uint16_t*>(rev ? Q2 : Q1);
  a.Ka = static_cast<const uint16_t*>(rev ? K2 : K1);
  a.Qb = static_cast<const uint16_t*>(rev ? Q1 : Q2);
  a.Kb = static_cast<const uint16_t*>(rev ? K1 : K2);
  a.BH = B * H;
  a.NQ = N_Q;
  a.NK = N_K;
  a.dra = rev ? d2 : d1;
  a.drb = rev ? d1 : d2;
  a.ca = (rev ? s2 : s1) * kLog2e;
  a.cb = (rev ? s1 : s2) * kLog2e;
  a.kl = kl;
  a.lse_a = rev ? stat2 : stat1;
  a.lse_b = rev ? stat1 : stat2;
  a.stream = stream;
  return hip_status(streamkl::launch_fwd_sigmoid(kernel_dim(a.dra), kernel_dim(a.drb), causal == 1, a));
}

extern "C" int streamkl_fwd_split(const void* Q1, const void* K1, const void* Q2, const void* K2, int B, int H,
                                  int N_Q, int N_K, int d1, int d2, float s1, float s2, int causal, int direction,
                                  int splits, void* workspace, size_t workspace_bytes, float* kl, float* lse1,
                                  float* lse2, hipStream_t stream) {
  return fwd_common(Q1, K1, Q2, K2, B, H, N_Q, N_K, d1, d2, s1, s2, causal, direction, splits, workspace,
                    workspace_bytes, false, kl, lse1, lse2, stream);
}

extern "C" int streamkl_fwd_split_noalloc(const void* Q1, const void* K1, const void* Q2, const void* K2, int B,
                                          int H, int N_Q, int N_K, int d1, int d2, float s1, float s2, int causal,
                                          int direction, int splits, float* kl, float* lse1, float* lse2,
                                          hipStream_t stream) {
  return fwd_common(Q1, K1, Q2, K2, B, H, N_Q, N_K, d1, d2, s1, s2, causal, direction, splits, nullptr, 0, true, kl,
                    lse1, lse2, stream);
}

extern "C" size_t streamkl_fwd_split_workspace_bytes(int B, int H, int N_Q, int splits) {
  if (B < 0 || H < 0 || N_Q < 0 || splits <= 1) return 0;
  return (size_t)20 * (size_t)splits * (size_t)B * (size_t)H * (size_t)N_Q;
}

extern "C" int streamkl_fwd_split_count(int B, int H, int N_Q, int N_K, int d1, int d2) {
  if (B < 0 || H < 0 || N_Q < 0 || N_K < 0) return 0;
  if (!supported_dim(d1) || !supported_dim(d2)) return 0;
  constexpr long long kTarget = 512;   // two workgroups per CU on 256 CUs
  const int bq = streamkl::fwd_rows_per_workgroup(kernel_dim(d1), kernel_dim(d2), N_Q, (long long)B * H, false,
                                                  d1 % 64 != 0 || d2 % 64 != 0);
  // base = B*H * query blocks, compared with the target without forming a
  // product that could overflow
  const long long bh = (long long)B * H, qb = ((long long)N_Q + bq - 1) / bq;
  if (bh == 0 || qb == 0 || bh >= kTarget || qb >= kTarget || bh * qb >= kTarget) return 1;
  const long long base = bh * qb;
  const long long tiles = (N_K + 31LL) / 32;
  const long long w = kTarget / base < tiles ? kTarget / base : tiles;
  return w < 1 ? 1 : (int)w;
}

namespace {

// Gradient masks of the first- and second-slot distributions ("a", "b").
struct BwdModes {
  int q, k;   // bit 0: b, bit 1: a
};

BwdModes bwd_modes(bool rev, bool dq1, bool dk1, bool dq2, bool dk2) {
  const bool dqa = rev ? dq2 : dq1, dqb = rev ? dq1 : dq2, dka = rev ? dk2 : dk1, dkb = rev ? dk1 : dk2;
  return BwdModes{(dqb ? 1 : 0) | (dqa ? 2 : 0), (dkb ? 1 : 0) | (dka ? 2 : 0)};
}

// Adaptive strategy rule (Sec. 4.2) over 128-row tiles: fused when
// T_Q * C <= T_K, C = 8, and in addition T_Q <= 4. Measured on MI355X
// (16 heads, d = 128, N_K from 4K to 64K): the fused kernel is 1.5-10x faster
// up to 512 query rows and slower from 1024 on, whatever N_K is, because its
// per-pair cost (atomic adds, the shared dS tile) exceeds that of the
// separate kernels once both have enough workgroups.
constexpr long long kFusedRatio = 8;
constexpr long long kFusedMaxQueryTiles = 4;

bool fused_preferred(int N_Q, int N_K) {
  const long long tq = (N_Q + 127LL) / 128, tk = (N_K + 127LL) / 128;
  return tq * kFusedRatio <= tk && tq <= kFusedMaxQueryTiles;
}

// act: STREAMKL_ACT_SOFTMAX or STREAMKL_ACT_SIGMOID (kl, lse1, lse2 unused
// and not required; separate kernels only).
int bwd_common(const void* Q1, const void* K1, const void* Q2, const void* K2, int B, int H, int N_Q, int N_K,
               int d1, int d2, float s1, float s2, int causal, int direction, const float* kl, const float* lse1,
               const float* lse2, const float* dkl, float* dQ1, float* dK1, float* dQ2, float* dK2, int strategy,
               int act, hipStream_t stream) {
  if (!dQ1 && !dK1 && !dQ2 && !dK2) return STREAMKL_ERR_INVALID_ARG;
  if (strategy != STREAMKL_BWD_AUTO && strategy != STREAMKL_BWD_SEPARATE && strategy != STREAMKL_BWD_FUSED)
    return STREAMKL_ERR_INVALID_ARG;
  bool empty = false;
  int st = check_common(Q1, K1, Q2, K2, B, H, N_Q, N_K, d1, d2, s1, s2, causal, direction, &empty);
  if (st != STREAMKL_OK) return st;
  const bool rev = direction == STREAMKL_KL_REV;
  const int da = rev ? d2 : d1, db = rev ? d1 : d2;                  // real head dims
  const int kda = kernel_dim(da), kdb = kernel_dim(db);              // the kernels' head dims
  const BwdModes m = bwd_modes(rev, dQ1, dK1, dQ2, dK2);
  const bool sig = act == STREAMKL_ACT_SIGMOID;
  const bool fused_ok =
      !sig && m.q != 0 && da == kda && db == kdb && streamkl::bwd_fused_fits(kda, kdb, m.q | m.k);
  if (strategy == STREAMKL_BWD_FUSED && m.q != 0 && !fused_ok) return STREAMKL_ERR_UNSUPPORTED;
  const bool fused = fused_ok && (strategy == STREAMKL_BWD_FUSED ||
                                  (strategy == STREAMKL_BWD_AUTO && fused_preferred(N_Q, N_K)));
  const long long bh = (long long)B * H;
  // With N_Q = 0 every dK is zero and there is no dQ; with N_K = 0 every dQ is zero.
  if (bh == 0) return STREAMKL_OK;
  if (N_Q == 0) {
    if ((dK1 && !aligned(dK1, 4)) || (dK2 && !aligned(dK2, 4))) return STREAMKL_ERR_INVALID_ARG;
    hipError_t e = hipSuccess;
    e = zero_fill(dK1, (size_t)bh * N_K * d1, stream);
    if (e == hipSuccess) e = zero_fill(dK2, (size_t)bh * N_K * d2, stream);
    return hip_status(e);
  }
  if (!sig && (!kl || !lse1 || !lse2)) return STREAMKL_ERR_INVALID_ARG;
  const void* ptrs[] = {kl, lse1, lse2, dkl, dQ1, dK1, dQ2, dK2};
  for (const void* p : ptrs)
    if (p && !aligned(p, 4)) return STREAMKL_ERR_INVALID_ARG;
  BwdArgs a;
  a.Qa = static_cast<const uint16_t*>(rev ? Q2 : Q1);
  a.Ka = static_cast<const uint16_t*>(rev ? K2 : K1);
  a.Qb = static_cast<const uint16_t*>(rev ? Q1 : Q2);
  a.Kb = static_cast<const uint16_t*>(rev ? K1 : K2);
  a.BH = (int)bh;
  a.NQ = N_Q;
  a.NK = N_K;
  a.dra = da;
  a.drb = db;
  a.sa = rev ? s2 : s1;
  a.sb = rev ? s1 : s2;
  a.kl = kl;
  a.lse_a = rev ? lse2 : lse1;
  a.lse_b = rev ? lse1 : lse2;
  a.g = dkl;
  a.dQa = rev ? dQ2 : dQ1;
  a.dQb = rev ? dQ1 : dQ2;
  a.dKa = rev ? dK2 : dK1;
  a.dKb = rev ? dK1 : dK2;
  a.act = sig ? 1 : 0;
  a.stream = stream;
  hipError_t e = hipSuccess;
  if (m.q && N_K == 0) {   // every row is empty: zero gradients
    e = zero_fill(a.dQa, (size_t)bh * N_Q * da, stream);
    if (e == hipSuccess) e = zero_fill(a.dQb, (size_t)bh * N_Q * db, stream);
    return hip_status(e);
  }
  if (fused) {
    // dQ accumulates atomically over key blocks: start from zero
    e = zero_fill(a.dQa, (size_t)bh * N_Q * da, stream);
    if (e == hipSuccess) e = zero_fill(a.dQb, (size_t)bh * N_Q * db, stream);
    if (e == hipSuccess) e = streamkl::launch_bwd_fused(kda, kdb, causal == 1, m.q | m.k, a);
    return hip_status(e);
  }
  // Both gradient pairs (mode 3) at kernel head dims d1 + d2 >= 448: one
  // kernel holding the accumulators of both pairs spills to scratch there,
  // while the student-pair and teacher-pair kernels do not; run one after
  // the other they recompute the logits once more and measured 1.1-2.6x
  // faster. Below that the single mode-3 kernel is faster (1.2-1.6x).
  const bool split_pairs = kda + kdb >= streamkl::kSplitPairsDims;
  auto launch = [&](bool dk, int mode, const streamkl::BwdArgs& x) -> hipError_t {
    auto one = [&](int md) {
      return dk ? streamkl::launch_bwd_dk(kda, kdb, causal == 1, md, x)
                : streamkl::launch_bwd_dq(kda, kdb, causal == 1, md, x);
    };
    if (mode != 3 || !split_pairs) return one(mode);
    const hipError_t e1 = one(1);
    return e1 == hipSuccess ? one(2) : e1;
  };
  // With a dQ output and softmax scores, the dK kernel's row statistics are
  // prepared ahead (kl_bwd_rowstats_kernel) into that dQ output, which the
  // dQ kernel overwrites afterwards: dK then runs first. The stream orders
  // the launches; the caller sees only the final dQ.
  float* scratch = nullptr;
  if (m.k && m.q && !sig) {
    float* dq = a.dQb ? a.dQb : a.dQa;
    const size_t room = (size_t)bh * N_Q * (a.dQb ? db : da);
    if (streamkl::bwd_rowstats_floats(a.BH, N_Q) <= room) scratch = dq;
  }
  if (scratch) {
    BwdArgs ak = a;
    e = streamkl::launch_bwd_rowstats(ak, scratch);
    if (e == hipSuccess) e = launch(true, m.k, ak);
    if (e == hipSuccess) e = launch(false, m.q, a);
    return hip_status(e);
  }
  if (m.q) e = launch(false, m.q, a);
  if (e == hipSuccess && m.k && N_K > 0) e = launch(true, m.k, a);
  return hip_status(e);
}

}  // namespace

extern "C" int streamkl_bwd(const void* Q1, const void* K1, const void* Q2, const void* K2, int B, int H, int N_Q,
                            int N_K, int d1, int d2, float s1, float s2, int causal, int direction,
                            const float* kl, const float* lse1, const float* lse2, const float* dkl, float* dQ1,
                            float* dK1, float* dQ2, float* dK2, hipStream_t stream) {
  return bwd_common(Q1, K1, Q2, K2, B, H, N_Q, N_K, d1, d2, s1, s2, causal, direction, kl, lse1, lse2, dkl, dQ1,
                    dK1, dQ2, dK2, STREAMKL_BWD_SEPARATE, STREAMKL_ACT_SOFTMAX, stream);
}

extern "C" int streamkl_bwd_ex(const void* Q1, const void* K1, const void* Q2, const void* K2, int B, int H,
                               int N_Q, int N_K, int d1, int d2, float s1, float s2, int causal, int direction,
                               const float* kl, const float* lse1, const float* lse2, const float* dkl,
                               float* dQ1, float* dK1, float* dQ2, float* dK2, int strategy, hipStream_t stream) {
  return bwd_common(Q1, K1, Q2, K2, B, H, N_Q, N_K, d1, d2, s1, s2, causal, direction, kl, lse1, lse2, dkl, dQ1,
                    dK1, dQ2, dK2, strategy, STREAMKL_ACT_SOFTMAX, stream);
}

extern "C" int streamkl_bwd_act(const void* Q1, const void* K1, const void* Q2, const void* K2, int B, int H,
                                int N_Q, int N_K, int d1, int d2, float s1, float s2, int causal, int direction,
                                int activation, const float* kl, const float* stat1, const float* stat2,
                                const float* dkl, float* dQ1, float* dK1, float* dQ2, float* dK2, hipStream_t stream) {
  if (activation != STREAMKL_ACT_SOFTMAX && activation != STREAMKL_ACT_SIGMOID) return STREAMKL_ERR_INVALID_ARG;
  return bwd_common(Q1, K1, Q2, K2, B, H, N_Q, N_K, d1, d2, s1, s2, causal, direction, kl, stat1, stat2, dkl, dQ1,
                    dK1, dQ2, dK2, STREAMKL_BWD_SEPARATE, activation, stream);
}

extern "C" int streamkl_bwd_choose(int B, int H, int N_Q, int N_K, int d1, int d2, int causal, int direction,
                                   int grads) {
  if (B < 0 || H < 0 || N_Q < 0 || N_K < 0) return 0;
  if (causal != 0 && causal != 1) return 0;
  if (direction != STREAMKL_KL_FWD && direction != STREAMKL_KL_REV) return 0;
  if (!supported_dim(d1) || !supported_dim(d2) || grads <= 0 || grads > 15) return 0;
  const bool rev = direction == STREAMKL_KL_REV;
  const BwdModes m = bwd_modes(rev, grads & STREAMKL_GRAD_DQ1, grads & STREAMKL_GRAD_DK1, grads & STREAMKL_GRAD_DQ2,
                               grads & STREAMKL_GRAD_DK2);
  const int da = rev ? d2 : d1, db = rev ? d1 : d2;
  const bool fused_ok = m.q != 0 && da % 64 == 0 && db % 64 == 0 && streamkl::bwd_fused_fits(da, db, m.q | m.k);
  return fused_ok && fused_preferred(N_Q, N_K) ? STREAMKL_BWD_FUSED : STREAMKL_BWD_SEPARATE;
}

extern "C" const char* streamkl_strerror(int status) {
  switch (status) {
    case STREAMKL_OK: return "success";
    case STREAMKL_ERR_INVALID_ARG: return "invalid argument (null pointer, negative extent, flag, scale or alignment)";
    case STREAMKL_ERR_UNSUPPORTED:
      return "unsupported configuration (head dim not a multiple of 32 in [32, 256], or extent too large)";
    case STREAMKL_ERR_HIP: return "HIP runtime rejected a kernel launch";
    case STREAMKL_ERR_SCRATCH_LIMIT:
      return "request needs more partial-statistics space than the allocation-free forward's static scratch holds";
    default: return "unknown status";
  }
}

extern "C" const char* streamkl_version(void) { return "streamkl 0.1.0 gfx950"; }

extern "C" int streamkl_supported_head_dim(int d) { return supported_dim(d) ? 1 : 0; }

namespace streamkl {

hipError_t launch_bwd_dq(int da, int db, bool causal, int mode, const BwdArgs& a) {
  if (a.act == 1) {
    switch (mode) {
      case 1: return launch_bwd_dq_sig_m1(da, db, causal, a);
      case 2: return launch_bwd_dq_sig_m2(da, db, causal, a);
      case 3: return launch_bwd_dq_sig_m3(da, db, causal, a);
      default: return hipErrorInvalidValue;
    }
  }
  switch (mode) {
    case 1: return launch_bwd_dq_m1(da, db, causal, a);
    case 2: return launch_bwd_dq_m2(da, db, causal, a);
    case 3: return launch_bwd_dq_m3(da, db, causal, a);
    default: return hipErrorInvalidValue;
  }
}

bool bwd_fused_fits(int da, int db, int mode) {
  switch (mode) {
    case 1: return bwd_fused_fits_m1(da, db);
    case 2: return bwd_fused_fits_m2(da, db);
    case 3: return bwd_fused_fits_m3(da, db);
    default: return false;
  }
}

hipError_t launch_bwd_fused(int da, int db, bool causal, int mode, const BwdArgs& a) {
  switch (mode) {
    case 1: return launch_bwd_fused_m1(da, db, causal, a);
    case 2: return launch_bwd_fused_m2(da, db, causal, a);
    case 3: return launch_bwd_fused_m3(da, db, causal, a);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_bwd_dk(int da, int db, bool causal, int mode, const BwdArgs& a) {
  if (a.act == 1) {
    switch (mode) {
      case 1: return launch_bwd_dk_sig_m1(da, db, causal, a);
      case 2: return launch_bwd_dk_sig_m2(da, db, causal, a);
      case 3: return launch_bwd_dk_sig_m3(da, db, causal, a);
      default: return hipErrorInvalidValue;
    }
  }
  switch (mode) {
    case 1: return launch_bwd_dk_m1(da, db, causal, a);
    case 2: return launch_bwd_dk_m2(da, db, causal, a);
    case 3: return launch_bwd_dk_m3(da, db, causal, a);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace streamkl
