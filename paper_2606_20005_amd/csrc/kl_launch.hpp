// Internal launch interface between the C ABI (streamkl_api.hip) and the
// translation units that instantiate the kernels for each head-dim pair.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace streamkl {

// Arguments after the host has resolved the KL direction: "a" is the
// distribution in the first KL slot, "b" the one in the second.
// Head dims: the kernels are instantiated for multiples of 64 (da, db of the
// launch functions); dra, drb are the row lengths of the tensors in memory,
// equal to da, db or, for 32, 96, 160 and 224, 32 less (the kernels treat
// the missing columns as zeros).
struct FwdArgs {
  const uint16_t *Qa, *Ka, *Qb, *Kb;
  int BH, NQ, NK;
  int dra, drb;
  float ca, cb;                 // s * log2(e)
  float *kl, *lse_a, *lse_b;
  hipStream_t stream;
};

struct BwdArgs {
  const uint16_t *Qa, *Ka, *Qb, *Kb;
  int BH, NQ, NK;
  int dra, drb;
  float sa, sb;
  const float *kl, *lse_a, *lse_b, *g;
  float *dQa, *dQb, *dKa, *dKb;
  int act;                      // 0: softmax scores; 1: sigmoid scores (kl and the LSEs unused)
  hipStream_t stream;
  // row statistics prepared by launch_bwd_rowstats for the dK kernel (null: it forms them itself)
  const float* pstats = nullptr;
  const int* pfold = nullptr;
};

// Each returns hipErrorInvalidValue for a head-dim pair it does not hold,
// otherwise the status of the launch (hipGetLastError).
// W <= 1: one pass over all keys. W > 1: split-K (Sec. 3.3) with W key chunks;
// part holds 5 * W * BH * NQ floats of partial row statistics.
hipError_t launch_fwd(int da, int db, bool causal, const FwdArgs& a, int W, float* part);
// Sigmoid-score forward (one pass): kl, and the row masses of the first and
// second slot in lse_a / lse_b (either may be null). ca, cb are s * log2(e).
hipError_t launch_fwd_sigmoid(int da, int db, bool causal, const FwdArgs& a);
// Query rows per workgroup of the forward for these (kernel) head dims, rows
// per head, number of heads and mask; padded: the real dims are narrower.
int fwd_rows_per_workgroup(int da, int db, int n_q, long long bh, bool causal, bool padded);
// Rows per workgroup of the split-K merge.
int fwd_merge_rows_per_workgroup();
// Kernel head dims d1 + d2 from which the host runs all four gradients as
// the student-pair kernels followed by the teacher-pair kernels: a kernel
// holding both pairs' accumulators would spill there (and is not built).
constexpr int kSplitPairsDims = 448;
hipError_t launch_bwd_dq(int da, int db, bool causal, int mode, const BwdArgs& a);
hipError_t launch_bwd_dk(int da, int db, bool causal, int mode, const BwdArgs& a);
// Floats of the prepared row statistics of the dK kernel (kl_bwd_rowstats_kernel):
// 128 per 32-row tile plus one int flag per tile.
size_t bwd_rowstats_floats(int bh, int nq);
// Prepares them into stats (the flags follow the 128-float tiles) and points
// a.pstats, a.pfold at them; softmax scores only.
hipError_t launch_bwd_rowstats(BwdArgs& a, float* stats);
hipError_t launch_bwd_dq_m1(int da, int db, bool causal, const BwdArgs& a);
hipError_t launch_bwd_dq_m2(int da, int db, bool causal, const BwdArgs& a);
hipError_t launch_bwd_dq_m3(int da, int db, bool causal, const BwdArgs& a);
hipError_t launch_bwd_dk_m1(int da, int db, bool causal, const BwdArgs& a);
hipError_t launch_bwd_dk_m2(int da, int db, bool causal, const BwdArgs& a);
hipError_t launch_bwd_dk_m3(int da, int db, bool causal, const BwdArgs& a);
hipError_t launch_bwd_dq_sig_m1(int da, int db, bool causal, const BwdArgs& a);
hipError_t launch_bwd_dq_sig_m2(int da, int db, bool causal, const BwdArgs& a);
hipError_t launch_bwd_dq_sig_m3(int da, int db, bool causal, const BwdArgs& a);
hipError_t launch_bwd_dk_sig_m1(int da, int db, bool causal, const BwdArgs& a);
hipError_t launch_bwd_dk_sig_m2(int da, int db, bool causal, const BwdArgs& a);
hipError_t launch_bwd_dk_sig_m3(int da, int db, bool causal, const BwdArgs& a);
// Fused backward (Sec. 4.2): one key-owned kernel writes dK and adds dQ with
// atomics; dQ must be zeroed first. bwd_fused_fits says whether the kernel
// exists for these head dims and mode (its working set must fit in LDS).
bool bwd_fused_fits(int da, int db, int mode);
hipError_t launch_bwd_fused(int da, int db, bool causal, int mode, const BwdArgs& a);
bool bwd_fused_fits_m1(int da, int db);
bool bwd_fused_fits_m2(int da, int db);
bool bwd_fused_fits_m3(int da, int db);
hipError_t launch_bwd_fused_m1(int da, int db, bool causal, const BwdArgs& a);
hipError_t launch_bwd_fused_m2(int da, int db, bool causal, const BwdArgs& a);
hipError_t launch_bwd_fused_m3(int da, int db, bool causal, const BwdArgs& a);

// Expands F(DA, DB) for every supported head-dim pair.
#define STREAMKL_FOR_EACH_DIM_PAIR(F)                                        \
  F(64, 64) F(64, 128) F(64, 192) F(64, 256)                                 \
  F(128, 64) F(128, 128) F(128, 192) F(128, 256)                             \
  F(192, 64) F(192, 128) F(192, 192) F(192, 256)                             \
  F(256, 64) F(256, 128) F(256, 192) F(256, 256)

}  // namespace streamkl
