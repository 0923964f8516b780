// Instantiations and launchers of the forward kernels for every head-dim pair.
#include "kl_fwd.hpp"
#include "kl_launch.hpp"

namespace streamkl {

// Waves per workgroup follow the query rows of a head: one wave for at most 32
// rows, four for at most 128, otherwise the default configuration.
template <int DA, int DB, bool CAUSAL, class C>
static hipError_t run_cfg(const FwdArgs& a, int W, float* part) {
  const int tq = (a.NQ + C::BQ - 1) / C::BQ;
  if (W <= 1) {
    const dim3 grid((unsigned)((long long)a.BH * tq));
    hipLaunchKernelGGL((kl_fwd_kernel<C, CAUSAL>), grid, dim3(C::NT), 0, a.stream,
                       a.Qa, a.Ka, a.Qb, a.Kb, a.NQ, a.NK, a.ca, a.cb, a.kl, a.lse_a, a.lse_b);
    return hipGetLastError();
  }
  const int nkt = (a.NK + C::BK - 1) / C::BK;
  const int chunk = (nkt + W - 1) / W;
  const dim3 grid((unsigned)((long long)a.BH * tq * W));
  hipLaunchKernelGGL((kl_fwd_partial_kernel<C, CAUSAL>), grid, dim3(C::NT), 0, a.stream,
                     a.Qa, a.Ka, a.Qb, a.Kb, a.NQ, a.NK, a.ca, a.cb, W, chunk, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t rows = (size_t)a.BH * a.NQ;
  hipLaunchKernelGGL(kl_fwd_merge_kernel, dim3((unsigned)((rows + kMergeRowsPerBlock - 1) / kMergeRowsPerBlock)),
                     dim3(64 * kMergeRowsPerBlock), 0, a.stream,
                     part, W, rows, a.kl, a.lse_a, a.lse_b);
  return hipGetLastError();
}

// Causal heads whose 256-row workgroups would number fewer than four per CU
// run 128-row ones instead (FwdCausalSmallCfg): twice the workgroups, so the
// two waves sharing a SIMD come from different workgroups (their phases are
// not tied by one barrier) and the rows that see the most keys are spread
// over more CUs. Measured 10-16% faster on such shapes; non-causal shapes of
// the same size measured 4-6% slower, so they keep the default.
constexpr long long kCausalSmallGrid = 1024;
static bool causal_small_grid(long long bh, int n_q) { return bh * ((n_q + 255) / 256) < kCausalSmallGrid; }

template <int DA, int DB, bool CAUSAL>
static hipError_t run_fwd(const FwdArgs& a, int W, float* part) {
  if (a.NQ <= 32) return run_cfg<DA, DB, CAUSAL, FwdSmallCfg<DA, DB, 1>>(a, W, part);
  if constexpr (DA + DB <= 256) {
    if (a.NQ <= 128) return run_cfg<DA, DB, CAUSAL, FwdSmallCfg<DA, DB, 4>>(a, W, part);
    if (CAUSAL && causal_small_grid(a.BH, a.NQ)) return run_cfg<DA, DB, CAUSAL, FwdCausalSmallCfg<DA, DB>>(a, W, part);
  }
  return run_cfg<DA, DB, CAUSAL, FwdCfg<DA, DB>>(a, W, part);
}

int fwd_merge_rows_per_workgroup() { return kMergeRowsPerBlock; }

int fwd_rows_per_workgroup(int da, int db, int n_q, long long bh, bool causal) {
  if (n_q <= 32) return 32;
  if (da + db <= 256) return (n_q <= 128 || (causal && causal_small_grid(bh, n_q))) ? 128 : 256;
  return 128;
}

hipError_t launch_fwd(int da, int db, bool causal, const FwdArgs& a, int W, float* part) {
#define STREAMKL_CASE(DA, DB) \
  if (da == DA && db == DB) return causal ? run_fwd<DA, DB, true>(a, W, part) : run_fwd<DA, DB, false>(a, W, part);
  STREAMKL_FOR_EACH_DIM_PAIR(STREAMKL_CASE)
#undef STREAMKL_CASE
  return hipErrorInvalidValue;
}

}  // namespace streamkl
