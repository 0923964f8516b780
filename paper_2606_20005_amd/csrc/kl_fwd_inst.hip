// Instantiations and launchers of the forward kernels for every head-dim pair.
#include "kl_fwd.hpp"
#include "kl_launch.hpp"

namespace streamkl {

// Waves per workgroup follow the query rows of a head: one wave for at most 32
// rows, four for at most 128, otherwise the default configuration.
template <int DA, int DB, bool CAUSAL, class C, bool PD = false>
static hipError_t run_cfg(const FwdArgs& a, int W, float* part) {
  const int tq = (a.NQ + C::BQ - 1) / C::BQ;
  if (W <= 1) {
    const dim3 grid((unsigned)((long long)a.BH * tq));
    hipLaunchKernelGGL((kl_fwd_kernel<C, CAUSAL, PD>), grid, dim3(C::NT), 0, a.stream,
                       a.Qa, a.Ka, a.Qb, a.Kb, a.NQ, a.NK, a.dra, a.drb, a.ca, a.cb, a.kl, a.lse_a, a.lse_b);
    return hipGetLastError();
  }
  if constexpr (C::KS > 1) {
    return hipErrorInvalidValue;   // the split pass takes configurations of one tile per stage
  } else {
    const int nkt = (a.NK + C::BK - 1) / C::BK;
    const int chunk = (nkt + W - 1) / W;
    const dim3 grid((unsigned)((long long)a.BH * tq * W));
    hipLaunchKernelGGL((kl_fwd_partial_kernel<C, CAUSAL, PD>), grid, dim3(C::NT), 0, a.stream,
                       a.Qa, a.Ka, a.Qb, a.Kb, a.NQ, a.NK, a.dra, a.drb, a.ca, a.cb, W, chunk, part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const size_t rows = (size_t)a.BH * a.NQ;
    hipLaunchKernelGGL(kl_fwd_merge_kernel, dim3((unsigned)((rows + kMergeRowsPerBlock - 1) / kMergeRowsPerBlock)),
                       dim3(64 * kMergeRowsPerBlock), 0, a.stream,
                       part, W, rows, a.kl, a.lse_a, a.lse_b);
    return hipGetLastError();
  }
}

template <int DA, int DB, bool CAUSAL>
static hipError_t run_fwd(const FwdArgs& a, int W, float* part) {
  if (a.dra != DA || a.drb != DB) return run_cfg<DA, DB, CAUSAL, FwdPadDimCfg<DA, DB>, true>(a, W, part);
  switch (fwd_shape(DA, DB, a.NQ, a.BH, CAUSAL)) {
    case FwdShape::kOneWave: return run_cfg<DA, DB, CAUSAL, FwdSmallCfg<DA, DB, 1>>(a, W, part);
    case FwdShape::kFourWaves:
      if constexpr (DA + DB <= 256) return run_cfg<DA, DB, CAUSAL, FwdSmallCfg<DA, DB, 4>>(a, W, part);
      break;
    case FwdShape::kCausalSmall:
      if constexpr (DA + DB <= 256) return run_cfg<DA, DB, CAUSAL, FwdCausalSmallCfg<DA, DB>>(a, W, part);
      break;
    case FwdShape::kCausalKeySplit:
      if constexpr (DA + DB <= 192) {
        if (W <= 1) return run_cfg<DA, DB, CAUSAL, FwdCausalKeySplitCfg<DA, DB>>(a, W, part);
        return run_cfg<DA, DB, CAUSAL, FwdCausalSmallCfg<DA, DB>>(a, W, part);   // split pass: single tiles
      }
      break;
    case FwdShape::kDefault: break;
  }
  return run_cfg<DA, DB, CAUSAL, FwdCfg<DA, DB>>(a, W, part);
}

int fwd_merge_rows_per_workgroup() { return kMergeRowsPerBlock; }

int fwd_rows_per_workgroup(int da, int db, int n_q, long long bh, bool causal, bool padded) {
  if (padded) return 128;   // FwdPadDimCfg
  switch (fwd_shape(da, db, n_q, bh, causal)) {
    case FwdShape::kOneWave: return 32;
    case FwdShape::kFourWaves:
    case FwdShape::kCausalSmall:
    case FwdShape::kCausalKeySplit: return 128;
    case FwdShape::kDefault: break;
  }
  return da + db <= 256 ? 256 : 128;
}

hipError_t launch_fwd(int da, int db, bool causal, const FwdArgs& a, int W, float* part) {
#define STREAMKL_CASE(DA, DB) \
  if (da == DA && db == DB) return causal ? run_fwd<DA, DB, true>(a, W, part) : run_fwd<DA, DB, false>(a, W, part);
  STREAMKL_FOR_EACH_DIM_PAIR(STREAMKL_CASE)
#undef STREAMKL_CASE
  return hipErrorInvalidValue;
}

}  // namespace streamkl
