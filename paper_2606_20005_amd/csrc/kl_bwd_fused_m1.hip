// Instantiations and launcher of the fused backward kernel, gradient mode 1
// (bit 0: second-slot distribution, bit 1: first-slot distribution). Head-dim
// pairs whose fused working set does not fit in LDS are not instantiated.
#include "kl_bwd_fused.hpp"
#include "kl_launch.hpp"

namespace streamkl {

template <int DA, int DB, bool CAUSAL>
static hipError_t run(const BwdArgs& a) {
  if constexpr (FusedCfg<DA, DB, 1>::FITS) {
    using C = FusedCfg<DA, DB, 1>;
    const int tiles = (a.NK + C::BR - 1) / C::BR;
    const dim3 grid((unsigned)((long long)a.BH * tiles));
    hipLaunchKernelGGL((kl_bwd_fused_kernel<DA, DB, CAUSAL, 1>), grid, dim3(kThreads), 0, a.stream,
                       a.Qa, a.Ka, a.Qb, a.Kb, a.NQ, a.NK, a.sa, a.sb, a.kl, a.lse_a, a.lse_b, a.g,
                       a.dQa, a.dQb, a.dKa, a.dKb);
    return hipGetLastError();
  } else {
    return hipErrorNotSupported;
  }
}

bool bwd_fused_fits_m1(int da, int db) {
#define STREAMKL_CASE(DA, DB) \
  if (da == DA && db == DB) return FusedCfg<DA, DB, 1>::FITS;
  STREAMKL_FOR_EACH_DIM_PAIR(STREAMKL_CASE)
#undef STREAMKL_CASE
  return false;
}

hipError_t launch_bwd_fused_m1(int da, int db, bool causal, const BwdArgs& a) {
#define STREAMKL_CASE(DA, DB) \
  if (da == DA && db == DB) return causal ? run<DA, DB, true>(a) : run<DA, DB, false>(a);
  STREAMKL_FOR_EACH_DIM_PAIR(STREAMKL_CASE)
#undef STREAMKL_CASE
  return hipErrorInvalidValue;
}

}  // namespace streamkl
