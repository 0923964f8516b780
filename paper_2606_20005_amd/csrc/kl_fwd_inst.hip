// Instantiations and launcher of the forward kernels for every head-dim pair.
#include "kl_fwd.hpp"
#include "kl_launch.hpp"

namespace streamkl {

template <int DA, int DB, bool CAUSAL>
static hipError_t run_fwd(const FwdArgs& a) {
  using C = FwdCfg<DA, DB>;
  const int tq = (a.NQ + C::BQ - 1) / C::BQ;
  const dim3 grid((unsigned)((long long)a.BH * tq));
  hipLaunchKernelGGL((kl_fwd_kernel<C, CAUSAL>), grid, dim3(C::NT), 0, a.stream,
                     a.Qa, a.Ka, a.Qb, a.Kb, a.NQ, a.NK, a.ca, a.cb, a.kl, a.lse_a, a.lse_b);
  return hipGetLastError();
}

hipError_t launch_fwd(int da, int db, bool causal, const FwdArgs& a) {
#define STREAMKL_CASE(DA, DB) \
  if (da == DA && db == DB) return causal ? run_fwd<DA, DB, true>(a) : run_fwd<DA, DB, false>(a);
  STREAMKL_FOR_EACH_DIM_PAIR(STREAMKL_CASE)
#undef STREAMKL_CASE
  return hipErrorInvalidValue;
}

}  // namespace streamkl
