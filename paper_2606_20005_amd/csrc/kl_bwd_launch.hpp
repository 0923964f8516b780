// Launchers of the separate backward kernels, shared by the translation units
// that instantiate them: one unit per (kernel, gradient mode, activation)
// keeps the instantiations of a unit few and the units compiling in parallel.
#pragma once

#include "kl_bwd.hpp"
#include "kl_launch.hpp"

namespace streamkl {

template <int DA, int DB, bool CAUSAL, int MODE, int ACT, bool PD>
hipError_t run_bwd_dq(const BwdArgs& a) {
  using C = BwdCfg<DA, DB, MODE>;
  const int tiles = (a.NQ + C::BR - 1) / C::BR;
  const dim3 grid((unsigned)((long long)a.BH * tiles));
  hipLaunchKernelGGL((kl_bwd_dq_kernel<DA, DB, CAUSAL, MODE, ACT, PD>), grid, dim3(kThreads), 0, a.stream,
                     a.Qa, a.Ka, a.Qb, a.Kb, a.NQ, a.NK, a.dra, a.drb, a.sa, a.sb, a.kl, a.lse_a, a.lse_b, a.g,
                     a.dQa, a.dQb);
  return hipGetLastError();
}

template <int DA, int DB, bool CAUSAL, int MODE, int ACT, bool PD>
hipError_t run_bwd_dk(const BwdArgs& a) {
  using C = BwdCfg<DA, DB, MODE>;
  const int tiles = (a.NK + C::BR - 1) / C::BR;
  const dim3 grid((unsigned)((long long)a.BH * tiles));
  hipLaunchKernelGGL((kl_bwd_dk_kernel<DA, DB, CAUSAL, MODE, ACT, PD>), grid, dim3(kThreads), 0, a.stream,
                     a.Qa, a.Ka, a.Qb, a.Kb, a.NQ, a.NK, a.dra, a.drb, a.sa, a.sb, a.kl, a.lse_a, a.lse_b, a.g,
                     a.dKa, a.dKb, a.pstats, a.pfold);
  return hipGetLastError();
}

template <int DA, int DB, int MODE, int ACT, bool DK, bool PD>
hipError_t run_bwd_kernel(bool causal, const BwdArgs& a) {
  if constexpr (DK)
    return causal ? run_bwd_dk<DA, DB, true, MODE, ACT, PD>(a) : run_bwd_dk<DA, DB, false, MODE, ACT, PD>(a);
  else
    return causal ? run_bwd_dq<DA, DB, true, MODE, ACT, PD>(a) : run_bwd_dq<DA, DB, false, MODE, ACT, PD>(a);
}

// Launches the dQ (DK = false) or dK (DK = true) kernel of gradient mode
// MODE and activation ACT for the kernel head-dim pair (da, db); the
// instantiation for padded head dims when the real ones (a.dra, a.drb) are
// narrower.
template <int MODE, int ACT, bool DK>
hipError_t launch_bwd_unit(int da, int db, bool causal, const BwdArgs& a) {
#define STREAMKL_CASE(DA, DB)                                                                       \
  if (da == DA && db == DB) {                                                                       \
    if constexpr (MODE == 3 && DA + DB >= kSplitPairsDims) {                                        \
      return hipErrorInvalidValue; /* the host runs modes 1 and 2 instead */                        \
    } else {                                                                                        \
      if (a.dra != DA || a.drb != DB) return run_bwd_kernel<DA, DB, MODE, ACT, DK, true>(causal, a); \
      return run_bwd_kernel<DA, DB, MODE, ACT, DK, false>(causal, a);                               \
    }                                                                                               \
  }
  STREAMKL_FOR_EACH_DIM_PAIR(STREAMKL_CASE)
#undef STREAMKL_CASE
  return hipErrorInvalidValue;
}

}  // namespace streamkl
