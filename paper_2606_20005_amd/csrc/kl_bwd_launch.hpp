// Launchers of the separate backward kernels, shared by the translation units
// that instantiate them: one unit per (kernel, gradient mode, activation)
// keeps the instantiations of a unit few and the units compiling in parallel.
#pragma once

#include "kl_bwd.hpp"
#include "kl_launch.hpp"

namespace streamkl {

template <int DA, int DB, bool CAUSAL, int MODE, int ACT>
hipError_t run_bwd_dq(const BwdArgs& a) {
  using C = BwdCfg<DA, DB, MODE>;
  const int tiles = (a.NQ + C::BR - 1) / C::BR;
  const dim3 grid((unsigned)((long long)a.BH * tiles));
  hipLaunchKernelGGL((kl_bwd_dq_kernel<DA, DB, CAUSAL, MODE, ACT>), grid, dim3(kThreads), 0, a.stream,
                     a.Qa, a.Ka, a.Qb, a.Kb, a.NQ, a.NK, a.sa, a.sb, a.kl, a.lse_a, a.lse_b, a.g, a.dQa, a.dQb);
  return hipGetLastError();
}

template <int DA, int DB, bool CAUSAL, int MODE, int ACT>
hipError_t run_bwd_dk(const BwdArgs& a) {
  using C = BwdCfg<DA, DB, MODE>;
  const int tiles = (a.NK + C::BR - 1) / C::BR;
  const dim3 grid((unsigned)((long long)a.BH * tiles));
  hipLaunchKernelGGL((kl_bwd_dk_kernel<DA, DB, CAUSAL, MODE, ACT>), grid, dim3(kThreads), 0, a.stream,
                     a.Qa, a.Ka, a.Qb, a.Kb, a.NQ, a.NK, a.sa, a.sb, a.kl, a.lse_a, a.lse_b, a.g, a.dKa, a.dKb);
  return hipGetLastError();
}

// Launches the dQ (DK = false) or dK (DK = true) kernel of gradient mode
// MODE and activation ACT for the head-dim pair (da, db).
template <int MODE, int ACT, bool DK>
hipError_t launch_bwd_unit(int da, int db, bool causal, const BwdArgs& a) {
#define STREAMKL_CASE(DA, DB)                                                                               \
  if (da == DA && db == DB) {                                                                               \
    if constexpr (DK)                                                                                       \
      return causal ? run_bwd_dk<DA, DB, true, MODE, ACT>(a) : run_bwd_dk<DA, DB, false, MODE, ACT>(a);    \
    else                                                                                                    \
      return causal ? run_bwd_dq<DA, DB, true, MODE, ACT>(a) : run_bwd_dq<DA, DB, false, MODE, ACT>(a);    \
  }
  STREAMKL_FOR_EACH_DIM_PAIR(STREAMKL_CASE)
#undef STREAMKL_CASE
  return hipErrorInvalidValue;
}

}  // namespace streamkl
