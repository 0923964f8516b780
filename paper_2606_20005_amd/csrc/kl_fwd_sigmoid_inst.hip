// Instantiations and launcher of the sigmoid-score forward for every
// head-dim pair, in the configurations the softmax forward takes for the same
// shapes (one pass over the keys; no split-K variant).
#include "kl_fwd.hpp"
#include "kl_launch.hpp"

namespace streamkl {

template <int DA, int DB, bool CAUSAL, class C, bool PD = false>
static hipError_t run_sig(const FwdArgs& a) {
  const int tq = (a.NQ + C::BQ - 1) / C::BQ;
  const dim3 grid((unsigned)((long long)a.BH * tq));
  hipLaunchKernelGGL((kl_fwd_sigmoid_kernel<C, CAUSAL, PD>), grid, dim3(C::NT), 0, a.stream,
                     a.Qa, a.Ka, a.Qb, a.Kb, a.NQ, a.NK, a.dra, a.drb, a.ca, a.cb, a.kl, a.lse_a, a.lse_b);
  return hipGetLastError();
}

template <int DA, int DB, bool CAUSAL>
static hipError_t run_fwd_sig(const FwdArgs& a) {
  if (a.dra != DA || a.drb != DB) return run_sig<DA, DB, CAUSAL, FwdPadDimCfg<DA, DB>, true>(a);
  switch (fwd_shape(DA, DB, a.NQ, a.BH, CAUSAL)) {
    case FwdShape::kOneWave: return run_sig<DA, DB, CAUSAL, FwdSmallCfg<DA, DB, 1>>(a);
    case FwdShape::kFourWaves:
      if constexpr (DA + DB <= 256) return run_sig<DA, DB, CAUSAL, FwdSmallCfg<DA, DB, 4>>(a);
      break;
    case FwdShape::kCausalSmall:
    case FwdShape::kCausalKeySplit:   // measured 1-1.5% slower with the key split: more vector work per tile
      if constexpr (DA + DB <= 256) return run_sig<DA, DB, CAUSAL, FwdCausalSmallCfg<DA, DB>>(a);
      break;
    case FwdShape::kDefault: break;
  }
  return run_sig<DA, DB, CAUSAL, FwdCfg<DA, DB>>(a);
}

hipError_t launch_fwd_sigmoid(int da, int db, bool causal, const FwdArgs& a) {
#define STREAMKL_CASE(DA, DB) \
  if (da == DA && db == DB) return causal ? run_fwd_sig<DA, DB, true>(a) : run_fwd_sig<DA, DB, false>(a);
  STREAMKL_FOR_EACH_DIM_PAIR(STREAMKL_CASE)
#undef STREAMKL_CASE
  return hipErrorInvalidValue;
}

}  // namespace streamkl
