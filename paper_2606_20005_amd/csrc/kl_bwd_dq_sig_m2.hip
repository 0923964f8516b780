// Instantiations of the query-owned dQ backward kernel for gradient mode 2
// (first-slot distribution (Setting 2)), sigmoid scores.
#include "kl_bwd_launch.hpp"

namespace streamkl {

hipError_t launch_bwd_dq_sig_m2(int da, int db, bool causal, const BwdArgs& a) {
  return launch_bwd_unit<2, kActSigmoid, false>(da, db, causal, a);
}

}  // namespace streamkl
