// Instantiations of the query-owned dQ backward kernel for gradient mode 3
// (both distributions), sigmoid scores.
#include "kl_bwd_launch.hpp"

namespace streamkl {

hipError_t launch_bwd_dq_sig_m3(int da, int db, bool causal, const BwdArgs& a) {
  return launch_bwd_unit<3, kActSigmoid, false>(da, db, causal, a);
}

}  // namespace streamkl
