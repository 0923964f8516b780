// Instantiations of the query-owned dQ backward kernel for gradient mode 3
// (both distributions), softmax scores.
#include "kl_bwd_launch.hpp"

namespace streamkl {

hipError_t launch_bwd_dq_m3(int da, int db, bool causal, const BwdArgs& a) {
  return launch_bwd_unit<3, kActSoftmax, false>(da, db, causal, a);
}

}  // namespace streamkl
