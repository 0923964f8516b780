// Instantiations of the key-owned dK backward kernel for gradient mode 2
// (first-slot distribution (Setting 2)), softmax scores.
#include "kl_bwd_launch.hpp"

namespace streamkl {

hipError_t launch_bwd_dk_m2(int da, int db, bool causal, const BwdArgs& a) {
  return launch_bwd_unit<2, kActSoftmax, true>(da, db, causal, a);
}

}  // namespace streamkl
