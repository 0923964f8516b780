// Instantiations of the key-owned dK backward kernel for gradient mode 1
// (second-slot distribution (Setting 1)), softmax scores.
#include "kl_bwd_launch.hpp"

namespace streamkl {

hipError_t launch_bwd_dk_m1(int da, int db, bool causal, const BwdArgs& a) {
  return launch_bwd_unit<1, kActSoftmax, true>(da, db, causal, a);
}

}  // namespace streamkl
