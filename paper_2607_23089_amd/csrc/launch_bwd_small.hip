// Softmax backward, small-row family.
#include "launch_bwd.hpp"

namespace rowsm {
int launch_bwd_small(const Call& c, int in_dt, int out_dt) {
  return dispatch<BwdSmallLaunch, kBackward>(c, in_dt, out_dt);
}
}  // namespace rowsm
