// Softmax backward, medium-row family.
#include "launch_bwd.hpp"

namespace rowsm {
int launch_bwd_medium(const Call& c, int in_dt, int out_dt) {
  return dispatch<BwdMediumLaunch, kBackward>(c, in_dt, out_dt);
}
}  // namespace rowsm
