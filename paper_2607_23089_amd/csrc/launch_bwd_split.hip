// Softmax backward, split-row family.
#include "launch_bwd.hpp"

namespace rowsm {
int launch_bwd_split(const Call& c, int in_dt, int out_dt) {
  return dispatch<BwdSplitLaunch, kBackward>(c, in_dt, out_dt);
}
}  // namespace rowsm
