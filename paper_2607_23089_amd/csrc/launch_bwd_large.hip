// Softmax backward, large-row family.
#include "launch_bwd.hpp"

namespace rowsm {
int launch_bwd_large(const Call& c, int in_dt, int out_dt) {
  return dispatch<BwdLargeLaunch, kBackward>(c, in_dt, out_dt);
}
}  // namespace rowsm
