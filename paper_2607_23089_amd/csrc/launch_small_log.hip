// Small-row family, log-softmax instantiations.
#include "launch_small.hpp"

namespace rowsm {
template int launch_small<kLog>(const Call& c, int in_dt, int out_dt);
}  // namespace rowsm
