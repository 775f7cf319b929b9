// Split-row family, log-softmax instantiations.
#include "split_launch.hpp"

namespace rowsm {
template int launch_split<kLog>(const Call& c, int in_dt, int out_dt);
}  // namespace rowsm
