// Split-row family, softmax instantiations.
#include "split_launch.hpp"

namespace rowsm {
template int launch_split<kPlain>(const Call& c, int in_dt, int out_dt);
}  // namespace rowsm
