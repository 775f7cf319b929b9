// Split-row family, scaled, causally masked softmax instantiations.
#include "split_launch.hpp"

namespace rowsm {
template int launch_split<kFused>(const Call& c, int in_dt, int out_dt);
}  // namespace rowsm
