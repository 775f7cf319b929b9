// Medium-row family, scaled, causally masked softmax instantiations.
#include "launch_medium.hpp"

namespace rowsm {
template int launch_medium<kFused>(const Call& c, int in_dt, int out_dt);
}  // namespace rowsm
