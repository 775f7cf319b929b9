// Small-row family, scaled, causally masked softmax instantiations.
#include "launch_small.hpp"

namespace rowsm {
template int launch_small<kFused>(const Call& c, int in_dt, int out_dt);
}  // namespace rowsm
