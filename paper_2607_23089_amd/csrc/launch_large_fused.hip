// Large-row family, scaled, causally masked softmax instantiations.
#include "launch_large.hpp"

namespace rowsm {
template int launch_large<kFused>(const Call& c, int in_dt, int out_dt);
}  // namespace rowsm
