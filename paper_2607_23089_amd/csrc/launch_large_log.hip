// Large-row family, log-softmax instantiations.
#include "launch_large.hpp"

namespace rowsm {
template int launch_large<kLog>(const Call& c, int in_dt, int out_dt);
}  // namespace rowsm
