// Small-row family, softmax instantiations.
#include "launch_small.hpp"

namespace rowsm {
template int launch_small<kPlain>(const Call& c, int in_dt, int out_dt);
}  // namespace rowsm
