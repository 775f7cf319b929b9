// Medium-row family, softmax instantiations.
#include "launch_medium.hpp"

namespace rowsm {
template int launch_medium<kPlain>(const Call& c, int in_dt, int out_dt);
}  // namespace rowsm
