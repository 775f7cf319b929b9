// Large-row family, softmax instantiations.
#include "launch_large.hpp"

namespace rowsm {
template int launch_large<kPlain>(const Call& c, int in_dt, int out_dt);
}  // namespace rowsm
