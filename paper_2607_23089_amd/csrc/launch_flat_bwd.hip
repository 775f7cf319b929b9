// Flat short rows of ragged widths, softmax-backward instantiations.
#include "launch_flat.hpp"

namespace rowsm {
template int launch_flat<kBackward>(const Call& c, int in_dt, int out_dt);
}  // namespace rowsm
