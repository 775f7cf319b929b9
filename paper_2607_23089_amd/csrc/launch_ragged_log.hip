// Ragged-width medium rows, log-softmax instantiations.
#include "launch_ragged.hpp"

namespace rowsm {
template int launch_ragged<kLog>(const Call& c, int in_dt, int out_dt);
}  // namespace rowsm
