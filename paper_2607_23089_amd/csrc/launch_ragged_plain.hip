// Ragged-width medium rows, softmax instantiations.
#include "launch_ragged.hpp"

namespace rowsm {
template int launch_ragged<kPlain>(const Call& c, int in_dt, int out_dt);
}  // namespace rowsm
