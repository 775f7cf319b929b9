// Stand-ins for the kernel-family launchers in the host-logic check build:
// that build compiles the planner, the argument checks and the C ABI with
// the host compiler's address and undefined-behaviour sanitizers, without the
// kernel families.  Each launcher here reports a HIP error and launches
// nothing, which is what the full library returns on a machine without a GPU.
#include "launch.hpp"

namespace rowsm {

template <int MODE> int launch_small(const Call&, int, int) { return ROWSM_EHIP; }
template <int MODE> int launch_medium(const Call&, int, int) { return ROWSM_EHIP; }
template <int MODE> int launch_large(const Call&, int, int) { return ROWSM_EHIP; }
template <int MODE> int launch_split(const Call&, int, int) { return ROWSM_EHIP; }
template int launch_small<kPlain>(const Call&, int, int);
template int launch_small<kFused>(const Call&, int, int);
template int launch_small<kLog>(const Call&, int, int);
template int launch_medium<kPlain>(const Call&, int, int);
template int launch_medium<kFused>(const Call&, int, int);
template int launch_medium<kLog>(const Call&, int, int);
template int launch_large<kPlain>(const Call&, int, int);
template int launch_large<kFused>(const Call&, int, int);
template int launch_large<kLog>(const Call&, int, int);
template int launch_split<kPlain>(const Call&, int, int);
template int launch_split<kFused>(const Call&, int, int);
template int launch_split<kLog>(const Call&, int, int);
template <int MODE> int launch_ragged(const Call&, int, int) { return ROWSM_EHIP; }
template int launch_ragged<kPlain>(const Call&, int, int);
template int launch_ragged<kLog>(const Call&, int, int);
template <int MODE> int launch_flat(const Call&, int, int) { return ROWSM_EHIP; }
template int launch_flat<kPlain>(const Call&, int, int);
template int launch_flat<kLog>(const Call&, int, int);
template int launch_flat<kBackward>(const Call&, int, int);

int launch_bwd_small(const Call&, int, int) { return ROWSM_EHIP; }
int launch_bwd_medium(const Call&, int, int) { return ROWSM_EHIP; }
int launch_bwd_split(const Call&, int, int) { return ROWSM_EHIP; }
int launch_bwd_large(const Call&, int, int) { return ROWSM_EHIP; }
int launch_moe_f32(const Call&, int) { return ROWSM_EHIP; }
int launch_moe_bf16(const Call&, int) { return ROWSM_EHIP; }

}  // namespace rowsm
